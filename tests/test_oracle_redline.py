"""Pins of the Redline oracle against the paper's printed worked examples,
brute force, textbook equivalences and the Monte Carlo validity check."""
import csv
import itertools
import os
from fractions import Fraction

import mpmath
import numpy as np
import pytest

from oracle import redline as rl

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
GRIDS = ["grid_llada2_math", "grid_llada2_code", "grid_sdar_math", "grid_sdar_code",
         "grid_llada2_math_L256", "grid_llada2_code_L256", "learncert"]
BUDGETS = [(0.05, "05"), (0.10, "10"), (0.15, "15"), (0.20, "20")]


def load(name):
    with open(os.path.join(GOLDEN, name + ".csv")) as f:
        rows = list(csv.reader(l for l in f if not l.startswith("#")))
    return [dict(zip(rows[0], r)) for r in rows[1:]]


def ref_index(rows):
    return next(i for i, r in enumerate(rows) if "reference" in r["config"])


def printed_match(p, s):
    """Printed p-values are 3 decimals, or one significant digit below 1e-3."""
    p = float(p)
    if "e" in s:
        return float("%.0e" % p) == float(s)
    return round(p, 3) == float(s)


@pytest.mark.parametrize("grid", GRIDS)
@pytest.mark.parametrize("alpha,col", BUDGETS)
def test_grid_table(grid, alpha, col):
    """Every printed p equals Pr[Bin(n, alpha) <= k]; Holm at delta = 0.10
    reproduces the bold (valid) marks and argmax TPF the underlined row."""
    rows = load(grid)
    ps = [rl.binom_pvalue(int(r["n"]), alpha, int(r["k"])) for r in rows]
    for r, p in zip(rows, ps):
        assert printed_match(p, r["p" + col]), (r["config"], float(p), r["p" + col])
    valid = rl.holm(ps, 0.10)
    assert valid.tolist() == [r["v" + col] == "1" for r in rows]
    dep = rl.deploy([float(r["tpf"]) for r in rows], valid, ref_index(rows))
    assert [i for i, r in enumerate(rows) if r["d" + col] == "1"] == [dep]


def test_unlock_table():
    """Deployed gains and the smallest budget with a gain on the fine (0.01)
    budget grid.  Gains are re-derived from 3-decimal TPFs, so they may differ
    from the printed one-decimal gain by one unit in the last digit."""
    for u in load("unlock"):
        rows = load(u["grid"])
        ref = ref_index(rows)
        tpf = [float(r["tpf"]) for r in rows]
        assert int(u["m"]) == len(rows) and all(int(r["n"]) == int(u["n"]) for r in rows)
        amin = None
        for ai in range(1, 31):
            a = ai / 100
            ps = [rl.binom_pvalue(int(r["n"]), a, int(r["k"])) for r in rows]
            dep = rl.deploy(tpf, rl.holm(ps, 0.10), ref)
            if dep != ref and amin is None:
                amin = a
            if ai in (10, 15, 20):
                gain = 100.0 * (tpf[dep] / tpf[ref] - 1.0)
                assert abs(gain - float(u["gain%d" % ai])) <= 0.1 + 1e-9, (u["grid"], a, gain)
        assert amin == pytest.approx(float(u["alpha_min"]))


def test_holm_beats_bonferroni_at_alpha_007():
    """App. D.3: on LLaDA2 math at alpha = 0.07, acc90/semi90 (p = 0.0190)
    fails Bonferroni's 0.1/7 and passes Holm's threshold at its rank."""
    rows = load("grid_llada2_math")
    tpf = [float(r["tpf"]) for r in rows]
    ps = [rl.binom_pvalue(1012, 0.07, int(r["k"])) for r in rows]
    holm = rows[rl.deploy(tpf, rl.holm(ps, 0.10), ref_index(rows))]["config"]
    bonf = rows[rl.deploy(tpf, rl.bonferroni(ps, 0.10), ref_index(rows))]["config"]
    assert (holm, bonf) == ("acc90/semi90", "acc95/semi70")
    assert rl.bonferroni(ps, 0.10).sum() < rl.holm(ps, 0.10).sum()


def test_spot_pvalues():
    for r in load("spot_pvalues"):
        p = float(rl.binom_pvalue(int(r["n"]), float(r["alpha"]), int(r["k"])))
        digits = len(r["p"].split("e")[0].replace("0.", "").lstrip("0")) if "e" not in r["p"] else 2
        assert float("%.*g" % (digits, p)) == pytest.approx(float(r["p"])), (r, p)


def test_samplesize_margin():
    """Largest passing k at alpha = 0.10 for thresholds delta/8, delta/50 and
    delta; the printed percentages round half up (169/2000 prints 8.5)."""
    for r in load("samplesize_margin"):
        n = int(r["n"])
        for thr, col in ((0.10 / 8, "pct_d8"), (0.10 / 50, "pct_d50"), (0.10, "pct_d")):
            k = max(k for k in range(n) if rl.binom_pvalue(n, 0.10, k) <= thr)
            pct = Fraction(100 * k, n)
            printed = Fraction(r[col])
            assert printed - Fraction(1, 20) <= pct < printed + Fraction(1, 20), (n, col, k)


@pytest.mark.parametrize("delta", [0.05, 0.01])
def test_delta_sensitivity_math(delta):
    """App. D.3: the math deployments at alpha = 0.10 survive delta = 0.05 and 0.01."""
    for grid, want in (("grid_llada2_math", "acc85/semi70"), ("grid_sdar_math", "acc90/semi90")):
        rows = load(grid)
        ps = [rl.binom_pvalue(1012, 0.10, int(r["k"])) for r in rows]
        dep = rl.deploy([float(r["tpf"]) for r in rows], rl.holm(ps, delta), ref_index(rows))
        assert rows[dep]["config"] == want


def test_bonferroni_over_grids_sdar():
    """App. A.6: at delta/4 = 0.025 the SDAR math deployment at alpha = 0.10 is still valid."""
    rows = load("grid_sdar_math")
    ps = [rl.binom_pvalue(1012, 0.10, int(r["k"])) for r in rows]
    dep = rl.deploy([float(r["tpf"]) for r in rows], rl.holm(ps, 0.025), ref_index(rows))
    assert rows[dep]["config"] == "acc90/semi90"


@pytest.mark.parametrize("n", [1, 5, 12, 16])
def test_binomial_by_enumeration(n):
    """Pr[Bin(n, a) <= v] by enumerating all 2**n loss vectors, in exact rationals."""
    a = Fraction(0.1)
    counts = np.zeros(n + 1, dtype=np.int64)
    for mask in range(2 ** n):
        counts[bin(mask).count("1")] += 1
    for v in range(n + 1):
        exact = sum(Fraction(int(counts[k])) * a ** k * (1 - a) ** (n - k) for k in range(v + 1))
        got = rl.binom_pvalue(n, 0.1, v)
        with mpmath.workdps(80):
            assert abs(got - mpmath.mpf(exact.numerator) / exact.denominator) <= mpmath.mpf(10) ** -70


def closed_testing(p, delta):
    """Closed testing with Bonferroni local tests: H_j is rejected iff every
    intersection I containing j has min_{i in I} p_i <= delta / |I|."""
    m = len(p)
    rej = []
    for j in range(m):
        ok = True
        for size in range(1, m + 1):
            for I in itertools.combinations(range(m), size):
                if j in I and not min(p[i] for i in I) <= delta / size:
                    ok = False
        rej.append(ok)
    return np.array(rej)


def test_holm_equals_closed_testing():
    rng = np.random.default_rng(5)
    for trial in range(400):
        m = int(rng.integers(1, 7))
        p = list(rng.uniform(0, 0.12, size=m) ** rng.uniform(0.5, 3))
        if trial % 5 == 0:          # exact ties and boundary values
            p = [0.1 / m, 0.1 / m, 0.05, 0.1][:m]
        assert rl.holm(p, 0.1).tolist() == closed_testing(p, 0.1).tolist(), p


def test_violation_count_construction():
    """V counts prompts with the reference right and the candidate wrong only."""
    n = 50
    ref = np.ones(n, dtype=np.uint8)
    ref[:10] = 0
    cand = np.ones(n, dtype=np.uint8)
    cand[5:22] = 0           # 5..9 reference wrong too: not violations; 10..21: 12 violations
    better = np.ones(n, dtype=np.uint8)   # also right where the reference is wrong
    flipped = 1 - ref                     # wrong exactly where the reference is right
    V = rl.violations(np.stack([ref, cand, better, flipped]), 0)
    assert V.tolist() == [0, 12, 0, 40]


def test_deploy_rule():
    assert rl.deploy([1.0, 3.0, 3.0, 2.0], [True, True, True, False], 0) == 1   # lowest index on ties
    assert rl.deploy([1.0, 3.0], [False, False], 0) == 0                         # nothing valid -> reference
    assert rl.deploy([5.0, 3.0], [False, True], 0) == 1


def test_monte_carlo_fwer():
    """App. A.7: true risks {0.01, 0.02, 0.07, 0.07, 0.07}, alpha = 0.05,
    n = 800, 4000 trials, losses from one shared uniform per prompt; the
    family-wise error of Holm (a configuration with R > alpha found valid)
    stays at or below delta = 0.10 (the paper observed 0.0003)."""
    R = np.array([0.01, 0.02, 0.07, 0.07, 0.07])
    n, alpha, delta, trials = 800, 0.05, 0.10, 4000
    table = [rl.binom_pvalue(n, alpha, v) for v in range(n + 1)]
    rng = np.random.default_rng(2026)
    errors = 0
    for _ in range(trials):
        u = rng.uniform(size=n)
        V = (u[None, :] < R[:, None]).sum(axis=1)
        valid = rl.holm([table[v] for v in V], delta)
        errors += bool(np.any(valid & (R > alpha)))
    fwer = errors / trials
    assert fwer <= delta
    assert fwer <= 0.01          # the shared uniform makes the three nulls identical


# ---- variants and the validity harness (App. A.3-A.7, App. D) --------------

def closed_testing_fixed_sequence(p, delta, order):
    """Closed testing whose local test of an intersection I rejects iff the
    member of I that comes first in ``order`` has p <= delta (the
    fixed-sequence walk is this closed procedure)."""
    m = len(p)
    rank = {j: i for i, j in enumerate(order)}
    rej = []
    for j in range(m):
        ok = True
        for size in range(1, m + 1):
            for I in itertools.combinations(range(m), size):
                if j in I and not p[min(I, key=lambda i: rank[i])] <= delta:
                    ok = False
        rej.append(ok)
    return np.array(rej)


def test_fixed_sequence_equals_closed_testing():
    rng = np.random.default_rng(11)
    for trial in range(300):
        m = int(rng.integers(1, 7))
        p = list(rng.uniform(0, 0.25, size=m))
        if trial % 7 == 0:
            p = [0.1, 0.05, 0.1000001, 0.0, 0.1, 0.2][:m]          # boundary values
        order = list(rng.permutation(m))
        assert rl.fixed_sequence(p, 0.1, order).tolist() == \
            closed_testing_fixed_sequence(p, 0.1, order).tolist(), (p, order)


def test_procedures_nest_and_coincide_for_one_hypothesis():
    """Bonferroni's valid set lies inside Holm's (§4.2), Holm's inside the
    uncorrected test's; with m = 1 Holm, Bonferroni, the fixed sequence and
    the uncorrected test are the same single test at level delta."""
    rng = np.random.default_rng(12)
    for _ in range(300):
        m = int(rng.integers(1, 9))
        p = list(rng.uniform(0, 0.2, size=m) ** 2)
        b, h, u = rl.bonferroni(p, 0.1), rl.holm(p, 0.1), rl.uncorrected(p, 0.1)
        assert np.all(b <= h) and np.all(h <= u)
        if m == 1:
            assert b[0] == h[0] == u[0] == rl.fixed_sequence(p, 0.1, [0])[0] == (p[0] <= 0.1)


@pytest.mark.parametrize("grid", GRIDS)
def test_plugin_rule_reads_the_printed_risk(grid):
    """The plug-in rule keeps exactly the rows whose printed empirical risk
    k / n (the tables' R_hat column, re-derived from k and n as printed) is
    at most the budget; the reference (k = 0) is always kept."""
    rows = load(grid)
    V = [int(r["k"]) for r in rows]
    n = int(rows[0]["n"])
    for alpha, _ in BUDGETS:
        keep = rl.plugin(V, n, alpha)
        assert keep[ref_index(rows)]
        assert keep.tolist() == [Fraction(k, n) <= Fraction(alpha) for k in V]


def _matrix_with_k(rows):
    n = int(rows[0]["n"])
    c = np.ones((len(rows), n), dtype=np.uint8)
    for j, r in enumerate(rows):
        c[j, :int(r["k"])] = 0
    return c


def test_alpha_sweep_reproduces_unlock_table():
    """App. A.6 / §5 table: alpha_hat on the 0.01 budget grid and the gains at
    0.10, 0.15, 0.20 from one sweep per grid."""
    alphas = [i / 100 for i in range(1, 31)]
    for u in load("unlock"):
        rows = load(u["grid"])
        ref = ref_index(rows)
        tpf = [float(r["tpf"]) for r in rows]
        sel, nval, hat = rl.alpha_sweep(_matrix_with_k(rows), tpf, ref, alphas, 0.10)
        assert hat == pytest.approx(float(u["alpha_min"]))
        for ai in (10, 15, 20):
            gain = 100.0 * (tpf[sel[ai - 1]] / tpf[ref] - 1.0)
            assert abs(gain - float(u["gain%d" % ai])) <= 0.1 + 1e-9
        # the number valid never falls as the budget grows (p-values fall in alpha)
        assert all(a <= b for a, b in zip(nval, nval[1:]))


def test_alpha_sweep_bonferroni_example():
    """App. D.3 at alpha = 0.07: the sweep under Bonferroni deploys acc95/semi70
    where Holm deploys acc90/semi90."""
    rows = load("grid_llada2_math")
    tpf = [float(r["tpf"]) for r in rows]
    c = _matrix_with_k(rows)
    h, _, _ = rl.alpha_sweep(c, tpf, ref_index(rows), [0.07], 0.10, "holm")
    b, _, _ = rl.alpha_sweep(c, tpf, ref_index(rows), [0.07], 0.10, "bonferroni")
    assert (rows[h[0]]["config"], rows[b[0]]["config"]) == ("acc90/semi90", "acc95/semi70")


def _hyper(n, k, c, t):
    """Pr[t of the k marked prompts fall in a uniformly random c-subset of n]."""
    from math import comb
    return Fraction(comb(k, t) * comb(n - k, c - t), comb(n, c))


def test_split_exceedance_plugin_over_every_split():
    """Exhaustive half splits of n = 12 prompts, one candidate with k = 4
    violations: the plug-in rule deploys it iff t / 6 <= alpha for the t
    violations in the calibration half, and the test half then reads
    (4 - t) / 6.  The exceedance count over all C(12, 6) splits equals the
    hypergeometric sum."""
    from math import comb
    n, k, half, alpha = 12, 4, 6, 0.2
    correct = np.ones((2, n), dtype=np.uint8)
    correct[1, [1, 4, 7, 10]] = 0
    masks = []
    for cal in itertools.combinations(range(n), half):
        mk = np.zeros(n, dtype=np.uint8)
        mk[list(cal)] = 1
        masks.append(mk)
    r = rl.split_exceedance(correct, [1.0, 2.0], 0, alpha, 0.1, masks, method="plugin")
    want = sum(_hyper(n, k, half, t) for t in range(k + 1)
               if Fraction(t, half) <= Fraction(alpha) and Fraction(k - t, half) > Fraction(alpha))
    assert Fraction(r.exceed_test, comb(n, half)) == want
    # pooled risk 4/12 > 0.2: every deployment of the candidate exceeds it
    deployed = sum(_hyper(n, k, half, t) for t in range(k + 1) if Fraction(t, half) <= Fraction(alpha))
    assert Fraction(r.exceed_pooled, comb(n, half)) == deployed
    assert r.fwer_pooled == r.exceed_pooled
    assert r.gain_sum == pytest.approx(float(deployed * comb(n, half)))
    assert r.deployed.count(1) == int(deployed * comb(n, half))


def test_split_exceedance_holm_matches_hypergeometric_rate():
    """Random half splits of n = 400 prompts with one candidate of k = 52
    violations (risk 0.13 against alpha = 0.10): Holm deploys the candidate
    iff its calibration count t has Pr[Bin(200, 0.1) <= t] <= delta (the
    reference, with p = 0.9**200, is rejected first at delta / 2).  Over 600
    seeded splits the exceedance rate lies within 4 standard errors of the
    hypergeometric probability of {t <= t*, (k - t) / 200 > alpha}."""
    import bd_synth
    n, k, half, alpha, delta = 400, 52, 200, 0.10, 0.10
    correct = np.ones((2, n), dtype=np.uint8)
    correct[1, np.arange(0, 7 * k, 7)] = 0
    masks = bd_synth.split_masks(n, 600, 0.5, seed=3)
    r = rl.split_exceedance(correct, [1.0, 2.0], 0, alpha, delta, masks)
    tstar = max(t for t in range(half + 1) if rl.binom_pvalue(half, alpha, t) <= delta)
    rate = float(sum(_hyper(n, k, half, t) for t in range(k + 1)
                     if t <= tstar and Fraction(k - t, half) > Fraction(alpha)))
    se = (rate * (1 - rate) / len(masks)) ** 0.5
    assert abs(r.exceed_test / len(masks) - rate) <= 4 * se + 1e-12
    assert 0.0 < rate < 1.0


def test_monte_carlo_independent_bonferroni_matches_exact_rates():
    """Independent draws, Bonferroni: configuration j is valid with the exact
    probability Pr[Bin(n, r_j) <= v*] (v* the largest count with
    Pr[Bin(n, alpha) <= v*] <= delta / m), independently across j.  The Monte
    Carlo counts match within 4 standard errors."""
    import bd_synth
    risks = [0.02, 0.06, 0.11, 0.12]
    n, alpha, delta, trials = 300, 0.10, 0.20, 3000
    u = bd_synth.mc_uniforms(trials, len(risks), n, seed=5)
    false_trials, counts = rl.monte_carlo(risks, alpha, delta, u, method="bonferroni")
    vstar = max(v for v in range(n + 1) if rl.binom_pvalue(n, alpha, v) <= delta / len(risks))
    with mpmath.workdps(40):
        q = [float(sum(mpmath.binomial(n, i) * mpmath.mpf(r) ** i * (1 - mpmath.mpf(r)) ** (n - i)
                       for i in range(vstar + 1))) for r in risks]
    for j in range(len(risks)):
        se = (q[j] * (1 - q[j]) / trials) ** 0.5
        assert abs(counts[j] / trials - q[j]) <= 4 * se + 1e-12, (j, counts[j], q[j])
    fw = 1 - (1 - q[2]) * (1 - q[3])
    se = (fw * (1 - fw) / trials) ** 0.5
    assert abs(false_trials / trials - fw) <= 4 * se + 1e-12
    assert q[0] > 0.5 and 0.001 < fw < 0.2        # a powered test and a visible error rate


def test_monte_carlo_shared_holm_matches_multinomial_enumeration():
    """Shared uniforms make the violation counts nested: with risks sorted,
    V_j counts the prompts whose uniform falls below r_j, so the counts in the
    intervals between consecutive risks are multinomial.  Enumerating every
    multinomial outcome for n = 30 gives the exact family-wise error of Holm;
    the Monte Carlo estimate lies within 4 standard errors and below delta."""
    import bd_synth
    from math import factorial
    risks = [0.05, 0.25, 0.30]
    n, alpha, delta, trials = 30, 0.20, 0.10, 4000
    cuts = [0.0] + risks + [1.0]
    probs = [Fraction(cuts[i + 1]) - Fraction(cuts[i]) for i in range(len(cuts) - 1)]
    table = [rl.binom_pvalue(n, alpha, v) for v in range(n + 1)]
    exact = Fraction(0)
    for c0 in range(n + 1):
        for c1 in range(n + 1 - c0):
            for c2 in range(n + 1 - c0 - c1):
                c3 = n - c0 - c1 - c2
                V = [c0, c0 + c1, c0 + c1 + c2]
                valid = rl.holm([table[v] for v in V], delta)
                if valid[1] or valid[2]:
                    w = Fraction(factorial(n), factorial(c0) * factorial(c1) * factorial(c2) * factorial(c3))
                    exact += w * probs[0] ** c0 * probs[1] ** c1 * probs[2] ** c2 * probs[3] ** c3
    u = bd_synth.mc_uniforms(trials, 1, n, seed=6)
    false_trials, _ = rl.monte_carlo(risks, alpha, delta, u, method="holm")
    e = float(exact)
    se = (e * (1 - e) / trials) ** 0.5
    assert abs(false_trials / trials - e) <= 4 * se + 1e-12, (false_trials / trials, e)
    assert e <= delta and e > 0.005
