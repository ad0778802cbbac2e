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
    """App. D.2: on LLaDA2 math at alpha = 0.07, acc90/semi90 (p = 0.0190)
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
    """App. D.2: the math deployments at alpha = 0.10 survive delta = 0.05 and 0.01."""
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
