"""Oracle for Redline's selection (test infrastructure only; see ``oracle/__init__``).

Follows §4.2 steps (i)-(iv) and App. A:

* (ii) violation count V = number of calibration prompts that the reference
  answers correctly and the candidate does not (the empirical form of the
  reference-relative risk of Eq. 1, App. A.1);
* exact binomial p-value p = Pr[Bin(n, alpha) <= V] (App. A.2), evaluated here
  as an exact sum in 80-digit arithmetic;
* (iii) Holm step-down at family-wise level delta (App. A.3): sort p
  ascending, reject while p_(i) <= delta / (m - i + 1), stop at the first
  failure; the rejected hypotheses are the valid configurations;
* (iv) deploy the valid configuration with the largest cost measure (TPF),
  or the reference when none is valid (App. A.5 and the baselines of App. D).

Variants and the validity harness:

* the other procedures of App. A.3 and the baselines of App. D: Bonferroni
  (p <= delta / m), the fixed-sequence walk (a data-independent order tested
  at full delta until the first failure), the uncorrected exact test
  (p <= delta for every configuration) and the plug-in rule (R_hat <= alpha);
* the budget sweep and its smallest budget with a gain, alpha_hat (App. A.6:
  the smallest grid budget at which a configuration with a larger cost measure
  than the reference is valid);
* split-half exceedance (§5 and App. D): select on a calibration half, score
  the deployed configuration -- and every valid one -- on the other half and
  against the risk pooled over all prompts;
* the synthetic Monte Carlo with known risks (App. A.7): losses are drawn as
  u < r from prompt-level uniforms, shared across configurations or drawn
  independently, and the family-wise error is the share of trials in which a
  configuration with true risk above alpha is declared valid.

Random numbers (split masks, uniforms) are inputs, drawn by the callers.
"""
from __future__ import annotations

import functools
from dataclasses import dataclass

import mpmath
import numpy as np

__all__ = ["violations", "binom_pvalue", "holm", "bonferroni", "fixed_sequence", "uncorrected",
           "plugin", "deploy", "risk_select", "select", "SelectResult", "METHODS", "alpha_sweep",
           "split_exceedance", "SplitResult", "monte_carlo"]

# procedure codes (the same numbering as the library's)
METHODS = {"holm": 0, "bonferroni": 1, "fixed_sequence": 2, "uncorrected": 3, "plugin": 4}

_DPS = 80


def violations(correct: np.ndarray, ref_index: int) -> np.ndarray:
    """V_lambda = sum_i [ref correct on i] and [lambda incorrect on i].
    ``correct`` is [m][n] of 0/1."""
    c = np.asarray(correct).astype(bool)
    ref = c[ref_index]
    return np.array([int(np.count_nonzero(ref & ~c[j])) for j in range(c.shape[0])], dtype=np.int64)


@functools.lru_cache(maxsize=64)
def _cdf_table(n: int, alpha: float):
    """Cumulative sums of the Bin(n, alpha) probabilities, term by term."""
    with mpmath.workdps(_DPS):
        a = mpmath.mpf(alpha)
        b = 1 - a
        out, total = [], mpmath.mpf(0)
        for j in range(0, n + 1):
            total += mpmath.binomial(n, j) * a ** j * b ** (n - j)
            out.append(+total)
        return out


def binom_pvalue(n: int, alpha: float, v: int) -> mpmath.mpf:
    """Pr[Bin(n, alpha) <= v] = sum_{j<=v} C(n, j) alpha^j (1-alpha)^(n-j).
    ``alpha`` is taken at its exact binary value."""
    if v < 0:
        return mpmath.mpf(0)
    return _cdf_table(int(n), float(alpha))[min(int(v), int(n))]


def holm(p, delta: float) -> np.ndarray:
    """Holm step-down; returns a boolean 'rejected' (valid) mask.
    Equal p-values keep index order (this cannot change the rejected set,
    because the thresholds are non-decreasing in rank)."""
    m = len(p)
    order = sorted(range(m), key=lambda j: (p[j], j))
    valid = np.zeros(m, dtype=bool)
    with mpmath.workdps(_DPS):
        d = mpmath.mpf(delta)
        for i, j in enumerate(order, start=1):
            if mpmath.mpf(p[j]) <= d / (m - i + 1):
                valid[j] = True
            else:
                break
    return valid


def bonferroni(p, delta: float) -> np.ndarray:
    m = len(p)
    with mpmath.workdps(_DPS):
        d = mpmath.mpf(delta)
        return np.array([mpmath.mpf(x) <= d / m for x in p], dtype=bool)


def fixed_sequence(p, delta: float, order) -> np.ndarray:
    """Test in a data-independent order at full delta until the first failure."""
    valid = np.zeros(len(p), dtype=bool)
    with mpmath.workdps(_DPS):
        d = mpmath.mpf(delta)
        for j in order:
            if mpmath.mpf(p[j]) <= d:
                valid[j] = True
            else:
                break
    return valid


def uncorrected(p, delta: float) -> np.ndarray:
    """Each configuration tested alone at level delta (no multiplicity
    correction; a baseline of App. D)."""
    with mpmath.workdps(_DPS):
        d = mpmath.mpf(delta)
        return np.array([mpmath.mpf(x) <= d for x in p], dtype=bool)


def plugin(V, n: int, alpha: float) -> np.ndarray:
    """Plug-in rule R_hat = V / n <= alpha (no finite-sample margin; a baseline
    of App. D).  The ratio is formed and compared in double precision."""
    return np.array([float(v) / float(n) <= alpha for v in V], dtype=bool)


def deploy(cost, valid, ref_index: int) -> int:
    """Largest cost among valid configurations, lowest index among equals;
    the reference when nothing is valid."""
    best = -1
    for j in range(len(cost)):
        if valid[j] and (best < 0 or cost[j] > cost[best]):
            best = j
    return ref_index if best < 0 else best


@dataclass
class SelectResult:
    V: np.ndarray
    p: list
    valid: np.ndarray
    selected: int


def risk_select(correct: np.ndarray, cost, ref_index: int, alpha: float, delta: float) -> SelectResult:
    correct = np.asarray(correct)
    n = correct.shape[1]
    V = violations(correct, ref_index)
    p = [binom_pvalue(n, alpha, int(v)) for v in V]
    valid = holm(p, delta)
    return SelectResult(V, p, valid, deploy(cost, valid, ref_index))


def _valid(method: str, p, V, n: int, alpha: float, delta: float, order) -> np.ndarray:
    if method == "holm":
        return holm(p, delta)
    if method == "bonferroni":
        return bonferroni(p, delta)
    if method == "fixed_sequence":
        return fixed_sequence(p, delta, order)
    if method == "uncorrected":
        return uncorrected(p, delta)
    if method == "plugin":
        return plugin(V, n, alpha)
    raise ValueError(method)


def select(correct: np.ndarray, cost, ref_index: int, alpha: float, delta: float,
           method: str = "holm", order=None, mask=None) -> SelectResult:
    """Steps (ii)-(iv) with any of the procedures, on the prompts where
    ``mask`` is true (all prompts when None)."""
    correct = np.asarray(correct)
    if mask is not None:
        correct = correct[:, np.asarray(mask).astype(bool)]
    n = correct.shape[1]
    V = violations(correct, ref_index)
    p = [binom_pvalue(n, alpha, int(v)) for v in V]
    valid = _valid(method, p, V, n, alpha, delta, order)
    return SelectResult(V, p, valid, deploy(cost, valid, ref_index))


def alpha_sweep(correct, cost, ref_index: int, alphas, delta: float, method: str = "holm",
                order=None):
    """Selection at every budget of ``alphas``.  Returns (selected, n_valid,
    alpha_hat) where alpha_hat is the smallest budget at which some valid
    configuration has a larger cost measure than the reference (None if no
    budget has one)."""
    sel, nval, hat = [], [], None
    for a in alphas:
        r = select(correct, cost, ref_index, a, delta, method, order)
        sel.append(r.selected)
        nval.append(int(r.valid.sum()))
        if any(r.valid[j] and cost[j] > cost[ref_index] for j in range(len(cost))):
            hat = a if hat is None else min(hat, a)
    return sel, nval, hat


@dataclass
class SplitResult:
    deployed: list        # per split
    test_violations: list # per split: violations of the deployed configuration on the test half
    exceed_test: int      # splits whose deployed configuration has test-half R > alpha
    exceed_pooled: int    # ... pooled R (all n prompts) > alpha
    fwer_test: int        # splits with any valid configuration at test-half R > alpha
    fwer_pooled: int      # ... pooled R > alpha
    gain_sum: float       # sum over splits of cost[deployed] / cost[ref] - 1


def split_exceedance(correct, cost, ref_index: int, alpha: float, delta: float, cal_masks,
                     method: str = "holm", order=None) -> SplitResult:
    """For each calibration mask: select on the calibration prompts, then
    measure risks R = V / n_prompts on the complementary test prompts and on
    all prompts (ratios and comparisons in double precision)."""
    correct = np.asarray(correct)
    n = correct.shape[1]
    V_all = violations(correct, ref_index)
    out = SplitResult([], [], 0, 0, 0, 0, 0.0)
    for cal in cal_masks:
        cal = np.asarray(cal).astype(bool)
        r = select(correct, cost, ref_index, alpha, delta, method, order, mask=cal)
        test = ~cal
        V_test = violations(correct[:, test], ref_index)
        n_test = int(test.sum())
        r_test = [float(v) / float(n_test) for v in V_test]
        r_pool = [float(v) / float(n) for v in V_all]
        d = r.selected
        out.deployed.append(d)
        out.test_violations.append(int(V_test[d]))
        out.exceed_test += r_test[d] > alpha
        out.exceed_pooled += r_pool[d] > alpha
        out.fwer_test += any(r.valid[j] and r_test[j] > alpha for j in range(len(cost)))
        out.fwer_pooled += any(r.valid[j] and r_pool[j] > alpha for j in range(len(cost)))
        out.gain_sum += float(cost[d]) / float(cost[ref_index]) - 1.0
    return out


def monte_carlo(true_risk, alpha: float, delta: float, u, method: str = "holm", order=None):
    """App. A.7.  ``u`` is [trials][k][n] uniforms with k = 1 (one uniform per
    prompt shared by every configuration) or k = m (independent draws).  In
    trial t configuration j loses prompt i when u[t][j or 0][i] < true_risk[j];
    its violation count is its number of losses.  Returns (false_trials,
    valid_counts): the trials in which some configuration with true risk
    above alpha is valid, and per configuration the trials in which it is."""
    u = np.asarray(u)
    m = len(true_risk)
    n = u.shape[2]
    false_trials, counts = 0, np.zeros(m, dtype=np.int64)
    for t in range(u.shape[0]):
        V = [int(np.count_nonzero(u[t, 0 if u.shape[1] == 1 else j] < true_risk[j])) for j in range(m)]
        p = [binom_pvalue(n, alpha, v) for v in V]
        valid = _valid(method, p, V, n, alpha, delta, order)
        counts += valid
        false_trials += any(valid[j] and true_risk[j] > alpha for j in range(m))
    return false_trials, counts
