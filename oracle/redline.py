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

Secondary procedures of App. A.3/A.4 (Bonferroni, fixed sequence) are given
for comparison tests.
"""
from __future__ import annotations

import functools
from dataclasses import dataclass

import mpmath
import numpy as np

__all__ = ["violations", "binom_pvalue", "holm", "bonferroni", "fixed_sequence", "deploy",
           "risk_select", "SelectResult"]

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
