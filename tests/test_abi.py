"""CPU checks of the C ABI: the library loads, exports every declared entry
point, and the host-only Redline selection matches the oracle bit for bit
on integer counts, valid sets and the selected index."""
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    src = open(os.path.join(ROOT, "include", "bd.h")).read()
    return sorted(set(re.findall(r"^\s*(?:bd_status|const char\*)\s+(\w+)\s*\(", src, re.M)))


def test_library_exports_every_declared_symbol():
    import ctypes
    from paper_2609_33887_amd import bd
    names = _declared()
    assert "bd_denoise_step" in names and "rl_risk_select" in names
    lib = ctypes.CDLL(bd.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n
    assert sorted(bd.EXPORTED) == names


def test_redline_matches_oracle_on_paper_tables():
    from paper_2609_33887_amd import bd
    from oracle import redline as rl
    from tests.test_oracle_redline import GRIDS, BUDGETS, load, ref_index
    for grid in GRIDS:
        rows = load(grid)
        n = int(rows[0]["n"])
        m = len(rows)
        ref = ref_index(rows)
        # build a correctness matrix with exactly k violations per row
        correct = np.ones((m, n), dtype=np.uint8)
        for j, r in enumerate(rows):
            correct[j, :int(r["k"])] = 0
        tpf = [float(r["tpf"]) for r in rows]
        for alpha, col in BUDGETS:
            V, p, valid, sel, near = bd.rl_risk_select(correct, tpf, ref, alpha, 0.10)
            o = rl.risk_select(correct, tpf, ref, alpha, 0.10)
            assert V.tolist() == o.V.tolist()
            assert valid.tolist() == o.valid.tolist()
            assert sel == o.selected
            assert near == 0
            for a, b in zip(p, o.p):
                assert abs(a - float(b)) <= 1e-12 * float(b) + 1e-300


def test_redline_matches_oracle_on_random_matrices():
    from paper_2609_33887_amd import bd
    from oracle import redline as rl
    rng = np.random.default_rng(7)
    for trial in range(60):
        m = int(rng.integers(1, 14))
        n = int(rng.integers(1, 400))
        risk = rng.uniform(0, 0.3, size=m)
        ref_i = int(rng.integers(0, m))
        base = (rng.uniform(size=n) < 0.8).astype(np.uint8)
        correct = np.array([base & (rng.uniform(size=n) >= r) for r in risk], dtype=np.uint8)
        correct[ref_i] = base
        cost = rng.choice([1.0, 2.0, 3.0, 4.0], size=m)            # ties on purpose
        alpha = float(rng.choice([0.05, 0.1, 0.15, 0.2]))
        delta = float(rng.choice([0.05, 0.1]))
        V, p, valid, sel, near = bd.rl_risk_select(correct, cost, ref_i, alpha, delta)
        o = rl.risk_select(correct, cost, ref_i, alpha, delta)
        assert V.tolist() == o.V.tolist()
        if near == 0:
            assert valid.tolist() == o.valid.tolist() and sel == o.selected
        for a, b in zip(p, o.p):
            assert abs(a - float(b)) <= 1e-11 * float(b) + 1e-300


def test_redline_rejects_bad_arguments():
    from paper_2609_33887_amd import bd
    ok = np.ones((2, 5), dtype=np.uint8)
    for args in ((ok, [1, 2], 2, 0.1, 0.1), (ok, [1, 2], 0, 0.0, 0.1), (ok, [1, 2], 0, 0.1, 0.0),
                 (ok, [1, 2], -1, 0.1, 0.1), (ok, [1, 2], 0, 1.0, 0.1)):
        with pytest.raises(bd.BDError) as e:
            bd.rl_risk_select(*args)
        assert e.value.status == bd.BD_EINVAL
        assert "rl_risk_select" in bd.bd_last_error()


def test_redline_nothing_valid_deploys_reference():
    from paper_2609_33887_amd import bd
    correct = np.zeros((3, 40), dtype=np.uint8)
    correct[0] = 1                       # reference right everywhere, others wrong everywhere
    V, p, valid, sel, _ = bd.rl_risk_select(correct, [1.0, 5.0, 9.0], 0, 0.1, 0.1)
    assert V.tolist() == [0, 40, 40] and valid.tolist() == [True, False, False] and sel == 0
    correct[0] = 0                       # reference wrong everywhere: no violations anywhere
    V, p, valid, sel, _ = bd.rl_risk_select(correct, [1.0, 5.0, 9.0], 0, 0.1, 0.1)
    assert V.tolist() == [0, 0, 0] and sel == 2
