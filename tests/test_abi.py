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


def test_binding_structs_match_the_header(tmp_path):
    """The ctypes mirrors of bd_model_cfg and bd_decode_cfg have the sizes
    and field offsets the C compiler gives the header's structs."""
    import ctypes
    import subprocess
    from paper_2609_33887_amd import bd
    fields = {"bd_model_cfg": [f[0] for f in bd.bd_model_cfg._fields_],
              "bd_decode_cfg": [f[0] for f in bd.bd_decode_cfg._fields_]}
    lines = ['#include <stdio.h>', '#include <stddef.h>', '#include "bd.h"', "int main(void) {"]
    for t, fs in fields.items():
        lines.append(f'  printf("{t} %zu\\n", sizeof({t}));')
        for f in fs:
            lines.append(f'  printf("{t}.{f} %zu\\n", offsetof({t}, {f}));')
    lines.append("  return 0; }")
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines))
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe)], check=True)
    out = dict(l.split() for l in subprocess.run([str(exe)], check=True, capture_output=True,
                                                 text=True).stdout.splitlines())
    for t, fs in fields.items():
        cls = getattr(bd, t)
        assert int(out[t]) == ctypes.sizeof(cls), t
        for f in fs:
            assert int(out[f"{t}.{f}"]) == getattr(cls, f).offset, (t, f)


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


# ---- Redline variants and validity harness: library against the oracle ----

def _no_near_ties(p_oracle, delta, m):
    """True when no oracle p-value sits within 1e-9 (relative) of any
    threshold a procedure can compare it with."""
    thr = [delta / k for k in range(1, m + 1)]
    return all(abs(float(p) / t - 1.0) >= 1e-9 for p in p_oracle for t in thr)


def _planted_cases(seed, count):
    import bd_synth
    rng = np.random.default_rng(seed)
    for case in range(count):
        m = int(rng.integers(1, 12))
        n = int(rng.integers(30, 700))
        ref = int(rng.integers(0, m))
        risks = list(rng.uniform(0.0, 0.25, size=m))
        c = bd_synth.planted_correctness(n, risks, ref, seed=seed * 1000 + case, shared=bool(case % 2))
        cost = list(rng.choice([1.0, 2.0, 3.0, 4.5], size=m))
        order = list(rng.permutation(m))
        yield m, n, ref, c, cost, order, rng


@pytest.mark.parametrize("method", ["holm", "bonferroni", "fixed_sequence", "uncorrected", "plugin"])
def test_rl_select_matches_oracle(method):
    from paper_2609_33887_amd import bd
    from oracle import redline as rl
    for m, n, ref, c, cost, order, rng in _planted_cases(21, 40):
        alpha = float(rng.choice([0.05, 0.1, 0.15, 0.2]))
        delta = float(rng.choice([0.05, 0.1]))
        mask = (rng.random(n) < 0.6).astype(np.uint8) if rng.random() < 0.5 else None
        if mask is not None and mask.sum() == 0:
            mask[0] = 1
        V, p, valid, sel = bd.rl_select(c, cost, ref, alpha, delta, method, order, mask)
        o = rl.select(c, cost, ref, alpha, delta, method, order, mask)
        assert V.tolist() == o.V.tolist()
        for a, b in zip(p, o.p):
            assert abs(a - float(b)) <= 1e-11 * float(b) + 1e-300
        if method == "plugin" or _no_near_ties(o.p, delta, m):
            assert valid.tolist() == o.valid.tolist() and sel == o.selected


def test_rl_select_holm_equals_rl_risk_select():
    from paper_2609_33887_amd import bd
    for m, n, ref, c, cost, order, rng in _planted_cases(22, 20):
        a = bd.rl_risk_select(c, cost, ref, 0.1, 0.1)
        b = bd.rl_select(c, cost, ref, 0.1, 0.1, "holm")
        assert a[0].tolist() == b[0].tolist() and a[1].tolist() == b[1].tolist()
        assert a[2].tolist() == b[2].tolist() and a[3] == b[3]


def test_rl_alpha_sweep_matches_oracle_and_unlock_table():
    from paper_2609_33887_amd import bd
    from oracle import redline as rl
    from tests.test_oracle_redline import load, ref_index
    alphas = [i / 100 for i in range(1, 31)]
    for u in load("unlock"):
        rows = load(u["grid"])
        n = int(rows[0]["n"])
        c = np.ones((len(rows), n), dtype=np.uint8)
        for j, r in enumerate(rows):
            c[j, :int(r["k"])] = 0
        tpf = [float(r["tpf"]) for r in rows]
        for method in ("holm", "bonferroni"):
            sel, nval, hat = bd.rl_alpha_sweep(c, tpf, ref_index(rows), alphas[::-1], 0.10, method)
            osel, onval, ohat = rl.alpha_sweep(c, tpf, ref_index(rows), alphas[::-1], 0.10, method)
            assert sel.tolist() == osel and nval.tolist() == onval and hat == ohat
        _, _, hat = bd.rl_alpha_sweep(c, tpf, ref_index(rows), alphas, 0.10)
        assert hat == pytest.approx(float(u["alpha_min"]))
    # no configuration faster than the reference: alpha_hat is undefined
    c = np.ones((2, 50), dtype=np.uint8)
    _, _, hat = bd.rl_alpha_sweep(c, [3.0, 1.0], 0, alphas, 0.10)
    assert hat is None


@pytest.mark.parametrize("method", ["holm", "bonferroni", "fixed_sequence", "uncorrected", "plugin"])
def test_rl_split_exceedance_matches_oracle(method):
    import bd_synth
    from paper_2609_33887_amd import bd
    from oracle import redline as rl
    for case, (m, n, ref, c, cost, order, rng) in enumerate(_planted_cases(23, 6)):
        masks = bd_synth.split_masks(n, 150, cal_frac=float(rng.choice([0.3, 0.5, 0.7])), seed=case)
        alpha = float(rng.choice([0.05, 0.1, 0.15]))
        dep, tv, counts, gain = bd.rl_split_exceedance(c, cost, ref, alpha, 0.1, masks, method, order)
        o = rl.split_exceedance(c, cost, ref, alpha, 0.1, masks, method, order)
        assert dep.tolist() == o.deployed and tv.tolist() == o.test_violations
        assert counts.tolist() == [o.exceed_test, o.exceed_pooled, o.fwer_test, o.fwer_pooled]
        assert gain == o.gain_sum


@pytest.mark.parametrize("shared", [True, False])
@pytest.mark.parametrize("method", ["holm", "bonferroni", "fixed_sequence", "uncorrected", "plugin"])
def test_rl_monte_carlo_matches_oracle(method, shared):
    import bd_synth
    from paper_2609_33887_amd import bd
    from oracle import redline as rl
    risks = [0.01, 0.02, 0.07, 0.07, 0.07]             # App. A.7's configurations
    u = bd_synth.mc_uniforms(300, 1 if shared else len(risks), 800, seed=8)
    order = [0, 1, 2, 3, 4]
    ft, counts = bd.rl_monte_carlo(risks, 0.05, 0.10, u, method, order)
    oft, ocounts = rl.monte_carlo(risks, 0.05, 0.10, u, method, order)
    assert ft == oft and counts.tolist() == ocounts.tolist()


def test_redline_variants_reject_bad_arguments():
    from paper_2609_33887_amd import bd
    c = np.ones((3, 20), dtype=np.uint8)
    cost = [1.0, 2.0, 3.0]
    bad = [
        lambda: bd.rl_select(c, cost, 0, 0.1, 0.1, "fixed_sequence", None),          # no order
        lambda: bd.rl_select(c, cost, 0, 0.1, 0.1, "fixed_sequence", [0, 0, 1]),     # not a permutation
        lambda: bd.rl_select(c, cost, 0, 0.1, 0.1, "holm", None, np.zeros(20)),      # empty prompt set
        lambda: bd.rl_alpha_sweep(c, cost, 0, [0.1, 1.0], 0.1),                      # budget out of range
        lambda: bd.rl_split_exceedance(c, cost, 0, 0.1, 0.1, np.ones((2, 20))),      # no test prompts
        lambda: bd.rl_monte_carlo([0.1, 0.2, 0.3], 0.1, 0.1, np.zeros((4, 2, 20))),  # k neither 1 nor m
    ]
    for f in bad:
        with pytest.raises(bd.BDError) as e:
            f()
        assert e.value.status == bd.BD_EINVAL
        assert bd.bd_last_error().startswith("rl_")
    code = bd.lib.rl_select(20, 3, 0, c.ctypes.data_as(bd._u8), None,
                            np.asarray(cost).ctypes.data_as(bd._f64), 0.1, 0.1, 7, None, None, None, None,
                            bd.ctypes.byref(bd.ctypes.c_int32()))
    assert code == bd.BD_EINVAL and "unknown procedure" in bd.bd_last_error()


def test_weight_bytes_counts_every_tensor():
    """The weight-memory cost of the precision sweep against a count over
    the ABI tensor list: bf16 matrices 2 bytes, fp32 norms and router 4;
    with fp8 the decoder-layer projections take 1 byte plus a 4-byte scale
    per output row, with MXFP4 half a byte plus a 1-byte exponent per 32
    elements."""
    import numpy as np
    from bd_synth import Workload, tensor_specs
    from oracle.quant import quantized_layer_slots
    from paper_2609_33887_amd.sweep import weight_bytes
    for kw in (dict(ffn_dim=512), dict(ffn_dim=0, n_experts=8, top_k=2, expert_ffn=128, n_shared=1),
               dict(ffn_dim=0, n_experts=4, top_k=1, expert_ffn=128, n_shared=0)):
        w = Workload(name="wb", seed=1, n_layers=3, d_model=256, n_heads=4, n_kv_heads=2, head_dim=64,
                     vocab=1024, dtype="bf16", batch=1, prompt_len=8, block_size=4, n_inflight=1, gen_len=8,
                     **kw)
        specs = tensor_specs(w)
        slots = set(quantized_layer_slots(w))
        bf16 = fp8 = mx = 0
        for i, (name, shape, kind) in enumerate(specs):
            n = int(np.prod(shape))
            if n == 0:
                continue
            size = 4 * n if kind in ("norm", "router") else 2 * n
            bf16 += size
            fp8 += (n + 4 * (n // shape[-1])) if i in slots else size
            mx += (n // 2 + n // 32) if i in slots else size
        assert weight_bytes(w) == bf16
        assert weight_bytes(w, "fp8") == fp8
        assert weight_bytes(w, "mxfp4") == mx


def test_argument_errors_before_any_device_work():
    """Argument checks of the entry points that return before any HIP call
    (so they run without a GPU): fp8 quantization of a NULL or empty matrix,
    an unknown weight precision, fp8 weights on an fp32 model, and NULL
    handles."""
    import ctypes
    from paper_2609_33887_amd import bd
    from bd_synth import Workload
    lib = bd.lib
    assert lib.bd_quantize_fp8(None, 4, 4, None, None, None) == bd.BD_EINVAL
    assert lib.bd_quantize_fp8(ctypes.c_void_p(16), 0, 4, ctypes.c_void_p(16), ctypes.c_void_p(16),
                               None) == bd.BD_EINVAL
    assert "rows, cols" in bd.bd_last_error()
    w = Workload(name="e", seed=1, n_layers=1, d_model=256, n_heads=4, n_kv_heads=2, head_dim=64,
                 ffn_dim=512, vocab=1024, dtype="bf16", batch=1, prompt_len=8, block_size=4,
                 n_inflight=1, gen_len=8)
    out = ctypes.c_void_p()
    arr = (ctypes.c_void_p * 10)()
    cfg = bd.model_cfg_from(w)
    cfg.wq = 7
    assert lib.bd_init_model(ctypes.byref(cfg), arr, 10, None, ctypes.byref(out)) == bd.BD_EINVAL
    cfg.wq = bd.BD_WQ_FP8
    cfg.dtype = bd.BD_F32
    assert lib.bd_init_model(ctypes.byref(cfg), arr, 10, None, ctypes.byref(out)) == bd.BD_EUNSUPPORTED
    dc = bd.decode_cfg(0.9, 1, 4, skip_masked=True)
    assert lib.bd_prefill(None, None, 1, 8, 8, ctypes.byref(dc), ctypes.byref(out)) == bd.BD_EINVAL
    stats = (ctypes.c_int64 * 12)()
    assert lib.bd_state_stats(None, None, stats, 12) == bd.BD_EINVAL
