"""Pins of the oracle's fp8 weight quantization (E4M3 with a power-of-two
scale per output row) against the format's own definition and an
independent library conversion."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle.quant import (e4m3_value, e4m3_encode, row_exponent, row_exponents, quantize_fp8_rows,
                          dequantize_fp8_rows)


def _torch_codes(x):
    return torch.tensor(np.asarray(x, dtype=np.float32)).to(torch.float8_e4m3fn).view(torch.uint8).numpy()


def test_every_code_decodes_like_torch_and_round_trips():
    codes = np.arange(256, dtype=np.uint8)
    ours = e4m3_value(codes)
    ref = torch.tensor(codes).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    nan = np.isnan(ref)
    assert nan.sum() == 2 and np.array_equal(np.isnan(ours), nan)
    np.testing.assert_array_equal(ours[~nan], ref[~nan])
    finite = codes[~nan]
    back = e4m3_encode(e4m3_value(finite))
    # -0 and +0 both encode; compare values, then the codes of the non-zeros
    np.testing.assert_array_equal(e4m3_value(back), e4m3_value(finite))
    nz = e4m3_value(finite) != 0
    np.testing.assert_array_equal(back[nz], finite[nz])
    assert np.nanmax(ours) == 448.0 and ours[1] == 2.0 ** -9


def test_midpoints_round_to_even_mantissa():
    """Every midpoint between neighbouring non-negative values goes to the
    neighbour with the even code; points just off the midpoint go to the
    nearer one."""
    vals = np.sort(np.unique(e4m3_value(np.arange(0, 127, dtype=np.uint8))))
    lo, hi = vals[:-1], vals[1:]
    mid = (lo + hi) / 2
    got = e4m3_encode(mid)
    lo_c, hi_c = e4m3_encode(lo), e4m3_encode(hi)
    want = np.where(lo_c % 2 == 0, lo_c, hi_c)
    np.testing.assert_array_equal(got, want)
    eps = (hi - lo) * 1e-6
    np.testing.assert_array_equal(e4m3_encode(mid - eps), lo_c)
    np.testing.assert_array_equal(e4m3_encode(mid + eps), hi_c)
    np.testing.assert_array_equal(e4m3_encode(-mid), got | 0x80)


def test_encode_matches_torch_on_random_values():
    rng = np.random.default_rng(7)
    x = np.concatenate([rng.uniform(-448, 448, 20000), rng.normal(0, 0.01, 20000),
                        rng.normal(0, 1e-3, 5000)]).astype(np.float32).astype(np.float64)
    ours = e4m3_encode(x)
    ref = _torch_codes(x)
    zero = e4m3_value(ours) == 0
    np.testing.assert_array_equal(ours[~zero], ref[~zero])
    assert np.all(e4m3_value(ref[zero]) == 0)


def test_row_exponent_is_the_smallest_fitting_power():
    rng = np.random.default_rng(8)
    for a in np.concatenate([rng.uniform(1e-6, 1e3, 2000), [448.0, 224.0, 448.0 * 2 ** -12, 1.0, 0.875]]):
        e = row_exponent(float(a))
        assert a / 2.0 ** e <= 448.0 < a / 2.0 ** (e - 1)
        assert row_exponents(np.array([a]))[0] == e
    assert row_exponent(0.0) == 0 and row_exponents(np.zeros(1))[0] == 0


def test_quantize_rows_bounds_and_exact_bf16():
    """Per-row quantization of bf16-valued weights: each element lies within
    half a spacing of its value, the row maximum fits, and every dequantized
    weight is an exact bf16 number."""
    from oracle.model import round_bf16
    rng = np.random.default_rng(9)
    w = round_bf16(rng.normal(0, 0.02, (64, 256)))
    w[3] = 0.0
    codes, exps = quantize_fp8_rows(w)
    dq = dequantize_fp8_rows(codes, exps)
    assert exps[3] == 0 and np.all(dq[3] == 0)
    np.testing.assert_array_equal(round_bf16(dq), dq)
    scaled = np.ldexp(w, -exps[:, None])
    assert np.max(np.abs(scaled)) <= 448.0
    a = np.abs(scaled)
    spacing = np.where(a >= 2.0 ** -6, np.ldexp(1.0, np.floor(np.log2(np.maximum(a, 1e-300))).astype(int) - 3),
                       2.0 ** -9)
    assert np.all(np.abs(np.ldexp(dq, -exps[:, None]) - scaled) <= spacing / 2 + 1e-18)
    # relative error of the format: at most 2**-4 of the value in the normal range
    big = a >= 2.0 ** -6
    assert np.all(np.abs(dq - w)[big] <= np.abs(w)[big] * 2.0 ** -4)


def test_fp8_weights_replace_exactly_the_layer_projections():
    """The fp8 configuration quantizes every decoder-layer projection and
    leaves the embeddings, norms, router and LM head as they are (the paper
    keeps embeddings and output head in bf16)."""
    from bd_synth import Workload, make_weights, tensor_specs
    from oracle.quant import fp8_weights, quantized_layer_slots
    for kw in (dict(ffn_dim=256), dict(ffn_dim=0, n_experts=4, top_k=2, expert_ffn=128, n_shared=1)):
        w = Workload(name="q", seed=3, n_layers=2, d_model=128, n_heads=2, n_kv_heads=1, head_dim=64,
                     vocab=256, dtype="bf16", batch=1, prompt_len=8, block_size=4, n_inflight=1,
                     gen_len=8, **kw)
        ws = make_weights(w)
        q = fp8_weights(w, ws)
        names = [n for n, _, _ in tensor_specs(w)]
        slots = set(quantized_layer_slots(w))
        for i, (n, a, b) in enumerate(zip(names, ws, q)):
            base = n.split(".")[-1]
            expect = base.startswith("w_") and base != "w_router"
            assert (i in slots) == expect, n
            fa = (np.asarray(a).astype(np.uint32) << 16).view(np.float32) if np.asarray(a).dtype == np.uint16 else a
            if i in slots:
                assert b.dtype == np.float32 and b.shape == fa.shape
                assert not np.array_equal(b, fa)
                # per output row: within 2**-4 relative, or half the subnormal
                # spacing 2**(E - 10) of that row's scale
                rows = fa.reshape(-1, fa.shape[-1]).astype(np.float64)
                e = np.array([row_exponent(float(m)) for m in np.max(np.abs(rows), axis=1)])
                bound = np.maximum(np.abs(rows) * 2.0 ** -4, np.ldexp(1.0, e - 10)[:, None])
                assert np.all(np.abs(b.reshape(rows.shape) - rows) <= bound)
            else:
                assert b is a


# ---------------------------------------------------------------- MXFP4
E2M1_MAGNITUDES = [0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0]   # the format's value set


def test_e2m1_codes_are_the_format_values():
    from oracle.quant import e2m1_value
    v = e2m1_value(np.arange(16))
    np.testing.assert_array_equal(v[:8], E2M1_MAGNITUDES)
    np.testing.assert_array_equal(v[8:], [-m for m in E2M1_MAGNITUDES])


def _nearest_code(x):
    """Exhaustive search: the magnitude nearest |x| after saturation at 6,
    the even code on a tie, then the sign bit."""
    a = min(abs(x), 6.0)
    d = [abs(a - m) for m in E2M1_MAGNITUDES]
    best = min(d)
    cands = [i for i, di in enumerate(d) if di == best]
    code = cands[0] if len(cands) == 1 else next(i for i in cands if i % 2 == 0)
    return code | (8 if x < 0 else 0)


def test_e2m1_encode_matches_exhaustive_nearest_search():
    from oracle.quant import e2m1_encode
    grid = np.concatenate([np.arange(-9.0, 9.0, 0.03125), np.arange(-9.0, 9.0, 0.0137),
                           np.random.default_rng(3).normal(0, 3, 4000), [0.25, 0.75, 1.25, 2.5, 3.5, 5.0, 7.0]])
    got = e2m1_encode(grid)
    want = np.array([_nearest_code(float(x)) for x in grid], dtype=np.uint8)
    # the sign of zero is free: compare values where the result is zero
    from oracle.quant import e2m1_value
    zero = e2m1_value(want) == 0
    np.testing.assert_array_equal(got[~zero], want[~zero])
    assert np.all(e2m1_value(got[zero]) == 0)


def test_mx_block_scale_and_saturation():
    """The shared exponent puts the block maximum in [4, 8) (so it codes to
    4, 6 or saturates to 6); an all-zero block takes the smallest scale."""
    from oracle.quant import mx_block_exponent, quantize_mxfp4_rows, dequantize_mxfp4_rows, e2m1_value
    rng = np.random.default_rng(4)
    amax = np.abs(rng.normal(0, 1, 5000)) + 1e-12
    e = mx_block_exponent(amax)
    r = amax / np.ldexp(1.0, e)
    assert np.all((r >= 4) & (r < 8))
    assert mx_block_exponent(np.zeros(1))[0] == -127
    w = rng.normal(0, 0.02, (16, 128))
    w[3, 32:64] = 0.0
    codes, exps = quantize_mxfp4_rows(w)
    assert exps.shape == (16, 4) and exps[3, 1] == -127
    dq = dequantize_mxfp4_rows(codes, exps)
    scaled = np.abs(w.reshape(16, 4, 32)) / np.ldexp(1.0, exps)[:, :, None]
    vals = np.abs(e2m1_value(codes)).reshape(16, 4, 32)
    # within half a spacing of the scaled value, or saturated at 6
    spacing = np.where(scaled >= 4, 2.0, np.where(scaled >= 2, 1.0, 0.5))
    ok = (np.abs(vals - scaled) <= spacing / 2 + 1e-12) | ((scaled > 6) & (vals == 6))
    assert np.all(ok)
    assert np.all(np.abs(dq) <= 6 * np.ldexp(1.0, np.repeat(exps, 32, axis=1)))


def test_mxfp4_weights_are_exact_bf16_and_touch_only_layer_projections():
    from bd_synth import Workload, make_weights
    from oracle.model import round_bf16
    from oracle.quant import mxfp4_weights, quantized_layer_slots
    w = Workload(name="mx", seed=5, n_layers=2, d_model=128, n_heads=2, n_kv_heads=1, head_dim=64,
                 ffn_dim=256, vocab=256, dtype="bf16", batch=1, prompt_len=8, block_size=4, n_inflight=1,
                 gen_len=8)
    ws = make_weights(w)
    q = mxfp4_weights(w, ws)
    slots = set(quantized_layer_slots(w))
    for i, (a, b) in enumerate(zip(ws, q)):
        if i in slots:
            assert b.dtype == np.float32
            np.testing.assert_array_equal(round_bf16(b.astype(np.float64)), b.astype(np.float64))
        else:
            assert b is a


def test_planted_mxfp4_mistakes_are_caught(monkeypatch):
    """Ties away from zero, a scale one binade too large, and no saturation
    are each caught by the pins above."""
    import oracle.quant as oq
    good_enc, good_exp = oq.e2m1_encode, oq.mx_block_exponent

    def enc_ties_away(x):
        x = np.asarray(x, dtype=np.float64)
        a = np.abs(x)
        _, ex = np.frexp(a)
        qe = np.where(a >= 1.0, ex - 2, -1)
        q = np.minimum(np.ldexp(np.floor(np.ldexp(a, -qe) + 0.5), qe), 6.0)
        return good_enc(np.where(x < 0, -q, q))

    def exp_one_up(amax):
        return good_exp(amax) + 1

    def enc_no_saturation(x):
        x = np.asarray(x, dtype=np.float64)
        if np.any(np.abs(x) > 6.5):
            raise ValueError("out of range")
        return good_enc(x)

    checks = [test_e2m1_encode_matches_exhaustive_nearest_search, test_mx_block_scale_and_saturation]
    for name, fn in (("e2m1_encode", enc_ties_away), ("mx_block_exponent", exp_one_up),
                     ("e2m1_encode", enc_no_saturation)):
        monkeypatch.setattr(oq, name, fn)
        caught = False
        for chk in checks:
            try:
                chk()
            except (AssertionError, ValueError):
                caught = True
        monkeypatch.setattr(oq, name, good_enc if name == "e2m1_encode" else good_exp)
        assert caught, f"planted mistake in {name} went unnoticed"
