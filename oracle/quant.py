"""Oracle weight quantization (test infrastructure only; see ``oracle/__init__``).

The paper treats numeric precision as one axis of a serving configuration and
calibrates weight quantization against bf16 weights as the reference, with the
embeddings and the output head kept in bf16 (§4.2 (iv) and the quantization grid
of App. E).  The format here is the OCP fp8 E4M3 encoding that gfx950's
matrix cores read, with one power-of-two scale per output row:

* E4M3 (the "fn" variant: no infinities, 0x7F/0xFF are NaN): sign, 4 exponent
  bits with bias 7, 3 mantissa bits.  Normal numbers (1 + m/8) * 2**(e - 7)
  for e in 1..15 (largest finite value 448 = 1.75 * 2**8); subnormal numbers
  (m/8) * 2**-6 for e = 0, i.e. multiples of 2**-9 below 2**-6.
* Row scale 2**E with E the smallest integer such that max|w| / 2**E <= 448
  (E = 0 for an all-zero row), so no scaled value exceeds the format.
* Each scaled value w / 2**E (exact: a power-of-two division) is rounded to
  the nearest representable value, ties to the even mantissa; the quantized
  weight is code_value * 2**E, which a bf16 number holds exactly (8
  significant bits >= 4, and the exponents stay far inside bf16's range).

The MXFP4 format of the OCP microscaling specification is the second
low-precision candidate: blocks of 32 consecutive elements along a row share
one E8M0 scale 2**X, X = floor(log2(block max)) - 2 (2 is the largest E2M1
exponent), and each element is the E2M1 value (sign, 2 exponent bits with
bias 1, 1 mantissa bit: 0, 0.5, 1, 1.5, 2, 3, 4, 6) nearest to w / 2**X,
ties to the even mantissa, magnitudes above 6 saturating to 6.
"""
from __future__ import annotations

import math

import numpy as np

__all__ = ["e4m3_value", "e4m3_encode", "row_exponent", "row_exponents", "quantize_fp8_rows", "dequantize_fp8_rows",
           "quantized_layer_slots", "fp8_weights", "e2m1_value", "e2m1_encode", "mx_block_exponent",
           "quantize_mxfp4_rows", "dequantize_mxfp4_rows", "mxfp4_weights", "MX_BLOCK"]

E4M3_MAX = 448.0


def e4m3_value(code: np.ndarray) -> np.ndarray:
    """float64 value of E4M3 codes (uint8); NaN for the two NaN codes."""
    c = np.asarray(code, dtype=np.int64)
    s = np.where(c >> 7, -1.0, 1.0)
    e = (c >> 3) & 15
    m = (c & 7).astype(np.float64)
    mag = np.where(e == 0, m / 8.0 * 2.0 ** -6, (1.0 + m / 8.0) * np.ldexp(1.0, e - 7))
    mag = np.where((c & 0x7F) == 0x7F, np.nan, mag)
    return s * mag


def e4m3_encode(x: np.ndarray) -> np.ndarray:
    """Round float64 values with |x| <= 448 to the nearest E4M3 code (ties to
    even).  The spacing of representable values is 2**(floor(log2|x|) - 3) in
    the normal range and 2**-9 below 2**-6."""
    x = np.asarray(x, dtype=np.float64)
    if np.any(~np.isfinite(x)) or np.any(np.abs(x) > E4M3_MAX):
        raise ValueError("value outside the E4M3 range")
    a = np.abs(x)
    _, ex = np.frexp(a)                 # a = f * 2**ex, 0.5 <= f < 1  ->  floor(log2 a) = ex - 1
    quantum_exp = np.where(a >= 2.0 ** -6, (ex - 1) - 3, -9)
    q = np.ldexp(np.rint(np.ldexp(a, -quantum_exp)), quantum_exp)   # nearest, ties to even
    # encode the rounded magnitude (rounding may have moved it to the next binade)
    _, eq = np.frexp(q)
    normal = q >= 2.0 ** -6
    e_field = np.where(normal, (eq - 1) + 7, 0)
    m_field = np.where(normal, np.ldexp(q, -(eq - 1)) * 8.0 - 8.0, np.ldexp(q, 9))
    code = (e_field.astype(np.int64) << 3) | np.rint(m_field).astype(np.int64)
    code = np.where(x < 0, code | 0x80, code)
    return code.astype(np.uint8)


def row_exponent(amax: float) -> int:
    """Smallest integer E with amax / 2**E <= 448 (0 when amax is 0)."""
    if amax == 0.0:
        return 0
    e = math.ceil(math.log2(amax / E4M3_MAX))
    # guard the floating-point logarithm: step to the exact boundary
    while amax / 2.0 ** (e - 1) <= E4M3_MAX:
        e -= 1
    while amax / 2.0 ** e > E4M3_MAX:
        e += 1
    return e


def row_exponents(amax: np.ndarray) -> np.ndarray:
    """``row_exponent`` for an array: with amax = f * 2**x (0.5 <= f < 1),
    448 = 0.875 * 2**9 gives E = x - 9 when f <= 0.875, else x - 8."""
    f, x = np.frexp(np.asarray(amax, dtype=np.float64))
    return np.where(f == 0, 0, x - 9 + (f > 0.875)).astype(np.int64)


def quantize_fp8_rows(w: np.ndarray):
    """Quantize a matrix [rows][cols] row by row; returns (codes uint8
    [rows][cols], exponents int64 [rows])."""
    w = np.asarray(w, dtype=np.float64)
    exps = row_exponents(np.max(np.abs(w), axis=1))
    codes = e4m3_encode(np.ldexp(w, -exps[:, None]))
    return codes, exps


def dequantize_fp8_rows(codes: np.ndarray, exps: np.ndarray) -> np.ndarray:
    """code_value * 2**E per row, float64."""
    return np.ldexp(e4m3_value(codes), np.asarray(exps)[:, None])


def _as_float(t: np.ndarray) -> np.ndarray:
    t = np.asarray(t)
    if t.dtype == np.uint16:   # bf16 bit patterns
        return (t.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return t.astype(np.float64)


def quantized_layer_slots(cfg):
    """Indices, in the ABI weight order, of the matrices that fp8 quantization
    replaces: every decoder-layer projection (QKV, O, gate, up, down, and for
    MoE the expert and shared-expert matrices), not the embeddings, norms,
    router or LM head."""
    per = 7 if cfg.n_experts == 0 else 11
    mats = (1, 2, 4, 5, 6) if cfg.n_experts == 0 else (1, 2, 5, 6, 7, 8, 9, 10)
    return [1 + l * per + j for l in range(cfg.n_layers) for j in mats]


def fp8_weights(cfg, weights):
    """The weight list of the fp8 configuration: each quantized matrix
    replaced by its dequantized values (float32, exactly bf16 numbers),
    quantized row by row (an expert tensor [E][out][in] row by row of every
    expert)."""
    out = list(weights)
    for i in quantized_layer_slots(cfg):
        t = weights[i]
        if t is None:
            continue
        w = _as_float(t)
        rows = w.reshape(-1, w.shape[-1])
        codes, exps = quantize_fp8_rows(rows)
        out[i] = dequantize_fp8_rows(codes, exps).reshape(w.shape).astype(np.float32)
    return out


# ---------------------------------------------------------------- MXFP4
MX_BLOCK = 32
E2M1_MAX = 6.0


def e2m1_value(code: np.ndarray) -> np.ndarray:
    """float64 value of E2M1 codes (0..15): bit 3 sign, bits 2-1 exponent
    (bias 1), bit 0 mantissa; exponent 0 is subnormal (m * 0.5)."""
    c = np.asarray(code, dtype=np.int64)
    s = np.where(c >> 3, -1.0, 1.0)
    e = (c >> 1) & 3
    m = (c & 1).astype(np.float64)
    mag = np.where(e == 0, m * 0.5, (1.0 + m / 2.0) * np.ldexp(1.0, e - 1))
    return s * mag


def e2m1_encode(x: np.ndarray) -> np.ndarray:
    """Nearest E2M1 code (ties to even), magnitudes above 6 saturating to 6.
    The spacing is 2**(floor(log2|x|) - 1) from 1 up and 0.5 below."""
    x = np.asarray(x, dtype=np.float64)
    if np.any(~np.isfinite(x)):
        raise ValueError("non-finite value")
    a = np.abs(x)
    _, ex = np.frexp(a)
    quantum_exp = np.where(a >= 1.0, (ex - 1) - 1, -1)
    q = np.minimum(np.ldexp(np.rint(np.ldexp(a, -quantum_exp)), quantum_exp), E2M1_MAX)
    _, eq = np.frexp(q)
    normal = q >= 1.0
    e_field = np.where(normal, (eq - 1) + 1, 0)
    m_field = np.where(normal, np.ldexp(q, -(eq - 1)) * 2.0 - 2.0, q * 2.0)
    code = (e_field.astype(np.int64) << 1) | np.rint(m_field).astype(np.int64)
    code = np.where(x < 0, code | 8, code)
    return code.astype(np.uint8)


def mx_block_exponent(amax: np.ndarray) -> np.ndarray:
    """Shared scale exponent of MX blocks: floor(log2(amax)) - 2; -127 (the
    smallest E8M0 scale) for an all-zero block."""
    f, x = np.frexp(np.asarray(amax, dtype=np.float64))
    return np.where(f == 0, -127, (x - 1) - 2).astype(np.int64)


def quantize_mxfp4_rows(w: np.ndarray):
    """Quantize a matrix [rows][cols] (cols a multiple of 32) in MX blocks of
    32 consecutive columns; returns (codes uint8 [rows][cols], exponents
    int64 [rows][cols / 32])."""
    w = np.asarray(w, dtype=np.float64)
    rows, cols = w.shape
    if cols % MX_BLOCK:
        raise ValueError("columns must be a multiple of the MX block")
    blocks = w.reshape(rows, cols // MX_BLOCK, MX_BLOCK)
    exps = mx_block_exponent(np.max(np.abs(blocks), axis=2))
    codes = e2m1_encode(np.ldexp(blocks, -exps[:, :, None]))
    return codes.reshape(rows, cols), exps


def dequantize_mxfp4_rows(codes: np.ndarray, exps: np.ndarray) -> np.ndarray:
    rows, cols = codes.shape
    v = e2m1_value(codes).reshape(rows, cols // MX_BLOCK, MX_BLOCK)
    return np.ldexp(v, np.asarray(exps)[:, :, None]).reshape(rows, cols)


def mxfp4_weights(cfg, weights):
    """The weight list of the MXFP4 configuration: the layer projections of
    ``quantized_layer_slots`` replaced by their dequantized MXFP4 values
    (float32, exactly bf16 numbers), blocks running along each row."""
    out = list(weights)
    for i in quantized_layer_slots(cfg):
        t = weights[i]
        if t is None:
            continue
        w = _as_float(t)
        rows = w.reshape(-1, w.shape[-1])
        codes, exps = quantize_mxfp4_rows(rows)
        out[i] = dequantize_mxfp4_rows(codes, exps).reshape(w.shape).astype(np.float32)
    return out
