"""ctypes binding of ``libbd.so`` (argument marshalling only).

The functions keep the C names and argument order of ``include/bd.h``; device
pointers are plain integers (``tensor.data_ptr()``).  PyTorch is used by the
helpers at the bottom only to allocate device memory and to name the stream.
No computation of the decoding path happens in Python, and there is no
fallback: importing this module fails loudly when the library is missing.
"""
from __future__ import annotations

import ctypes
import os
from typing import Sequence

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libbd.so")

BD_OK, BD_EINVAL, BD_ENOMEM, BD_EHIP, BD_ESTATE, BD_EUNSUPPORTED = 0, -1, -2, -3, -4, -5
BD_F32, BD_BF16 = 0, 1

EXPORTED = ["bd_init_model", "bd_quantize_fp8", "bd_quantize_mxfp4", "bd_prefill", "bd_denoise_step", "bd_commit", "bd_state_read",
            "bd_decode", "bd_decode_static", "bd_state_reset", "bd_state_steps", "bd_state_stats", "bd_profile",
            "bd_profile_read", "bd_plan_projection", "bd_state_free", "bd_model_free", "bd_last_error", "rl_risk_select",
            "rl_select", "rl_alpha_sweep", "rl_split_exceedance", "rl_monte_carlo"]
RL_METHODS = {"holm": 0, "bonferroni": 1, "fixed_sequence": 2, "uncorrected": 3, "plugin": 4}
PROF_KINDS = ["embed", "norm", "gemm_qkv", "rope", "attn", "gemm_o", "gemm_gu", "gemm_down", "lm_head",
              "commit", "moe_route"]


class bd_model_cfg(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("n_layers", "d_model", "n_heads", "n_kv_heads", "head_dim",
                                              "ffn_dim", "vocab", "n_experts", "top_k", "expert_ffn",
                                              "n_shared")] + \
               [("rms_eps", ctypes.c_float), ("rope_theta", ctypes.c_float), ("logit_scale", ctypes.c_float),
                ("mask_id", ctypes.c_int32), ("dtype", ctypes.c_int32), ("wq", ctypes.c_int32)]


BD_WQ_NONE, BD_WQ_FP8, BD_WQ_MXFP4 = 0, 1, 2
WQ = {None: BD_WQ_NONE, "bf16": BD_WQ_NONE, "fp8": BD_WQ_FP8, "mxfp4": BD_WQ_MXFP4}
MX_BLOCK = 32


class bd_decode_cfg(ctypes.Structure):
    _fields_ = [("tau", ctypes.c_float), ("n_inflight", ctypes.c_int32), ("block_size", ctypes.c_int32),
                ("tau_semi", ctypes.c_float), ("tau_add", ctypes.c_float), ("skip_masked", ctypes.c_int32)]


def decode_cfg(tau: float, n_inflight: int, block_size: int, tau_semi=None, tau_add: float = 0.0,
               skip_masked: bool = False):
    """The C configuration; ``tau_semi=None`` switches semi-completion off."""
    return bd_decode_cfg(tau=tau, n_inflight=n_inflight, block_size=block_size,
                         tau_semi=-1.0 if tau_semi is None else tau_semi, tau_add=tau_add,
                         skip_masked=1 if skip_masked else 0)


STAT_NAMES = ("forwards", "rows", "lm_rows", "pairs", "keys", "committed", "active_forwards",
              "zero_commit", "static_saved", "static_deferred", "cache_writes", "skipped")


class BDError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"bd status {status}: {msg}")
        self.status = status


def _load():
    # torch ships its own libamdhip64; load it first so that libbd.so binds to
    # the same HIP runtime instance instead of pulling in a second one.
    import torch  # noqa: F401
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with `python -m paper_2609_33887_amd.build`")
    lib = ctypes.CDLL(LIB_PATH)
    P, I32, VP = ctypes.POINTER, ctypes.c_int32, ctypes.c_void_p
    sig = {
        "bd_init_model": [P(bd_model_cfg), P(VP), I32, VP, P(VP)],
        "bd_quantize_fp8": [VP, I32, I32, VP, VP, VP],
        "bd_quantize_mxfp4": [VP, I32, I32, I32, VP, VP, VP],
        "bd_prefill": [VP, VP, I32, I32, I32, P(bd_decode_cfg), P(VP)],
        "bd_denoise_step": [VP, VP, VP, VP, VP],
        "bd_commit": [VP, VP, P(I32)],
        "bd_state_read": [VP, VP, VP, VP, VP],
        "bd_decode": [VP, VP, I32, I32, I32, P(bd_decode_cfg), VP, VP, VP],
        "bd_decode_static": [VP, VP, I32, I32, I32, P(bd_decode_cfg), VP, VP, VP],
        "bd_state_reset": [VP, VP],
        "bd_state_steps": [VP, P(I32)],
        "bd_state_stats": [VP, VP, P(ctypes.c_int64), I32],
        "bd_profile": [VP, I32],
        "bd_profile_read": [VP, P(ctypes.c_double), P(I32)],
        "bd_plan_projection": [I32, I32, I32, I32, P(I32), P(I32), P(I32), P(ctypes.c_int64)],
        "bd_state_free": [VP],
        "bd_model_free": [VP],
        "rl_risk_select": [I32, I32, I32, P(ctypes.c_uint8), P(ctypes.c_double), ctypes.c_double,
                           ctypes.c_double, P(I32), P(ctypes.c_double), P(ctypes.c_uint8), P(I32), P(I32)],
        "rl_select": [I32, I32, I32, P(ctypes.c_uint8), P(ctypes.c_uint8), P(ctypes.c_double),
                      ctypes.c_double, ctypes.c_double, I32, P(I32), P(I32), P(ctypes.c_double),
                      P(ctypes.c_uint8), P(I32)],
        "rl_alpha_sweep": [I32, I32, I32, P(ctypes.c_uint8), P(ctypes.c_double), P(ctypes.c_double), I32,
                           ctypes.c_double, I32, P(I32), P(I32), P(I32), P(ctypes.c_double)],
        "rl_split_exceedance": [I32, I32, I32, P(ctypes.c_uint8), P(ctypes.c_double), ctypes.c_double,
                                ctypes.c_double, I32, P(I32), I32, P(ctypes.c_uint8), P(I32), P(I32),
                                P(I32), P(ctypes.c_double)],
        "rl_monte_carlo": [I32, I32, P(ctypes.c_double), ctypes.c_double, ctypes.c_double, I32, P(I32),
                           I32, I32, P(ctypes.c_double), P(I32), P(I32)],
    }
    for name, args in sig.items():
        f = getattr(lib, name)
        f.argtypes = args
        f.restype = I32
    lib.bd_last_error.argtypes = []
    lib.bd_last_error.restype = ctypes.c_char_p
    return lib


lib = _load()


def bd_last_error() -> str:
    return lib.bd_last_error().decode()


def _check(st: int):
    if st != BD_OK:
        raise BDError(st, bd_last_error())


# ---------------------------------------------------------------- thin wrappers
def bd_init_model(cfg: bd_model_cfg, weight_ptrs: Sequence[int], stream: int = 0) -> int:
    arr = (ctypes.c_void_p * len(weight_ptrs))(*weight_ptrs)
    out = ctypes.c_void_p()
    _check(lib.bd_init_model(ctypes.byref(cfg), arr, len(weight_ptrs), ctypes.c_void_p(stream),
                             ctypes.byref(out)))
    return out.value


def bd_quantize_fp8(w_ptr: int, rows: int, cols: int, codes_ptr: int, scale_ptr: int, stream: int = 0):
    _check(lib.bd_quantize_fp8(w_ptr, rows, cols, codes_ptr, scale_ptr, ctypes.c_void_p(stream)))


def quantize_fp8(w_bf16_bits, device: str = "cuda:0"):
    """fp8 E4M3 codes and row scales of a bf16 matrix given as uint16 bit
    patterns [rows][cols] (numpy); returns numpy (codes uint8, scale float32)."""
    import numpy as np
    import torch
    a = np.ascontiguousarray(w_bf16_bits)
    rows, cols = a.shape
    w = torch.from_numpy(a.view(np.int16)).to(device)
    codes = torch.empty((rows, cols), dtype=torch.uint8, device=device)
    scale = torch.empty((rows,), dtype=torch.float32, device=device)
    bd_quantize_fp8(w.data_ptr(), rows, cols, codes.data_ptr(), scale.data_ptr(),
                    torch.cuda.current_stream(device).cuda_stream)
    torch.cuda.synchronize(device)
    return codes.cpu().numpy(), scale.cpu().numpy()


def bd_quantize_mxfp4(w_ptr: int, rows: int, cols: int, group_rows: int, codes_ptr: int, exps_ptr: int,
                      stream: int = 0):
    _check(lib.bd_quantize_mxfp4(w_ptr, rows, cols, group_rows, codes_ptr, exps_ptr, ctypes.c_void_p(stream)))


def quantize_mxfp4(w_bf16_bits, group_rows=None, device: str = "cuda:0"):
    """MXFP4 codes and block exponents of a bf16 matrix given as uint16 bit
    patterns [rows][cols] (numpy), in the library's layout (see
    bd_quantize_mxfp4); returns numpy (codes uint8 [groups][cols/32][group_rows][16],
    exps uint8 [groups][cols/32][group_rows])."""
    import numpy as np
    import torch
    a = np.ascontiguousarray(w_bf16_bits)
    rows, cols = a.shape
    gr = rows if group_rows is None else group_rows
    w = torch.from_numpy(a.view(np.int16)).to(device)
    nb = cols // MX_BLOCK
    codes = torch.empty((rows // gr, nb, gr, 16), dtype=torch.uint8, device=device)
    exps = torch.empty((rows // gr, nb, gr), dtype=torch.uint8, device=device)
    bd_quantize_mxfp4(w.data_ptr(), rows, cols, gr, codes.data_ptr(), exps.data_ptr(),
                      torch.cuda.current_stream(device).cuda_stream)
    torch.cuda.synchronize(device)
    return codes.cpu().numpy(), exps.cpu().numpy()


def bd_prefill(model: int, prompt_ptr: int, b: int, P: int, G: int, cfg: bd_decode_cfg) -> int:
    out = ctypes.c_void_p()
    _check(lib.bd_prefill(model, prompt_ptr, b, P, G, ctypes.byref(cfg), ctypes.byref(out)))
    return out.value


def bd_denoise_step(model: int, state: int, conf_ptr: int = 0, tok_ptr: int = 0, logits_ptr: int = 0):
    _check(lib.bd_denoise_step(model, state, conf_ptr or None, tok_ptr or None, logits_ptr or None))


def bd_commit(model: int, state: int, want_done: bool = False):
    if want_done:
        d = ctypes.c_int32(0)
        _check(lib.bd_commit(model, state, ctypes.byref(d)))
        return bool(d.value)
    _check(lib.bd_commit(model, state, None))
    return None


def bd_state_read(model: int, state: int, tokens_ptr: int = 0, commit_ptr: int = 0, fwd_ptr: int = 0):
    _check(lib.bd_state_read(model, state, tokens_ptr or None, commit_ptr or None, fwd_ptr or None))


def bd_decode(model: int, prompt_ptr: int, b: int, P: int, G: int, cfg: bd_decode_cfg, tokens_ptr: int,
              commit_ptr: int, fwd_ptr: int):
    _check(lib.bd_decode(model, prompt_ptr, b, P, G, ctypes.byref(cfg), tokens_ptr, commit_ptr, fwd_ptr))


def bd_decode_static(model: int, prompt_ptr: int, b: int, P: int, G: int, cfg: bd_decode_cfg, tokens_ptr: int,
                     commit_ptr: int, fwd_ptr: int):
    _check(lib.bd_decode_static(model, prompt_ptr, b, P, G, ctypes.byref(cfg), tokens_ptr, commit_ptr,
                                fwd_ptr))


def bd_state_reset(model: int, state: int):
    _check(lib.bd_state_reset(model, state))


def bd_state_steps(state: int) -> int:
    n = ctypes.c_int32(0)
    _check(lib.bd_state_steps(state, ctypes.byref(n)))
    return n.value


def bd_state_stats(model: int, state: int):
    out = (ctypes.c_int64 * len(STAT_NAMES))()
    _check(lib.bd_state_stats(model, state, out, len(STAT_NAMES)))
    return dict(zip(STAT_NAMES, list(out)))


def bd_profile(model: int, enable: bool):
    _check(lib.bd_profile(model, 1 if enable else 0))


def bd_profile_read(model: int):
    ms = (ctypes.c_double * len(PROF_KINDS))()
    n = (ctypes.c_int32 * len(PROF_KINDS))()
    _check(lib.bd_profile_read(model, ms, n))
    return {k: (ms[i], n[i]) for i, k in enumerate(PROF_KINDS)}


def bd_plan_projection(N: int, K: int, rows_cap: int, resid: bool):
    """Tile plan of a bf16 projection: (bm, bn, zmax, workspace floats)."""
    bm, bn, zm = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int32()
    wsf = ctypes.c_int64()
    _check(lib.bd_plan_projection(N, K, rows_cap, 1 if resid else 0, ctypes.byref(bm), ctypes.byref(bn),
                                  ctypes.byref(zm), ctypes.byref(wsf)))
    return bm.value, bn.value, zm.value, wsf.value


def bd_state_free(state: int):
    _check(lib.bd_state_free(state))


def bd_model_free(model: int):
    _check(lib.bd_model_free(model))


def rl_risk_select(correct, cost, ref_index: int, alpha: float, delta: float):
    """correct: uint8 numpy [m][n]; cost: float64 [m].  Returns
    (V int32[m], p float64[m], valid bool[m], selected, near_ties)."""
    import numpy as np
    c = np.ascontiguousarray(correct, dtype=np.uint8)
    m, n = c.shape
    k = np.ascontiguousarray(cost, dtype=np.float64)
    V = np.zeros(m, dtype=np.int32)
    p = np.zeros(m, dtype=np.float64)
    valid = np.zeros(m, dtype=np.uint8)
    sel = ctypes.c_int32(-1)
    near = ctypes.c_int32(0)
    u8, f64, i32 = ctypes.POINTER(ctypes.c_uint8), ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_int32)
    _check(lib.rl_risk_select(n, m, ref_index, c.ctypes.data_as(u8), k.ctypes.data_as(f64), alpha, delta,
                              V.ctypes.data_as(i32), p.ctypes.data_as(f64), valid.ctypes.data_as(u8),
                              ctypes.byref(sel), ctypes.byref(near)))
    return V, p, valid.astype(bool), sel.value, near.value


_u8, _f64, _i32 = ctypes.POINTER(ctypes.c_uint8), ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_int32)


def _method_order(method: str, order, m: int):
    import numpy as np
    code = RL_METHODS[method]
    o = None if order is None else np.ascontiguousarray(order, dtype=np.int32)
    if o is not None and o.shape != (m,):
        raise ValueError("order must hold m entries")
    return code, o, (None if o is None else o.ctypes.data_as(_i32))


def rl_select(correct, cost, ref_index: int, alpha: float, delta: float, method: str = "holm",
              order=None, mask=None):
    """Returns (V int32[m], p float64[m], valid bool[m], selected)."""
    import numpy as np
    c = np.ascontiguousarray(correct, dtype=np.uint8)
    m, n = c.shape
    k = np.ascontiguousarray(cost, dtype=np.float64)
    code, o, op = _method_order(method, order, m)
    mk = None if mask is None else np.ascontiguousarray(mask, dtype=np.uint8)
    V = np.zeros(m, dtype=np.int32)
    p = np.zeros(m, dtype=np.float64)
    valid = np.zeros(m, dtype=np.uint8)
    sel = ctypes.c_int32(-1)
    _check(lib.rl_select(n, m, ref_index, c.ctypes.data_as(_u8), None if mk is None else mk.ctypes.data_as(_u8),
                         k.ctypes.data_as(_f64), alpha, delta, code, op, V.ctypes.data_as(_i32),
                         p.ctypes.data_as(_f64), valid.ctypes.data_as(_u8), ctypes.byref(sel)))
    return V, p, valid.astype(bool), sel.value


def rl_alpha_sweep(correct, cost, ref_index: int, alphas, delta: float, method: str = "holm", order=None):
    """Returns (selected int32[n_alpha], n_valid int32[n_alpha], alpha_hat or None)."""
    import math
    import numpy as np
    c = np.ascontiguousarray(correct, dtype=np.uint8)
    m, n = c.shape
    k = np.ascontiguousarray(cost, dtype=np.float64)
    a = np.ascontiguousarray(alphas, dtype=np.float64)
    code, o, op = _method_order(method, order, m)
    sel = np.zeros(len(a), dtype=np.int32)
    nval = np.zeros(len(a), dtype=np.int32)
    hat = ctypes.c_double(0.0)
    _check(lib.rl_alpha_sweep(n, m, ref_index, c.ctypes.data_as(_u8), k.ctypes.data_as(_f64),
                              a.ctypes.data_as(_f64), len(a), delta, code, op, sel.ctypes.data_as(_i32),
                              nval.ctypes.data_as(_i32), ctypes.byref(hat)))
    return sel, nval, (None if math.isnan(hat.value) else hat.value)


def rl_split_exceedance(correct, cost, ref_index: int, alpha: float, delta: float, cal_masks,
                        method: str = "holm", order=None):
    """Returns (deployed int32[S], test_violations int32[S], counts int32[4], gain_sum);
    counts = (exceed_test, exceed_pooled, fwer_test, fwer_pooled)."""
    import numpy as np
    c = np.ascontiguousarray(correct, dtype=np.uint8)
    m, n = c.shape
    k = np.ascontiguousarray(cost, dtype=np.float64)
    masks = np.ascontiguousarray(cal_masks, dtype=np.uint8)
    if masks.ndim != 2 or masks.shape[1] != n:
        raise ValueError("cal_masks must be [n_splits][n]")
    S = masks.shape[0]
    code, o, op = _method_order(method, order, m)
    dep = np.zeros(S, dtype=np.int32)
    tv = np.zeros(S, dtype=np.int32)
    counts = np.zeros(4, dtype=np.int32)
    gain = ctypes.c_double(0.0)
    _check(lib.rl_split_exceedance(n, m, ref_index, c.ctypes.data_as(_u8), k.ctypes.data_as(_f64), alpha,
                                   delta, code, op, S, masks.ctypes.data_as(_u8), dep.ctypes.data_as(_i32),
                                   tv.ctypes.data_as(_i32), counts.ctypes.data_as(_i32), ctypes.byref(gain)))
    return dep, tv, counts, gain.value


def rl_monte_carlo(true_risk, alpha: float, delta: float, u, method: str = "holm", order=None):
    """u: float64 [trials][1 or m][n].  Returns (false_trials, valid_counts int32[m])."""
    import numpy as np
    r = np.ascontiguousarray(true_risk, dtype=np.float64)
    m = r.shape[0]
    uu = np.ascontiguousarray(u, dtype=np.float64)
    if uu.ndim != 3:
        raise ValueError("u must be [trials][k][n]")
    trials, kk, n = uu.shape
    code, o, op = _method_order(method, order, m)
    ft = ctypes.c_int32(0)
    counts = np.zeros(m, dtype=np.int32)
    _check(lib.rl_monte_carlo(n, m, r.ctypes.data_as(_f64), alpha, delta, code, op, trials, kk,
                              uu.ctypes.data_as(_f64), ctypes.byref(ft), counts.ctypes.data_as(_i32)))
    return ft.value, counts


# ---------------------------------------------------------------- torch helpers
def model_cfg_from(w) -> bd_model_cfg:
    """Build the C config from a workload description (attribute access)."""
    return bd_model_cfg(n_layers=w.n_layers, d_model=w.d_model, n_heads=w.n_heads, n_kv_heads=w.n_kv_heads,
                        head_dim=w.head_dim, ffn_dim=w.ffn_dim, vocab=w.vocab, n_experts=w.n_experts,
                        top_k=w.top_k, expert_ffn=w.expert_ffn, n_shared=w.n_shared, rms_eps=w.rms_eps,
                        rope_theta=w.rope_theta, logit_scale=w.logit_scale, mask_id=w.vocab - 1,
                        dtype=BD_BF16 if w.dtype == "bf16" else BD_F32)


class Model:
    """Device copy of the weights plus the library handle."""

    def __init__(self, workload, weights, device: str = "cuda:0", wq=None):
        """``wq``: None (weights in the model dtype), "fp8" or "mxfp4"
        (decoder-layer projections quantized by the library, see
        bd_quantize_fp8 and bd_quantize_mxfp4)."""
        import numpy as np
        import torch
        self.torch = torch
        self.device = torch.device(device)
        self.w = workload
        self.tensors = []
        for a in weights:
            a = np.ascontiguousarray(a)
            if a.dtype == np.uint16:
                t = torch.from_numpy(a.view(np.int16)).to(self.device)
            else:
                t = torch.from_numpy(a.astype(np.float32)).to(self.device)
            self.tensors.append(t)
        self.stream = torch.cuda.current_stream(self.device)
        torch.cuda.synchronize(self.device)
        self.cfg = model_cfg_from(workload)
        self.cfg.wq = WQ[wq]
        self.wq = wq
        self.handle = bd_init_model(self.cfg, [t.data_ptr() for t in self.tensors], self.stream.cuda_stream)

    def close(self):
        if self.handle:
            bd_model_free(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class State:
    """A decode state of ``b`` sequences (prefill done on creation)."""

    def __init__(self, model: Model, prompts, G: int, tau: float, n_inflight: int, block_size: int,
                 tau_semi=None, tau_add: float = 0.0, skip_masked: bool = False):
        torch = model.torch
        self.m = model
        self.prompts = torch.as_tensor(prompts, dtype=torch.int32).to(model.device).contiguous()
        self.b, self.P = self.prompts.shape
        self.G = G
        self.cfg = decode_cfg(tau, n_inflight, block_size, tau_semi, tau_add, skip_masked)
        self.handle = bd_prefill(model.handle, self.prompts.data_ptr(), self.b, self.P, G, self.cfg)

    def step(self, conf=None, tok=None, logits=None):
        ptr = lambda t: 0 if t is None else t.data_ptr()
        bd_denoise_step(self.m.handle, self.handle, ptr(conf), ptr(tok), ptr(logits))

    def commit(self, want_done: bool = False):
        return bd_commit(self.m.handle, self.handle, want_done)

    def read(self):
        torch = self.m.torch
        t = torch.empty((self.b, self.G), dtype=torch.int32, device=self.m.device)
        c = torch.empty((self.b, self.G), dtype=torch.int32, device=self.m.device)
        f = torch.empty((self.b,), dtype=torch.int32, device=self.m.device)
        bd_state_read(self.m.handle, self.handle, t.data_ptr(), c.data_ptr(), f.data_ptr())
        return t.cpu().numpy(), c.cpu().numpy(), f.cpu().numpy()

    def reset(self):
        bd_state_reset(self.m.handle, self.handle)

    @property
    def steps(self) -> int:
        return bd_state_steps(self.handle)

    def stats(self) -> dict:
        return bd_state_stats(self.m.handle, self.handle)

    def close(self):
        if self.handle:
            bd_state_free(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def decode(model: Model, prompts, G: int, tau: float, n_inflight: int, block_size: int, tau_semi=None,
           tau_add: float = 0.0, skip_masked: bool = False, static: bool = False):
    """Whole decode through ``bd_decode`` (``bd_decode_static`` with
    ``static``); returns numpy (tokens, commit_step, forwards)."""
    torch = model.torch
    pr = torch.as_tensor(prompts, dtype=torch.int32).to(model.device).contiguous()
    b, P = pr.shape
    t = torch.empty((b, G), dtype=torch.int32, device=model.device)
    c = torch.empty((b, G), dtype=torch.int32, device=model.device)
    f = torch.empty((b,), dtype=torch.int32, device=model.device)
    cfg = decode_cfg(tau, n_inflight, block_size, tau_semi, tau_add, skip_masked)
    entry = bd_decode_static if static else bd_decode
    entry(model.handle, pr.data_ptr(), b, P, G, cfg, t.data_ptr(), c.data_ptr(), f.data_ptr())
    return t.cpu().numpy(), c.cpu().numpy(), f.cpu().numpy()
