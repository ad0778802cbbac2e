"""Oracle decoder forward (test infrastructure only; see ``oracle/__init__``).

What is computed, and where it comes from:

* Block-diffusion factorisation (paper §2.1): the sequence is cut into blocks of
  ``B`` positions aligned at absolute position 0; attention is bidirectional
  inside a block and causal across blocks, so a query at position ``p`` sees
  exactly the keys ``j`` with ``j // B <= p // B``.  Generated blocks are
  cached like an autoregressive prefix.
* The paper does not specify the architecture of its models; the readings used
  here (pre-norm RMSNorm decoder, rotate-half RoPE, SwiGLU or top-k MoE FFN,
  untied LM head scaled by ``logit_scale``) are the documented workload
  definition.
* The engine commits from the mask-suppressed softmax (App. B.1): the logit of
  the mask token is removed before the softmax, confidence is the largest
  probability and the committed token is its argmax.

Precision modes
  ``"f64"``  every operand and every operation in float64.
  ``"bf16"`` bf16 weights; every stored activation -- the matmul operands
             (RMSNorm outputs, attention output, SwiGLU product, final-norm
             output) and Q, K, V after RoPE (the KV cache) -- is fp32(x)
             carried as the bf16 pair hi = bf16(x), lo = bf16(x - hi), i.e.
             x to 16 significant bits (nearest-even at both roundings);
             matmuls run as float32 BLAS on those operands; residual stream,
             attention softmax, norms and router in float64.
"""
from __future__ import annotations

import math

import numpy as np

__all__ = ["round_bf16", "split_bf16x2", "OracleModel", "KVCache", "lm_stats"]


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round to the nearest bfloat16 (ties to even) after first rounding to
    float32, as a kernel that holds an fp32 value and stores bf16 does.

    Implemented through the binary exponent: with x = m * 2**e, 0.5 <= |m| < 1,
    bfloat16 keeps 8 significant bits, i.e. round(m * 2**8) * 2**(e-8), and
    ``np.rint`` rounds half to even.
    """
    x32 = np.asarray(x, dtype=np.float64).astype(np.float32).astype(np.float64)
    m, e = np.frexp(x32)
    return np.ldexp(np.rint(np.ldexp(m, 8)), e - 8)


def split_bf16x2(x: np.ndarray) -> np.ndarray:
    """Value of the bf16 pair (hi, lo) that carries fp32(x): hi = bf16(x),
    lo = bf16(x - hi) (the difference is exact), returned as hi + lo."""
    x32 = np.asarray(x, dtype=np.float64).astype(np.float32).astype(np.float64)
    hi = round_bf16(x32)
    return hi + round_bf16(x32 - hi)


def _bits_to_float(a: np.ndarray) -> np.ndarray:
    if a.dtype == np.uint16:   # bfloat16 bit patterns: high half of an fp32
        return (a.astype(np.uint32) << 16).view(np.float32)
    return a


def _rmsnorm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    """x / sqrt(mean(x^2) + eps) * g, per row, in float64."""
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * g


def _silu(x: np.ndarray) -> np.ndarray:
    return x / (1.0 + np.exp(-x))


def _block_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, scale: float, use_torch: bool) -> np.ndarray:
    """softmax(scale * q @ k.T) @ v per row, in float64: the scores, their row
    maximum, exp(s - max), the sum, the normalised weights and the weighted
    sum of v -- as numpy operations, or as torch CPU operations (which use
    every host core) when ``use_torch``."""
    if not use_torch:
        return _softmax_rows((q @ k.T) * scale) @ v
    import torch
    s = (torch.from_numpy(q) @ torch.from_numpy(k).T) * scale
    e = torch.exp(s - torch.amax(s, dim=-1, keepdim=True))
    p = e / torch.sum(e, dim=-1, keepdim=True)
    return (p @ torch.from_numpy(v)).numpy()


def _softmax_rows(s: np.ndarray) -> np.ndarray:
    m = np.max(s, axis=-1, keepdims=True)
    e = np.exp(s - m)
    return e / np.sum(e, axis=-1, keepdims=True)


class KVCache:
    """Per-layer key/value arrays indexed by absolute position."""

    def __init__(self, n_layers: int, max_pos: int, n_kv_heads: int, head_dim: int, dtype):
        self.k = [np.zeros((max_pos, n_kv_heads, head_dim), dtype=dtype) for _ in range(n_layers)]
        self.v = [np.zeros((max_pos, n_kv_heads, head_dim), dtype=dtype) for _ in range(n_layers)]


class OracleModel:
    """Decoder forward over a window of absolute positions ``[start, end)``.

    ``cfg`` supplies the dimensions (see the workload definition); ``weights``
    is the list of tensors in ABI order, either float arrays or uint16 bf16
    bit patterns.
    """

    def __init__(self, cfg, weights, precision: str = "f64"):
        if precision not in ("f64", "bf16"):
            raise ValueError(precision)
        self.cfg = cfg
        self.precision = precision
        self.H, self.Hkv, self.hd = cfg.n_heads, cfg.n_kv_heads, cfg.head_dim
        self.d, self.V = cfg.d_model, cfg.vocab
        self.mask_id = cfg.vocab - 1
        wdt = np.float64 if precision == "f64" else np.float32

        def widen(t):
            return _bits_to_float(np.asarray(t)).astype(wdt)

        # the conversions of large models take minutes one after another;
        # numpy releases the GIL while casting, so a thread pool runs them at once
        import concurrent.futures as cf
        import os
        with cf.ThreadPoolExecutor(max_workers=min(16, len(os.sched_getaffinity(0)))) as ex:
            ws = list(ex.map(widen, weights))
        it = iter(ws)
        self.embed = next(it)
        self.layers = []
        for _ in range(cfg.n_layers):
            L = {"attn_norm": next(it).astype(np.float64), "w_qkv": next(it), "w_o": next(it),
                 "ffn_norm": next(it).astype(np.float64)}
            if cfg.n_experts == 0:
                L.update(w_gate=next(it), w_up=next(it), w_down=next(it))
            else:
                L.update(w_router=next(it).astype(np.float64), w_gate_e=next(it), w_up_e=next(it),
                         w_down_e=next(it), w_gate_s=next(it), w_up_s=next(it), w_down_s=next(it))
            self.layers.append(L)
        self.final_norm = next(it).astype(np.float64)
        self.lm_head = next(it)
        rest = list(it)
        if rest:
            raise ValueError(f"{len(rest)} unexpected weight tensors")
        # RoPE inverse frequencies theta^(-2i/hd) for the rotate-half pairs (i, i + hd/2).
        i = np.arange(self.hd // 2, dtype=np.float64)
        self.inv_freq = cfg.rope_theta ** (-2.0 * i / self.hd)
        self.router_gaps = []

    # -- storage points ---------------------------------------------------
    def _store(self, x: np.ndarray) -> np.ndarray:
        """Q/K/V as stored in the cache: the bf16 pair value in bf16 mode."""
        return split_bf16x2(x) if self.precision == "bf16" else x

    def _operand(self, x: np.ndarray) -> np.ndarray:
        """Matmul activation operand: the bf16 pair value in bf16 mode."""
        return split_bf16x2(x) if self.precision == "bf16" else x

    def _mm(self, a: np.ndarray, w: np.ndarray) -> np.ndarray:
        """a @ w.T for a [rows][in] and a weight stored [out][in], evaluated
        as (w @ a.T).T: the same dot products, with the weight as the left
        operand, the orientation in which BLAS runs these few-row products
        fastest."""
        if self.precision == "f64":
            return (w @ a.T).T
        return (w @ a.astype(np.float32).T).T.astype(np.float64)

    def kv_cache(self, max_pos: int) -> KVCache:
        dt = np.float64 if self.precision == "f64" else np.float32
        return KVCache(self.cfg.n_layers, max_pos, self.Hkv, self.hd, dt)

    # -- pieces -----------------------------------------------------------
    def rope(self, x: np.ndarray, pos: np.ndarray) -> np.ndarray:
        """Rotate-half RoPE: pair (i, i + hd/2) rotated by pos * inv_freq[i].
        x: [rows][heads][hd], pos: [rows] absolute positions."""
        ang = pos.astype(np.float64)[:, None] * self.inv_freq[None, :]
        c, s = np.cos(ang)[:, None, :], np.sin(ang)[:, None, :]
        h = self.hd // 2
        x1, x2 = x[..., :h], x[..., h:]
        return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)

    def attention(self, q: np.ndarray, qpos: np.ndarray, K: np.ndarray, V: np.ndarray,
                  B: int) -> np.ndarray:
        """Block-causal attention (§2.1).  q: [W][H][hd] at positions qpos;
        K, V: [e][Hkv][hd] for keys at positions 0..e-1.  Query at p attends to
        key j iff j // B <= p // B, i.e. to the keys [0, (p // B + 1) B): every
        query of one block sees the same keys, so each block's queries are
        taken together over exactly those keys.  GQA: q-head h reads kv-head
        h // (H/Hkv).  Scores, softmax (max, exponentials, normalisation) and
        the weighted sum of values in float64."""
        group = self.H // self.Hkv
        scale = 1.0 / math.sqrt(self.hd)
        Kd = np.ascontiguousarray(K, dtype=np.float64)
        Vd = np.ascontiguousarray(V, dtype=np.float64)
        out = np.empty(q.shape, dtype=np.float64)
        blk = np.asarray(qpos) // B
        # long prefixes: torch's thread pool for the whole call (switching
        # between it and numpy's BLAS threads per block costs more than small
        # blocks gain from it)
        use_torch = q.shape[0] * self.H * K.shape[0] >= (1 << 24)
        for b in np.unique(blk):
            rows = np.nonzero(blk == b)[0]
            r0, r1 = int(rows[0]), int(rows[-1]) + 1
            assert r1 - r0 == rows.size, "a block's queries are consecutive window rows"
            kend = int((b + 1) * B)
            for kv in range(self.Hkv):
                hs = slice(kv * group, (kv + 1) * group)
                qb = q[r0:r1, hs, :].reshape(-1, self.hd).astype(np.float64)     # [rows * group][hd]
                o = _block_attention(qb, Kd[:kend, kv, :], Vd[:kend, kv, :], scale, use_torch)
                out[r0:r1, hs, :] = o.reshape(r1 - r0, group, self.hd)
        return out

    def dense_ffn(self, a: np.ndarray, L) -> np.ndarray:
        act = self._operand(_silu(self._mm(a, L["w_gate"])) * self._mm(a, L["w_up"]))
        return self._mm(act, L["w_down"])

    def router(self, a: np.ndarray, L):
        """Top-k routing: softmax over all experts, k largest (lowest expert id
        first among equals), weights renormalised to sum to one.  The gap
        between the k-th and (k+1)-th largest router logits of every row is
        appended to ``self.router_gaps`` (used to recognise routing near-ties)."""
        logits = a @ L["w_router"].T
        probs = _softmax_rows(logits)
        k = self.cfg.top_k
        order = np.argsort(-probs, axis=-1, kind="stable")[:, :k]
        w = np.take_along_axis(probs, order, axis=-1)
        if k < logits.shape[1]:
            srt = -np.sort(-logits, axis=-1)
            self.router_gaps.append(srt[:, k - 1] - srt[:, k])
        return order, w / np.sum(w, axis=-1, keepdims=True), logits

    def moe_ffn(self, a: np.ndarray, L) -> np.ndarray:
        experts, wts, _ = self.router(a, L)
        out = np.zeros((a.shape[0], self.d), dtype=np.float64)
        for e in range(self.cfg.n_experts):
            rows, slot = np.nonzero(experts == e)
            if rows.size == 0:
                continue
            ae = a[rows]
            g = self._mm(ae, L["w_gate_e"][e])
            u = self._mm(ae, L["w_up_e"][e])
            y = self._mm(self._operand(_silu(g) * u), L["w_down_e"][e])
            out[rows] += wts[rows, slot][:, None] * y
        g = self._mm(a, L["w_gate_s"])
        u = self._mm(a, L["w_up_s"])
        return out + self._mm(self._operand(_silu(g) * u), L["w_down_s"])

    # -- forward ------------------------------------------------------------
    def forward(self, tokens: np.ndarray, start: int, end: int, cache: KVCache, B: int) -> np.ndarray:
        """Run every layer over window positions [start, end) of one sequence.

        K/V of the window are written into ``cache`` at their absolute
        positions before attention reads keys 0..end-1, so keys below
        ``start`` come from the cache.  Returns the final-norm hidden states of
        the window rows (bf16-stored in bf16 mode), one row per position.
        """
        cfg = self.cfg
        pos = np.arange(start, end)
        x = self.embed[tokens[start:end]].astype(np.float64)
        H, Hkv, hd = self.H, self.Hkv, self.hd
        for li, L in enumerate(self.layers):
            a = self._operand(_rmsnorm(x, L["attn_norm"], cfg.rms_eps))
            qkv = self._mm(a, L["w_qkv"])
            q = qkv[:, :H * hd].reshape(-1, H, hd)
            k = qkv[:, H * hd:(H + Hkv) * hd].reshape(-1, Hkv, hd)
            v = qkv[:, (H + Hkv) * hd:].reshape(-1, Hkv, hd)
            q = self._store(self.rope(q, pos))
            cache.k[li][start:end] = self._store(self.rope(k, pos))
            cache.v[li][start:end] = self._store(v)
            o = self.attention(q, pos, cache.k[li][:end], cache.v[li][:end], B)
            x = x + self._mm(self._operand(o.reshape(len(pos), H * hd)), L["w_o"])
            a = self._operand(_rmsnorm(x, L["ffn_norm"], cfg.rms_eps))
            x = x + (self.dense_ffn(a, L) if cfg.n_experts == 0 else self.moe_ffn(a, L))
        return self._operand(_rmsnorm(x, self.final_norm, cfg.rms_eps))

    def logits(self, h: np.ndarray) -> np.ndarray:
        """Scaled LM-head logits with the mask token's column suppressed."""
        z = self.cfg.logit_scale * self._mm(h, self.lm_head)
        z[:, self.mask_id] = -np.inf
        return z


def lm_stats(z: np.ndarray):
    """Mask-suppressed softmax statistics per row (App. B.1).

    Returns ``conf`` = largest probability = 1 / sum(exp(z - max z)), ``tok`` =
    its argmax (lowest token id among equal maxima), and ``p2`` = the second
    largest probability (used to recognise near-ties)."""
    zmax = np.max(z, axis=-1)
    tok = np.argmax(z, axis=-1)                 # first maximum = lowest id
    ssum = np.sum(np.exp(z - zmax[:, None]), axis=-1)
    conf = 1.0 / ssum
    z2 = z.copy()
    z2[np.arange(z.shape[0]), tok] = -np.inf
    p2 = np.exp(np.max(z2, axis=-1) - zmax) / ssum
    return conf, tok.astype(np.int64), p2
