"""Seeded synthetic inputs shared by the oracle and the GPU path.

This module holds only input generation: workload shapes, random-init weights
and random prompts.  It contains none of the decoding arithmetic (no forward
pass, no softmax, no commit rule), so that the oracle and the HIP library can
both consume the same host arrays without sharing any of the method's code.

Weights follow a random-init recipe: every matrix and embedding is drawn from
N(0, 0.02) with a counter-style seed ``[1000 + seed, tensor_index]``; RMSNorm
gains are ones.  For bf16 models the float32 draw is rounded to bfloat16
(round to nearest even) and returned as ``uint16`` bit patterns.  Prompts are
uniform on ``[0, vocab - 2]`` so the mask token (``vocab - 1``) never appears in
a prompt.
"""
from __future__ import annotations

import copy
from dataclasses import dataclass, field, asdict
from typing import List, Tuple

import numpy as np

__all__ = [
    "Workload", "WORKLOADS", "workload", "tensor_specs", "make_weights",
    "make_prompts", "bf16_bits_to_f32", "f32_to_bf16_bits", "n_weight_tensors",
]


@dataclass
class Workload:
    """Model architecture plus decode setting of one synthetic workload."""
    name: str
    seed: int
    n_layers: int
    d_model: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    ffn_dim: int
    vocab: int
    dtype: str                 # "f32" or "bf16"
    batch: int
    prompt_len: int
    block_size: int
    n_inflight: int
    gen_len: int
    taus: Tuple[float, ...] = (0.9,)
    n_experts: int = 0         # 0 => dense SwiGLU FFN
    top_k: int = 0
    expert_ffn: int = 0
    n_shared: int = 0
    rms_eps: float = 1e-6
    rope_theta: float = 1e4
    logit_scale: float = 20.0

    @property
    def mask_id(self) -> int:
        return self.vocab - 1

    @property
    def qkv_dim(self) -> int:
        return (self.n_heads + 2 * self.n_kv_heads) * self.head_dim

    def replace(self, **kw) -> "Workload":
        w = copy.deepcopy(self)
        for k, v in kw.items():
            if not hasattr(w, k):
                raise KeyError(k)
            setattr(w, k, v)
        return w

    def as_dict(self) -> dict:
        return asdict(self)


# The five workloads of the benchmark description.  Index 0 is the tiny fp32
# model, 1 the small-batch dense bf16 model, 2 the multi-block GQA model, 3 the
# long-prefix variant of 2, and 4 the MoE model used for the selection sweep.
WORKLOADS = {
    0: Workload("tiny-f32", 0, n_layers=2, d_model=256, n_heads=4, n_kv_heads=4, head_dim=64,
                ffn_dim=1024, vocab=4096, dtype="f32", batch=1, prompt_len=32, block_size=4,
                n_inflight=1, gen_len=64, taus=(0.9,)),
    1: Workload("dense-1024", 1, n_layers=12, d_model=1024, n_heads=16, n_kv_heads=16, head_dim=64,
                ffn_dim=4096, vocab=32768, dtype="bf16", batch=16, prompt_len=512, block_size=32,
                n_inflight=1, gen_len=256, taus=(0.95, 0.9, 0.8, 0.7)),
    2: Workload("gqa-2048-multiblock", 2, n_layers=24, d_model=2048, n_heads=16, n_kv_heads=4,
                head_dim=128, ffn_dim=8192, vocab=152064, dtype="bf16", batch=32, prompt_len=1024,
                block_size=32, n_inflight=3, gen_len=1024, taus=(0.9, 0.7)),
    3: Workload("gqa-2048-longprefix", 3, n_layers=24, d_model=2048, n_heads=16, n_kv_heads=4,
                head_dim=128, ffn_dim=8192, vocab=152064, dtype="bf16", batch=8, prompt_len=8192,
                block_size=64, n_inflight=2, gen_len=512, taus=(0.8,)),
    4: Workload("moe-2048", 4, n_layers=20, d_model=2048, n_heads=16, n_kv_heads=4, head_dim=128,
                ffn_dim=0, vocab=152064, dtype="bf16", batch=64, prompt_len=256, block_size=32,
                n_inflight=1, gen_len=128, taus=(0.95, 0.9, 0.8, 0.7), n_experts=64, top_k=8,
                expert_ffn=512, n_shared=1),
}


def workload(idx: int, **overrides) -> Workload:
    return WORKLOADS[idx].replace(**overrides) if overrides else copy.deepcopy(WORKLOADS[idx])


def tensor_specs(w: Workload) -> List[Tuple[str, Tuple[int, ...], str]]:
    """Names, shapes and storage kinds of the weight tensors, in ABI order.

    Kind "mat" tensors are random N(0, 0.02) in the model dtype; kind "norm"
    tensors are float32 ones; kind "router" is float32 N(0, 0.02).
    Matrices are stored [out_features][in_features] (row-major).
    """
    d, hd = w.d_model, w.head_dim
    specs = [("tok_embed", (w.vocab, d), "mat")]
    for layer in range(w.n_layers):
        p = f"l{layer}."
        specs += [
            (p + "attn_norm", (d,), "norm"),
            (p + "w_qkv", (w.qkv_dim, d), "mat"),
            (p + "w_o", (d, w.n_heads * hd), "mat"),
            (p + "ffn_norm", (d,), "norm"),
        ]
        if w.n_experts == 0:
            specs += [
                (p + "w_gate", (w.ffn_dim, d), "mat"),
                (p + "w_up", (w.ffn_dim, d), "mat"),
                (p + "w_down", (d, w.ffn_dim), "mat"),
            ]
        else:
            e, fe, fs = w.n_experts, w.expert_ffn, w.n_shared * w.expert_ffn
            specs += [
                (p + "w_router", (e, d), "router"),
                (p + "w_gate_e", (e, fe, d), "mat"),
                (p + "w_up_e", (e, fe, d), "mat"),
                (p + "w_down_e", (e, d, fe), "mat"),
                (p + "w_gate_s", (fs, d), "mat"),
                (p + "w_up_s", (fs, d), "mat"),
                (p + "w_down_s", (d, fs), "mat"),
            ]
    specs += [("final_norm", (d,), "norm"), ("lm_head", (w.vocab, d), "mat")]
    return specs


def n_weight_tensors(w: Workload) -> int:
    return len(tensor_specs(w))


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (nearest, ties to even); returns uint16 bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    bias = np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
    return ((u + bias) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def _draw(seed: int, t: int, shape) -> np.ndarray:
    rng = np.random.default_rng([1000 + seed, t])
    a = rng.standard_normal(shape, dtype=np.float32)
    a *= np.float32(0.02)
    return a


def make_weights(w: Workload, threads: int | None = None) -> List[np.ndarray]:
    """Weights in ABI order.  "mat" tensors are float32 (f32 models) or uint16
    bf16 bit patterns (bf16 models); "norm" and "router" tensors are float32.
    Each tensor has its own seeded stream, so drawing them on a thread pool
    (numpy's generators release the GIL while filling an array) gives the
    same arrays as drawing them one after another."""
    import concurrent.futures as cf
    import os

    def one(item):
        t, (_, shape, kind) = item
        if kind == "norm":
            return np.ones(shape, dtype=np.float32)
        a = _draw(w.seed, t, shape)
        if kind == "router" or w.dtype == "f32":
            return a
        return f32_to_bf16_bits(a)

    items = list(enumerate(tensor_specs(w)))
    n = threads or min(16, len(os.sched_getaffinity(0)))
    if n <= 1:
        return [one(it) for it in items]
    with cf.ThreadPoolExecutor(max_workers=n) as ex:
        return list(ex.map(one, items))


def make_prompts(w: Workload, n: int | None = None, offset: int = 0) -> np.ndarray:
    """int32 [n][prompt_len] uniform on [0, vocab-2]; rows ``offset..offset+n``
    of one seeded stream, so a subset of rows is reproducible on its own."""
    n = w.batch if n is None else n
    rng = np.random.default_rng(2000 + w.seed)
    allp = rng.integers(0, w.vocab - 1, size=(offset + n, w.prompt_len), dtype=np.int64)
    return allp[offset:offset + n].astype(np.int32)


# ---- Redline harness inputs -------------------------------------------------
# Random draws only: which prompts form a calibration half, the prompt-level
# uniforms of a Monte Carlo trial, and planted correctness matrices.

def split_masks(n: int, n_splits: int, cal_frac: float = 0.5, seed: int = 0) -> np.ndarray:
    """[n_splits][n] uint8: 1 for the round(cal_frac * n) prompts of each
    split's calibration half (a uniformly random subset), 0 for its test half."""
    rng = np.random.default_rng([3000, seed])
    k = int(round(cal_frac * n))
    out = np.zeros((n_splits, n), dtype=np.uint8)
    for s in range(n_splits):
        out[s, rng.permutation(n)[:k]] = 1
    return out


def mc_uniforms(trials: int, k: int, n: int, seed: int = 0) -> np.ndarray:
    """[trials][k][n] float64 uniforms on [0, 1)."""
    return np.random.default_rng([4000, seed]).random((trials, k, n))


def planted_correctness(n: int, risks, ref_index: int, ref_acc: float = 0.8, seed: int = 0,
                        shared: bool = False) -> np.ndarray:
    """[m][n] uint8 matrix: the reference is right on a random ref_acc share of
    prompts; configuration j keeps each of those with probability 1 - risks[j]
    (one uniform per prompt for every configuration when ``shared``) and is
    right elsewhere with probability ref_acc."""
    rng = np.random.default_rng([5000, seed])
    m = len(risks)
    ref = rng.random(n) < ref_acc
    u_shared = rng.random(n)
    out = np.zeros((m, n), dtype=np.uint8)
    for j in range(m):
        u = u_shared if shared else rng.random(n)
        other = rng.random(n) < ref_acc
        out[j] = np.where(ref, u >= risks[j], other)
    out[ref_index] = ref
    return out
