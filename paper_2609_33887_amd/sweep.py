"""Redline selection sweep over serving configurations (§4.2, App. A).

Every configuration lambda = (tau, n_inflight) or (tau, n_inflight, tau_semi,
tau_add) decodes the same calibration prompts through ``bd_decode``; a decode
is *correct* when its final ``tail`` generated tokens equal the reference
configuration's.  The correctness matrix and the TPF of each configuration
then go to ``rl_select`` (Holm by default), which deploys the fastest
configuration whose reference-relative risk passes the exact binomial test,
and to ``rl_alpha_sweep`` for the smallest budget with a gain.

Grids: ``tau-nb`` -- accept threshold x in-flight blocks against the
one-token-per-step reference; ``engine`` -- accept {0.85, 0.90, 0.95, 0.99} x
semi-completion {0.70, 0.90} at admission 0.10 and two blocks in flight, with
the engine default acc95/semi90 as the reference (the shape of the paper's
grids, App. D); ``precision`` -- the same decode configuration served with
bf16 weights (the reference) and with fp8 E4M3 layer weights, deploying the
valid configuration with the least weight memory (the paper's quantization
grid: §4.2 (iv) "for quantization the one with the least memory").

Run: ``python -m paper_2609_33887_amd.sweep --prompts 1000 [--grid engine]``
(prints JSON).
"""
from __future__ import annotations

import argparse
import json
import sys
import time

import numpy as np

from . import bd


ENGINE_REFERENCE = (0.95, 2, 0.90, 0.10)
ENGINE_GRID = [(acc, 2, semi, 0.10) for acc in (0.85, 0.90, 0.95, 0.99) for semi in (0.70, 0.90)
               if (acc, semi) != (0.95, 0.90)]


def label(cfg) -> str:
    """acc85/semi70/add0.10-style label (nb suffix for the tau x nb grid)."""
    tau, nb = cfg[0], cfg[1]
    if len(cfg) == 2:
        return f"acc{round(100 * tau)}/nb{nb}" if tau <= 1 else f"one-token/nb{nb}"
    return f"acc{round(100 * tau)}/semi{round(100 * cfg[2])}/add{cfg[3]:.2f}"


def decode_all(model, prompts, G, cfg, B, batch):
    """Decode ``prompts`` in batches under cfg = (tau, nb[, tau_semi, tau_add]);
    returns tokens [n][G] and forwards [n]."""
    tau, nb = cfg[0], cfg[1]
    ts, ta = (cfg[2], cfg[3]) if len(cfg) == 4 else (None, 0.0)
    toks, fwd = [], []
    for i in range(0, prompts.shape[0], batch):
        t, _, f = bd.decode(model, prompts[i:i + batch], G, tau, nb, B, ts, ta)
        toks.append(t)
        fwd.append(f)
    return np.concatenate(toks), np.concatenate(fwd)


def redline_sweep(model, prompts, G, B, candidates, reference, alpha, delta, tail=16, batch=64,
                  progress=None, method="holm", alphas=None):
    """candidates / reference: (tau, n_inflight[, tau_semi, tau_add]).  The
    reference is the first row of the grid (the grid includes it, §4.2 (i))."""
    grid = [tuple(reference)] + [tuple(c) for c in candidates]
    outs, tpf = [], []
    for j, cfg in enumerate(grid):
        t0 = time.perf_counter()
        toks, fwd = decode_all(model, prompts, G, cfg, B, batch)
        outs.append(toks)
        tpf.append(toks.size / float(fwd.sum()))
        if progress:
            progress(f"config {j} {label(cfg)}: TPF {tpf[-1]:.4f} ({time.perf_counter() - t0:.1f} s)")
    ref_tail = outs[0][:, -tail:]
    correct = np.stack([np.all(o[:, -tail:] == ref_tail, axis=1) for o in outs]).astype(np.uint8)
    V, p, valid, sel = bd.rl_select(correct, np.array(tpf), 0, alpha, delta, method)
    out = {"grid": grid, "labels": [label(c) for c in grid], "tpf": tpf, "correct": correct, "V": V,
           "p": p, "valid": valid, "selected": sel, "tokens": outs}
    if alphas is not None:
        sweep_sel, n_valid, hat = bd.rl_alpha_sweep(correct, np.array(tpf), 0, alphas, delta, method)
        out.update(alphas=list(alphas), alpha_selected=sweep_sel.tolist(), alpha_n_valid=n_valid.tolist(),
                   alpha_hat=hat)
    return out


def weight_bytes(w, wq=None) -> int:
    """Weight memory of a model as the library holds it: decoder-layer
    projections in bf16 (2 bytes), fp8 (1 byte plus a 4-byte scale per row)
    or MXFP4 (half a byte plus a 1-byte exponent per 32 elements);
    embeddings and LM head in bf16; norms and router in fp32."""
    d, hd = w.d_model, w.head_dim
    proj = [((w.n_heads + 2 * w.n_kv_heads) * hd, d), (d, w.n_heads * hd)]
    if w.n_experts == 0:
        proj += [(2 * w.ffn_dim, d), (d, w.ffn_dim)]
    else:
        Fe, Fs = w.expert_ffn, w.n_shared * w.expert_ffn
        proj += [(w.n_experts * 2 * Fe, d), (w.n_experts * d, Fe)]
        if Fs:
            proj += [(2 * Fs, d), (d, Fs)]
    if wq == "fp8":
        per_row = lambda r, c: r * c + 4 * r
    elif wq == "mxfp4":
        per_row = lambda r, c: r * c // 2 + r * c // 32
    else:
        per_row = lambda r, c: 2 * r * c
    layer = sum(per_row(r, c) for r, c in proj) + 4 * 2 * d + (4 * w.n_experts * d if w.n_experts else 0)
    return w.n_layers * layer + 2 * 2 * w.vocab * d + 4 * d


def precision_sweep(w, models, prompts, G, B, reference, candidates, alpha, delta, tail=16, batch=64,
                    progress=None, method="holm"):
    """reference / candidates: (precision, decode config) with precision a
    key of ``models`` ("bf16", "fp8" or "mxfp4").  Correctness as in redline_sweep;
    the cost measure is the weight-memory reduction against the reference
    (larger is better), so the deployed configuration is the valid one with
    the least weight memory (first listed among equals)."""
    grid = [tuple(reference)] + [tuple(c) for c in candidates]
    outs, tpf, mem = [], [], []
    for j, (prec, cfg) in enumerate(grid):
        t0 = time.perf_counter()
        toks, fwd = decode_all(models[prec], prompts, G, cfg, B, batch)
        outs.append(toks)
        tpf.append(toks.size / float(fwd.sum()))
        mem.append(weight_bytes(w, None if prec == "bf16" else prec))
        if progress:
            progress(f"config {j} {prec} {label(cfg)}: TPF {tpf[-1]:.4f}, weights {mem[-1] / 2**20:.1f} MiB "
                     f"({time.perf_counter() - t0:.1f} s)")
    ref_tail = outs[0][:, -tail:]
    correct = np.stack([np.all(o[:, -tail:] == ref_tail, axis=1) for o in outs]).astype(np.uint8)
    cost = mem[0] / np.array(mem, dtype=np.float64)
    V, p, valid, sel = bd.rl_select(correct, cost, 0, alpha, delta, method)
    return {"grid": grid, "labels": [f"{prec}/{label(cfg)}" for prec, cfg in grid], "tpf": tpf,
            "weight_bytes": mem, "cost": cost, "correct": correct, "V": V, "p": p, "valid": valid,
            "selected": sel, "tokens": outs}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--config", type=int, default=4)
    ap.add_argument("--prompts", type=int, default=1000)
    ap.add_argument("--alpha", type=float, default=0.10)
    ap.add_argument("--delta", type=float, default=0.05)
    ap.add_argument("--grid", choices=["tau-nb", "engine", "precision"], default="tau-nb")
    ap.add_argument("--method", choices=list(bd.RL_METHODS), default="holm")
    args = ap.parse_args()
    import os
    sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
    from bd_synth import workload, make_weights, make_prompts
    w = workload(args.config)
    weights = make_weights(w)
    model = bd.Model(w, weights)
    prompts = make_prompts(w, args.prompts)
    say = lambda m: print(m, file=sys.stderr, flush=True)
    if args.grid == "precision":
        models = {"bf16": model, "fp8": bd.Model(w, weights, wq="fp8"), "mxfp4": bd.Model(w, weights, wq="mxfp4")}
        ref = ("bf16", (0.9, w.n_inflight))
        cands = [(prec, (t, w.n_inflight)) for prec in ("fp8", "mxfp4") for t in (0.9, 0.8)]
        r = precision_sweep(w, models, prompts, w.gen_len, w.block_size, ref, cands, args.alpha, args.delta,
                            batch=w.batch, progress=say, method=args.method)
        print(json.dumps({"workload": w.name, "prompts": args.prompts, "alpha": args.alpha,
                          "delta": args.delta, "method": args.method, "grid": r["labels"], "tpf": r["tpf"],
                          "weight_bytes": r["weight_bytes"], "V": r["V"].tolist(), "p": r["p"].tolist(),
                          "valid": r["valid"].tolist(), "selected": r["selected"],
                          "selected_config": r["labels"][r["selected"]]}))
        return
    if args.grid == "engine":
        cands, ref = ENGINE_GRID, ENGINE_REFERENCE
    else:
        cands, ref = [(t, nb) for t in (0.95, 0.9, 0.8, 0.7) for nb in (1, 2, 3)], (2.0, 1)
    r = redline_sweep(model, prompts, w.gen_len, w.block_size, cands, ref, args.alpha, args.delta,
                      batch=w.batch, progress=say, method=args.method,
                      alphas=[i / 100 for i in range(1, 31)])
    print(json.dumps({"workload": w.name, "prompts": args.prompts, "alpha": args.alpha,
                      "delta": args.delta, "method": args.method, "grid": r["labels"], "tpf": r["tpf"],
                      "V": r["V"].tolist(), "p": r["p"].tolist(), "valid": r["valid"].tolist(),
                      "selected": r["selected"], "selected_config": r["labels"][r["selected"]],
                      "alpha_hat": r["alpha_hat"]}))


if __name__ == "__main__":
    main()
