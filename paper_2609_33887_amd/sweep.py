"""Redline selection sweep over serving configurations (§4.2, App. A).

Every configuration lambda = (tau, n_inflight) decodes the same calibration
prompts through ``bd_decode``; a decode is *correct* when its final ``tail``
generated tokens equal the reference configuration's.  The correctness
matrix and the TPF of each configuration then go to ``rl_risk_select``,
which deploys the fastest configuration whose reference-relative risk passes
the exact binomial test under Holm's correction.

Run: ``python -m paper_2609_33887_amd.sweep --prompts 1000`` (prints JSON).
"""
from __future__ import annotations

import argparse
import json
import sys
import time

import numpy as np

from . import bd


def decode_all(model, prompts, G, tau, nb, B, batch):
    """Decode ``prompts`` in batches; returns tokens [n][G] and forwards [n]."""
    toks, fwd = [], []
    for i in range(0, prompts.shape[0], batch):
        t, _, f = bd.decode(model, prompts[i:i + batch], G, tau, nb, B)
        toks.append(t)
        fwd.append(f)
    return np.concatenate(toks), np.concatenate(fwd)


def redline_sweep(model, prompts, G, B, candidates, reference, alpha, delta, tail=16, batch=64,
                  progress=None):
    """candidates / reference: (tau, n_inflight) pairs.  The reference is the
    first row of the grid (the grid includes it, §4.2 (i))."""
    grid = [tuple(reference)] + [tuple(c) for c in candidates]
    outs, tpf = [], []
    for j, (tau, nb) in enumerate(grid):
        t0 = time.perf_counter()
        toks, fwd = decode_all(model, prompts, G, tau, nb, B, batch)
        outs.append(toks)
        tpf.append(toks.size / float(fwd.sum()))
        if progress:
            progress(f"config {j} tau={tau} nb={nb}: TPF {tpf[-1]:.4f} ({time.perf_counter() - t0:.1f} s)")
    ref_tail = outs[0][:, -tail:]
    correct = np.stack([np.all(o[:, -tail:] == ref_tail, axis=1) for o in outs]).astype(np.uint8)
    V, p, valid, sel, near = bd.rl_risk_select(correct, np.array(tpf), 0, alpha, delta)
    return {"grid": grid, "tpf": tpf, "correct": correct, "V": V, "p": p, "valid": valid,
            "selected": sel, "near_ties": near, "tokens": outs}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--config", type=int, default=4)
    ap.add_argument("--prompts", type=int, default=1000)
    ap.add_argument("--alpha", type=float, default=0.10)
    ap.add_argument("--delta", type=float, default=0.05)
    args = ap.parse_args()
    import os
    sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
    from bd_synth import workload, make_weights, make_prompts
    w = workload(args.config)
    model = bd.Model(w, make_weights(w))
    prompts = make_prompts(w, args.prompts)
    cands = [(t, nb) for t in (0.95, 0.9, 0.8, 0.7) for nb in (1, 2, 3)]
    say = lambda m: print(m, file=sys.stderr, flush=True)
    r = redline_sweep(model, prompts, w.gen_len, w.block_size, cands, (2.0, 1), args.alpha, args.delta,
                      batch=w.batch, progress=say)
    print(json.dumps({"workload": w.name, "prompts": args.prompts, "alpha": args.alpha,
                      "delta": args.delta, "grid": r["grid"], "tpf": r["tpf"],
                      "V": r["V"].tolist(), "p": r["p"].tolist(), "valid": r["valid"].tolist(),
                      "selected": r["selected"], "selected_config": r["grid"][r["selected"]],
                      "near_ties": r["near_ties"]}))


if __name__ == "__main__":
    main()
