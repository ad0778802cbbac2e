#!/usr/bin/env python3
"""Throughput of the block-diffusion denoising path on one MI355X.

A bench "step" is one full decode of the workload's batch: every denoising
step (window forward + fused LM head + commit) until all b x G tokens are
committed.  Prompts are encoded once before timing (prefill is not part of
the step); each timed decode starts from the post-prefill state
(bd_state_reset, a single small kernel, inside the timed region).  The
number of denoising steps per decode is learnt in an untimed first decode
(the trace is deterministic), so timed decodes launch exactly that many
steps with no host synchronisation.

Prints one JSON line: committed tokens/s, TPF, step latency, the roofline
of the dominant kernel class (HIP events on the library's stream in a
second, profiled pass over the same decodes), and the CPU oracle timed on a
bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0          # MI355X HBM3E
PEAK_BF16_TFLOPS = 2500.0      # dense bf16 MFMA
PEAK_F32_TFLOPS = 157.3        # fp32 vector


def algorithmic_work(w, stats, wq="bf16"):
    """FLOPs and HBM bytes per kernel class for the work recorded in ``stats``
    (counters summed over one decode).  Bytes count each weight once per
    forward (for MoE layers, every expert: an upper bound, as nearly all of
    the 64 experts receive rows at these batch sizes), the K/V read once per
    (sequence, kv head, layer) and the window K/V written; FLOPs count only
    visible query-key pairs and masked LM rows.  With fp8 layer weights the
    layer projections read 1 byte per weight (the per-row scales are
    negligible); the LM head stays bf16."""
    esz = 2 if w.dtype == "bf16" else 4     # LM-head weights
    lsz = 1 if wq == "fp8" else esz         # decoder-layer projection weights
    asz = 4                                  # activations / KV: fp32 or a bf16 hi/lo pair
    d, H, Hkv, hd, F, V, L = w.d_model, w.n_heads, w.n_kv_heads, w.head_dim, w.ffn_dim, w.vocab, w.n_layers
    qkv = (H + 2 * Hkv) * hd
    rows, lm_rows, fw = stats["rows"], stats["lm_rows"], stats["forwards"]
    gemm = {"gemm_qkv": (qkv, d), "gemm_o": (d, H * hd)}
    if not w.n_experts:
        gemm.update({"gemm_gu": (2 * F, d), "gemm_down": (d, F)})
    out = {}
    for k, (N, K) in gemm.items():
        flops = 2.0 * rows * N * K * L
        byts = (N * K * lsz * fw + rows * K * asz + rows * N * 4) * L
        out[k] = (flops, byts)
    if w.n_experts:
        # routed experts: each row meets top_k experts; the shared experts see every row
        Fe, Fs, E, k = w.expert_ffn, w.n_shared * w.expert_ffn, w.n_experts, w.top_k
        out["gemm_gu"] = (2.0 * rows * (k * 2 * Fe + 2 * Fs) * d * L,
                          ((E + w.n_shared) * 2 * Fe * d * lsz * fw + rows * (k + 1) * d * asz) * L)
        out["gemm_down"] = (2.0 * rows * (k * Fe + Fs) * d * L,
                            ((E + w.n_shared) * Fe * d * lsz * fw + rows * (k + 1) * (Fe * asz + d * 4)) * L)
    out["attn"] = (4.0 * hd * H * stats["pairs"] * L,
                   (stats["keys"] * Hkv * hd * 2 * asz + rows * H * hd * asz
                    + rows * H * hd * asz) * L)
    out["lm_head"] = (2.0 * lm_rows * V * d, V * d * esz * fw + lm_rows * d * asz)
    return out


def source_tag(path):
    """First 12 hex digits of the SHA-256 of a source file (to tell whether a
    kernel changed since its counters were taken)."""
    import hashlib
    with open(path, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:12]


def measured_traffic(workload_name, kernel_class):
    """HBM bytes per launch of ``kernel_class`` from the committed counter
    summary of this workload (FETCH_SIZE and WRITE_SIZE passes, scaled by the
    plain-copy calibration), or None when there is none or when the kernel
    source has changed since the counters were taken."""
    path = os.path.join(ROOT, "profiles", f"{workload_name}_hbm_counters.md")
    if not os.path.exists(path):
        return None
    rec = {}
    with open(path) as f:
        for line in f:
            if line.startswith("counters:"):
                r = dict(kv.split("=", 1) for kv in line.split()[1:])
                if r.get("class") == kernel_class:
                    rec = r
    if not rec or source_tag(os.path.join(ROOT, rec["source"])) != rec["source_sha256_12"]:
        return None
    return {"bytes_per_launch": float(rec["bytes_per_launch"]),
            "algorithmic_bytes_per_launch": float(rec["algorithmic_bytes_per_launch"]),
            "launches": rec["launches"]}


def cpu_baseline(w, weights, prompts, tau, target_s=12.0, tau_semi=None, tau_add=0.0, skip_masked=False):
    """The oracle as it stands, on the host cores, over whole sequences of the
    same batch until about ``target_s`` seconds of decode work (prefill
    excluded, as on the GPU)."""
    import numpy as np
    from oracle.model import OracleModel
    from oracle.decode import SeqDecoder
    try:
        from threadpoolctl import threadpool_info
        cores = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        cores = len(os.sched_getaffinity(0))
    om = OracleModel(w, weights, "f64" if w.dtype == "f32" else "bf16")
    spent, tokens, seqs = 0.0, 0, 0
    for i in range(prompts.shape[0]):
        d = SeqDecoder(om, prompts[i], w.gen_len, w.block_size, w.n_inflight, tau, tau_semi, tau_add,
                       skip_masked)
        d.prefill()
        t0 = time.perf_counter()
        s = 0
        while not d.done:
            d.step(s)
            s += 1
        spent += time.perf_counter() - t0
        tokens += w.gen_len
        seqs += 1
        if spent >= target_s:
            break
    return {"value": tokens / spent, "unit": "committed tokens/s", "cores": int(cores), "kind": "oracle",
            "sample": f"{seqs} of {prompts.shape[0]} sequences of workload {w.name}, whole decodes at "
                      f"tau={tau}, prefill excluded, {spent:.1f} s"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5, help="timed decodes of the whole batch")
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--config", type=int, default=1)
    ap.add_argument("--tau", type=float, default=0.9)
    ap.add_argument("--tau-semi", type=float, default=None,
                    help="semi-completion threshold (default: off)")
    ap.add_argument("--tau-add", type=float, default=0.0,
                    help="admission threshold (default 0: refill every free slot)")
    ap.add_argument("--wq", choices=["bf16", "fp8"], default="bf16",
                    help="weight precision of the decoder-layer projections")
    ap.add_argument("--skip-masked", action="store_true",
                    help="static skip rule: leave fully masked blocks behind an active one out of the forward")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--trace-steps", type=int, default=0, metavar="N",
                    help="only encode the prompts and run N denoising steps (a short program for "
                         "rocprofv3 counter passes), print the per-step work counters and exit")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only copy MIB MiB device-to-device 5 times (a known-size kernel that scales "
                         "the FETCH_SIZE / WRITE_SIZE counters) and exit")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py runs on one GPU only: the library has no multi-GPU path (batch rows would shard "
              "across GPUs with no exchange during decode)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    if args.copy_calibration:
        n = args.copy_calibration << 20
        src = torch.ones(n // 4, dtype=torch.int32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_per_launch": n, "launches": 5}))
        return
    from bd_synth import workload, make_weights, make_prompts
    from paper_2609_33887_amd import bd

    w = workload(args.config)
    print(f"[bench] workload {w.name}: building weights", file=sys.stderr, flush=True)
    weights = make_weights(w)
    prompts = make_prompts(w)
    model = bd.Model(w, weights, wq=None if args.wq == "bf16" else args.wq)
    st = bd.State(model, prompts, w.gen_len, args.tau, w.n_inflight, w.block_size, args.tau_semi,
                  args.tau_add, args.skip_masked)
    if args.trace_steps:
        torch.cuda.synchronize()
        print(f"[bench] prefill done; running {args.trace_steps} denoising steps", file=sys.stderr, flush=True)
        for _ in range(args.trace_steps):
            st.step()
            st.commit()
        torch.cuda.synchronize()
        print(json.dumps({"workload": w.name, "trace_steps": args.trace_steps, "stats": st.stats()}))
        st.close()
        model.close()
        return
    # untimed reference decode: learn the step count, keep the trace
    done, S = False, 0
    while not done:
        st.step()
        done = st.commit(want_done=True)
        S += 1
    ref_tokens, ref_cs, ref_fw = st.read()
    stats = st.stats()
    tpf = float(w.batch * w.gen_len) / float(ref_fw.sum())
    print(f"[bench] {S} denoising steps per decode, TPF {tpf:.4f}", file=sys.stderr, flush=True)

    def one_decode():
        st.reset()
        for _ in range(S):
            st.step()
            st.commit()

    for _ in range(args.warmup):
        one_decode()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t_wall = time.perf_counter()
    e0.record()
    for _ in range(args.steps):
        one_decode()
    e1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_wall
    ms = e0.elapsed_time(e1) / args.steps
    tok, cs, fw = st.read()
    if not (np.array_equal(tok, ref_tokens) and np.array_equal(cs, ref_cs)):
        raise RuntimeError("timed decode differs from the reference decode")
    value = w.batch * w.gen_len / (ms / 1e3)

    # profiled pass: per-kernel-class HIP events on the library stream
    bd.bd_profile(model.handle, True)
    for _ in range(args.steps):
        one_decode()
    prof = bd.bd_profile_read(model.handle)
    bd.bd_profile(model.handle, False)
    work = algorithmic_work(w, stats, args.wq)
    kernels = {}
    for k, (tms, n) in prof.items():
        if n == 0:
            continue
        entry = {"ms_per_decode": tms / args.steps, "launches_per_decode": n // args.steps}
        if k in work:
            fl, by = work[k]
            sec = tms / args.steps / 1e3
            entry["tflops"] = fl / sec / 1e12
            entry["gbs"] = by / sec / 1e9
        kernels[k] = entry
    dom = max((k for k in kernels if k in work), key=lambda k: kernels[k]["ms_per_decode"])
    fl, by = work[dom]
    ai = fl / by
    peak_f = PEAK_BF16_TFLOPS if w.dtype == "bf16" else PEAK_F32_TFLOPS
    ridge = peak_f * 1e12 / (PEAK_HBM_GBS * 1e9)
    if ai >= ridge:
        roof = {"bound": "mfma", "achieved": kernels[dom]["tflops"], "peak": peak_f, "unit": "TFLOP/s"}
    else:
        roof = {"bound": "hbm", "achieved": kernels[dom]["gbs"], "peak": PEAK_HBM_GBS, "unit": "GB/s"}
    roof["frac"] = roof["achieved"] / roof["peak"]
    mt = measured_traffic(w.name, dom)
    roof["traffic"] = mt["bytes_per_launch"] if mt else None
    if mt:
        roof["traffic_note"] = (f"HBM bytes per launch (FETCH_SIZE x2 + WRITE_SIZE x1) over {mt['launches'].replace('_', ' ')}; "
                                f"algorithmic bytes per launch over the same launches: "
                                f"{mt['algorithmic_bytes_per_launch']:.4g}")
    roof["kernel"] = dom
    roof["avg_launch_us"] = 1e3 * kernels[dom]["ms_per_decode"] / kernels[dom]["launches_per_decode"]

    cpu = None
    if not args.no_cpu_baseline:
        print("[bench] timing the CPU oracle", file=sys.stderr, flush=True)
        ow = weights
        if args.wq == "fp8":
            from oracle.quant import fp8_weights
            ow = fp8_weights(w, weights)
        cpu = cpu_baseline(w, ow, prompts, args.tau, args.cpu_seconds, args.tau_semi, args.tau_add,
                           args.skip_masked)

    line = {
        "metric": "committed tokens/sec/GPU (TPF at tau=0.9; step latency; HBM GB/s, MFMA util)",
        "value": value, "unit": "committed tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": w.dtype, "data": "synthetic (seeded random-init weights and prompts)",
        "config": {"workload": w.name, "batch": w.batch, "prompt_len": w.prompt_len, "gen_len": w.gen_len,
                   "block_size": w.block_size, "n_inflight": w.n_inflight, "tau": args.tau,
                   **({"tau_semi": args.tau_semi, "tau_add": args.tau_add}
                      if args.tau_semi is not None or args.tau_add else {}),
                   **({"skip_masked": True} if args.skip_masked else {}),
                   **({"weights": args.wq} if args.wq != "bf16" else {})},
        "tpf": tpf, "denoise_steps_per_decode": S, "step_latency_us": 1e3 * ms / S,
        "wall_s": wall, "roofline": roof, "kernels": kernels, "cpu_baseline": cpu,
        "participation": {k: stats[k] for k in ("active_forwards", "zero_commit", "static_saved",
                                                "static_deferred", "cache_writes", "skipped")},
    }
    print(json.dumps(line))
    st.close()
    model.close()


if __name__ == "__main__":
    main()
