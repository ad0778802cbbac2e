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
second, profiled pass over the same decodes) and of the whole step, the
prefill time (reported apart), whether the timed decodes reproduced the
reference decode bit for bit, the CPU oracle timed on a bounded sample of the
same workload, and shorter runs of the batch-16 dense and batch-64 MoE
workloads as sub-entries.
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
    (counters summed over one decode), at the method's widths: bf16
    activations, Q/K/V and K/V cache entries count 2 bytes (4 for fp32
    models), whatever representation the kernels carry them in; FLOPs count
    one product per multiply-add of the method (the extra products of the
    kernels' high/low bf16 operand pairs are not counted).  Bytes count each
    weight once per forward (for MoE layers every expert: nearly all of the
    64 receive rows at these batch sizes), each kernel's activation operand
    and output once, the K/V read once per (sequence, kv head, layer) and the
    window K/V written; FLOPs count only visible query-key pairs and masked
    LM rows.  With fp8 layer weights the layer projections read 1 byte per
    weight (the per-row scales are negligible); the LM head stays bf16."""
    esz = 2 if w.dtype == "bf16" else 4     # LM-head / embedding weights
    # decoder-layer projection weights: fp8 1 byte, MXFP4 half a byte + an exponent per 32
    lsz = 1 if wq == "fp8" else (0.5 + 1 / 32 if wq == "mxfp4" else esz)
    asz = esz                                # activations, Q/K/V, K/V cache
    d, H, Hkv, hd, F, V, L = w.d_model, w.n_heads, w.n_kv_heads, w.head_dim, w.ffn_dim, w.vocab, w.n_layers
    qkv = (H + 2 * Hkv) * hd
    rows, lm_rows, fw = stats["rows"], stats["lm_rows"], stats["forwards"]
    out = {}
    # (N, K, output bytes per element): QKV writes Q/K/V, O and down add into
    # the fp32 residual stream (read and written), gate/up writes the SwiGLU product
    gemm = {"gemm_qkv": (qkv, d, asz), "gemm_o": (d, H * hd, 8)}
    if not w.n_experts:
        gemm["gemm_gu"] = (2 * F, d, None)
        gemm["gemm_down"] = (d, F, 8)
    for k, (N, K, osz) in gemm.items():
        flops = 2.0 * rows * N * K * L
        outb = rows * (N // 2) * asz if osz is None else rows * N * osz
        out[k] = (flops, (N * K * lsz * fw + rows * K * asz + outb) * L)
    if w.n_experts:
        # routed experts: each row meets top_k experts; the shared experts see every row
        Fe, Fs, E, k = w.expert_ffn, w.n_shared * w.expert_ffn, w.n_experts, w.top_k
        out["gemm_gu"] = (2.0 * rows * (k * 2 * Fe + 2 * Fs) * d * L,
                          ((E + w.n_shared) * 2 * Fe * d * lsz * fw
                           + rows * (k + 1) * (d + Fe) * asz) * L)
        out["gemm_down"] = (2.0 * rows * (k * Fe + Fs) * d * L,
                            ((E + w.n_shared) * Fe * d * lsz * fw + rows * (k + 1) * (Fe * asz + d * 4)) * L)
    # attention: keys read once per (sequence, kv head) and step (K and V),
    # Q read and O written once per row and head, window K/V written once
    out["attn"] = (4.0 * hd * H * stats["pairs"] * L,
                   (stats["keys"] * Hkv * hd * 2 * asz + 2 * rows * H * hd * asz
                    + rows * Hkv * hd * 2 * asz) * L)
    out["lm_head"] = (2.0 * lm_rows * V * d, V * d * esz * fw + lm_rows * d * asz)
    return out


def step_work(w, stats, wq="bf16"):
    """Whole-step algorithmic work of one decode (the roofline of the step):
    FLOPs of every projection, the LM head on masked rows and the visible
    attention pairs; HBM bytes of every weight read once per forward (MoE:
    every expert), the K/V cache read once per (sequence, kv head, layer),
    the window K/V written, the embedding rows gathered and the per-row
    token/confidence I/O.  Activations passed between kernels are not
    counted (a fused step would not move them)."""
    work = algorithmic_work(w, stats, wq)
    flops = sum(f for f, _ in work.values())
    esz = 2 if w.dtype == "bf16" else 4
    lsz = 1 if wq == "fp8" else (0.5 + 1 / 32 if wq == "mxfp4" else esz)
    d, H, Hkv, hd, L = w.d_model, w.n_heads, w.n_kv_heads, w.head_dim, w.n_layers
    qkv = (H + 2 * Hkv) * hd
    if w.n_experts:
        Fe, Fs, E = w.expert_ffn, w.n_shared * w.expert_ffn, w.n_experts
        layer_w = qkv * d + d * H * hd + (E * 3 * Fe + 3 * Fs) * d
    else:
        layer_w = qkv * d + d * H * hd + 3 * w.ffn_dim * d
    fw, rows = stats["forwards"], stats["rows"]
    byts = (layer_w * L * lsz + w.vocab * d * esz) * fw
    byts += (stats["keys"] * Hkv * hd * 2 + rows * Hkv * hd * 2) * esz * L
    byts += rows * d * esz + stats["lm_rows"] * 8
    return flops, byts


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


def cpu_baseline(w, weights, prompts, tau, target_s=15.0, tau_semi=None, tau_add=0.0, skip_masked=False):
    """The oracle as it stands, on the host cores: sequences of the same
    batch decoded step by step (prefill excluded, as on the GPU) until about
    ``target_s`` seconds of denoising work; committed tokens / time."""
    import numpy as np
    from oracle.model import OracleModel
    from oracle.decode import SeqDecoder
    try:
        from threadpoolctl import threadpool_info
        cores = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        cores = len(os.sched_getaffinity(0))
    om = OracleModel(w, weights, "f64" if w.dtype == "f32" else "bf16")
    spent, tokens, steps, seqs = 0.0, 0, 0, 0
    for i in range(prompts.shape[0]):
        d = SeqDecoder(om, prompts[i], w.gen_len, w.block_size, w.n_inflight, tau, tau_semi, tau_add,
                       skip_masked)
        d.prefill()
        seqs += 1
        s = 0
        while not d.done and spent < target_s:
            before = int(np.count_nonzero(d.tokens == d.mask_id))
            t0 = time.perf_counter()
            d.step(s)
            spent += time.perf_counter() - t0
            tokens += before - int(np.count_nonzero(d.tokens == d.mask_id))
            s += 1
            steps += 1
        if spent >= target_s:
            break
    return {"value": tokens / spent, "unit": "committed tokens/s", "cores": int(cores), "kind": "oracle",
            "sample": f"{steps} denoising steps over {seqs} of the {prompts.shape[0]} sequences of workload "
                      f"{w.name} (each decoded from its first step; prefill excluded), tau={tau}: "
                      f"{tokens} tokens committed in {spent:.1f} s"}


def measure(w, tau, steps, warmup, wq="bf16", tau_semi=None, tau_add=0.0, skip_masked=False,
            weights=None, prof_decodes=None, say=None):
    """Decode the workload's batch on the GPU: one untimed reference decode
    (learns the step count), ``warmup`` untimed and ``steps`` timed decodes
    (HIP events on the library's stream, no host synchronisation inside),
    then a profiled pass with per-kernel-class HIP events.  Returns the
    measurement (and the host weights, for the CPU baseline)."""
    import numpy as np
    import torch
    from bd_synth import make_weights, make_prompts
    from paper_2609_33887_amd import bd
    say = say or (lambda m: None)
    say(f"workload {w.name}: building weights")
    if weights is None:
        weights = make_weights(w)
    prompts = make_prompts(w)
    model = bd.Model(w, weights, wq=None if wq == "bf16" else wq)
    torch.cuda.synchronize()
    t_pre = time.perf_counter()
    st = bd.State(model, prompts, w.gen_len, tau, w.n_inflight, w.block_size, tau_semi, tau_add, skip_masked)
    torch.cuda.synchronize()
    prefill_s = time.perf_counter() - t_pre
    say(f"{w.name}: prefill of {w.batch} x {w.prompt_len} prompt tokens in {1e3 * prefill_s:.1f} ms")
    done, S = False, 0
    while not done:
        st.step()
        done = st.commit(want_done=True)
        S += 1
    ref_tokens, ref_cs, ref_fw = st.read()
    stats = st.stats()
    tpf = float(w.batch * w.gen_len) / float(ref_fw.sum())
    say(f"{w.name}: {S} denoising steps per decode, TPF {tpf:.4f}")

    stream = model.stream          # the torch stream the library launches on

    def one_decode():
        st.reset()
        for _ in range(S):
            st.step()
            st.commit()

    for _ in range(warmup):
        one_decode()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t_wall = time.perf_counter()
    e0.record(stream)
    for _ in range(steps):
        one_decode()
    e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_wall
    ms = e0.elapsed_time(e1) / steps
    tok, cs, fw = st.read()
    if not (np.array_equal(tok, ref_tokens) and np.array_equal(cs, ref_cs)):
        raise RuntimeError("timed decode differs from the reference decode")
    value = w.batch * w.gen_len / (ms / 1e3)
    say(f"{w.name}: {value:.0f} committed tokens/s, {ms:.2f} ms per decode")

    # profiled pass: per-kernel-class HIP events on the library stream
    npd = prof_decodes or min(steps, 3)
    bd.bd_profile(model.handle, True)
    for _ in range(npd):
        one_decode()
    prof = bd.bd_profile_read(model.handle)
    bd.bd_profile(model.handle, False)
    work = algorithmic_work(w, stats, wq)
    kernels = {}
    for k, (tms, n) in prof.items():
        if n == 0:
            continue
        entry = {"ms_per_decode": tms / npd, "launches_per_decode": n // npd}
        if k in work:
            fl, by = work[k]
            sec = tms / npd / 1e3
            entry["tflops"] = fl / sec / 1e12
            entry["gbs"] = by / sec / 1e9
            entry["avg_launch_us"] = 1e3 * tms / n
        kernels[k] = entry
    dom = max((k for k in kernels if k in work), key=lambda k: kernels[k]["ms_per_decode"])
    fl, by = work[dom]
    peak_f = PEAK_BF16_TFLOPS if w.dtype == "bf16" else PEAK_F32_TFLOPS
    ridge = peak_f * 1e12 / (PEAK_HBM_GBS * 1e9)
    if fl / by >= ridge:
        roof = {"bound": "mfma", "achieved": kernels[dom]["tflops"], "peak": peak_f, "unit": "TFLOP/s"}
    else:
        roof = {"bound": "hbm", "achieved": kernels[dom]["gbs"], "peak": PEAK_HBM_GBS, "unit": "GB/s"}
    roof["frac"] = roof["achieved"] / roof["peak"]
    # the counter summaries are of the bf16-weight kernels
    mt = measured_traffic(w.name, dom) if wq == "bf16" else None
    roof["traffic"] = mt["bytes_per_launch"] if mt else None
    launches = kernels[dom]["launches_per_decode"]
    roof["algorithmic_per_launch"] = {"flops": fl / launches, "bytes": by / launches}
    if mt:
        roof["traffic_note"] = (f"HBM bytes per launch (FETCH_SIZE x2 + WRITE_SIZE x1, copy-calibrated) over "
                                f"{mt['launches'].replace('_', ' ')}; algorithmic bytes per launch over the "
                                f"same launches: {mt['algorithmic_bytes_per_launch']:.4g}")
    roof["kernel"] = dom
    roof["avg_launch_us"] = kernels[dom]["avg_launch_us"]
    # whole step: the larger of its HBM and MFMA times at peak, against the measured step
    sfl, sby = step_work(w, stats, wq)
    t_hbm = sby / (PEAK_HBM_GBS * 1e9) / S
    t_mfma = sfl / (peak_f * 1e12) / S
    step_s = ms / 1e3 / S
    step_roof = {"bytes_per_step": sby / S, "flops_per_step": sfl / S,
                 "t_hbm_us": 1e6 * t_hbm, "t_mfma_us": 1e6 * t_mfma, "step_us": 1e6 * step_s,
                 "frac_hbm": t_hbm / step_s, "frac_mfma": t_mfma / step_s,
                 "frac": max(t_hbm, t_mfma) / step_s,
                 "bound": "hbm" if t_hbm >= t_mfma else "mfma"}
    res = {"workload": w, "value": value, "ms": ms, "wall": wall, "tpf": tpf, "S": S, "stats": stats,
           "roofline": roof, "step_roofline": step_roof, "kernels": kernels, "weights": weights,
           "prompts": prompts,
           "prefill": {"wall_ms": 1e3 * prefill_s,
                       "prompt_tokens_per_s": w.batch * w.prompt_len / prefill_s,
                       "note": "first bd_prefill of the batch, host clock around the state's creation "
                               "(its device allocation included); outside the timed decodes"}}
    st.close()
    model.close()
    return res


SUB_WORKLOADS = (1, 4)      # batch <= 16 (HBM target) and batch >= 64 (MFMA target)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5, help="timed decodes of the whole batch")
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--config", type=int, default=2,
                    help="workload index (default 2: the multi-block GQA model, the largest per-step work)")
    ap.add_argument("--tau", type=float, default=0.9)
    ap.add_argument("--tau-semi", type=float, default=None,
                    help="semi-completion threshold (default: off)")
    ap.add_argument("--tau-add", type=float, default=0.0,
                    help="admission threshold (default 0: refill every free slot)")
    ap.add_argument("--wq", choices=["bf16", "fp8", "mxfp4"], default="bf16",
                    help="weight precision of the decoder-layer projections")
    ap.add_argument("--skip-masked", action="store_true",
                    help="static skip rule: leave fully masked blocks behind an active one out of the forward")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-sub", action="store_true",
                    help="skip the sub-entries (dense-1024 and moe-2048 at tau 0.9)")
    ap.add_argument("--sub-steps", type=int, default=3, help="timed decodes of each sub-entry")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
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

    import torch

    def say(msg):
        print(f"[bench] {msg}", file=sys.stderr, flush=True)

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
    if args.trace_steps:
        say(f"workload {w.name}: building weights")
        weights = make_weights(w)
        model = bd.Model(w, weights, wq=None if args.wq == "bf16" else args.wq)
        st = bd.State(model, make_prompts(w), w.gen_len, args.tau, w.n_inflight, w.block_size, args.tau_semi,
                      args.tau_add, args.skip_masked)
        torch.cuda.synchronize()
        say(f"prefill done; running {args.trace_steps} denoising steps")
        for _ in range(args.trace_steps):
            st.step()
            st.commit()
        torch.cuda.synchronize()
        print(json.dumps({"workload": w.name, "trace_steps": args.trace_steps, "stats": st.stats()}))
        st.close()
        model.close()
        return

    r = measure(w, args.tau, args.steps, args.warmup, args.wq, args.tau_semi, args.tau_add, args.skip_masked,
                say=say)
    weights, prompts = r.pop("weights"), r.pop("prompts")
    cpu = None
    if not args.no_cpu_baseline:
        say("timing the CPU oracle")
        ow = weights
        if args.wq == "fp8":
            from oracle.quant import fp8_weights
            ow = fp8_weights(w, weights)
        elif args.wq == "mxfp4":
            from oracle.quant import mxfp4_weights
            ow = mxfp4_weights(w, weights)
        cpu = cpu_baseline(w, ow, prompts, args.tau, args.cpu_seconds, args.tau_semi, args.tau_add,
                           args.skip_masked)
    del weights
    subs = {}
    if not args.no_sub and args.config not in SUB_WORKLOADS:
        for c in SUB_WORKLOADS:
            sw = workload(c)
            q = measure(sw, 0.9, args.sub_steps, 1, say=say)
            subs[sw.name] = {"value": q["value"], "unit": "committed tokens/s", "tpf": q["tpf"],
                             "ms_per_decode": q["ms"], "denoise_steps_per_decode": q["S"],
                             "step_latency_us": 1e3 * q["ms"] / q["S"], "batch": sw.batch, "tau": 0.9,
                             "roofline": q["roofline"], "step_roofline": q["step_roofline"]}
            del q

    line = {
        "metric": "committed tokens/sec/GPU (TPF at tau=0.9; step latency; HBM GB/s, MFMA util)",
        "value": r["value"], "unit": "committed tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": r["ms"], "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": w.dtype, "data": "synthetic (seeded random-init weights and prompts)",
        "config": {"workload": w.name, "batch": w.batch, "prompt_len": w.prompt_len, "gen_len": w.gen_len,
                   "block_size": w.block_size, "n_inflight": w.n_inflight, "tau": args.tau,
                   **({"tau_semi": args.tau_semi, "tau_add": args.tau_add}
                      if args.tau_semi is not None or args.tau_add else {}),
                   **({"skip_masked": True} if args.skip_masked else {}),
                   **({"weights": args.wq} if args.wq != "bf16" else {})},
        "tpf": r["tpf"], "denoise_steps_per_decode": r["S"], "step_latency_us": 1e3 * r["ms"] / r["S"],
        "wall_s": r["wall"], "prefill": r["prefill"],
        "deterministic": True,       # every timed decode reproduced the reference decode bit for bit
        "roofline": r["roofline"], "step_roofline": r["step_roofline"],
        "kernels": r["kernels"], "cpu_baseline": cpu,
        "participation": {k: r["stats"][k] for k in ("active_forwards", "zero_commit", "static_saved",
                                                     "static_deferred", "cache_writes", "skipped")},
        "sub_workloads": subs,
    }
    print(json.dumps(line))


if __name__ == "__main__":
    main()
