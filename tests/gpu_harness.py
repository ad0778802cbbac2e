"""Step-by-step GPU trace capture and lockstep comparison with the oracle.

The GPU decodes the whole batch through the C ABI, one bd_denoise_step +
bd_commit at a time, and records for every step the confidence and argmax of
each masked position (and, optionally, its logits).  The oracle then decodes
chosen sequences on the CPU; at every step it compares its statistics with the
GPU's and its own commit decision with the GPU's.  A differing decision is
excused only when the oracle's numbers make it a near-tie:

  T1  |conf - tau| <= 1e-3 at a position committed by one side only;
  T2  the two most probable tokens are within 1e-3 of probability;
  T3  a forced commit (of the sequence, or of one block under semi-completion)
      whose two best confidences are within 1e-3;
  T4  (MoE) a step whose forward, in the oracle, routed some row with a gap of
      at most 1e-4 between its k-th and (k+1)-th router logits: expert choice
      there can differ from the GPU's (float32 router logits of 16-bit
      activations carry errors of order 1e-5), so when such a step differs,
      its statistics and decisions are excused as a whole; such a step that
      agrees is counted like any other.

After an excused difference the oracle adopts the GPU's decision, so that the
rest of the trace stays comparable.  Any other difference is a failure.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

NEAR = 1e-3
ROUTER_NEAR = 1e-4


@dataclass
class GpuTrace:
    steps: list                      # per step: dict seq -> (positions, conf, tok, logits or None)
    tokens: np.ndarray               # [b][G]
    commit_step: np.ndarray          # [b][G]
    forwards: np.ndarray             # [b]
    stats: dict = None               # bd_state_stats after the decode


def capture_gpu_trace(model, prompts, G, tau, nb, B, logits_for=(), max_steps=None, logit_steps=None,
                      progress=None, tau_semi=None, tau_add=0.0, skip_masked=False, logit_every=1):
    """Decode the batch step by step; logits of the sequences in
    ``logits_for`` are kept on every ``logit_every``-th step (and only on the
    first ``logit_steps`` steps when that is given)."""
    import torch
    from paper_2609_33887_amd import bd
    st = bd.State(model, prompts, G, tau, nb, B, tau_semi, tau_add, skip_masked)
    b = st.b
    dev = model.device
    V = model.w.vocab
    conf = torch.empty((b, G), dtype=torch.float32, device=dev)
    tok = torch.empty((b, G), dtype=torch.int32, device=dev)
    logits = torch.empty((b, G, V), dtype=torch.float32, device=dev) if logits_for else None
    steps = []
    limit = max_steps or (G + 2)
    for s in range(limit):
        conf.fill_(-1.0)
        tok.fill_(-1)
        want_logits = (logits is not None and (logit_steps is None or s < logit_steps)
                       and s % logit_every == 0)
        st.step(conf, tok, logits if want_logits else None)
        done = st.commit(want_done=True)
        c = conf.cpu().numpy()
        t = tok.cpu().numpy()
        rec = {}
        for i in range(b):
            pos = np.nonzero(c[i] >= 0)[0]
            if pos.size:
                lg = None
                if want_logits and i in logits_for:
                    lg = logits[i, torch.as_tensor(pos, device=dev)].cpu().numpy()
                rec[i] = (pos, c[i, pos], t[i, pos], lg)
        steps.append(rec)
        if progress and s % 50 == 0:
            progress(f"  gpu step {s}")
        if done:
            break
    tokens, cstep, fwd = st.read()
    stats = st.stats()
    st.close()
    return GpuTrace(steps, tokens, cstep, fwd, stats)


@dataclass
class Report:
    max_conf_diff: float = 0.0
    max_logit_diff: float = 0.0
    # the same maxima over the compared steps whose routing had no near-tie
    # (MoE: every row's k-th and (k+1)-th router logits more than ROUTER_NEAR
    # apart in the oracle's forward; equal to the above for dense models)
    max_conf_diff_routed: float = 0.0
    max_logit_diff_routed: float = 0.0
    route_near_steps: int = 0        # compared steps with a routing near-tie that still passed
    t1: int = 0
    t2: int = 0
    t3: int = 0
    t4: int = 0
    positions: int = 0
    failures: list = field(default_factory=list)
    participation: dict = None       # oracle counters summed over the replayed sequences
    complete: bool = True            # every replayed sequence ran to its end


def prefilled(oracle_model, prompt, G, B, nb, tau, tau_semi=None, tau_add=0.0, skip_masked=False,
              cache=None, key=None):
    """An oracle decoder of one sequence after its prefill.  The prefill (the
    prompt's forward) depends only on the prompt and the block grid, so with
    a ``cache`` dict the prefilled KV cache is kept under ``key`` and copied
    into later decoders of the same prompt and block size, whatever their
    thresholds and in-flight count."""
    import copy
    from oracle.decode import SeqDecoder
    d = SeqDecoder(oracle_model, prompt, G, B, nb, tau, tau_semi, tau_add, skip_masked)
    if cache is None or key is None:
        d.prefill()
        return d
    if key not in cache:
        d.prefill()
        cache[key] = (copy.deepcopy(d.cache), d.cache_len)
        return d
    kv, clen = cache[key]
    d.cache = copy.deepcopy(kv)
    d.cache_len = clen
    d._admit()
    return d


def lockstep(oracle_model, prompts, seq_ids, trace: GpuTrace, G, tau, nb, B, conf_tol, logit_tol,
             max_steps=None, progress=None, tau_semi=None, tau_add=0.0, skip_masked=False,
             prefill_cache=None, cache_tag=None):
    """Replay the chosen sequences in the oracle against ``trace`` (the first
    ``max_steps`` steps of each when given)."""
    from oracle.decode import PART_NAMES
    rep = Report()
    part = np.zeros(len(PART_NAMES), dtype=np.int64)
    tau32 = float(np.float32(tau))
    for i in seq_ids:
        if progress:
            progress(f"  oracle prefill of sequence {i}")
        d = prefilled(oracle_model, prompts[i], G, B, nb, tau, tau_semi, tau_add, skip_masked,
                      prefill_cache, None if cache_tag is None else (cache_tag, i, B))
        P = d.P
        step = 0
        while not d.done and (max_steps is None or step < max_steps):
            if progress and step % 10 == 0:
                progress(f"  oracle step {step} of sequence {i}")
            if step >= len(trace.steps) or i not in trace.steps[step]:
                rep.failures.append((i, step, "GPU finished this sequence earlier than the oracle"))
                break
            gpos, gconf, gtok, glog = trace.steps[step][i]
            oracle_model.router_gaps = []
            masked, conf, tok, p2, z = d.forward_step(with_logits=True)
            if not np.array_equal(masked - P, gpos):
                rep.failures.append((i, step, "masked position sets differ"))
                break
            gaps = oracle_model.router_gaps
            near_route = bool(gaps) and min(float(np.min(g)) for g in gaps) <= ROUTER_NEAR
            # the step's comparison; a step whose routing had a near-tie is
            # excused (T4) only when it differs, and then as a whole
            fails, t1, t2, t3 = [], 0, 0, 0
            cdiff = float(np.max(np.abs(conf - gconf)))
            ldiff = 0.0
            if glog is not None:
                fin = np.isfinite(z)
                if not np.array_equal(fin, np.isfinite(glog)):
                    fails.append((i, step, "suppressed logit columns differ"))
                ldiff = float(np.max(np.abs(z[fin] - glog[fin])))
                if ldiff > logit_tol:
                    fails.append((i, step, f"logits differ by {ldiff:.3g}"))
            if cdiff > conf_tol:
                fails.append((i, step, f"confidence differs by {cdiff:.3g}"))
            # decisions
            own, forced = d.decision(masked, conf)
            gsel = trace.commit_step[i, masked - P] == step

            def forced_near(k):
                for grp in forced:
                    if k in grp and len(grp) > 1:
                        c2 = np.sort(conf[grp])
                        if c2[-1] - c2[-2] <= NEAR:
                            return True
                return False

            for k in np.nonzero(own != gsel)[0]:
                if abs(conf[k] - tau32) <= NEAR:
                    t1 += 1
                elif forced_near(k):
                    t3 += 1
                else:
                    fails.append((i, step, f"commit decision differs at position {masked[k] - P} "
                                           f"(oracle conf {conf[k]:.6f}, GPU conf {gconf[k]:.6f})"))
            both = own & gsel
            gtoks = trace.tokens[i, masked - P]
            for k in np.nonzero(both & (tok != gtoks))[0]:
                if conf[k] - p2[k] <= NEAR:
                    t2 += 1
                else:
                    fails.append((i, step, f"token differs at position {masked[k] - P}"))
            if fails and near_route:
                rep.t4 += 1
            else:
                rep.failures += fails
                rep.t1 += t1
                rep.t2 += t2
                rep.t3 += t3
                rep.positions += len(masked)
                rep.max_conf_diff = max(rep.max_conf_diff, cdiff)
                rep.max_logit_diff = max(rep.max_logit_diff, ldiff)
                if near_route:
                    rep.route_near_steps += 1
                else:
                    rep.max_conf_diff_routed = max(rep.max_conf_diff_routed, cdiff)
                    rep.max_logit_diff_routed = max(rep.max_logit_diff_routed, ldiff)
            d.count_participation(masked[gsel])
            d.apply(masked[gsel], gtoks[gsel], step)
            step += 1
        if d.done and d.forwards != trace.forwards[i]:
            rep.failures.append((i, step, f"forwards {d.forwards} vs GPU {trace.forwards[i]}"))
        if d.done and not np.array_equal(d.tokens[P:], trace.tokens[i]):
            rep.failures.append((i, step, "final tokens differ"))
        rep.complete &= bool(d.done)
        part += d.part
    rep.participation = dict(zip(PART_NAMES, part.tolist()))
    return rep
