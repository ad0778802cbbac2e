"""Independent reference implementations used to pin the oracle.

These are written separately from ``oracle/`` on purpose:

* ``scalar_forward`` -- a scalar-loop float64 forward over a whole sequence
  (no cache), with an explicit (i, j) block-causal mask predicate and an
  explicit softmax; for tiny models only.
* ``torch_causal_logits`` -- a textbook causal transformer written with
  torch's scaled-dot-product attention (``is_causal=True``), float64 on CPU.
* ``brute_decode`` -- the decode rules restated compactly over block
  counters, re-running the full-sequence forward every step (no cache, no
  pending rows).
"""
import math

import numpy as np
import torch


class TinyCfg:
    def __init__(self, n_layers=2, d_model=16, n_heads=2, n_kv_heads=1, head_dim=8, ffn_dim=24,
                 vocab=11, n_experts=0, top_k=0, expert_ffn=0, n_shared=0, rms_eps=1e-6,
                 rope_theta=1e4, logit_scale=20.0):
        self.__dict__.update(locals())
        del self.__dict__["self"]
        self.qkv_dim = (n_heads + 2 * n_kv_heads) * head_dim
        self.mask_id = vocab - 1


def tiny_weights(cfg, seed=0, std=0.3):
    """Weights in ABI order with a large spread so that confidences vary."""
    rng = np.random.default_rng(seed)
    d, hd = cfg.d_model, cfg.head_dim
    g = lambda *s: rng.standard_normal(s) * std
    ws = [g(cfg.vocab, d)]
    for _ in range(cfg.n_layers):
        ws += [1.0 + 0.1 * rng.standard_normal(d), g(cfg.qkv_dim, d), g(d, cfg.n_heads * hd),
               1.0 + 0.1 * rng.standard_normal(d)]
        if cfg.n_experts == 0:
            ws += [g(cfg.ffn_dim, d), g(cfg.ffn_dim, d), g(d, cfg.ffn_dim)]
        else:
            e, fe, fs = cfg.n_experts, cfg.expert_ffn, cfg.n_shared * cfg.expert_ffn
            ws += [g(e, d), g(e, fe, d), g(e, fe, d), g(e, d, fe), g(fs, d), g(fs, d), g(d, fs)]
    ws += [1.0 + 0.1 * rng.standard_normal(d), g(cfg.vocab, d)]
    return [np.asarray(w, dtype=np.float64) for w in ws]


def _unpack(cfg, ws):
    it = iter(ws)
    emb = next(it)
    layers = []
    for _ in range(cfg.n_layers):
        L = dict(an=next(it), qkv=next(it), o=next(it), fn=next(it))
        if cfg.n_experts == 0:
            L.update(g=next(it), u=next(it), dn=next(it))
        else:
            L.update(r=next(it), ge=next(it), ue=next(it), de=next(it), gs=next(it), us=next(it),
                     ds=next(it))
        layers.append(L)
    return emb, layers, next(it), next(it)


# ---------------------------------------------------------------- scalar loops
def _matvec(W, x):
    return [sum(W[o][i] * x[i] for i in range(len(x))) for o in range(len(W))]


def _rms(x, g, eps):
    r = math.sqrt(sum(v * v for v in x) / len(x) + eps)
    return [x[i] / r * g[i] for i in range(len(x))]


def _silu(v):
    return v / (1.0 + math.exp(-v))


def _rope_vec(x, pos, hd, theta):
    h = hd // 2
    out = list(x)
    for i in range(h):
        a = pos * theta ** (-2.0 * i / hd)
        c, s = math.cos(a), math.sin(a)
        out[i] = x[i] * c - x[i + h] * s
        out[i + h] = x[i + h] * c + x[i] * s
    return out


def _ffn_scalar(cfg, L, a):
    if cfg.n_experts == 0:
        gv, uv = _matvec(L["g"], a), _matvec(L["u"], a)
        return _matvec(L["dn"], [_silu(gv[f]) * uv[f] for f in range(len(gv))])
    logits = _matvec(L["r"], a)
    mx = max(logits)
    ex = [math.exp(z - mx) for z in logits]
    probs = [e / sum(ex) for e in ex]
    chosen = sorted(range(cfg.n_experts), key=lambda e: (-probs[e], e))[:cfg.top_k]
    wsum = sum(probs[e] for e in chosen)
    out = [0.0] * cfg.d_model
    for e in chosen:
        gv, uv = _matvec(L["ge"][e], a), _matvec(L["ue"][e], a)
        y = _matvec(L["de"][e], [_silu(gv[f]) * uv[f] for f in range(len(gv))])
        out = [out[i] + probs[e] / wsum * y[i] for i in range(cfg.d_model)]
    gv, uv = _matvec(L["gs"], a), _matvec(L["us"], a)
    y = _matvec(L["ds"], [_silu(gv[f]) * uv[f] for f in range(len(gv))])
    return [out[i] + y[i] for i in range(cfg.d_model)]


def scalar_forward(cfg, ws, tokens, B):
    """Logits of every position of ``tokens`` under the block-causal mask:
    query i sees key j iff floor(j / B) <= floor(i / B)."""
    emb, layers, gfin, lm = _unpack(cfg, ws)
    T, H, Hkv, hd = len(tokens), cfg.n_heads, cfg.n_kv_heads, cfg.head_dim
    xs = [list(emb[t]) for t in tokens]
    for L in layers:
        qs, ks, vs = [], [], []
        for i in range(T):
            a = _rms(xs[i], L["an"], cfg.rms_eps)
            y = _matvec(L["qkv"], a)
            q = [_rope_vec(y[h * hd:(h + 1) * hd], i, hd, cfg.rope_theta) for h in range(H)]
            k = [_rope_vec(y[(H + h) * hd:(H + h + 1) * hd], i, hd, cfg.rope_theta) for h in range(Hkv)]
            v = [y[(H + Hkv + h) * hd:(H + Hkv + h + 1) * hd] for h in range(Hkv)]
            qs.append(q); ks.append(k); vs.append(v)
        new = []
        for i in range(T):
            o = []
            for h in range(H):
                kv = h // (H // Hkv)
                scores = {}
                for j in range(T):
                    if j // B <= i // B:
                        scores[j] = sum(qs[i][h][c] * ks[j][kv][c] for c in range(hd)) / math.sqrt(hd)
                mx = max(scores.values())
                w = {j: math.exp(s - mx) for j, s in scores.items()}
                tot = sum(w.values())
                o += [sum(w[j] / tot * vs[j][kv][c] for j in w) for c in range(hd)]
            x = [xs[i][c] + val for c, val in enumerate(_matvec(L["o"], o))]
            a = _rms(x, L["fn"], cfg.rms_eps)
            f = _ffn_scalar(cfg, L, a)
            new.append([x[c] + f[c] for c in range(cfg.d_model)])
        xs = new
    out = []
    for i in range(T):
        h = _rms(xs[i], gfin, cfg.rms_eps)
        z = [cfg.logit_scale * v for v in _matvec(lm, h)]
        z[cfg.mask_id] = -math.inf
        out.append(z)
    return np.array(out)


# ---------------------------------------------------------------- torch causal LM
def torch_causal_logits(cfg, ws, tokens):
    """Ordinary causal transformer (dense FFN), torch float64 on CPU."""
    emb, layers, gfin, lm = [None] * 4
    emb, layers, gfin, lm = _unpack(cfg, ws)
    t = lambda a: torch.tensor(np.asarray(a), dtype=torch.float64)
    T, H, Hkv, hd = len(tokens), cfg.n_heads, cfg.n_kv_heads, cfg.head_dim
    x = t(emb)[torch.tensor(tokens)]
    pos = torch.arange(T, dtype=torch.float64)
    inv = cfg.rope_theta ** (-torch.arange(0, hd, 2, dtype=torch.float64) / hd)
    ang = pos[:, None] * inv[None, :]
    rot = torch.polar(torch.ones_like(ang), ang)                   # e^{i pos w}

    def rope(v):  # v: [T, heads, hd]; complex pairs (i, i + hd/2)
        c = torch.complex(v[..., :hd // 2], v[..., hd // 2:]) * rot[:, None, :]
        return torch.cat([c.real, c.imag], dim=-1)

    def rms(v, g):
        return v * torch.rsqrt((v * v).mean(-1, keepdim=True) + cfg.rms_eps) * t(g)

    for L in layers:
        a = rms(x, L["an"])
        y = a @ t(L["qkv"]).T
        q = rope(y[:, :H * hd].reshape(T, H, hd))
        k = rope(y[:, H * hd:(H + Hkv) * hd].reshape(T, Hkv, hd))
        v = y[:, (H + Hkv) * hd:].reshape(T, Hkv, hd)
        rep = H // Hkv
        k = k.repeat_interleave(rep, dim=1)
        v = v.repeat_interleave(rep, dim=1)
        o = torch.nn.functional.scaled_dot_product_attention(
            q.transpose(0, 1), k.transpose(0, 1), v.transpose(0, 1), is_causal=True)
        x = x + o.transpose(0, 1).reshape(T, H * hd) @ t(L["o"]).T
        a = rms(x, L["fn"])
        x = x + (torch.nn.functional.silu(a @ t(L["g"]).T) * (a @ t(L["u"]).T)) @ t(L["dn"]).T
    z = cfg.logit_scale * (rms(x, gfin) @ t(lm).T)
    z[:, cfg.mask_id] = -math.inf
    return z.numpy()


# ---------------------------------------------------------------- brute decode
def brute_decode(cfg, ws, prompt, G, B, nb, tau, forward=scalar_forward, tau_semi=None, tau_add=0.0,
                 skip_masked=False, counters=None):
    """Decode by recomputing the whole sequence every step.

    Block k of the generation is committed once it and all blocks before it
    hold no mask; blocks in [committed, admitted) are active; at most ``nb``
    blocks are active; a step commits every masked position of an active block
    with confidence >= tau, or the single most confident one.  With
    ``tau_semi``: the single most confident position is taken per block, in
    every active block with none above tau whose previous block is committed
    or had at least the fraction tau_semi of its positions unmasked when the
    step began.  A further block is admitted while fewer than nb are active
    and either none is active or the last admitted one has at least the
    fraction tau_add of its positions unmasked (fractions in float32).
    With ``skip_masked`` an active block other than the first one that has
    no unmasked position yet stays out of the step.  ``counters`` (a dict)
    receives, summed over steps: "active_forwards" (active blocks in the
    step), "zero_commit" (of those, ones that commit nothing),
    "static_saved" / "static_deferred" (of those, ones other than the first
    active block with nothing unmasked before the step that commit nothing /
    something), "cache_writes" (blocks committed in the previous step, which
    this step recomputes) and "skipped" (active blocks left out)."""
    P = len(prompt)
    tokens = list(prompt) + [cfg.mask_id] * G
    nblk = G // B
    f32 = np.float32

    def unmasked(k):
        return sum(1 for p in range(P + k * B, P + (k + 1) * B) if tokens[p] != cfg.mask_id)

    def admit(committed, admitted):
        while admitted < nblk and admitted - committed < nb and \
                (admitted == committed or f32(unmasked(admitted - 1)) / f32(B) >= f32(tau_add)):
            admitted += 1
        return admitted

    committed = 0
    admitted = admit(0, 0)
    commit_step = [-1] * G
    steps = 0
    tau32 = float(np.float32(tau))
    cnt = {k: 0 for k in ("active_forwards", "zero_commit", "static_saved", "static_deferred",
                          "cache_writes", "skipped")}
    newly_committed = 0
    while committed < nblk:
        live = [k for k in range(committed, admitted)
                if not (skip_masked and k > committed and unmasked(k) == 0)]
        cnt["skipped"] += (admitted - committed) - len(live)
        cnt["cache_writes"] += newly_committed
        before = {k: unmasked(k) for k in live}
        end = P + (live[-1] + 1) * B
        z = forward(cfg, ws, tokens[:end], B)
        cand = [p for p in range(P + committed * B, end)
                if tokens[p] == cfg.mask_id and (p - P) // B in live]
        stats = []
        for p in cand:
            row = z[p]
            mx = max(row)
            tot = sum(math.exp(v - mx) for v in row if v != -math.inf)
            tok = min(i for i, v in enumerate(row) if v == mx)
            stats.append((1.0 / tot, tok))
        chosen = [i for i, (c, _) in enumerate(stats) if c >= tau32]
        if tau_semi is None:
            if not chosen:
                best = max(c for c, _ in stats)
                chosen = [min(i for i, (c, _) in enumerate(stats) if c == best)]
        else:
            done_before = {k: unmasked(k) for k in range(committed, admitted)}
            for k in range(committed, admitted):
                mine = [i for i, p in enumerate(cand) if (p - P) // B == k]
                if not mine or any(i in chosen for i in mine):
                    continue
                if k == committed or f32(done_before[k - 1]) / f32(B) >= f32(tau_semi):
                    best = max(stats[i][0] for i in mine)
                    chosen.append(min(i for i in mine if stats[i][0] == best))
        for i in chosen:
            tokens[cand[i]] = stats[i][1]
            commit_step[cand[i] - P] = steps
        for k in live:
            n = sum(1 for i in chosen if (cand[i] - P) // B == k)
            cnt["active_forwards"] += 1
            cnt["zero_commit"] += n == 0
            if k > committed and before[k] == 0:
                cnt["static_saved" if n == 0 else "static_deferred"] += 1
        was = committed
        while committed < admitted and cfg.mask_id not in tokens[P + committed * B:P + (committed + 1) * B]:
            committed += 1
        newly_committed = committed - was
        admitted = admit(committed, admitted)
        steps += 1
    if counters is not None:
        counters.update(cnt)
    return np.array(tokens[P:]), np.array(commit_step), steps
