"""Pins of the decode oracle: closed forms, brute force, textbook special
cases and invariants (block size 1 = causal decoding; cached step = full
recompute; at least one token per step; tau > 1 gives one token per step;
maximal exact commit)."""
import itertools
import math

import numpy as np
import pytest
import torch

from oracle.model import OracleModel, round_bf16, lm_stats
from oracle.decode import (SeqDecoder, decode_batch, commit_set, ACTIVE, PENDING, CACHED,
                           PLACEHOLDER, PART_NAMES)
from tests.refmodels import TinyCfg, tiny_weights, scalar_forward, torch_causal_logits, brute_decode


# ---------------------------------------------------------------- numerics pieces
def test_round_bf16_matches_torch():
    rng = np.random.default_rng(1)
    x = np.concatenate([rng.standard_normal(20000) * 10.0 ** rng.integers(-6, 6, 20000),
                        [1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -2.5, 0.0, 65504.0]])
    want = torch.tensor(x, dtype=torch.float64).to(torch.float32).to(torch.bfloat16).to(torch.float64)
    np.testing.assert_array_equal(round_bf16(x), want.numpy())
    assert round_bf16(np.array([1.0 + 2 ** -8]))[0] == 1.0              # tie -> even
    assert round_bf16(np.array([1.0 + 3 * 2 ** -8]))[0] == 1.0 + 2 ** -6


def test_split_bf16x2_carries_16_bits():
    """hi + lo represents fp32(x) to 16 significant bits; both halves are
    bf16 values; values that are already bf16 have lo = 0."""
    from oracle.model import split_bf16x2
    rng = np.random.default_rng(8)
    x = rng.standard_normal(50000) * 10.0 ** rng.integers(-4, 4, 50000)
    x32 = x.astype(np.float32).astype(np.float64)
    y = split_bf16x2(x)
    assert np.all(np.abs(y - x32) <= np.abs(x32) * 2.0 ** -16)
    hi = round_bf16(x32)
    np.testing.assert_array_equal(round_bf16(y - hi), y - hi)
    b = round_bf16(x)
    np.testing.assert_array_equal(split_bf16x2(b), b)


def _model(cfg=None, seed=0, precision="f64", std=0.3):
    cfg = cfg or TinyCfg()
    return cfg, tiny_weights(cfg, seed, std), OracleModel(cfg, tiny_weights(cfg, seed, std), precision)


def test_rope_is_complex_rotation_and_relative():
    cfg, _, m = _model(TinyCfg(head_dim=8))
    rng = np.random.default_rng(2)
    q = rng.standard_normal((5, 2, 8))
    pos = np.array([0, 1, 7, 100, 9000])
    got = m.rope(q, pos)
    z = (q[..., :4] + 1j * q[..., 4:]) * np.exp(1j * pos[:, None, None] * 1e4 ** (-np.arange(4) * 2 / 8))
    np.testing.assert_allclose(got, np.concatenate([z.real, z.imag], -1), rtol=0, atol=1e-12)
    np.testing.assert_allclose(m.rope(q[:1], np.array([0])), q[:1], atol=0)
    # the score between a rotated query and key depends only on the offset
    a, b = rng.standard_normal((1, 1, 8)), rng.standard_normal((1, 1, 8))
    s = lambda i, j: float(np.sum(m.rope(a, np.array([i])) * m.rope(b, np.array([j]))))
    assert s(10, 3) == pytest.approx(s(107, 100), abs=1e-9)


def test_rmsnorm_unit_rms():
    from oracle.model import _rmsnorm
    x = np.random.default_rng(3).standard_normal((4, 64)) * 7
    y = _rmsnorm(x, np.ones(64), 0.0)
    np.testing.assert_allclose(np.sqrt(np.mean(y * y, -1)), 1.0, rtol=1e-12)


@pytest.mark.parametrize("B,causal", [(64, False), (1, True)])
def test_attention_special_cases_match_torch(B, causal):
    """One block covering everything = full attention; B = 1 = causal attention."""
    cfg, _, m = _model(TinyCfg(n_heads=4, n_kv_heads=2, head_dim=8))
    rng = np.random.default_rng(4)
    T = 12
    q, k, v = rng.standard_normal((T, 4, 8)), rng.standard_normal((T, 2, 8)), rng.standard_normal((T, 2, 8))
    got = m.attention(q, np.arange(T), k, v, B)
    tq = torch.tensor(q).transpose(0, 1)
    tk = torch.tensor(k).repeat_interleave(2, 1).transpose(0, 1)
    tv = torch.tensor(v).repeat_interleave(2, 1).transpose(0, 1)
    want = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, is_causal=causal)
    np.testing.assert_allclose(got, want.transpose(0, 1).numpy(), atol=1e-12)


def test_lm_stats_identities():
    """conf = max softmax probability in (0, 1]; shift invariance; the
    suppressed mask column never wins; lowest id among equal maxima."""
    rng = np.random.default_rng(5)
    z = rng.standard_normal((50, 33)) * 5
    conf, tok, p2 = lm_stats(z)
    e = np.exp(z - z.max(1, keepdims=True))
    prob = e / e.sum(1, keepdims=True)
    np.testing.assert_allclose(conf, prob.max(1), rtol=1e-14)
    np.testing.assert_array_equal(tok, prob.argmax(1))
    np.testing.assert_allclose(p2, np.sort(prob, 1)[:, -2], rtol=1e-13)
    c2, t2, _ = lm_stats(z + 123.25)
    np.testing.assert_allclose(c2, conf, rtol=1e-12)
    np.testing.assert_array_equal(t2, tok)
    assert np.all((conf > 0) & (conf <= 1))
    tie = np.array([[0.0, 3.0, 1.0, 3.0]])
    assert lm_stats(tie)[1][0] == 1
    cfg, _, m = _model()
    h = np.zeros((1, cfg.d_model))
    h[0, 0] = 1.0
    m.lm_head[:] = 0.0
    m.lm_head[cfg.mask_id, 0] = 100.0        # mask column would win without suppression
    m.lm_head[3, 0] = 0.5
    zz = m.logits(h)
    assert zz[0, cfg.mask_id] == -np.inf and lm_stats(zz)[1][0] == 3


def test_commit_rule():
    assert commit_set(np.array([0.2, 0.95, 0.9, 0.91]), 0.9).tolist() == [False, True, True, True]
    assert commit_set(np.array([0.2, 0.5, 0.5]), 0.9).tolist() == [False, True, False]
    assert commit_set(np.array([1.0, 1.0]), 2.0).tolist() == [True, False]
    assert commit_set(np.array([0.1, 0.3]), 0.0).all()


# ---------------------------------------------------------------- P5: brute force
@pytest.mark.parametrize("B", [1, 2, 4, 8])
def test_forward_matches_scalar_loops(B):
    cfg, ws, m = _model(TinyCfg())
    toks = np.array([3, 1, 4, 1, 5, 9, 2, cfg.mask_id])
    want = scalar_forward(cfg, ws, list(toks), B)
    cache = m.kv_cache(8)
    got = m.logits(m.forward(toks, 0, 8, cache, B))
    np.testing.assert_allclose(got, want, atol=1e-10)


def test_moe_forward_matches_scalar_loops():
    cfg, ws, m = _model(TinyCfg(n_experts=4, top_k=2, expert_ffn=6, n_shared=1, ffn_dim=0))
    toks = np.array([3, 1, 4, 1, 5, 9, 2, 6])
    got = m.logits(m.forward(toks, 0, 8, m.kv_cache(8), 2))
    np.testing.assert_allclose(got, scalar_forward(cfg, ws, list(toks), 2), atol=1e-10)


def test_moe_all_experts_is_dense_mixture():
    cfg, ws, m = _model(TinyCfg(n_experts=3, top_k=3, expert_ffn=5, n_shared=1, ffn_dim=0))
    L = m.layers[0]
    a = np.random.default_rng(6).standard_normal((7, cfg.d_model))
    lg = a @ L["w_router"].T
    pr = np.exp(lg - lg.max(1, keepdims=True))
    pr /= pr.sum(1, keepdims=True)
    silu = lambda x: x / (1 + np.exp(-x))
    want = sum(pr[:, e:e + 1] * ((silu(a @ L["w_gate_e"][e].T) * (a @ L["w_up_e"][e].T)) @ L["w_down_e"][e].T)
               for e in range(3))
    want = want + (silu(a @ L["w_gate_s"].T) * (a @ L["w_up_s"].T)) @ L["w_down_s"].T
    np.testing.assert_allclose(m.moe_ffn(a, L), want, atol=1e-12)


CASES = [(P, B, nb, tau) for B in (1, 2, 4, 8) for P in range(0, 8, B)
         for nb in (1, 2, 3) for tau in (0.0, 0.5, 0.9, 2.0)]


@pytest.mark.parametrize("P,B,nb,tau", CASES)
def test_decode_matches_brute_force(P, B, nb, tau):
    """2-layer model, 8 tokens, vocabulary 11: the cached oracle decode equals
    full recomputation with independently restated rules."""
    G = 8 - P
    cfg, ws, m = _model(TinyCfg())
    prompt = np.random.default_rng(P * 100 + B).integers(0, cfg.vocab - 1, P)
    bt, bs, bsteps = brute_decode(cfg, ws, list(prompt), G, B, nb, tau)
    r = decode_batch(m, prompt[None, :], G, B, nb, tau)
    np.testing.assert_array_equal(r.tokens[0], bt)
    np.testing.assert_array_equal(r.commit_step[0], bs)
    assert r.forwards[0] == bsteps


SEMI_CASES = [(P, B, nb, tau, ts, ta) for B in (2, 4) for P in range(0, 8 - B, B) for nb in (2, 3)
              for tau in (0.5, 0.9, 2.0) for ts, ta in ((0.5, 0.0), (0.5, 0.5), (1.0, 0.25), (0.0, 1.0))]


@pytest.mark.parametrize("P,B,nb,tau,tau_semi,tau_add", SEMI_CASES)
def test_decode_with_semi_and_add_matches_brute_force(P, B, nb, tau, tau_semi, tau_add):
    """The semi-completion and admission thresholds (App. F): cached oracle
    decode = full recomputation with the rules restated independently."""
    G = 8 - P
    cfg, ws, m = _model(TinyCfg())
    prompt = np.random.default_rng(P * 100 + B + 7).integers(0, cfg.vocab - 1, P)
    bt, bs, bsteps = brute_decode(cfg, ws, list(prompt), G, B, nb, tau, tau_semi=tau_semi, tau_add=tau_add)
    r = decode_batch(m, prompt[None, :], G, B, nb, tau, tau_semi=tau_semi, tau_add=tau_add)
    np.testing.assert_array_equal(r.tokens[0], bt)
    np.testing.assert_array_equal(r.commit_step[0], bs)
    assert r.forwards[0] == bsteps


@pytest.mark.parametrize("nb", [2, 3])
def test_semi_zero_forces_one_token_per_block(nb):
    """tau > 1 and tau_semi = 0: every active block is fully activated and
    resolves one position per step, so nb blocks finish together every B
    steps: forwards = G / nb, TPF = nb (G / B a multiple of nb)."""
    cfg, ws, m = _model(TinyCfg(vocab=29))
    P, B = 4, 4
    G = B * nb * 2
    prompts = np.random.default_rng(16).integers(0, cfg.vocab - 1, (2, P))
    r = decode_batch(m, prompts, G, B, nb, 2.0, tau_semi=0.0, tau_add=0.0)
    assert r.forwards.tolist() == [G // nb] * 2 and r.tpf == nb
    np.testing.assert_array_equal(np.sort(r.commit_step[0]), np.repeat(np.arange(G // nb), nb))


@pytest.mark.parametrize("nb", [2, 3])
def test_semi_above_one_forces_only_the_oldest_block(nb):
    """tau > 1 and tau_semi > 1: only the oldest active block (whose
    predecessor is committed) may force a commit: one token per step."""
    cfg, ws, m = _model(TinyCfg(vocab=29))
    P, G, B = 4, 24, 4
    prompts = np.random.default_rng(17).integers(0, cfg.vocab - 1, (2, P))
    r = decode_batch(m, prompts, G, B, nb, 2.0, tau_semi=1.5)
    assert r.forwards.tolist() == [G, G] and r.tpf == 1.0


@pytest.mark.parametrize("tau", [0.4, 0.8])
def test_add_one_or_single_block_reduces_to_one_block_decoding(tau):
    """tau_add = 1 admits a block only when no other is in flight, and with
    one block in flight the semi-completion rule is the base rule: both give
    the n_inflight = 1 trace."""
    cfg, ws, m = _model(TinyCfg(vocab=31), seed=5, std=0.4)
    P, G, B = 4, 32, 4
    prompts = np.random.default_rng(18).integers(0, cfg.vocab - 1, (2, P))
    base = decode_batch(m, prompts, G, B, 1, tau)
    for nb, ts in ((3, 0.7), (2, None), (3, 0.0)):
        r = decode_batch(m, prompts, G, B, nb, tau, tau_semi=ts, tau_add=1.0)
        np.testing.assert_array_equal(r.commit_step, base.commit_step)
        np.testing.assert_array_equal(r.tokens, base.tokens)
    r = decode_batch(m, prompts, G, B, 1, tau, tau_semi=0.9, tau_add=0.3)
    np.testing.assert_array_equal(r.commit_step, base.commit_step)


# ------------------------------------------- static skip rule and participation
SKIP_CASES = [(P, B, nb, tau, ts, skip) for B in (1, 2, 4) for P in range(0, 8 - B, B) for nb in (2, 3)
              for tau in (0.0, 0.5, 0.9, 2.0) for ts in (None, 0.5) for skip in (False, True)]


@pytest.mark.parametrize("P,B,nb,tau,tau_semi,skip", SKIP_CASES)
def test_participation_and_skip_match_brute_force(P, B, nb, tau, tau_semi, skip):
    """Participation counters (App. B.3) and the live
    static skip rule (§3.3): cached oracle decode = full
    recomputation with the rule and the counts restated independently."""
    G = 8 - P
    cfg, ws, m = _model(TinyCfg())
    prompt = np.random.default_rng(P * 100 + B + 11).integers(0, cfg.vocab - 1, P)
    cnt = {}
    bt, bs, bsteps = brute_decode(cfg, ws, list(prompt), G, B, nb, tau, tau_semi=tau_semi,
                                  skip_masked=skip, counters=cnt)
    r = decode_batch(m, prompt[None, :], G, B, nb, tau, tau_semi=tau_semi, skip_masked=skip)
    np.testing.assert_array_equal(r.tokens[0], bt)
    np.testing.assert_array_equal(r.commit_step[0], bs)
    assert r.forwards[0] == bsteps
    assert dict(zip(PART_NAMES, r.participation.tolist())) == cnt


def _sweep_steps(commit_step, B):
    """Step at which each block leaves the active set: the latest commit of
    the block and of every block before it (in-order sweep)."""
    last = commit_step.reshape(-1, B).max(axis=1)
    return np.maximum.accumulate(last)


@pytest.mark.parametrize("nb,tau,ts", [(2, 0.5, None), (3, 0.8, None), (2, 0.8, 0.6), (3, 2.0, None),
                                       (3, 0.3, 0.0)])
def test_skip_rule_reduces_to_one_block_in_flight(nb, tau, ts):
    """A fully masked block can only gain a token by being forwarded, and the
    skip rule forwards it only once no older block is active; so only the
    oldest active block ever takes part and the decode is the n_inflight = 1
    decode, position by position, while the n_inflight - 1 admitted blocks
    behind it are skipped at every step where they exist."""
    cfg, ws, m = _model(TinyCfg(vocab=31), seed=5, std=0.4)
    P, G, B = 4, 32, 4
    prompts = np.random.default_rng(19).integers(0, cfg.vocab - 1, (3, P))
    base = decode_batch(m, prompts, G, B, 1, tau, tau_semi=ts)
    r = decode_batch(m, prompts, G, B, nb, tau, tau_semi=ts, skip_masked=True)
    np.testing.assert_array_equal(r.tokens, base.tokens)
    np.testing.assert_array_equal(r.commit_step, base.commit_step)
    np.testing.assert_array_equal(r.forwards, base.forwards)
    part = dict(zip(PART_NAMES, r.participation.tolist()))
    assert part["active_forwards"] == int(base.forwards.sum())
    assert part["static_saved"] == part["static_deferred"] == 0
    # skipped: at each step min(nb, blocks not yet swept) - 1 blocks wait
    nblk = G // B
    expect = 0
    for i in range(len(prompts)):
        sw = _sweep_steps(r.commit_step[i], B)
        for t in range(int(r.forwards[i])):
            left = nblk - int(np.count_nonzero(sw < t))
            expect += min(nb, left) - 1
    assert part["skipped"] == expect


@pytest.mark.parametrize("nb,tau,ts", [(1, 0.7, None), (2, 0.7, None), (3, 0.5, 0.5), (2, 0.0, None),
                                       (3, 2.0, None), (1, 2.0, None)])
def test_participation_closed_forms(nb, tau, ts):
    """Counter identities that follow from the rules alone:
    * every step of a sequence forwards each active block once, so the active
      block-forwards are the sum over steps of the blocks neither swept nor
      unadmitted, min(nb, blocks not yet swept) without admission thresholds;
    * cache writes: every block swept before a sequence's final step is
      recomputed by the next one (App. F.2);
    * n_inflight = 1: no block has an older active block;
    * tau > 1 without semi-completion: exactly one block commits per step,
      so the zero-commit forwards are the active forwards minus the forwards;
    * tau = 0: every forwarded block resolves at once, so none commits
      nothing and each block is forwarded once while active."""
    cfg, ws, m = _model(TinyCfg(vocab=31), seed=5, std=0.4)
    P, G, B = 4, 24, 4
    prompts = np.random.default_rng(23).integers(0, cfg.vocab - 1, (3, P))
    r = decode_batch(m, prompts, G, B, nb, tau, tau_semi=ts)
    part = dict(zip(PART_NAMES, r.participation.tolist()))
    nblk = G // B
    act = cw = 0
    for i in range(len(prompts)):
        sw = _sweep_steps(r.commit_step[i], B)
        final = int(r.forwards[i]) - 1
        assert sw.max() == final
        cw += int(np.count_nonzero(sw < final))
        for t in range(int(r.forwards[i])):
            act += min(nb, nblk - int(np.count_nonzero(sw < t)))
    assert part["active_forwards"] == act
    assert part["cache_writes"] == cw
    assert part["skipped"] == 0
    if nb == 1:
        assert part["static_saved"] == part["static_deferred"] == 0
    if tau > 1 and ts is None:
        assert part["zero_commit"] == act - int(r.forwards.sum())
    if tau == 0:
        assert part["zero_commit"] == 0 and act == nblk * len(prompts)
    assert part["static_saved"] + part["static_deferred"] <= part["active_forwards"]


# ---------------------------------------------------------------- P2: causal decoding
def test_block_size_one_is_greedy_causal_decoding():
    cfg, ws, m = _model(TinyCfg(vocab=23, n_kv_heads=2), seed=3)
    P, G = 5, 9
    prompt = list(np.random.default_rng(9).integers(0, cfg.vocab - 1, P))
    toks = list(prompt)
    for p in range(P, P + G):
        z = torch_causal_logits(cfg, ws, toks + [cfg.mask_id])[p]
        toks.append(int(np.argmax(z)))
    for tau in (0.0, 0.7, 2.0):
        r = decode_batch(m, np.array([prompt]), G, 1, 1, tau)
        assert r.tokens[0].tolist() == toks[P:]
        assert r.forwards[0] == G


# ---------------------------------------------------------------- P1: cache = recompute
@pytest.mark.parametrize("precision", ["f64", "bf16"])
def test_cached_step_equals_full_recompute(precision):
    cfg = TinyCfg(n_layers=3, d_model=32, n_heads=4, n_kv_heads=2, head_dim=8, ffn_dim=48, vocab=37)
    ws = tiny_weights(cfg, 11, 0.2)
    m = OracleModel(cfg, ws, precision)
    P, G, B, nb = 8, 24, 4, 2
    prompt = np.random.default_rng(12).integers(0, cfg.vocab - 1, P)
    d = SeqDecoder(m, prompt, G, B, nb, 0.6)
    d.prefill()
    checked = 0
    step = 0
    while not d.done:
        s, e = d.window()
        fresh = m.kv_cache(P + G)
        full = m.forward(d.tokens, 0, e, fresh, B)[s:]
        cached = m.forward(d.tokens, s, e, d.cache, B)
        # bf16 mode: BLAS may accumulate the two row sets in different orders
        # before the 16-bit operand roundings
        tol = 1e-12 if precision == "f64" else 2e-4
        np.testing.assert_allclose(cached, full, atol=tol, rtol=0)
        checked += 1
        d.step(step)
        step += 1
    assert checked == d.forwards and checked >= 3


# ---------------------------------------------------------------- P3 / P4: closed forms
@pytest.mark.parametrize("nb", [1, 2, 3])
def test_tau_above_one_commits_one_token_per_step(nb):
    cfg, ws, m = _model(TinyCfg(vocab=29))
    P, G, B = 4, 24, 4
    prompts = np.random.default_rng(13).integers(0, cfg.vocab - 1, (2, P))
    r = decode_batch(m, prompts, G, B, nb, 2.0)
    assert r.forwards.tolist() == [G, G] and r.tpf == 1.0
    for i in range(2):
        assert sorted(r.commit_step[i].tolist()) == list(range(G))


@pytest.mark.parametrize("nb", [1, 2, 3])
def test_tau_zero_resolves_each_block_in_one_step(nb):
    cfg, ws, m = _model(TinyCfg(vocab=29))
    P, G, B = 4, 28, 4
    prompts = np.random.default_rng(14).integers(0, cfg.vocab - 1, (1, P))
    r = decode_batch(m, prompts, G, B, nb, 0.0)
    nblk = G // B
    assert r.forwards[0] == math.ceil(nblk / nb)
    assert r.tpf == G / math.ceil(nblk / nb)
    np.testing.assert_array_equal(r.commit_step[0], np.repeat(np.arange(nblk) // nb, B))


# ---------------------------------------------------------------- P6: invariants
@pytest.mark.parametrize("tau,nb", [(0.3, 3), (0.6, 2), (0.9, 3), (0.99, 1)])
def test_commit_invariants(tau, nb):
    cfg, ws, m = _model(TinyCfg(vocab=31), seed=5, std=0.4)
    P, G, B = 4, 32, 4
    prompt = np.random.default_rng(15).integers(0, cfg.vocab - 1, P)
    d = SeqDecoder(m, prompt, G, B, nb, tau)
    d.keep_records = True
    d.prefill()
    s = 0
    while not d.done:
        before = d.status.copy()
        d.step(s)
        rec = d.records[-1]
        assert len(rec.committed) >= 1                       # at least one token per step
        st = rec.status_after
        # slot order: cached / pending blocks form a prefix, then active, then placeholders
        order = [{CACHED: 0, PENDING: 0, ACTIVE: 1, PLACEHOLDER: 2}[x] for x in st]
        assert order == sorted(order)
        # maximal exact commit: no active complete block preceded only by committed blocks
        first_active = next((b for b in range(len(st)) if st[b] == ACTIVE), None)
        if first_active is not None:
            lo = P + first_active * B
            assert np.any(d.tokens[lo:lo + B] == cfg.mask_id)
        assert np.count_nonzero(st == ACTIVE) <= nb
        # transitions are one-way: placeholder -> active -> pending -> cached
        rank = {PLACEHOLDER: 0, ACTIVE: 1, PENDING: 2, CACHED: 3}
        assert all(rank[a] <= rank[b] for a, b in zip(before, st))
        s += 1
    cs = d.commit_step
    assert np.all(cs >= 0) and np.all(d.tokens != cfg.mask_id)
    assert sum(len(r.committed) for r in d.records) == G
    # blocks enter the cache in order
    done_step = [cs[b * B:(b + 1) * B].max() for b in range(G // B)]
    assert all(np.maximum.accumulate(done_step) >= done_step)


def test_bf16_mode_differs_only_at_storage_points(monkeypatch):
    """With the storage rounding switched off, bf16 mode equals f64 mode up to
    float32 matmul accumulation."""
    import oracle.model as om
    cfg = TinyCfg(n_layers=2, d_model=32, n_heads=4, n_kv_heads=2, head_dim=8, ffn_dim=48, vocab=37)
    ws = [np.float32(w).astype(np.float64) for w in tiny_weights(cfg, 21, 0.2)]
    toks = np.array([1, 2, 3, 4, 5, 6, 7, 8])
    a = OracleModel(cfg, ws, "f64")
    za = a.logits(a.forward(toks, 0, 8, a.kv_cache(8), 4))
    monkeypatch.setattr(om, "round_bf16", lambda x: np.asarray(x, dtype=np.float64))
    monkeypatch.setattr(om, "split_bf16x2", lambda x: np.asarray(x, dtype=np.float64))
    b = OracleModel(cfg, ws, "bf16")
    zb = b.logits(b.forward(toks, 0, 8, b.kv_cache(8), 4))
    np.testing.assert_allclose(zb, za, atol=2e-4)
