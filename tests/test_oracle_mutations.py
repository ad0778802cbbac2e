"""Plants plausible mistakes in the oracle (on the CPU) and checks that the
independent pins catch each of them."""
import math

import numpy as np
import pytest

import oracle.model as om
import oracle.decode as od
from oracle.model import OracleModel
from tests.refmodels import TinyCfg, tiny_weights, scalar_forward, brute_decode


def _rope_wrong_sign(self, x, pos):
    ang = pos.astype(np.float64)[:, None] * self.inv_freq[None, :]
    c, s = np.cos(ang)[:, None, :], np.sin(ang)[:, None, :]
    h = self.hd // 2
    x1, x2 = x[..., :h], x[..., h:]
    return np.concatenate([x1 * c + x2 * s, x2 * c - x1 * s], axis=-1)


def _attention_strict_mask(self, q, qpos, K, V, B):
    e = K.shape[0]
    visible = (np.arange(e)[None, :] // B) < (qpos[:, None] // B)
    visible |= np.arange(e)[None, :] == qpos[:, None]
    out = np.empty(q.shape)
    for h in range(self.H):
        kv = h // (self.H // self.Hkv)
        s = np.where(visible, q[:, h] @ K[:, kv].T / math.sqrt(self.hd), -np.inf)
        out[:, h] = om._softmax_rows(s) @ V[:, kv]
    return out


def _attention_wrong_gqa(self, q, qpos, K, V, B):
    e = K.shape[0]
    visible = (np.arange(e)[None, :] // B) <= (qpos[:, None] // B)
    out = np.empty(q.shape)
    for h in range(self.H):
        kv = h % self.Hkv
        s = np.where(visible, q[:, h] @ K[:, kv].T / math.sqrt(self.hd), -np.inf)
        out[:, h] = om._softmax_rows(s) @ V[:, kv]
    return out


def _rms_no_gain(x, g, eps):
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps)


def _commit_strict(conf, tau):
    s = conf > float(np.float32(tau))
    if not s.any():
        s[int(np.argmax(conf))] = True
    return s


def _commit_last_argmax(conf, tau):
    s = conf >= float(np.float32(tau))
    if not s.any():
        s[len(conf) - 1 - int(np.argmax(conf[::-1]))] = True
    return s


def _apply_no_chain(self, positions, toks, step):
    for b in np.nonzero(self.status == od.PENDING)[0]:
        self.status[b] = od.CACHED
        self.cache_len += self.B
    self.tokens[positions] = toks
    self.commit_step[positions - self.P] = step
    for b in range(len(self.status)):            # commits at most one block per step
        if self.status[b] == od.ACTIVE:
            lo = self.P + b * self.B
            if not np.any(self.tokens[lo:lo + self.B] == self.mask_id):
                self.status[b] = od.PENDING
            break
    self._admit()
    self.forwards += 1


def _apply_skip_cache_write(self, positions, toks, step):
    # forgets that pending rows were written: cache_len jumps ahead one step early
    self.tokens[positions] = toks
    self.commit_step[positions - self.P] = step
    for b in range(len(self.status)):
        if self.status[b] in (od.CACHED, od.PENDING):
            continue
        if self.status[b] != od.ACTIVE:
            break
        lo = self.P + b * self.B
        if np.any(self.tokens[lo:lo + self.B] == self.mask_id):
            break
        self.status[b] = od.CACHED
        self.cache_len += self.B
    self._admit()
    self.forwards += 1


def _count_static_oldest(self, committed):
    # counts the oldest active block as one the skip rule could leave out
    act = np.nonzero(self.status == od.ACTIVE)[0]
    blk = (np.asarray(committed, dtype=np.int64) - self.P) // self.B
    for b in act:
        n_commit = int(np.count_nonzero(blk == int(b)))
        self.part[0] += 1
        self.part[1] += n_commit == 0
        if self.resolved(int(b)) == 0:
            self.part[2 if n_commit == 0 else 3] += 1
    self.part[4] += int(np.count_nonzero(self.status == od.PENDING))


def _forward_ignores_skip(self):
    return np.nonzero(self.status == od.ACTIVE)[0]


MUTATIONS = {
    "rope_sign": ("OracleModel.rope", _rope_wrong_sign),
    "mask_strict": ("OracleModel.attention", _attention_strict_mask),
    "gqa_modulo": ("OracleModel.attention", _attention_wrong_gqa),
    "norm_no_gain": ("_rmsnorm", _rms_no_gain),
    "commit_strict": ("commit_set", _commit_strict),
    "forced_top1_last": ("commit_set", _commit_last_argmax),
    "sweep_no_chain": ("SeqDecoder.apply", _apply_no_chain),
    "cache_write_early": ("SeqDecoder.apply", _apply_skip_cache_write),
    "static_counts_oldest": ("SeqDecoder.count_participation", _count_static_oldest),
    "skip_not_applied": ("SeqDecoder.forwarded", _forward_ignores_skip),
}


def _pins_pass():
    """A compact run of the independent pins; False as soon as one fails
    (a crash of the mutated oracle counts as caught)."""
    try:
        return _run_pins()
    except (ValueError, IndexError, RuntimeError):
        return False


def _run_pins():
    cfg = TinyCfg(n_heads=4, n_kv_heads=2)
    ws = tiny_weights(cfg, 0, 0.3)
    m = OracleModel(cfg, ws, "f64")
    toks = np.array([3, 1, 4, 1, 5, 9, 2, cfg.mask_id])
    for B in (1, 2, 4):
        got = m.logits(m.forward(toks, 0, 8, m.kv_cache(8), B))
        if not np.allclose(got, scalar_forward(cfg, ws, list(toks), B), atol=1e-9):
            return False
    t32 = float(np.float32(0.9))
    if od.commit_set(np.array([t32, t32, 0.1]), 0.9).tolist() != [True, True, False]:
        return False
    if od.commit_set(np.array([0.3, 0.5, 0.5]), 0.9).tolist() != [False, True, False]:
        return False
    for P, G, B, nb, tau in ((4, 12, 2, 3, 0.0), (2, 6, 2, 2, 0.5), (4, 12, 4, 3, 0.3)):
        prompt = np.random.default_rng(P + G).integers(0, cfg.vocab - 1, P)
        bt, bs, steps = brute_decode(cfg, ws, list(prompt), G, B, nb, tau)
        r = od.decode_batch(m, prompt[None], G, B, nb, tau)
        if not (np.array_equal(r.tokens[0], bt) and np.array_equal(r.commit_step[0], bs)):
            return False
    for skip in (False, True):
        prompt = np.random.default_rng(5).integers(0, cfg.vocab - 1, 2)
        cnt = {}
        bt, bs, steps = brute_decode(cfg, ws, list(prompt), 6, 2, 3, 0.5, skip_masked=skip,
                                     counters=cnt)
        r = od.decode_batch(m, prompt[None], 6, 2, 3, 0.5, skip_masked=skip)
        if not (np.array_equal(r.commit_step[0], bs)
                and dict(zip(od.PART_NAMES, r.participation.tolist())) == cnt):
            return False
    return True


def test_unmutated_oracle_passes():
    assert _pins_pass()


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_planted_mistake_is_caught(name, monkeypatch):
    target, fn = MUTATIONS[name]
    if target.startswith("OracleModel."):
        monkeypatch.setattr(OracleModel, target.split(".")[1], fn)
    elif target.startswith("SeqDecoder."):
        monkeypatch.setattr(od.SeqDecoder, target.split(".")[1], fn)
    elif target == "commit_set":
        monkeypatch.setattr(od, "commit_set", fn)
    else:
        monkeypatch.setattr(om, target, fn)
    assert not _pins_pass(), f"planted mistake {name} went unnoticed"
