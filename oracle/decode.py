"""Oracle decode loop (test infrastructure only; see ``oracle/__init__``).

One sequence is decoded as a state machine over generation blocks, following
the engine description of the paper:

* Block slots (App. F): a generation block is a placeholder (all mask, not
  admitted), active (admitted, being denoised), committed and awaiting its
  cache write, or cached.  Here a committed block waiting for its cache write
  is called *pending*.
* Commit rule (stated for one block in App. B.2, applied per sequence): every
  masked position of an active block whose confidence is at least ``tau`` is
  committed; when none clears ``tau`` the single most confident position is
  committed (lowest position among equals).
* Commit sweep (App. C.2, part 1): blocks are visited oldest first; a complete
  active block whose predecessors are all committed becomes committed, chains
  commit in one step, and the sweep stops at the first incomplete block.
* One-step cache write (App. F.2): a committed block's K/V are recomputed
  from its clean tokens in the next forward, where its rows ride along in
  front of the active blocks; after that forward it is cached.
* Admission (App. F: the admission threshold turns a placeholder into an
  active block): at the end of a step, and after the prefill, placeholders
  are admitted in order while fewer than ``n_inflight`` blocks are active and
  either no block is active or the youngest active block has resolved a
  fraction >= ``tau_add`` of its positions.  ``tau_add <= 0`` refills every
  free slot at once.
* Semi-completion (App. F: the accept and semi-completion thresholds decide
  which positions an active block resolves): with ``tau_semi`` given, an
  active block whose predecessor is still active and has resolved a fraction
  < ``tau_semi`` of its positions is semi-activated and commits only positions
  with confidence >= ``tau``; every other active block is fully activated and,
  when none of its masked positions clears ``tau``, commits its single most
  confident one.  Later blocks thus start committing at the engine's pace once
  the predecessor's top-1 context is mostly in place, before it is cached.
  Without ``tau_semi`` the forced commit is one per sequence, over all active
  blocks (the base rule above).  Resolved fractions are float32 ratios
  compared with float32 thresholds.
* Static skip rule (§3.3, App. B.3): with ``skip_masked`` an active block
  that is still fully masked at the start of a step is left out of that
  step's forward while an older block is active; it gets no confidences and
  no commits.
* Participation counters (the same appendix, measured here on the live
  decode rather than on a replayed trace), summed over steps: active
  block-forwards, those that commit nothing, those the static rule would
  skip (fully masked with an older active block) split into the ones that
  commit nothing (the FLOPs the rule saves) and the ones that commit
  (deferred), the one-step cache writes forwarded, and the active blocks a
  live skip rule left out.
* TPF (§2.1): tokens committed per model forward; a forward is a step in
  which the sequence has at least one active block.  Prefill is not counted
  (App. F.1).
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Callable, List, Optional

import numpy as np

from .model import OracleModel, lm_stats

PLACEHOLDER, ACTIVE, PENDING, CACHED = 0, 1, 2, 3

PART_NAMES = ("active_forwards", "zero_commit", "static_saved", "static_deferred", "cache_writes",
              "skipped")

__all__ = ["PART_NAMES", "SeqDecoder", "commit_set", "commit_set_semi", "frac_at_least", "decode_batch", "PLACEHOLDER", "ACTIVE", "PENDING", "CACHED"]


def frac_at_least(resolved: int, B: int, thr: float) -> bool:
    """resolved / B >= thr, as a float32 division and comparison."""
    return bool(np.float32(resolved) / np.float32(B) >= np.float32(thr))


def commit_set_semi(conf: np.ndarray, block: np.ndarray, resolved, B: int, tau: float,
                    tau_semi: float):
    """Semi-completion commit rule.  ``block[i]`` is the index (0 = oldest
    active) of the block holding masked position i; ``resolved[k]`` is active
    block k's resolved count before this step.  Returns (commit mask, list of
    the index arrays of the blocks that took a forced commit)."""
    t = float(np.float32(tau))
    s = conf >= t
    forced = []
    for k in range(len(resolved)):
        idx = np.nonzero(block == k)[0]
        if idx.size == 0:
            continue
        full = k == 0 or frac_at_least(int(resolved[k - 1]), B, tau_semi)
        if full and not s[idx].any():
            s[idx[int(np.argmax(conf[idx]))]] = True   # first maximum = lowest position
            forced.append(idx)
    return s, forced


def commit_set(conf: np.ndarray, tau: float) -> np.ndarray:
    """Boolean commit mask over masked positions listed in position order.
    conf >= tau (inclusive, tau held as float32); at least the argmax."""
    t = float(np.float32(tau))
    s = conf >= t
    if not s.any():
        s[int(np.argmax(conf))] = True          # first maximum = lowest position
    return s


@dataclass
class StepRecord:
    step: int
    masked: np.ndarray          # absolute positions that were masked in active blocks
    conf: np.ndarray
    tok: np.ndarray
    p2: np.ndarray
    committed: np.ndarray       # absolute positions committed this step
    status_after: np.ndarray    # block slot states after the sweep and admission


class SeqDecoder:
    """Decoder state of one sequence: prompt ``[0, P)``, ``G`` generated
    positions in ``G // B`` blocks, at most ``n_inflight`` active blocks."""

    def __init__(self, model: OracleModel, prompt: np.ndarray, G: int, B: int, n_inflight: int,
                 tau: float, tau_semi: Optional[float] = None, tau_add: float = 0.0,
                 skip_masked: bool = False):
        P = len(prompt)
        if B < 1 or n_inflight < 1 or P % B or G % B:
            raise ValueError("need B >= 1, n_inflight >= 1, P % B == 0 and G % B == 0")
        self.model, self.P, self.G, self.B, self.nb, self.tau = model, P, G, B, n_inflight, tau
        self.tau_semi, self.tau_add, self.skip_masked = tau_semi, tau_add, skip_masked
        self.part = np.zeros(len(PART_NAMES), dtype=np.int64)
        self.mask_id = model.mask_id
        self.tokens = np.concatenate([np.asarray(prompt, dtype=np.int64),
                                      np.full(G, self.mask_id, dtype=np.int64)])
        self.status = np.full(G // B, PLACEHOLDER, dtype=np.int64)
        self.cache = model.kv_cache(P + G)
        self.cache_len = 0
        self.forwards = 0
        self.commit_step = np.full(G, -1, dtype=np.int64)
        self.records: List[StepRecord] = []
        self.keep_records = False

    # -- slots --------------------------------------------------------------
    def resolved(self, b: int) -> int:
        """Unmasked positions of generation block b."""
        lo = self.P + b * self.B
        return int(np.count_nonzero(self.tokens[lo:lo + self.B] != self.mask_id))

    def _admit(self):
        while np.count_nonzero(self.status == ACTIVE) < self.nb:
            free = np.nonzero(self.status == PLACEHOLDER)[0]
            if free.size == 0:
                break
            act = np.nonzero(self.status == ACTIVE)[0]
            if act.size and not frac_at_least(self.resolved(int(act[-1])), self.B, self.tau_add):
                break
            self.status[free[0]] = ACTIVE

    @property
    def done(self) -> bool:
        return not np.any((self.status == ACTIVE) | (self.status == PLACEHOLDER))

    def forwarded(self) -> np.ndarray:
        """Active blocks that take part in this step's forward: all of them,
        or under the static skip rule those that are the oldest active block
        or already hold a resolved position."""
        act = np.nonzero(self.status == ACTIVE)[0]
        if not self.skip_masked:
            return act
        return np.array([b for j, b in enumerate(act) if j == 0 or self.resolved(int(b)) > 0],
                        dtype=np.int64)

    def window(self):
        """Absolute positions [start, end) of this step's forward: pending
        blocks (clean rows for their cache write) followed by the forwarded
        active blocks (the skip rule only ever leaves out the youngest)."""
        fwd = self.forwarded()
        live = np.concatenate([np.nonzero(self.status == PENDING)[0], fwd])
        if self.skip_masked:
            assert np.array_equal(live, np.arange(live[0], live[-1] + 1)), "window not contiguous"
        return self.cache_len, self.P + self.B * (int(live[-1]) + 1)

    def count_participation(self, committed: np.ndarray):
        """Add this step's participation counters (see the module notes);
        ``committed`` are the absolute positions committed by the step."""
        act = np.nonzero(self.status == ACTIVE)[0]
        fwd = set(int(b) for b in self.forwarded())
        blk = (np.asarray(committed, dtype=np.int64) - self.P) // self.B
        for j, b in enumerate(act):
            b = int(b)
            if b not in fwd:
                self.part[5] += 1
                continue
            n_commit = int(np.count_nonzero(blk == b))
            self.part[0] += 1
            self.part[1] += n_commit == 0
            if j > 0 and self.resolved(b) == 0:
                self.part[2 if n_commit == 0 else 3] += 1
        self.part[4] += int(np.count_nonzero(self.status == PENDING))

    # -- prefill --------------------------------------------------------------
    def prefill(self):
        """Encode the prompt (no LM head) and admit the first blocks."""
        if self.P > 0:
            self.model.forward(self.tokens, 0, self.P, self.cache, self.B)
        self.cache_len = self.P
        self._admit()

    # -- one denoising step -------------------------------------------------
    def forward_step(self, with_logits: bool = False):
        """Forward over the window; statistics for every masked position
        (and their logits when ``with_logits``)."""
        s, e = self.window()
        h = self.model.forward(self.tokens, s, e, self.cache, self.B)
        masked = np.nonzero(self.tokens[s:e] == self.mask_id)[0] + s
        z = self.model.logits(h[masked - s])
        conf, tok, p2 = lm_stats(z)
        if with_logits:
            return masked, conf, tok, p2, z
        return masked, conf, tok, p2

    def apply(self, positions: np.ndarray, toks: np.ndarray, step: int):
        """Commit ``toks`` at ``positions``; cache write, sweep, admission."""
        # Pending blocks had their K/V written by this step's forward.
        for b in np.nonzero(self.status == PENDING)[0]:
            self.status[b] = CACHED
            self.cache_len += self.B
        self.tokens[positions] = toks
        self.commit_step[positions - self.P] = step
        # In-order sweep over the block buffer, oldest block first.
        for b in range(len(self.status)):
            if self.status[b] in (CACHED, PENDING):
                continue
            if self.status[b] != ACTIVE:
                break
            lo = self.P + b * self.B
            if np.any(self.tokens[lo:lo + self.B] == self.mask_id):
                break
            self.status[b] = PENDING
        self._admit()
        self.forwards += 1

    def decision(self, masked: np.ndarray, conf: np.ndarray):
        """This step's own commit mask over ``masked`` and the index arrays of
        the groups that took a forced commit (the whole set under the base
        rule, single blocks under semi-completion)."""
        if self.tau_semi is None:
            own = commit_set(conf, self.tau)
            forced = [] if (conf >= np.float32(self.tau)).any() else [np.arange(len(conf))]
            return own, forced
        act = np.nonzero(self.status == ACTIVE)[0]
        block = (masked - self.P) // self.B - int(act[0])
        resolved = [self.resolved(int(b)) for b in act]
        return commit_set_semi(conf, block, resolved, self.B, self.tau, self.tau_semi)

    def step(self, step: int, decide: Optional[Callable] = None):
        masked, conf, tok, p2 = self.forward_step()
        own, _ = self.decision(masked, conf)
        if decide is None:
            sel = own
            toks = tok[sel]
            positions = masked[sel]
        else:
            positions, toks = decide(self, step, masked, conf, tok, p2, own)
        self.count_participation(np.asarray(positions, dtype=np.int64))
        self.apply(np.asarray(positions, dtype=np.int64), np.asarray(toks, dtype=np.int64), step)
        if self.keep_records:
            self.records.append(StepRecord(step, masked, conf, tok, p2, np.asarray(positions),
                                           self.status.copy()))


@dataclass
class BatchResult:
    tokens: np.ndarray          # [b][G] generated tokens
    commit_step: np.ndarray     # [b][G] step index at which each position committed
    forwards: np.ndarray        # [b]
    steps: int
    participation: np.ndarray = None   # [len(PART_NAMES)], summed over sequences

    @property
    def tpf(self) -> float:
        """Tokens per forward: sum of generated tokens over sum of forwards."""
        return float(self.tokens.size) / float(np.sum(self.forwards))


def decode_batch(model: OracleModel, prompts: np.ndarray, G: int, B: int, n_inflight: int,
                 tau: float, decide: Optional[Callable] = None, max_steps: int | None = None,
                 keep_records: bool = False, tau_semi: Optional[float] = None,
                 tau_add: float = 0.0, skip_masked: bool = False) -> BatchResult:
    """Decode independent sequences; batch rows never interact, so each runs
    its own state machine and the global step index equals its forward index
    while it is active."""
    b = prompts.shape[0]
    toks = np.zeros((b, G), dtype=np.int64)
    cs = np.zeros((b, G), dtype=np.int64)
    fw = np.zeros(b, dtype=np.int64)
    part = np.zeros(len(PART_NAMES), dtype=np.int64)
    steps = 0
    for i in range(b):
        d = SeqDecoder(model, prompts[i], G, B, n_inflight, tau, tau_semi, tau_add, skip_masked)
        d.keep_records = keep_records
        d.seq_index = i
        d.prefill()
        s = 0
        while not d.done:
            if max_steps is not None and s >= max_steps:
                raise RuntimeError("decode did not finish within max_steps")
            d.step(s, decide)
            s += 1
        steps = max(steps, s)
        toks[i] = d.tokens[d.P:]
        cs[i] = d.commit_step
        fw[i] = d.forwards
        part += d.part
    return BatchResult(toks, cs, fw, steps, part)
