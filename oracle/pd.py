"""numpy float64 oracle: block-wise P&D attention, scoring, eviction, compaction.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``): the product path never
imports this module.

One *unit* is one (sample, KV head) pair together with the G query heads that
share its KV head.  The paper bounds the cache separately for every attention
head of every sample (Sec. 3); with grouped-query attention there is one cache
per KV head, and its scores sum over the G query heads that read it
(reading R7).

The state of a unit is an *unordered* collection of entries
``(pos, k, v, score)``: ``pos`` is ``kv_ids`` and ``score`` is ``sum_weights``
of Sec. 3.2.  Storage order carries no meaning (every result below is a
function of the set), which is what licenses in-place hole-filling compaction
on the device.

Schedule (Sec. 3.1, Algorithm 1, under reading R1): the cache holds at most
``kv_max`` entries between steps.  Prefill runs in blocks of ``block`` tokens;
each block's keys are appended, every query of the block attends causally to
the cache plus the block's own keys up to itself, and afterwards the cache is
cut back to ``kv_max`` with ``curr_id`` = the last processed position.  Decode
does the same with one token per step (one eviction per step).

Everything is float64 on exactly the input values the device receives.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np


@dataclass
class EvictionEvent:
    """Record of one cut (the removal step of Algorithm 1, Sec. 3.1; rule of Sec. 3.2).

    ``all_pos``/``all_score``/``all_ave`` describe every entry present at the
    moment of the cut (sorted by position), so a comparison can evaluate any
    candidate kept set against the oracle's own averages.
    """

    kind: str
    curr_id: int
    n_before: int
    kept_pos: np.ndarray
    evicted_pos: np.ndarray
    all_pos: np.ndarray
    all_score: np.ndarray
    all_ave: np.ndarray
    gap: float  # smallest kept average minus largest evicted average


@dataclass
class UnitOracle:
    """State and steps of one unit (Sec. 3, 3.1, 3.2)."""

    head_dim: int
    group: int          # G query heads per KV head
    kv_max: int         # the paper's maximum cache size |kv|-bar
    sm_scale: float
    rule: str = "ave"   # ranking key of a cut, see ``ranking_key``
    pad: int = 0        # left pad tokens of the unit's sample (Sec. 3), reading R11
    pos: np.ndarray = field(default=None)
    k: np.ndarray = field(default=None)
    v: np.ndarray = field(default=None)
    score: np.ndarray = field(default=None)
    last_w: np.ndarray = field(default=None)   # weights of the last processed query
    queries_seen: int = 0
    evicted_score_total: float = 0.0

    def __post_init__(self):
        d = self.head_dim
        self.pos = np.zeros(0, dtype=np.int64)
        self.k = np.zeros((0, d), dtype=np.float64)
        self.v = np.zeros((0, d), dtype=np.float64)
        self.score = np.zeros(0, dtype=np.float64)
        self.last_w = np.zeros(0, dtype=np.float64)

    # -- state ----------------------------------------------------------------
    @property
    def n(self) -> int:
        return int(self.pos.shape[0])

    def append(self, first_pos: int, k: np.ndarray, v: np.ndarray) -> None:
        """Add the KV pairs of positions first_pos.. with zero scores.

        ``sum_weights`` is zero-initialised and grows with the cache
        (Sec. 3.2); ``kv_ids`` are the token positions.
        """
        m = k.shape[0]
        self.pos = np.concatenate([self.pos, first_pos + np.arange(m, dtype=np.int64)])
        self.k = np.concatenate([self.k, np.asarray(k, dtype=np.float64)])
        self.v = np.concatenate([self.v, np.asarray(v, dtype=np.float64)])
        self.score = np.concatenate([self.score, np.zeros(m)])
        self.last_w = np.concatenate([self.last_w, np.zeros(m)])

    # -- attention + score accumulation ----------------------------------------
    def attend(self, q: np.ndarray, first_pos: int) -> np.ndarray:
        """Queries at positions first_pos.. attend causally to the cache.

        ``q`` is ``[G, m, d]``.  A query at position i sees exactly the entries
        with pos <= i (causal attention; the block's own keys included, the
        query's own key included -- reading R5).  The probabilities are the
        softmax of ``sm_scale * q.k`` over those entries (Sec. 3.2 calls these
        ``attn_weights``; reading R6), and
        ``sum_weights += sum_i attn_weights[i]`` over every query of the block
        and every query head of the group (Sec. 3.2 update; reading R7).
        Returns the attention outputs ``[G, m, d]``.

        Left padding (Sec. 3, reading R11): the ``pad`` first positions of the
        sample are pad tokens.  Their keys are visible to no query (they keep
        score 0), and a pad query attends to nothing: its output is zero and it
        adds nothing to any score.
        """
        q = np.asarray(q, dtype=np.float64)
        g_heads, m, d = q.shape
        qpos = first_pos + np.arange(m, dtype=np.int64)
        real_q = qpos >= self.pad
        visible = (self.pos[None, :] <= qpos[:, None]) & (self.pos[None, :] >= self.pad)
        visible &= real_q[:, None]                                     # [m, n]
        out = np.zeros((g_heads, m, d))
        last = np.zeros(self.n)
        for g in range(g_heads):
            logits = self.sm_scale * (q[g] @ self.k.T)                # [m, n]
            logits = np.where(visible, logits, -np.inf)
            p = np.zeros_like(logits)
            if real_q.any():
                z = logits[real_q]
                z = z - z.max(axis=1, keepdims=True)
                w = np.exp(z)
                p[real_q] = w / w.sum(axis=1, keepdims=True)           # real rows sum to 1
            out[g] = p @ self.v
            self.score = self.score + p.sum(axis=0)
            last += p[m - 1]
        # the last query of the call, summed over the group's heads (TOVA's key)
        self.last_w = last
        self.queries_seen += g_heads * int(real_q.sum())
        return out

    # -- eviction rule ------------------------------------------------------------
    def averages(self, curr_id: int) -> np.ndarray:
        """``ave_weights = sum_weights / (curr_id + 1 - kv_ids)`` (Sec. 3.2).

        The denominator is the number of queries (per query head) that have
        attended the entry: positions pos..curr_id inclusive (reading R4).
        """
        return self.score / (curr_id + 1 - self.pos).astype(np.float64)

    def ranking_key(self, curr_id: int) -> np.ndarray:
        """The key whose smallest entries a cut removes.

        ``"ave"``: ``ave_weights`` (Sec. 3.2; the method).  ``"sum"``: the
        accumulated ``sum_weights`` itself, the cumulative rule that Sec. 3.2
        corrects because it favours early tokens.  ``"recent"``: the position,
        so the most recent pairs stay (the eviction of Algorithm 3, the
        extreme decoding-only comparator of Sec. 4).  ``"tova"``: the weights
        the last processed query gave each entry, summed over the group's
        heads (TOVA, one of the related policies of Sec. 2: the current query
        alone decides).
        """
        if self.rule == "ave":
            return self.averages(curr_id)
        if self.rule == "sum":
            return self.score.copy()
        if self.rule == "recent":
            return self.pos.astype(np.float64)
        if self.rule == "tova":
            return self.last_w.copy()
        raise ValueError(f"unknown ranking rule {self.rule!r}")

    def evict(self, curr_id: int, kind: str, target: int | None = None) -> EvictionEvent | None:
        """Cut the cache back to ``target`` (default ``kv_max``) entries (Sec. 3.1;
        Sec. 3.2 rule).

        The entries with the smallest ranking key (``ave_weights`` under the
        paper's rule) are removed; on an exact tie the older entry (smaller
        position) goes first (reading R8).  No-op while the cache holds at most
        ``target`` entries (reading R16).  Survivors keep their accumulated
        scores (reading R13).  ``all_ave`` and ``gap`` of the event are in the
        rule's key.
        """
        target = self.kv_max if target is None else target
        n = self.n
        if n <= target:
            return None
        ave = self.ranking_key(curr_id)
        order = np.lexsort((self.pos, ave))        # ascending ave, then ascending pos
        n_evict = n - target
        evict_idx = order[:n_evict]
        keep_idx = np.sort(order[n_evict:])
        # smallest kept average minus largest removed one (no tie when nothing is kept)
        gap = float(ave[order[n_evict]] - ave[order[n_evict - 1]]) if n_evict < n else np.inf
        by_pos = np.argsort(self.pos)
        ev = EvictionEvent(
            kind=kind, curr_id=int(curr_id), n_before=n,
            kept_pos=np.sort(self.pos[keep_idx]), evicted_pos=np.sort(self.pos[evict_idx]),
            all_pos=self.pos[by_pos].copy(), all_score=self.score[by_pos].copy(),
            all_ave=ave[by_pos].copy(), gap=gap)
        self.evicted_score_total += float(self.score[evict_idx].sum())
        self._keep(keep_idx)
        return ev

    def _keep(self, idx: np.ndarray) -> None:
        self.pos = self.pos[idx]
        self.k = self.k[idx]
        self.v = self.v[idx]
        self.score = self.score[idx]
        self.last_w = self.last_w[idx]

    # -- schedule steps -----------------------------------------------------------
    def prefill_block(self, t0: int, q: np.ndarray, k: np.ndarray, v: np.ndarray) -> np.ndarray:
        """Process prompt tokens [t0, t0+m): append their KV pairs, attend.

        The processing step of Algorithm 1 (Sec. 3.1) for tokens [t0, t1);
        no eviction here.
        """
        self.append(t0, k, v)
        return self.attend(q, t0)

    def decode_step(self, pos: int, q: np.ndarray, k: np.ndarray, v: np.ndarray,
                    bound: int | None = None):
        """One decode step at position ``pos`` with one eviction (reading R3).

        Algorithm 1 decode loop (Sec. 3.1) with one KV pair removed per step:
        append, attend with ``curr_id = pos``, then cut back to ``bound``
        (default ``kv_max``).  ``q`` is ``[G, d]``; returns (outputs ``[G, d]``,
        event or None).
        """
        self.append(pos, np.asarray(k)[None], np.asarray(v)[None])
        o = self.attend(np.asarray(q)[:, None, :], pos)[:, 0, :]
        return o, self.evict(pos, "decode", target=bound)

    def decode_step_alg1(self, pos: int, q: np.ndarray, k: np.ndarray, v: np.ndarray, p: int,
                         bound: int | None = None):
        """One decode step of Algorithm 1's decoding loop taken literally: when
        the cache holds ``bound`` (default ``kv_max``) entries or more, first
        cut it to ``bound - p`` (ranked with ``curr_id = pos - 1``, the last
        processed position, reading R4), then process the token at ``pos``
        (append and attend, no removal).  Algorithm 3's decoding loop is the
        case ``bound = 2``, ``p = 1`` under the ``"recent"`` rule.
        Returns (outputs ``[G, d]``, event or None)."""
        bound = self.kv_max if bound is None else bound
        ev = None
        if self.n >= bound:
            ev = self.evict(pos - 1, "decode", target=bound - p)
        self.append(pos, np.asarray(k)[None], np.asarray(v)[None])
        o = self.attend(np.asarray(q)[:, None, :], pos)[:, 0, :]
        return o, ev


class StepOracle(UnitOracle):
    """``UnitOracle`` that remembers the entries of its last cut, so that a
    comparison harness can adopt another valid kept set after a near-tie."""

    def evict(self, curr_id: int, kind: str, target: int | None = None):
        before = (self.pos.copy(), self.k.copy(), self.v.copy(), self.score.copy(),
                  self.evicted_score_total, self.last_w.copy())
        ev = super().evict(curr_id, kind, target)
        self._last = before if ev is not None else None
        self._last_target = self.kv_max if target is None else target
        return ev

    def adopt(self, kept_pos) -> None:
        """Replace the result of the last cut by another kept set of the same size.
        Call it right after that cut (before anything is appended)."""
        pos, k, v, score, evt, last_w = self._last
        kept_pos = np.asarray(sorted(int(p) for p in kept_pos), dtype=np.int64)
        size = getattr(self, "_last_target", None)
        size = self.kv_max if size is None else size
        if kept_pos.shape[0] != size:
            raise ValueError("adopted kept set has the wrong size")
        idx = np.searchsorted(pos[np.argsort(pos)], kept_pos)
        order = np.argsort(pos)
        sel = order[idx]
        if not np.array_equal(pos[sel], kept_pos):
            raise ValueError("adopted kept set is not a subset of the cut's entries")
        mask = np.ones(pos.shape[0], dtype=bool)
        mask[sel] = False
        self.pos, self.k, self.v, self.score = pos[sel], k[sel], v[sel], score[sel]
        self.last_w = last_w[sel]
        self.evicted_score_total = evt + float(score[mask].sum())


@dataclass
class Trace:
    """Everything one unit's P&D run produces."""

    out: np.ndarray                 # [G, s + D, d] attention outputs by position
    events: list                    # EvictionEvent per cut, in order
    final_pos: np.ndarray
    final_score: np.ndarray
    queries_seen: int
    evicted_score_total: float


def run_unit(q, k, v, *, s: int, kv_max: int, block: int, n_decode: int,
             sm_scale: float, p_dec: int = 0, rule: str = "ave",
             kv_dec: int | None = None, pad: int = 0) -> Trace:
    """Full P&D run of one unit (Sec. 3.1, Algorithm 1 under reading R1).

    ``q`` is ``[G, s + n_decode, d]``; ``k``, ``v`` are ``[s + n_decode, d]``,
    holding the prompt then the per-step decode inputs (reading R15: no model,
    the vectors of every position are given).  Prefill: for t0 = 0, block, ...
    process [t0, t1) with t1 = min(s, t0 + block) (reading R17), then cut with
    curr_id = t1 - 1.  Decode: step t processes position s + t (reading R12)
    and cuts with curr_id = s + t; with ``p_dec > 0`` it follows Algorithm 1's
    decoding loop literally instead (``decode_step_alg1``: remove ``p_dec``
    entries when the cache is full, before the token is processed).

    ``rule`` picks the ranking key (``UnitOracle.ranking_key``).  ``kv_dec``
    bounds the cache during decode (default ``kv_max``); with ``p_dec = 0`` a
    cache larger than ``kv_dec`` at the first step is first cut to ``kv_dec``
    with curr_id = the last processed position.  Algorithm 3 (ED): ``kv_max >=
    s`` (no removal while prefilling), ``kv_dec = 2``, ``p_dec = 1``,
    ``rule = "recent"``.  ``pad`` left pad tokens occupy positions 0..pad-1
    of the prompt (Sec. 3; see ``UnitOracle.attend``).
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    g_heads, total, d = q.shape
    unit = UnitOracle(head_dim=d, group=g_heads, kv_max=kv_max, sm_scale=sm_scale, rule=rule,
                      pad=pad)
    kd = kv_max if kv_dec is None else kv_dec
    out = np.zeros((g_heads, total, d))
    events = []
    t0 = 0
    while t0 < s:
        t1 = min(s, t0 + block)
        out[:, t0:t1] = unit.prefill_block(t0, q[:, t0:t1], k[t0:t1], v[t0:t1])
        ev = unit.evict(t1 - 1, "prefill")
        if ev is not None:
            events.append(ev)
        t0 = t1
    for t in range(n_decode):
        i = s + t
        if p_dec > 0:
            out[:, i], ev = unit.decode_step_alg1(i, q[:, i], k[i], v[i], p_dec, bound=kd)
        else:
            if unit.n > kd:
                events.append(unit.evict(i - 1, "decode", target=kd))
            out[:, i], ev = unit.decode_step(i, q[:, i], k[i], v[i], bound=kd)
        if ev is not None:
            events.append(ev)
    order = np.argsort(unit.pos)
    return Trace(out=out, events=events, final_pos=unit.pos[order],
                 final_score=unit.score[order], queries_seen=unit.queries_seen,
                 evicted_score_total=unit.evicted_score_total)


def run_paper_schedule(q, k, v, *, s: int, kv_max_paper: int, p: int, max_gen: int,
                       sm_scale: float):
    """Algorithm 1 of Sec. 3.1 as printed, for the schedule-equivalence pin.

    Prefill: t1 = min(s, |kv|-bar); process [0, t1 - 1]; while t1 < s: remove
    p pairs, t0 = t1, t1 = min(s, t0 + p), process [t0, t1 - 1].  Decode: for
    t = 1 .. max_gen - 1: if |kv| = |kv|-bar remove p pairs; process the token
    at position s + t - 1.  A removal uses curr_id = the last processed position
    (reading R4).  Returns (outputs [G, s + max_gen - 1, d], events).
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    g_heads, total, d = q.shape
    # the removal amount is p, so the cut target is |kv|-bar - p entries
    unit = UnitOracle(head_dim=d, group=g_heads, kv_max=kv_max_paper - p, sm_scale=sm_scale)
    out = np.zeros((g_heads, s + max_gen - 1, d))
    events = []
    t1 = min(s, kv_max_paper)
    out[:, 0:t1] = unit.prefill_block(0, q[:, 0:t1], k[0:t1], v[0:t1])
    last = t1 - 1
    while t1 < s:
        ev = unit.evict(last, "prefill")   # removes exactly p: the cache is full here
        events.append(ev)
        t0 = t1
        t1 = min(s, t0 + p)
        out[:, t0:t1] = unit.prefill_block(t0, q[:, t0:t1], k[t0:t1], v[t0:t1])
        last = t1 - 1
    for t in range(1, max_gen):
        if unit.n == kv_max_paper:
            events.append(unit.evict(last, "decode"))
        i = s + t - 1
        unit.append(i, k[i:i + 1], v[i:i + 1])
        out[:, i] = unit.attend(q[:, i:i + 1], i)[:, 0]
        last = i
    return out, events
