"""Pins of the CPU oracle against facts that do not come from the oracle itself.

Each check below ties ``oracle.pd`` (and ``oracle.micro``) to something
outside it: a library routine (torch's scaled-dot-product attention in
float64), a hand-derived exact example (tests/golden), the paper's stated
values (Sec. 3.2), brute-force subset enumeration, conservation of probability
mass, schedule equivalence with Algorithm 1 as printed, or permutation
invariance.  The last test plants plausible mistakes in a copy of the oracle
and checks that some pin fails for each.
"""
import itertools
import json
import os
from fractions import Fraction

import numpy as np
import pytest
import torch

from oracle import pd as opd
from oracle import micro

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "uniform_worked_example.json")


def _rand_unit(rng, G, T, d, kscale=1.0):
    q = rng.standard_normal((G, T, d))
    k = rng.standard_normal((T, d)) * kscale
    v = rng.standard_normal((T, d))
    return q, k, v


# ---------------------------------------------------------------------------
# pin helpers (parameterised by the oracle class so mutations can be planted)
# ---------------------------------------------------------------------------
def _run(cls, q, k, v, *, s, kv_max, block, n_decode, sm_scale):
    """run_unit with an arbitrary UnitOracle subclass (for planted mistakes)."""
    G, T, d = q.shape
    u = cls(head_dim=d, group=G, kv_max=kv_max, sm_scale=sm_scale)
    out = np.zeros((G, T, d))
    events = []
    t0 = 0
    while t0 < s:
        t1 = min(s, t0 + block)
        out[:, t0:t1] = u.prefill_block(t0, q[:, t0:t1], k[t0:t1], v[t0:t1])
        ev = u.evict(t1 - 1, "prefill")
        if ev is not None:
            events.append(ev)
        t0 = t1
    for t in range(n_decode):
        i = s + t
        out[:, i], ev = u.decode_step(i, q[:, i], k[i], v[i])
        if ev is not None:
            events.append(ev)
    return out, events, u


def pin_dense_fixed_point(cls):
    """No eviction (bound >= s + D): outputs equal causal softmax attention
    from torch SDPA, scores equal causal column sums of SDPA's probabilities."""
    rng = np.random.default_rng(7)
    G, s, D, d, block = 3, 19, 4, 16, 5
    T = s + D
    q, k, v = _rand_unit(rng, G, T, d)
    scale = 0.37
    out, events, u = _run(cls, q, k, v, s=s, kv_max=T + 3, block=block, n_decode=D, sm_scale=scale)
    assert events == []
    tq = torch.from_numpy(q)[None]                       # [1, G, T, d]
    tk = torch.from_numpy(k)[None, None].expand(1, G, T, d)
    tv = torch.from_numpy(v)[None, None].expand(1, G, T, d)
    ref = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, is_causal=True, scale=scale)
    np.testing.assert_allclose(out, ref[0].numpy(), rtol=0, atol=1e-12)
    # probabilities via one-hot values: output row i is row i of P
    eye = torch.eye(T, dtype=torch.float64)[None, None].expand(1, G, T, T)
    P = torch.nn.functional.scaled_dot_product_attention(tq, tk, eye, is_causal=True, scale=scale)[0]
    colsum = P.sum(dim=(0, 1)).numpy()                   # over heads and queries
    order = np.argsort(u.pos)
    np.testing.assert_allclose(u.score[order], colsum, rtol=0, atol=1e-12)


def pin_golden(cls):
    """The hand-derived exact example, run through the float64 oracle.  Exact
    ties of the example become ulp-level near-ties in float64; there the
    golden (exact) kept set is adopted, as a comparison harness would."""
    gold = json.load(open(GOLDEN))
    s, D, d = 6, 2, 8
    T = s + D
    q = np.ones((1, T, d))
    k = np.zeros((T, d))
    v = np.eye(T, d)
    u = cls(head_dim=d, group=1, kv_max=2, sm_scale=1.0)

    def check(ev, gev):
        assert ev is not None and ev.curr_id == gev["curr_id"]
        for p, sc in zip(ev.all_pos, ev.all_score):
            assert abs(sc - float(Fraction(gev["score"][str(p)]))) < 1e-12
        for p, a in zip(ev.all_pos, ev.all_ave):
            assert abs(a - float(Fraction(gev["ave"][str(p)]))) < 1e-12
        if list(ev.kept_pos) != gev["kept"]:
            assert ev.gap < 1e-12, "kept set differs outside an exact tie"
            u.adopt(gev["kept"])

    gi = 0
    outs = {}
    for t0 in range(0, s, 2):
        o = u.prefill_block(t0, q[:, t0:t0 + 2], k[t0:t0 + 2], v[t0:t0 + 2])
        outs[t0], outs[t0 + 1] = o[0, 0], o[0, 1]
        ev = u.evict(t0 + 1, "prefill")
        if t0 == 0:
            assert ev is None
        else:
            check(ev, gold["events"][gi])
            gi += 1
    for i in (6, 7):
        o, ev = u.decode_step(i, q[:, i], k[i], v[i])
        outs[i] = o[0]
        check(ev, gold["events"][gi])
        gi += 1
    for i, vis in gold["outputs_visible_sets"].items():
        if i.startswith("_"):
            continue
        want = np.zeros(d)
        want[vis] = 1.0 / len(vis)
        np.testing.assert_allclose(outs[int(i)], want, rtol=0, atol=1e-12)


def pin_selection_bruteforce(cls):
    """Kept set = the unique subset whose every member ranks above every
    evicted entry under (ave, pos); found by enumerating all subsets."""
    rng = np.random.default_rng(11)
    for trial in range(60):
        n = int(rng.integers(3, 11))
        kv_max = int(rng.integers(1, n))
        curr_id = 40
        pos = rng.choice(np.arange(0, curr_id + 1), size=n, replace=False)
        # integer-ish scores so exact ties in ave occur often
        score = rng.integers(0, 4, size=n).astype(np.float64) * (curr_id + 1 - pos) / 4.0
        if trial % 3 == 0:
            score = rng.random(n)
        u = cls(head_dim=2, group=1, kv_max=kv_max, sm_scale=1.0)
        u.pos, u.score, u.last_w = pos.astype(np.int64), score, np.zeros(n)
        u.k, u.v = np.zeros((n, 2)), np.zeros((n, 2))
        ev = u.evict(curr_id, "prefill")
        ave = score / (curr_id + 1 - pos)
        key = {int(p): (a, int(p)) for p, a in zip(pos, ave)}
        valid = []
        for kept in itertools.combinations(sorted(int(p) for p in pos), kv_max):
            ev_set = set(int(p) for p in pos) - set(kept)
            if min(key[p] for p in kept) > max(key[p] for p in ev_set):
                valid.append(list(kept))
        assert len(valid) == 1
        assert list(ev.kept_pos) == valid[0]


def pin_conservation_and_lengths(cls):
    """Every query head's probabilities sum to 1, so kept + evicted score mass
    equals the number of (head, query) pairs; the cache never exceeds the bound
    between steps and equals min(bound, tokens seen) after every cut."""
    rng = np.random.default_rng(3)
    for (G, s, D, d, kv_max, block) in [(1, 40, 6, 8, 8, 4), (4, 33, 5, 8, 10, 7), (2, 64, 9, 4, 16, 16)]:
        q, k, v = _rand_unit(rng, G, s + D, d)
        out, events, u = _run(cls, q, k, v, s=s, kv_max=kv_max, block=block, n_decode=D, sm_scale=0.5)
        total = u.score.sum() + u.evicted_score_total
        assert abs(total - G * (s + D)) < 1e-9 * G * (s + D)
        assert u.queries_seen == G * (s + D)
        assert u.n == min(kv_max, s + D)
        seen = 0
        for ev in events:
            assert len(ev.kept_pos) == kv_max
            assert len(ev.kept_pos) + len(ev.evicted_pos) == ev.n_before
            assert ev.curr_id + 1 >= ev.n_before    # never more entries than tokens
            assert ev.n_before <= kv_max + block
            assert max(ev.kept_pos.max(), ev.evicted_pos.max()) == ev.curr_id
            seen = ev.curr_id + 1
        assert seen > 0


def pin_paper_stated_values(cls):
    """Sec. 3.2: the first KV pair starts with a summed weight of 1 (query 0
    sees only itself), and a query that sees L entries spreads total weight 1,
    i.e. mean weight 1/L = 1/min(i+1, bound) without eviction in between."""
    rng = np.random.default_rng(5)
    d = 8
    q, k, v = _rand_unit(rng, 1, 12, d, kscale=3.0)
    u = cls(head_dim=d, group=1, kv_max=100, sm_scale=1.0)
    u.prefill_block(0, q[:, 0:1], k[0:1], v[0:1])
    assert u.score[0] == 1.0
    for i in range(1, 12):
        before = u.score.sum()
        u.prefill_block(i, q[:, i:i + 1], k[i:i + 1], v[i:i + 1])
        inc = u.score.sum() - before
        assert abs(inc / (i + 1) - 1.0 / min(i + 1, 100)) < 1e-15
    # key 0's average counts curr_id + 1 queries
    ave0 = u.averages(11)[np.argmin(u.pos)]
    assert abs(ave0 - u.score[np.argmin(u.pos)] / 12.0) < 1e-15


def pin_alg1_equivalence(cls_unused=None):
    """Algorithm 1 as printed, with bound K+B and removal amount p = B, matches
    the block loop with bound K (reading R1) on every prefill output, every
    prefill cut, the first decode removal and the first decode output."""
    rng = np.random.default_rng(19)
    for (G, d, kv, B, nblk) in [(1, 8, 8, 4, 6), (4, 16, 12, 4, 5), (2, 8, 16, 8, 4)]:
        s = kv + B * nblk
        D = 3
        q, k, v = _rand_unit(rng, G, s + D, d)
        tr = opd.run_unit(q, k, v, s=s, kv_max=kv, block=B, n_decode=D, sm_scale=0.6)
        out_p, ev_p = opd.run_paper_schedule(q, k, v, s=s, kv_max_paper=kv + B, p=B,
                                             max_gen=D + 1, sm_scale=0.6)
        np.testing.assert_allclose(out_p[:, :s + 1], tr.out[:, :s + 1], rtol=0, atol=1e-12)
        n_prefill_cuts = sum(1 for e in tr.events if e.kind == "prefill")
        assert n_prefill_cuts == nblk
        for a, b in zip(ev_p[:n_prefill_cuts], tr.events[:n_prefill_cuts]):
            assert a.curr_id == b.curr_id
            assert list(a.kept_pos) == list(b.kept_pos)
            np.testing.assert_allclose(a.all_score, b.all_score, rtol=0, atol=1e-12)
        # Algorithm 1's first decode removal is the block loop's last prefill cut
        assert ev_p[n_prefill_cuts - 1].curr_id == s - 1


def pin_permutation_invariance(cls):
    """Shuffling a unit's storage order between steps changes nothing but
    rounding: storage order carries no meaning."""
    rng = np.random.default_rng(23)
    G, s, D, d, kv, B = 2, 48, 8, 8, 12, 6
    q, k, v = _rand_unit(rng, G, s + D, d)
    ref = opd.run_unit(q, k, v, s=s, kv_max=kv, block=B, n_decode=D, sm_scale=0.5)
    u = cls(head_dim=d, group=G, kv_max=kv, sm_scale=0.5)
    evs, outs = [], np.zeros((G, s + D, d))

    def shuffle():
        perm = rng.permutation(u.n)
        u.pos, u.k, u.v, u.score = u.pos[perm], u.k[perm], u.v[perm], u.score[perm]

    for t0 in range(0, s, B):
        outs[:, t0:t0 + B] = u.prefill_block(t0, q[:, t0:t0 + B], k[t0:t0 + B], v[t0:t0 + B])
        shuffle()
        ev = u.evict(t0 + B - 1, "prefill")
        if ev is not None:
            evs.append(ev)
        shuffle()
    for t in range(D):
        i = s + t
        outs[:, i], ev = u.decode_step(i, q[:, i], k[i], v[i])
        evs.append(ev)
        shuffle()
    np.testing.assert_allclose(outs, ref.out, rtol=0, atol=1e-12)
    assert len(evs) == len(ref.events)
    for a, b in zip(evs, ref.events):
        assert list(a.kept_pos) == list(b.kept_pos) or b.gap < 1e-12


def pin_micro_agreement(cls):
    """The loop-based micro-oracle (independent code) agrees with the numpy
    oracle to rounding on random float inputs with several cuts."""
    rng = np.random.default_rng(29)
    for (G, s, D, d, kv, B) in [(2, 11, 3, 4, 3, 2), (1, 9, 4, 3, 4, 3), (4, 8, 2, 2, 2, 4)]:
        q, k, v = _rand_unit(rng, G, s + D, d)
        out, events, u = _run(cls, q, k, v, s=s, kv_max=kv, block=B, n_decode=D, sm_scale=0.8)
        mo, mev, mfinal = micro.micro_run(q.tolist(), k.tolist(), v.tolist(), s=s, kv_max=kv,
                                          block=B, n_decode=D, sm_scale=0.8)
        for (g, i), row in mo.items():
            np.testing.assert_allclose(out[g, i], row, rtol=0, atol=1e-12)
        assert len(mev) == len(events)
        for a, b in zip(events, mev):
            assert a.curr_id == b["curr_id"]
            assert list(a.kept_pos) == b["kept"]
            for p, sc in zip(a.all_pos, a.all_score):
                assert abs(sc - b["score"][int(p)]) < 1e-12
        order = np.argsort(u.pos)
        assert [int(p) for p in u.pos[order]] == sorted(mfinal)


def pin_super_key(cls):
    """A key aligned with every query at large norm is never evicted and
    collects almost all of the weight of every query after it."""
    rng = np.random.default_rng(31)
    G, s, D, d, kv, B = 2, 64, 8, 16, 8, 8
    q, k, v = _rand_unit(rng, G, s + D, d)
    u_dir = np.ones(d) / np.sqrt(d)
    q = q * 0.1 + u_dir * 2.0
    k[10] = u_dir * 12.0
    out, events, u = _run(cls, q, k, v, s=s, kv_max=kv, block=B, n_decode=D, sm_scale=1.0)
    for ev in events:
        if ev.curr_id >= 10:
            assert 10 in set(int(p) for p in ev.kept_pos)
    sc = u.score[list(u.pos).index(10)]
    n_after = G * (s + D - 10)
    assert sc > 0.99 * n_after


def pin_rule_keys_bruteforce(cls):
    """Under every ranking rule the kept set is the unique subset whose every
    member ranks above every removed entry under (key, pos), with the key
    written from its definition: ave_weights (Sec. 3.2), the accumulated
    sum_weights (the cumulative rule Sec. 3.2 corrects), the position
    (Algorithm 3 keeps the most recent pairs).  Includes a hand-made case where
    the three rules disagree."""
    curr_id = 10
    # pos 0 with sum 3 (ave 3/11), pos 9 with sum 1 (ave 1/2), pos 5 with sum 2 (ave 1/3)
    # last query's weights: pos 0 0.2, pos 9 0.1, pos 5 0.7
    want = {"ave": [9], "sum": [0], "recent": [9], "tova": [5]}
    for rule, kept in want.items():
        u = cls(head_dim=2, group=1, kv_max=1, sm_scale=1.0, rule=rule)
        u.pos, u.score = np.array([0, 9, 5], dtype=np.int64), np.array([3.0, 1.0, 2.0])
        u.last_w = np.array([0.2, 0.1, 0.7])
        u.k, u.v = np.zeros((3, 2)), np.zeros((3, 2))
        ev = u.evict(curr_id, "prefill")
        assert list(ev.kept_pos) == kept, rule
    rng = np.random.default_rng(37)
    for trial in range(80):
        rule = ("ave", "sum", "recent", "tova")[trial % 4]
        n = int(rng.integers(3, 10))
        kv_max = int(rng.integers(1, n))
        pos = rng.choice(np.arange(0, curr_id + 30), size=n, replace=False)
        score = rng.integers(0, 3, size=n).astype(np.float64) / 2.0   # frequent exact ties
        lw = rng.integers(0, 3, size=n).astype(np.float64) / 4.0
        u = cls(head_dim=2, group=1, kv_max=kv_max, sm_scale=1.0, rule=rule)
        u.pos, u.score, u.last_w = pos.astype(np.int64), score, lw
        u.k, u.v = np.zeros((n, 2)), np.zeros((n, 2))
        c = int(pos.max())
        ev = u.evict(c, "prefill")
        key = {"ave": lambda i, p: score[i] / (c + 1 - p), "sum": lambda i, p: score[i],
               "recent": lambda i, p: float(p), "tova": lambda i, p: lw[i]}[rule]
        rank = {int(p): (key(i, int(p)), int(p)) for i, p in enumerate(pos)}
        valid = [list(kept) for kept in itertools.combinations(sorted(rank), kv_max)
                 if min(rank[p] for p in kept) > max(rank[p] for p in set(rank) - set(kept))]
        assert len(valid) == 1 and list(ev.kept_pos) == valid[0], rule


def pin_alg3_closed_form(cls):
    """Algorithm 3 (ED): no removal while prefilling (bound >= s), then every
    decode step attends over exactly the previous token and itself, so each
    output is the two-term softmax average written out by hand; prefill outputs
    are dense causal attention (SDPA); the cache ends with the last two
    positions."""
    rng = np.random.default_rng(41)
    G, s, D, d = 2, 12, 6, 8
    q, k, v = _rand_unit(rng, G, s + D, d)
    sm = 0.7
    u = cls(head_dim=d, group=G, kv_max=s, sm_scale=sm, rule="recent")
    out = np.zeros((G, s + D, d))
    out[:, :s] = u.prefill_block(0, q[:, :s], k[:s], v[:s])
    for t in range(D):
        i = s + t
        out[:, i], _ = u.decode_step_alg1(i, q[:, i], k[i], v[i], 1, bound=2)
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.tensor(q[:, :s]), torch.tensor(k[:s])[None].expand(G, s, d),
        torch.tensor(v[:s])[None].expand(G, s, d), is_causal=True, scale=sm).numpy()
    np.testing.assert_allclose(out[:, :s], ref, rtol=0, atol=1e-12)
    for t in range(D):
        i = s + t
        for g in range(G):
            z0, z1 = sm * q[g, i] @ k[i - 1], sm * q[g, i] @ k[i]
            w0, w1 = 1.0 / (1.0 + np.exp(z1 - z0)), 1.0 / (1.0 + np.exp(z0 - z1))
            np.testing.assert_allclose(out[g, i], w0 * v[i - 1] + w1 * v[i], rtol=0, atol=1e-12)
    assert sorted(int(p) for p in u.pos) == [s + D - 2, s + D - 1]


def _run_padded(cls, q, k, v, *, s, kv_max, block, n_decode, sm_scale, pad):
    G, T, d = q.shape
    u = cls(head_dim=d, group=G, kv_max=kv_max, sm_scale=sm_scale, pad=pad)
    out = np.zeros((G, T, d))
    events = []
    for t0 in range(0, s, block):
        t1 = min(s, t0 + block)
        out[:, t0:t1] = u.prefill_block(t0, q[:, t0:t1], k[t0:t1], v[t0:t1])
        ev = u.evict(t1 - 1, "prefill")
        if ev is not None:
            events.append(ev)
    for t in range(n_decode):
        i = s + t
        out[:, i], ev = u.decode_step(i, q[:, i], k[i], v[i])
        if ev is not None:
            events.append(ev)
    return out, events, u


def pin_left_padding_is_a_shift(cls):
    """Left padding by a multiple of the block (Sec. 3): the real tokens' outputs,
    every cut that removes a real entry, and the final cache equal those of the
    unpadded run of the same real tokens, shifted by the pad; pad vectors are
    large junk, so a pad key that leaked into any softmax would show."""
    rng = np.random.default_rng(53)
    for (G, s_real, D, d, kv, B, n_blocks_pad) in [(2, 24, 5, 8, 6, 4, 2), (1, 18, 4, 4, 5, 3, 3)]:
        pad = n_blocks_pad * B
        q, k, v = _rand_unit(rng, G, s_real + D, d)
        ref, rev, ru = _run(cls, q, k, v, s=s_real, kv_max=kv, block=B, n_decode=D, sm_scale=0.6)
        jq = rng.standard_normal((G, pad, d)) * 30.0
        jk = rng.standard_normal((pad, d)) * 30.0
        jv = rng.standard_normal((pad, d)) * 30.0
        qp = np.concatenate([jq, q], axis=1)
        kp, vp = np.concatenate([jk, k]), np.concatenate([jv, v])
        out, ev, u = _run_padded(cls, qp, kp, vp, s=pad + s_real, kv_max=kv, block=B,
                                 n_decode=D, sm_scale=0.6, pad=pad)
        np.testing.assert_allclose(out[:, pad:], ref, rtol=0, atol=1e-12)
        assert not out[:, :pad].any()
        real_cuts = [list(e.kept_pos) for e in ev if any(p >= pad for p in e.evicted_pos)]
        assert real_cuts == [[p + pad for p in e.kept_pos] for e in rev]
        order, rorder = np.argsort(u.pos), np.argsort(ru.pos)
        assert list(u.pos[order]) == [p + pad for p in ru.pos[rorder]]
        np.testing.assert_allclose(u.score[order], ru.score[rorder], rtol=0, atol=1e-12)


def pin_left_padding_invariants(cls):
    """Any left pad: pad rows give zero outputs, pad keys keep score 0 and are
    removed before any real entry (ave 0, older), and the scores of the live
    and removed entries add up to G per real query."""
    rng = np.random.default_rng(59)
    G, s, D, d, kv, B, pad = 2, 23, 4, 6, 5, 4, 7
    q, k, v = _rand_unit(rng, G, s + D, d)
    out, ev, u = _run_padded(cls, q, k, v, s=s, kv_max=kv, block=B, n_decode=D, sm_scale=0.7,
                             pad=pad)
    assert not out[:, :pad].any()
    for e in ev:
        pads_kept = [p for p in e.kept_pos if p < pad]
        real_removed = [p for p in e.evicted_pos if p >= pad]
        assert not (pads_kept and real_removed)
        for p, sc in zip(e.all_pos, e.all_score):
            if p < pad:
                assert sc == 0.0
    total = float(u.score.sum()) + u.evicted_score_total
    assert abs(total - G * (s + D - pad)) < 1e-9


def pin_tova_last_query_weights(cls):
    """TOVA's key is the last processed query's attention (summed over the
    group's heads): with nothing removed it equals SDPA's output for that
    query against one-hot values; with all-zero keys every weight ties, so
    TOVA keeps exactly the most recent entries, like Algorithm 3's rule."""
    rng = np.random.default_rng(61)
    G, s, d = 2, 20, 8
    q, k, v = _rand_unit(rng, G, s, d)
    u = cls(head_dim=d, group=G, kv_max=64, sm_scale=0.5, rule="tova")
    for t0 in range(0, s, 6):
        t1 = min(s, t0 + 6)
        u.prefill_block(t0, q[:, t0:t1], k[t0:t1], v[t0:t1])
        onehot = torch.eye(t1, dtype=torch.float64)
        ref = torch.nn.functional.scaled_dot_product_attention(
            torch.tensor(q[:, t1 - 1:t1]), torch.tensor(k[:t1])[None].expand(G, t1, d),
            onehot[None].expand(G, t1, t1), scale=0.5).numpy()[:, 0].sum(axis=0)
        order = np.argsort(u.pos)
        np.testing.assert_allclose(u.last_w[order], ref, rtol=0, atol=1e-12)
    z = np.zeros((s + 4, d))
    qq = rng.standard_normal((G, s + 4, d))
    a = opd.run_unit(qq, z, v[:1].repeat(s + 4, 0), s=s, kv_max=5, block=4, n_decode=4,
                     sm_scale=1.0, rule="recent")
    u2 = cls(head_dim=d, group=G, kv_max=5, sm_scale=1.0, rule="tova")
    kept = []
    for t0 in range(0, s, 4):
        u2.prefill_block(t0, qq[:, t0:t0 + 4], z[t0:t0 + 4], z[t0:t0 + 4])
        ev = u2.evict(t0 + 3, "prefill")
        if ev is not None:
            kept.append(list(ev.kept_pos))
    for t in range(4):
        _, ev = u2.decode_step(s + t, qq[:, s + t], z[s + t], z[s + t])
        kept.append(list(ev.kept_pos))
    assert kept == [list(e.kept_pos) for e in a.events]


ALL_PINS = [pin_dense_fixed_point, pin_golden, pin_selection_bruteforce,
            pin_conservation_and_lengths, pin_paper_stated_values, pin_permutation_invariance,
            pin_micro_agreement, pin_super_key, pin_rule_keys_bruteforce, pin_alg3_closed_form,
            pin_left_padding_is_a_shift, pin_left_padding_invariants,
            pin_tova_last_query_weights]


@pytest.mark.parametrize("pin", ALL_PINS, ids=lambda f: f.__name__)
def test_pin(pin):
    pin(opd.StepOracle)


def test_alg1_schedule_equivalence():
    pin_alg1_equivalence()


def test_micro_exact_golden():
    """The exact micro-oracle reproduces the hand-derived example exactly,
    including both exact decode ties (older entry evicted)."""
    gold = json.load(open(GOLDEN))
    s, D, d = 6, 2, 8
    T = s + D
    F = Fraction
    q = [[[F(1)] * d for _ in range(T)]]
    k = [[F(0)] * d for _ in range(T)]
    v = [[F(int(i == j)) for j in range(d)] for i in range(T)]
    outs, events, final = micro.micro_run(q, k, v, s=s, kv_max=2, block=2, n_decode=D, sm_scale=F(1))
    assert len(events) == len(gold["events"])
    for ev, gev in zip(events, gold["events"]):
        assert ev["curr_id"] == gev["curr_id"]
        assert ev["kept"] == gev["kept"] and ev["evicted"] == gev["evicted"]
        assert {str(p): x for p, x in ev["score"].items()} == {p: F(x) for p, x in gev["score"].items()}
        assert {str(p): x for p, x in ev["ave"].items()} == {p: F(x) for p, x in gev["ave"].items()}
    assert {str(p): x for p, x in final.items()} == {p: F(x) for p, x in gold["final_score"].items()}
    for i, vis in gold["outputs_visible_sets"].items():
        if i.startswith("_"):
            continue
        want = [F(1, len(vis)) if j in vis else F(0) for j in range(d)]
        assert outs[(0, int(i))] == want


def test_uniform_prefill_keeps_oldest():
    """With all-zero keys (uniform attention) and the bound a multiple of the
    block, every prefill cut keeps exactly positions 0..bound-1: older entries
    average over strictly larger early 1/L terms.  Checked exactly."""
    F = Fraction
    for (kv, B, s) in [(2, 2, 10), (4, 2, 12), (3, 3, 12), (4, 4, 16)]:
        d = 1
        T = s
        q = [[[F(1)] for _ in range(T)]]
        k = [[F(0)] for _ in range(T)]
        v = [[F(0)] for _ in range(T)]
        _, events, _ = micro.micro_run(q, k, v, s=s, kv_max=kv, block=B, n_decode=0, sm_scale=F(1))
        assert events
        for ev in events:
            assert ev["kept"] == list(range(kv))


# ---------------------------------------------------------------------------
# planted mistakes: each must make at least one pin fail
# ---------------------------------------------------------------------------
class _DenomOffByOne(opd.StepOracle):
    def averages(self, curr_id):
        return self.score / np.maximum(curr_id - self.pos, 1).astype(np.float64)


class _NoSelfAttention(opd.StepOracle):
    def attend(self, q, first_pos):
        q = np.asarray(q, dtype=np.float64)
        G, m, d = q.shape
        qpos = first_pos + np.arange(m)
        vis = (self.pos[None, :] < qpos[:, None]) | (qpos[:, None] == 0)
        out = np.zeros((G, m, d))
        for g in range(G):
            z = np.where(vis, self.sm_scale * (q[g] @ self.k.T), -np.inf)
            w = np.exp(z - z.max(axis=1, keepdims=True))
            p = w / w.sum(axis=1, keepdims=True)
            out[g] = p @ self.v
            self.score = self.score + p.sum(axis=0)
        self.queries_seen += G * m
        return out


class _TieNewestFirst(opd.StepOracle):
    def evict(self, curr_id, kind, target=None):
        target = self.kv_max if target is None else target
        n = self.n
        if n <= target:
            return None
        ave = self.ranking_key(curr_id)
        order = np.lexsort((-self.pos, ave))
        n_evict = n - target
        keep = np.sort(order[n_evict:])
        by = np.argsort(self.pos)
        ev = opd.EvictionEvent(kind, curr_id, n, np.sort(self.pos[keep]),
                               np.sort(self.pos[order[:n_evict]]), self.pos[by], self.score[by],
                               ave[by], float(ave[order[n_evict]] - ave[order[n_evict - 1]]))
        self._last = (self.pos.copy(), self.k.copy(), self.v.copy(), self.score.copy(),
                      self.evicted_score_total, self.last_w.copy())
        self.evicted_score_total += float(self.score[order[:n_evict]].sum())
        self._keep(keep)
        return ev


class _FirstHeadOnly(opd.StepOracle):
    def attend(self, q, first_pos):
        before = self.score.copy()
        out = super().attend(q, first_pos)
        q = np.asarray(q, dtype=np.float64)
        G = q.shape[0]
        # keep only head 0's contribution to the scores
        inc = (self.score - before)
        self.score = before + inc / G
        return out


class _NoScale(opd.StepOracle):
    def attend(self, q, first_pos):
        saved = self.sm_scale
        self.sm_scale = 1.0
        try:
            return super().attend(q, first_pos)
        finally:
            self.sm_scale = saved


class _TransposedValues(opd.StepOracle):
    def attend(self, q, first_pos):
        out = super().attend(q, first_pos)
        return out[:, :, ::-1].copy()


class _EvictLargest(opd.StepOracle):
    def averages(self, curr_id):
        return -super().averages(curr_id)


class _SumRuleUsesAverages(opd.StepOracle):
    def ranking_key(self, curr_id):
        if self.rule == "sum":
            return self.averages(curr_id)
        return super().ranking_key(curr_id)


class _RecentKeepsOldest(opd.StepOracle):
    def ranking_key(self, curr_id):
        if self.rule == "recent":
            return -self.pos.astype(np.float64)
        return super().ranking_key(curr_id)


class _TovaFirstRow(opd.StepOracle):
    def attend(self, q, first_pos):
        out = super().attend(q, first_pos)
        saved = (self.score.copy(), self.queries_seen)
        q = np.asarray(q)
        super().attend(q[:, :1], first_pos)          # weights of the call's first row
        self.score, self.queries_seen = saved
        return out


class _TovaUsesScores(opd.StepOracle):
    def ranking_key(self, curr_id):
        if self.rule == "tova":
            return self.score.copy()
        return super().ranking_key(curr_id)


class _PadKeysVisible(opd.StepOracle):
    def attend(self, q, first_pos):
        saved = self.pad
        self.pad = 0
        try:
            return super().attend(q, first_pos)
        finally:
            self.pad = saved


class _PadQueriesScore(opd.StepOracle):
    def attend(self, q, first_pos):
        out = super().attend(q, first_pos)
        q = np.asarray(q)
        m = q.shape[1]
        n_pad_rows = int(np.clip(self.pad - first_pos, 0, m))
        if n_pad_rows and self.n:
            # each pad row spreads its weight uniformly over the visible keys
            self.score = self.score + q.shape[0] * n_pad_rows / self.n
        return out


@pytest.mark.parametrize("mutant", [_DenomOffByOne, _NoSelfAttention, _TieNewestFirst,
                                    _FirstHeadOnly, _NoScale, _TransposedValues, _EvictLargest,
                                    _SumRuleUsesAverages, _RecentKeepsOldest, _PadKeysVisible,
                                    _PadQueriesScore, _TovaFirstRow, _TovaUsesScores],
                         ids=lambda c: c.__name__)
def test_planted_mistake_is_caught(mutant):
    failures = 0
    for pin in ALL_PINS:
        try:
            pin(mutant)
        except AssertionError:
            failures += 1
        except (ValueError, IndexError):
            failures += 1
    assert failures >= 1, f"no pin catches {mutant.__name__}"


# --- Algorithm 1's decoding loop taken literally (remove p when full) ----------
def _alg1_inputs(seed, G=2, T=48, d=16):
    rng = np.random.default_rng(seed)
    q = rng.standard_normal((G, T, d)) / np.sqrt(d)
    k = rng.standard_normal((T, d)) / np.sqrt(d)
    v = rng.standard_normal((T, d))
    return q, k, v


@pytest.mark.parametrize("p", [1, 3, 8])
def test_alg1_decode_lengths_and_removal_rule(p):
    # lengths: full (kv_max) when a step starts -> remove p first, then append;
    # every removal takes the p smallest (ave, pos) with curr_id = pos - 1
    q, k, v = _alg1_inputs(5 + p)
    s, kv, B, D = 16, 8, 4, 32
    unit = opd.UnitOracle(head_dim=16, group=2, kv_max=kv, sm_scale=0.25)
    for t0 in range(0, s, B):
        unit.prefill_block(t0, q[:, t0:t0 + B], k[t0:t0 + B], v[t0:t0 + B])
        unit.evict(t0 + B - 1, "prefill")
    assert unit.n == kv
    cuts = 0
    for t in range(D):
        i = s + t
        full = unit.n == kv
        _, ev = unit.decode_step_alg1(i, q[:, i], k[i], v[i], p)
        assert (ev is not None) == full
        if ev is not None:
            cuts += 1
            assert ev.curr_id == i - 1 and ev.n_before == kv
            pairs = sorted(zip(ev.all_ave, ev.all_pos))
            assert sorted(int(x) for x in ev.evicted_pos) == sorted(int(b) for _, b in pairs[:p])
            # the averages come from the scores and ages at curr_id = i - 1
            assert np.allclose(ev.all_ave, ev.all_score / (i - ev.all_pos))
        assert unit.n == (kv - p + 1 if full else min(kv, unit.n))
        assert unit.n <= kv
    assert cuts == len(range(0, D, p)) if p > 1 else cuts == D


def test_alg1_decode_removing_everything_leaves_the_new_token():
    # p = kv_max: the cut empties the cache, so the new token attends to itself
    # alone and its output is exactly its own value row
    q, k, v = _alg1_inputs(3)
    s, kv, B = 16, 8, 8
    unit = opd.UnitOracle(head_dim=16, group=2, kv_max=kv, sm_scale=0.25)
    for t0 in range(0, s, B):
        unit.prefill_block(t0, q[:, t0:t0 + B], k[t0:t0 + B], v[t0:t0 + B])
        unit.evict(t0 + B - 1, "prefill")
    o, ev = unit.decode_step_alg1(s, q[:, s], k[s], v[s], kv)
    assert ev is not None and len(ev.kept_pos) == 0
    assert np.array_equal(o, np.broadcast_to(v[s], o.shape))
    assert np.allclose(unit.score, [2.0])       # both heads put weight 1 on it


def test_alg1_decode_matches_dense_when_bound_is_never_reached():
    q, k, v = _alg1_inputs(9)
    s, D = 16, 32
    a = opd.run_unit(q, k, v, s=s, kv_max=64, block=4, n_decode=D, sm_scale=0.25)
    b = opd.run_unit(q, k, v, s=s, kv_max=64, block=4, n_decode=D, sm_scale=0.25, p_dec=5)
    assert np.array_equal(a.out, b.out) and not b.events


def test_run_unit_ed_mode_is_algorithm_3():
    """run_unit's ED configuration (no prefill removal, decode bound 2, p = 1,
    most-recent rule) reproduces Algorithm 3 stepped by hand, and its decode
    outputs only ever see two entries."""
    rng = np.random.default_rng(43)
    G, s, D, d = 2, 10, 5, 4
    q, k, v = _rand_unit(rng, G, s + D, d)
    tr = opd.run_unit(q, k, v, s=s, kv_max=s, block=4, n_decode=D, sm_scale=0.5, p_dec=1,
                      rule="recent", kv_dec=2)
    u = opd.UnitOracle(head_dim=d, group=G, kv_max=s, sm_scale=0.5, rule="recent")
    u.prefill_block(0, q[:, :s], k[:s], v[:s])
    keep = u.evict(s - 1, "decode", target=1)          # remove all but the most recent
    assert list(keep.kept_pos) == [s - 1]
    for t in range(D):
        i = s + t
        u.append(i, k[i:i + 1], v[i:i + 1])
        assert u.n == 2
        o = u.attend(q[:, i:i + 1], i)[:, 0]
        np.testing.assert_allclose(tr.out[:, i], o, rtol=0, atol=1e-13)
        u.evict(i, "decode", target=1)
    assert len(tr.events) == D


def test_run_unit_decode_bound_with_one_removal_per_step():
    """p = 0 with a decode bound below the prefill bound: the first step cuts
    to the decode bound at the last processed position, then one removal per
    step keeps the bound."""
    rng = np.random.default_rng(47)
    G, s, D, d = 1, 16, 6, 4
    q, k, v = _rand_unit(rng, G, s + D, d)
    tr = opd.run_unit(q, k, v, s=s, kv_max=12, block=4, n_decode=D, sm_scale=0.5, kv_dec=5)
    dec = [e for e in tr.events if e.kind == "decode"]
    assert dec[0].curr_id == s - 1 and len(dec[0].kept_pos) == 5
    assert all(len(e.kept_pos) == 5 for e in dec[1:]) and len(dec) == D + 1
    assert len(tr.final_pos) == 5
