"""Pure-Python loop oracle for tiny inputs, exact where softmax is exact.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

An independent second implementation of the same method as ``oracle.pd``:
lists and explicit loops, no numpy.  It serves two pins:

* with ``fractions.Fraction`` inputs whose visible logits within a row are all
  equal (for instance all-zero keys), softmax is exactly uniform, 1/L for a row
  with L visible entries, so scores, averages, kept sets and outputs are exact
  rationals and exact ties are resolved exactly (reading R8);
* with float inputs it uses ``math.exp`` on Python floats (IEEE double), so
  it must agree with the numpy oracle to rounding.

Semantics follow Sec. 3.1 (Algorithm 1 under reading R1) and Sec. 3.2
(``sum_weights`` update, ``ave_weights`` rule), as in ``oracle.pd``.
"""
from __future__ import annotations

import math
from fractions import Fraction


def _softmax(logits):
    """Softmax of one row; exact 1/L when every logit is the same rational."""
    if all(isinstance(z, Fraction) for z in logits):
        if any(z != logits[0] for z in logits):
            raise ValueError("exact mode needs equal logits within a row")
        return [Fraction(1, len(logits))] * len(logits)
    m = max(logits)
    e = [math.exp(z - m) for z in logits]
    tot = sum(e)
    return [x / tot for x in e]


def micro_run(q, k, v, *, s, kv_max, block, n_decode, sm_scale):
    """Run one unit; returns (outputs, events, final entries).

    q: list [G][s+D][d]; k, v: list [s+D][d] (Fractions or floats).
    outputs: dict (g, position) -> list of d values.
    events: list of dicts with curr_id, kept (sorted positions), evicted,
            score (dict pos -> score before the cut), ave (dict pos -> ave).
    final: dict pos -> score of the entries left at the end.
    """
    G = len(q)
    cache = []          # entries: dict(pos=, k=, v=, score=)
    outputs = {}
    events = []

    def process(first, last):
        # append the KV pairs of positions first..last with zero score (Sec. 3.2)
        for i in range(first, last + 1):
            cache.append({"pos": i, "k": k[i], "v": v[i], "score": 0 * sm_scale})
        # every query head g and every position i in the span attends causally
        for g in range(G):
            for i in range(first, last + 1):
                vis = [e for e in cache if e["pos"] <= i]
                logits = []
                for e in vis:
                    dot = 0
                    for a, b in zip(q[g][i], e["k"]):
                        dot += a * b
                    logits.append(sm_scale * dot)
                probs = _softmax(logits)
                out = [0] * len(q[g][i])
                for p, e in zip(probs, vis):
                    for t in range(len(out)):
                        out[t] += p * e["v"][t]
                    e["score"] += p
                outputs[(g, i)] = out

    def cut(curr_id):
        if len(cache) <= kv_max:
            return
        ave = {e["pos"]: e["score"] / (curr_id + 1 - e["pos"]) for e in cache}
        ranked = sorted(cache, key=lambda e: (ave[e["pos"]], e["pos"]))
        n_evict = len(cache) - kv_max
        evicted = ranked[:n_evict]
        kept = ranked[n_evict:]
        events.append({
            "curr_id": curr_id,
            "kept": sorted(e["pos"] for e in kept),
            "evicted": sorted(e["pos"] for e in evicted),
            "score": {e["pos"]: e["score"] for e in cache},
            "ave": ave,
        })
        cache[:] = kept

    t0 = 0
    while t0 < s:
        t1 = min(s, t0 + block)
        process(t0, t1 - 1)
        cut(t1 - 1)
        t0 = t1
    for t in range(n_decode):
        i = s + t
        process(i, i)
        cut(i)
    final = {e["pos"]: e["score"] for e in cache}
    return outputs, events, final
