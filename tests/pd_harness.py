"""GPU-versus-oracle comparison of a full P&D run, event by event.

Both sides get exactly the same input values (the seeded unit streams).  After
every device call the checked units' state is copied back and compared with the
float64 oracle stepping in lockstep:

* cache length: exact;
* the set of live positions after every cut: exact, except inside the near-tie
  band -- if the device kept a different set, every entry it evicted must rank
  within ``band`` (in the oracle's own averages) of every entry it kept; the
  oracle then adopts the device's set so later steps stay comparable;
* scores of live entries, matched by position: relative tolerance 1e-3;
* attention outputs: max abs error <= 2e-2 (bf16) or 1e-4 (float32).

Counts of cuts, near-ties (oracle gap below ``band``) and adopted sets are
reported; any other difference is a failure.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np
import torch

from oracle import pd as opd
from paper_2412_05693_amd import synth
from paper_2412_05693_amd.batchmax import PDAttention

BAND = 1e-6
SCORE_RTOL = 1e-3
SCORE_ATOL = 1e-6
OUT_TOL = {"bf16": 2e-2, "f32": 1e-4}


@dataclass
class Stats:
    cuts: int = 0
    near_ties: int = 0
    adopted: int = 0
    max_out_err: float = 0.0
    max_score_rel: float = 0.0
    failures: list = field(default_factory=list)

    def fail(self, msg):
        if len(self.failures) < 20:
            self.failures.append(msg)

    def summary(self) -> str:
        return (f"cuts={self.cuts} near_ties={self.near_ties} adopted={self.adopted} "
                f"max_out_err={self.max_out_err:.3e} max_score_rel={self.max_score_rel:.3e} "
                f"failures={len(self.failures)}")


def make_pd(wl: synth.Workload, device="cuda", b=None) -> PDAttention:
    return PDAttention(b=wl.b if b is None else b, s=wl.s, kv_max=wl.kv_max, block=wl.block,
                       max_gen=wl.n_decode, n_heads=wl.n_heads, n_kv_heads=wl.n_kv_heads,
                       head_dim=wl.head_dim, dtype=wl.dtype, sm_scale=wl.sm_scale, device=device)


def _snapshot(pd: PDAttention, units, length):
    bi = torch.tensor([u[0] for u in units], device=pd.device)
    hk = torch.tensor([u[1] for u in units], device=pd.device)
    pos = pd.pos[bi, hk, :length].cpu().numpy()
    score = pd.score[bi, hk, :length].cpu().numpy().astype(np.float64)
    dlen = pd.len[bi, hk].cpu().numpy()
    return pos, score, dlen


def _compare_state(tag, orc, pos, score, dlen, length, st: Stats, scores=True):
    if np.any(dlen != length):
        st.fail(f"{tag}: device len {dlen.tolist()} != {length}")
        return False
    order = np.argsort(pos)
    gpos, gscore = pos[order], score[order]
    opos_order = np.argsort(orc.pos)
    opos, oscore = orc.pos[opos_order], orc.score[opos_order]
    if not np.array_equal(gpos, opos):
        st.fail(f"{tag}: live positions differ (device {len(gpos)}, oracle {len(opos)})")
        return False
    if not scores:
        return True
    err = np.abs(gscore - oscore)
    rel = err / np.maximum(np.abs(oscore), 1e-30)
    st.max_score_rel = max(st.max_score_rel, float(np.max(np.where(err > SCORE_ATOL, rel, 0.0))))
    bad = err > SCORE_RTOL * np.abs(oscore) + SCORE_ATOL
    if np.any(bad):
        i = int(np.argmax(bad))
        st.fail(f"{tag}: score of pos {gpos[i]} {gscore[i]:.8g} vs oracle {oscore[i]:.8g}")
        return False
    return True


def _compare_cut(tag, orc: opd.StepOracle, ev, gpu_pos, st: Stats):
    if ev is None:
        return
    st.cuts += 1
    if ev.gap < BAND:
        st.near_ties += 1
    gk = sorted(int(p) for p in gpu_pos)
    ok = list(int(p) for p in ev.kept_pos)
    if gk == ok:
        return
    ave = {int(p): float(a) for p, a in zip(ev.all_pos, ev.all_ave)}
    gset = set(gk)
    if len(gk) != len(ok) or not gset <= set(ave):
        st.fail(f"{tag}: device kept set is not a valid cut")
        return
    evicted = set(ave) - gset
    spread = max(ave[p] for p in evicted) - min(ave[p] for p in gset)
    if spread < BAND:
        st.adopted += 1
        orc.adopt(gk)
    else:
        st.fail(f"{tag}: device cut differs beyond the band (spread {spread:.3e}, "
                f"oracle gap {ev.gap:.3e})")


def run_parity(wl: synth.Workload, checked, *, sharp=False, device="cuda", decode_steps=None,
               inputs=None, pd=None, stop_on_failure=True, decode_p=0, rule="ave",
               decode_bound=None, accumulate=True, fused_cut=False) -> Stats:
    """Run the whole P&D schedule on the device and compare the checked units.

    ``decode_p > 0`` selects Algorithm 1's decoding loop taken literally (a step
    that starts with a full cache first removes ``decode_p`` entries); the cut
    is compared against the device's live set without the step's new entry.
    ``rule`` is the ranking rule of every cut, ``decode_bound`` the cache bound
    during decode (default kv_max).  ``accumulate=False`` runs the prefill
    without score sums: scores are then not compared (only positions).
    ``fused_cut`` runs each block and its cut as one call (the state between
    the two is then not observed)."""
    st = Stats()
    if inputs is None:
        inputs = synth.batch_inputs(wl, device, checked=checked, sharp=sharp)
    q, k, v = inputs
    o = torch.zeros_like(q)
    pd = pd or make_pd(wl, device)
    if decode_p:
        pd.set_decode_removal(decode_p)
    if rule != "ave":
        pd.set_rank_rule(rule)
    kd = wl.kv_max if decode_bound is None else decode_bound
    if decode_bound is not None:
        pd.set_decode_bound(decode_bound)
    if not accumulate:
        pd.set_score_accumulation(False)
    pads = synth.sample_pads(wl)
    if wl.pad_max > 0:
        pd.set_left_padding(torch.from_numpy(pads).to(pd.device))
    sc = accumulate
    G = wl.group
    uin = {u: synth.unit_inputs(wl, 0, u[0], u[1], sharp=sharp) for u in checked}
    orcs = {u: opd.StepOracle(head_dim=wl.head_dim, group=G, kv_max=wl.kv_max,
                              sm_scale=wl.sm_scale, rule=rule, pad=int(pads[u[0]]))
            for u in checked}
    tol = OUT_TOL[wl.dtype]
    D = wl.n_decode if decode_steps is None else decode_steps

    def check_out(tag, u, rows, ref):
        bi, hk = u
        got = o[bi, hk * G:(hk + 1) * G, rows].float().cpu().numpy().astype(np.float64)
        err = float(np.max(np.abs(got - ref))) if got.size else 0.0
        st.max_out_err = max(st.max_out_err, err)
        if not err <= tol:
            st.fail(f"{tag} unit {u}: output error {err:.3e} > {tol}")

    for t0 in range(0, wl.s, wl.block):
        n = min(wl.block, wl.s - t0)
        if fused_cut:
            pd.prefill_block_cut(t0, n, q, k, v, o)
            for u in checked:
                uq, uk, uv = uin[u]
                ref = orcs[u].prefill_block(t0, uq[:, t0:t0 + n], uk[t0:t0 + n], uv[t0:t0 + n])
                check_out(f"block {t0}", u, slice(t0, t0 + n), ref)
        else:
            pd.prefill_block(t0, n, q, k, v, o)
            length = pd.length
            pos, score, dlen = _snapshot(pd, checked, length)
            for i, u in enumerate(checked):
                uq, uk, uv = uin[u]
                ref = orcs[u].prefill_block(t0, uq[:, t0:t0 + n], uk[t0:t0 + n], uv[t0:t0 + n])
                check_out(f"block {t0}", u, slice(t0, t0 + n), ref)
                _compare_state(f"block {t0} unit {u}", orcs[u], pos[i], score[i], dlen[i], length,
                               st, sc)
            pd.evict_compact(t0 + n - 1)
        length = pd.length
        pos, score, dlen = _snapshot(pd, checked, length)
        for i, u in enumerate(checked):
            ev = orcs[u].evict(t0 + n - 1, "prefill")
            _compare_cut(f"cut {t0 + n - 1} unit {u}", orcs[u], ev, pos[i], st)
            _compare_state(f"cut {t0 + n - 1} unit {u}", orcs[u], pos[i], score[i], dlen[i],
                           length, st, sc)
        if stop_on_failure and st.failures:
            return st

    for t in range(D):
        p = wl.s + t
        pd.decode_step(p, q, k, v, o, row=p)
        length = pd.length
        pos, score, dlen = _snapshot(pd, checked, length)
        for i, u in enumerate(checked):
            uq, uk, uv = uin[u]
            orc = orcs[u]
            if decode_p:
                # the oracle's step taken apart (the cut, then append + attend, as in
                # UnitOracle.decode_step_alg1) so a near-tie cut can be adopted before
                # the new entry is attended
                if orc.n >= kd:
                    ev = orc.evict(p - 1, "decode", target=kd - decode_p)
                    _compare_cut(f"decode {p} unit {u}", orc, ev, pos[i][pos[i] != p], st)
                orc.append(p, uk[p][None], uv[p][None])
                ref = orc.attend(uq[:, p][:, None, :], p)[:, 0, :]
            else:
                if orc.n > kd:    # a lower decode bound: cut first (seen only in the end state)
                    orc.evict(p - 1, "decode", target=kd)
                ref, ev = orc.decode_step(p, uq[:, p], uk[p], uv[p], bound=kd)
                _compare_cut(f"decode {p} unit {u}", orc, ev, pos[i], st)
            check_out(f"decode {p}", u, slice(p, p + 1), ref[:, None, :])
            _compare_state(f"decode {p} unit {u}", orc, pos[i], score[i], dlen[i], length, st, sc)
        if stop_on_failure and st.failures:
            return st
    return st


def stack_params(wl: synth.Workload, layer: int, b: int):
    from paper_2412_05693_amd.batchmax import synth_params

    return synth_params(b=b, n_heads=wl.n_heads, n_kv_heads=wl.n_kv_heads, head_dim=wl.head_dim,
                        dtype=wl.dtype, seed=wl.seed, layer=layer, s=wl.s, hh_frac=wl.hh_frac,
                        hh_scale=wl.hh_scale, n_sinks=wl.n_sinks, sink_scale=wl.sink_scale,
                        heavy=wl.hh_mode != "none")


def run_stack_parity(wl: synth.Workload, checked, *, device="cuda", decode_steps=None,
                     stop_on_failure=True, fused_cut=False) -> Stats:
    """The layer stack: every layer's inputs come from the device generator one
    block (or decode row) at a time; the checked units ``(layer, sample,
    kv_head)`` are compared with the oracle fed by the host evaluation of the
    same counter-based stream.  ``fused_cut`` runs each block and its cut as
    one call (the benchmark's path; the state between the two is then not
    observed)."""
    from paper_2412_05693_amd.batchmax import PDStack, synth_qkv

    st = Stats()
    b, H, Hk, d, B, G = wl.b, wl.n_heads, wl.n_kv_heads, wl.head_dim, wl.block, wl.group
    tdt = torch.float32 if wl.dtype == "f32" else torch.bfloat16
    stack = PDStack(n_layers=wl.n_layers, b=b, s=wl.s, kv_max=wl.kv_max, block=B,
                    max_gen=wl.n_decode, n_heads=H, n_kv_heads=Hk, head_dim=d, dtype=wl.dtype,
                    sm_scale=wl.sm_scale, device=device)
    stack.reset()
    q = torch.empty((b, H, B, d), dtype=tdt, device=device)
    k = torch.empty((b, Hk, B, d), dtype=tdt, device=device)
    v = torch.empty_like(k)
    o = torch.zeros_like(q)
    qd = torch.empty((b, H, 1, d), dtype=tdt, device=device)
    kd = torch.empty((b, Hk, 1, d), dtype=tdt, device=device)
    vd = torch.empty_like(kd)
    od = torch.zeros_like(qd)
    params = [stack_params(wl, layer, b) for layer in range(wl.n_layers)]
    by_layer = {}
    for (layer, bi, hk) in checked:
        by_layer.setdefault(layer, []).append((bi, hk))
    uin = {u: synth.stack_unit_inputs(wl, *u) for u in checked}
    orcs = {u: opd.StepOracle(head_dim=d, group=G, kv_max=wl.kv_max, sm_scale=wl.sm_scale)
            for u in checked}
    tol = OUT_TOL[wl.dtype]
    D = wl.n_decode if decode_steps is None else decode_steps

    def check_out(tag, out, u, n, ref):
        _, bi, hk = u
        got = out[bi, hk * G:(hk + 1) * G, :n].float().cpu().numpy().astype(np.float64)
        err = float(np.max(np.abs(got - ref))) if got.size else 0.0
        st.max_out_err = max(st.max_out_err, err)
        if not err <= tol:
            st.fail(f"{tag} unit {u}: output error {err:.3e} > {tol}")

    for t0 in range(0, wl.s, B):
        n = min(B, wl.s - t0)
        for layer in range(wl.n_layers):
            pd = stack.layers[layer]
            synth_qkv(params[layer], t0, q, k, v)
            units = by_layer.get(layer)
            if fused_cut:
                pd.prefill_block_cut(t0, n, q, k, v, o, row=0)
                for (bi, hk) in units or ():
                    u = (layer, bi, hk)
                    uq, uk, uv = uin[u]
                    ref = orcs[u].prefill_block(t0, uq[:, t0:t0 + n], uk[t0:t0 + n], uv[t0:t0 + n])
                    check_out(f"block {t0}", o, u, n, ref)
            else:
                pd.prefill_block(t0, n, q, k, v, o, row=0)
            if units and not fused_cut:
                length = pd.length
                pos, score, dlen = _snapshot(pd, units, length)
                for i, (bi, hk) in enumerate(units):
                    u = (layer, bi, hk)
                    uq, uk, uv = uin[u]
                    ref = orcs[u].prefill_block(t0, uq[:, t0:t0 + n], uk[t0:t0 + n], uv[t0:t0 + n])
                    check_out(f"block {t0}", o, u, n, ref)
                    _compare_state(f"block {t0} unit {u}", orcs[u], pos[i], score[i], dlen[i],
                                   length, st)
            if not fused_cut:
                pd.evict_compact(t0 + n - 1)
            if units:
                length = pd.length
                pos, score, dlen = _snapshot(pd, units, length)
                for i, (bi, hk) in enumerate(units):
                    u = (layer, bi, hk)
                    ev = orcs[u].evict(t0 + n - 1, "prefill")
                    _compare_cut(f"cut {t0 + n - 1} unit {u}", orcs[u], ev, pos[i], st)
                    _compare_state(f"cut {t0 + n - 1} unit {u}", orcs[u], pos[i], score[i],
                                   dlen[i], length, st)
        if stop_on_failure and st.failures:
            return st

    for t in range(D):
        p = wl.s + t
        for layer in range(wl.n_layers):
            pd = stack.layers[layer]
            synth_qkv(params[layer], p, qd, kd, vd)
            pd.decode_step(p, qd, kd, vd, od, row=0)
            units = by_layer.get(layer)
            if units:
                length = pd.length
                pos, score, dlen = _snapshot(pd, units, length)
                for i, (bi, hk) in enumerate(units):
                    u = (layer, bi, hk)
                    uq, uk, uv = uin[u]
                    ref, ev = orcs[u].decode_step(p, uq[:, p], uk[p], uv[p])
                    check_out(f"decode {p}", od, u, 1, ref[:, None, :])
                    _compare_cut(f"decode {p} unit {u}", orcs[u], ev, pos[i], st)
                    _compare_state(f"decode {p} unit {u}", orcs[u], pos[i], score[i], dlen[i],
                                   length, st)
        if stop_on_failure and st.failures:
            return st
    stack.close()
    return st
