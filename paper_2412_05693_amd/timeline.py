"""Per-workgroup timeline of the prefill attention kernel (measurement only).

    python -m paper_2412_05693_amd.timeline [--config c2] [--batch B]
    python -m paper_2412_05693_amd.timeline --fit [--config c2]

The first form loads ``libbatchmax_timeline.so`` (``python -m
paper_2412_05693_amd.build --timeline``), runs one workload's prefill (every
block with its fused cut, twice), and summarises the records the kernel wrote
for the last block: where each workgroup's time goes (prologue, the two
sweeps, the step between them), how the prologue splits (query loads, tile
copies, the wait), and the time spent issuing copies, waiting for them and in
barriers inside the tile loops.  Tick length is calibrated against HIP events
around the same launch.

The second form uses the ordinary library and fits the prefill time per step
against the key tiles per workgroup over cache bounds 128 to 3072 (same
shape otherwise): the intercept is the cost per workgroup that does not grow
with its tiles.  Prints markdown.
"""
from __future__ import annotations

import argparse
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))


def _parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--config", default="c2")
    ap.add_argument("--batch", type=int, default=None)
    ap.add_argument("--fit", action="store_true")
    return ap.parse_args()


def _setup(wl, dev):
    import torch

    from . import batchmax as bmx
    from . import synth

    q, k, v = synth.batch_inputs(wl, dev)
    o = torch.zeros_like(q)
    pd = bmx.PDAttention(b=wl.b, s=wl.s, kv_max=wl.kv_max, block=wl.block, max_gen=wl.n_decode,
                         n_heads=wl.n_heads, n_kv_heads=wl.n_kv_heads, head_dim=wl.head_dim,
                         dtype=wl.dtype, sm_scale=wl.sm_scale, device=dev)
    return pd, (q, k, v, o)


def _prefill_timed(pd, qkvo, wl, stream):
    """One prefill of every block with its cut; returns per-block attention ms."""
    import torch

    blocks = [(t0, min(wl.block, wl.s - t0)) for t0 in range(0, wl.s, wl.block)]
    evs = []
    pd.reset()
    for t0, n in blocks:
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        pd.set_split_event(e1)
        e0.record(stream)
        pd.prefill_block_cut(t0, n, *qkvo)
        evs.append((e0, e1))
    torch.cuda.synchronize()
    return [a.elapsed_time(b) for a, b in evs]


def _tiles_per_step(wl, ppw):
    """Key tiles over all workgroups of one prefill step, and workgroups."""
    tiles = wgs = 0
    length = 0
    for t0 in range(0, wl.s, wl.block):
        n = min(wl.block, wl.s - t0)
        for p in range(-(-n // ppw)):
            in_rows = min(n, p * ppw + ppw)
            tiles += -(-length // 64) + -(-in_rows // 64)
            wgs += 1
        length = min(wl.kv_max, length + n)
    units = wl.b * wl.n_kv_heads
    return tiles * units, wgs * units


def timeline(args) -> None:
    import numpy as np
    import torch

    from . import batchmax as bmx
    from . import synth

    wl = synth.WORKLOADS[args.config].with_(n_decode=1)
    if args.batch:
        wl = wl.with_(b=args.batch)
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    pd, qkvo = _setup(wl, dev)
    stream = torch.cuda.current_stream(dev)
    for _ in range(2):
        ms = _prefill_timed(pd, qkvo, wl, stream)
    d = bmx.make_dims(b=wl.b, s=wl.s, kv_max=wl.kv_max, block=wl.block, max_gen=wl.n_decode,
                      n_heads=wl.n_heads, n_kv_heads=wl.n_kv_heads, head_dim=wl.head_dim,
                      dtype=wl.dtype)
    ppw = bmx.bm_prefill_positions_per_workgroup(d)
    last_n = wl.s - (len(ms) - 1) * wl.block
    nwg = wl.b * wl.n_kv_heads * -(-last_n // ppw)
    if nwg > bmx.TIMELINE_MAX_RECORDS:
        raise SystemExit(f"{nwg} workgroups: more than {bmx.TIMELINE_MAX_RECORDS} records; use --batch")
    r = bmx.bm_prefill_timeline(nwg).astype(np.int64)
    span = r[:, 7].max() - r[:, 0].min()
    us = ms[-1] * 1e3 / span                      # microseconds per tick
    ph = lambda a, b: (r[:, b] - r[:, a]) * us    # noqa: E731
    tot = ph(0, 7)
    print(f"# Prefill timeline: {wl.name}, b={wl.b}, last block ({nwg} workgroups)\n")
    print(f"Attention kernel {ms[-1] * 1e3:.1f} us by events; {us * 1e3:.2f} ns per tick "
          f"({1 / us:.1f} ticks per us).  Per workgroup, mean (p10 / p90):\n")
    print("| phase | us | p10 | p90 |\n|---|---:|---:|---:|")
    rows = [("entry -> block-row and query loads issued", ph(0, 1)), ("query loads -> first copies issued", ph(1, 2)),
            ("copies issued -> first tiles ready (wait, append, barrier)", ph(2, 3)),
            ("sweep 1 (online softmax, PV)", ph(3, 4)), ("output rows stored", ph(4, 5)),
            ("sweep 2 prologue", ph(5, 6)), ("sweep 2 (column sums)", ph(6, 7)), ("total", tot),
            ("sweep 1: issuing tile copies", r[:, 8] * us), ("sweep 1: waiting at tile ends", r[:, 9] * us),
            ("sweep 1: barriers", r[:, 10] * us), ("sweep 2: waiting at tile ends", r[:, 11] * us),
            ("sweep 2: barriers", r[:, 12] * us)]
    for name, x in rows:
        print(f"| {name} | {x.mean():.2f} | {np.percentile(x, 10):.2f} | {np.percentile(x, 90):.2f} |")
    tiles = r[:, 15]
    print(f"\nKey tiles per workgroup: {tiles.min()}-{tiles.max()} (mean {tiles.mean():.2f}); "
          f"sweep 1 {ph(3, 4).mean() / tiles.mean():.2f} us and sweep 2 "
          f"{ph(6, 7).mean() / tiles.mean():.2f} us per tile.")
    hw = r[:, 13] & 0xFFFFFFFF
    xcc = (r[:, 13] >> 32) & 0xF
    cu = ((xcc * 8 + ((hw >> 13) & 7)) * 2 + ((hw >> 12) & 1)) * 16 + ((hw >> 8) & 15)
    start, end = r[:, 0], r[:, 7]
    busy = []
    for c in np.unique(cu):
        idx = np.where(cu == c)[0]
        ev = sorted([(start[i], 1) for i in idx] + [(end[i], -1) for i in idx])
        acc, cur, last = np.zeros(4), 0, None
        for t, dlt in ev:
            if last is not None:
                acc[min(cur, 3)] += t - last
            cur += dlt
            last = t
        busy.append(acc)
    busy = np.sum(busy, 0)
    busy = busy / busy.sum()
    print(f"Per compute unit ({len(np.unique(cu))} seen): share of the time from a unit's first "
          f"workgroup start to its last workgroup end with 0 / 1 / 2 / 3+ workgroups resident "
          f"{busy[0]:.3f} / {busy[1]:.3f} / {busy[2]:.3f} / {busy[3]:.3f}.")
    pd.close()


def fit(args) -> None:
    import numpy as np
    import torch

    from . import batchmax as bmx
    from . import synth

    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream(dev)
    base = synth.WORKLOADS[args.config].with_(n_decode=1)
    if args.batch:
        base = base.with_(b=args.batch)
    rows = []
    print(f"# Prefill time against key tiles per workgroup: {base.name}, b={base.b}\n")
    print("| cache bound | workgroup tiles per step | workgroups per step | attention ms per step |")
    print("|---:|---:|---:|---:|")
    for kv in (128, 256, 512, 1024, 2048, 3072):
        wl = base.with_(kv_max=kv)
        pd, qkvo = _setup(wl, dev)
        _prefill_timed(pd, qkvo, wl, stream)
        ms = np.mean([sum(_prefill_timed(pd, qkvo, wl, stream)) for _ in range(3)])
        d = bmx.make_dims(b=wl.b, s=wl.s, kv_max=wl.kv_max, block=wl.block, max_gen=wl.n_decode,
                          n_heads=wl.n_heads, n_kv_heads=wl.n_kv_heads, head_dim=wl.head_dim,
                          dtype=wl.dtype)
        t, w = _tiles_per_step(wl, bmx.bm_prefill_positions_per_workgroup(d))
        rows.append((t, w, ms))
        print(f"| {kv} | {t} | {w} | {ms:.3f} |")
        pd.close()
        del pd, qkvo
        torch.cuda.empty_cache()
    t = np.array([x[0] for x in rows], float)
    ms = np.array([x[2] for x in rows])
    (slope, icpt), *_ = np.linalg.lstsq(np.stack([t, np.ones_like(t)], 1), ms, rcond=None)
    w = rows[0][1]
    print(f"\nFit: {slope * 1e6:.3f} ms per 1e6 workgroup-tiles + {icpt:.3f} ms per step; "
          f"the intercept is {icpt / slope / w:.2f} tile-times per workgroup "
          f"({icpt / ms.mean() * 100:.0f}% of the mean step).")


def main() -> None:
    args = _parse()
    if not args.fit:
        os.environ.setdefault("BATCHMAX_LIB", os.path.join(HERE, "libbatchmax_timeline.so"))
    sys.path.insert(0, os.path.dirname(HERE))
    if args.fit:
        fit(args)
    else:
        timeline(args)


if __name__ == "__main__":
    main()
