#!/usr/bin/env python3
"""Benchmark: Batch-Max P&D KV-compressed attention on one MI355X.

A *step* is one full P&D pass over one batch: reset the bounded cache, prefill
the prompt block by block (attention + score sums, then the cut back to the
bound and compaction after every block), then the decode steps (attention,
score update and one eviction per step).  Inputs are synthetic (seeded, the
distributions of the workload statement) and resident in HBM before timing.

Prints one JSON line:  metric/value (P&D tokens/s = b * (s + D) / step time),
roofline of the dominant kernel (algorithmic flops or bytes per launch over the
launch time measured with HIP events on the launch stream), and the CPU
baseline (the float64 oracle on a bounded sample of units, timed on the host
before the GPU is initialised).

    python bench.py [--config c2] [--steps K] [--warmup W] [--gpus 1]
"""
from __future__ import annotations

import argparse
import json
import math
import multiprocessing as mp
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_BF16_MFMA = 2.5e15      # dense bf16 MFMA, FLOP/s
PEAK_F32_MFMA = 157.3e12     # fp32 matrix/vector, FLOP/s
PEAK_HBM = 8.0e12            # bytes/s
HBM_PROBE_BYTES = 1 << 30    # the plain copy that calibrates the HBM byte counters


def source_digest() -> str:
    """sha256 over the prefill kernel's sources: a counter record applies only
    to the kernel it was measured on."""
    import hashlib

    h = hashlib.sha256()
    for rel in ("paper_2412_05693_amd/csrc/k_prefill.hip", "paper_2412_05693_amd/csrc/bm_internal.h"):
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def measured_traffic(workload: str):
    """HBM bytes per prefill launch from a committed counter record
    (`traffic-record:` line under profiles/), or None when there is none for
    this workload or the kernel sources changed since it was taken."""
    pdir = os.path.join(ROOT, "profiles")
    if not os.path.isdir(pdir):
        return None
    digest = source_digest()
    for fn in sorted(os.listdir(pdir)):
        if not fn.endswith((".md", ".txt")):
            continue
        with open(os.path.join(pdir, fn)) as f:
            for line in f:
                line = line.strip().strip("`")
                if not line.startswith("traffic-record:"):
                    continue
                kv = dict(item.split("=", 1) for item in line.split()[1:] if "=" in item)
                if kv.get("workload") == workload and kv.get("source_sha256") == digest:
                    return int(kv["bytes_per_launch"])
    return None


def hbm_probe():
    """A plain device copy of HBM_PROBE_BYTES, three times: run it under
    rocprofv3 --pmc FETCH_SIZE (then WRITE_SIZE) to calibrate the counters."""
    import torch

    a = torch.ones(HBM_PROBE_BYTES, dtype=torch.uint8, device="cuda")
    b = torch.empty_like(a)
    for _ in range(3):
        b.copy_(a)
    torch.cuda.synchronize()
    print(f"hbm probe: copied {HBM_PROBE_BYTES} bytes three times", flush=True)


# ---------------------------------------------------------------------------
# CPU baseline: the oracle as it stands, one unit per worker process
# ---------------------------------------------------------------------------
def _oracle_unit(args):
    name, overrides, bi, hk = args
    os.environ.setdefault("OMP_NUM_THREADS", "1")
    from oracle import pd as opd
    from paper_2412_05693_amd import synth

    wl = synth.WORKLOADS[name].with_(**overrides)
    q, k, v = synth.unit_inputs(wl, 0, bi, hk)
    t = time.perf_counter()
    opd.run_unit(q, k, v, s=wl.s, kv_max=wl.kv_max, block=wl.block, n_decode=wl.n_decode,
                 sm_scale=wl.sm_scale)
    return time.perf_counter() - t


def cpu_baseline(name, overrides, budget_s):
    from paper_2412_05693_amd import synth

    wl = synth.WORKLOADS[name].with_(**overrides)
    cores = len(os.sched_getaffinity(0))
    cores = max(1, min(cores, 16))
    for var in ("OMP_NUM_THREADS", "OPENBLAS_NUM_THREADS", "MKL_NUM_THREADS"):
        os.environ[var] = "1"
    ctx = mp.get_context("fork")     # forked before any GPU initialisation
    units = synth.checked_units(wl, min(wl.units, 100000), seed=7)
    done, t0 = 0, time.perf_counter()
    with ctx.Pool(cores) as pool:
        # first wave sizes the sample: keep to about budget_s of wall time
        first = pool.map(_oracle_unit, [(name, overrides, bi, hk) for (bi, hk) in units[:cores]])
        per_unit = sum(first) / len(first)
        want = max(cores, int(budget_s * cores / max(per_unit, 1e-6)))
        want = min(want, len(units))
        rest = units[cores:want]
        if rest:
            pool.map(_oracle_unit, [(name, overrides, bi, hk) for (bi, hk) in rest])
        done = cores + len(rest)
    wall = time.perf_counter() - t0
    t_full = wall * wl.units / done          # units are independent and equal in cost
    tok = wl.b * (wl.s + wl.n_decode)
    return {"value": tok / t_full, "unit": "tokens/s", "cores": cores, "kind": "oracle",
            "sample": f"{done} of {wl.units} (sample, KV head) units of {wl.name}, full P&D "
                      f"each, float64 numpy, one unit per process; {wall:.1f} s wall, "
                      f"scaled to all units"}


# ---------------------------------------------------------------------------
# GPU run
# ---------------------------------------------------------------------------
def gpu_bench(name, overrides, steps, warmup):
    import torch

    from paper_2412_05693_amd import batchmax as bmx
    from paper_2412_05693_amd import synth

    wl = synth.WORKLOADS[name].with_(**overrides)
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    q, k, v = synth.batch_inputs(wl, dev)
    o = torch.zeros_like(q)
    pd = bmx.PDAttention(b=wl.b, s=wl.s, kv_max=wl.kv_max, block=wl.block, max_gen=wl.n_decode,
                         n_heads=wl.n_heads, n_kv_heads=wl.n_kv_heads, head_dim=wl.head_dim,
                         dtype=wl.dtype, sm_scale=wl.sm_scale, device=dev)
    stream = torch.cuda.current_stream(dev)
    blocks = [(t0, min(wl.block, wl.s - t0)) for t0 in range(0, wl.s, wl.block)]

    def one_step(ev=None):
        pd.reset()
        for bi_, (t0, n) in enumerate(blocks):
            if ev is not None:
                ev["pf"][bi_][0].record(stream)
            pd.prefill_block(t0, n, q, k, v, o)
            if ev is not None:
                ev["pf"][bi_][1].record(stream)
                ev["ev"][bi_][0].record(stream)
            pd.evict_compact(t0 + n - 1)
            if ev is not None:
                ev["ev"][bi_][1].record(stream)
        if ev is not None:
            ev["dec"][0].record(stream)
        for t in range(wl.n_decode):
            pd.decode_step(wl.s + t, q, k, v, o, row=wl.s + t)
        if ev is not None:
            ev["dec"][1].record(stream)

    def new_events():
        mk = lambda: torch.cuda.Event(enable_timing=True)
        return {"pf": [(mk(), mk()) for _ in blocks], "ev": [(mk(), mk()) for _ in blocks],
                "dec": (mk(), mk())}

    for _ in range(warmup):
        one_step()
    torch.cuda.synchronize()
    evs = [new_events() for _ in range(steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(steps):
        one_step(evs[i])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0

    pf_ms = sum(a.elapsed_time(b) for e in evs for (a, b) in e["pf"]) / steps
    ev_ms = sum(a.elapsed_time(b) for e in evs for (a, b) in e["ev"]) / steps
    dec_ms = sum(e["dec"][0].elapsed_time(e["dec"][1]) for e in evs) / steps
    ms_step = wall * 1e3 / steps

    G = wl.group
    es = 4 if wl.dtype == "f32" else 2
    flops = bmx.prefill_flops(b=wl.b, n_kv_heads=wl.n_kv_heads, group=G, head_dim=wl.head_dim,
                              s=wl.s, kv_max=wl.kv_max, block=wl.block)
    dbytes = bmx.decode_bytes_per_step(b=wl.b, n_kv_heads=wl.n_kv_heads, group=G,
                                       head_dim=wl.head_dim, kv_max=wl.kv_max, elem_bytes=es)
    peak_f = PEAK_F32_MFMA if wl.dtype == "f32" else PEAK_BF16_MFMA
    prefill_tflops = flops / (pf_ms * 1e-3) / 1e12
    decode_gbs = dbytes * wl.n_decode / (dec_ms * 1e-3) / 1e9 if wl.n_decode else 0.0
    kernels = {
        "prefill_attention": {"bound": "mfma", "achieved": prefill_tflops,
                              "peak": peak_f / 1e12, "unit": "TFLOP/s",
                              "frac": prefill_tflops / (peak_f / 1e12),
                              "ms_per_step": pf_ms, "launches_per_step": len(blocks),
                              "algorithmic_per_launch": flops / len(blocks)},
        "evict_compact": {"ms_per_step": ev_ms, "launches_per_step": len(blocks)},
        "decode_step": {"bound": "hbm", "achieved": decode_gbs, "peak": PEAK_HBM / 1e9,
                        "unit": "GB/s", "frac": decode_gbs / (PEAK_HBM / 1e9),
                        "ms_per_step": dec_ms, "launches_per_step": wl.n_decode,
                        "algorithmic_per_launch": dbytes},
    }
    dom = "prefill_attention" if pf_ms >= dec_ms else "decode_step"
    kd = kernels[dom]
    traffic = measured_traffic(wl.name) if dom == "prefill_attention" else None
    roofline = {"bound": kd["bound"], "achieved": round(kd["achieved"], 3), "peak": kd["peak"],
                "unit": kd["unit"], "frac": round(kd["frac"], 5), "traffic": traffic,
                "kernel": dom}
    tokens = wl.b * (wl.s + wl.n_decode)
    return {
        "value": tokens / (ms_step * 1e-3),
        "ms_per_step": ms_step,
        "roofline": roofline,
        "kernels": kernels,
        "phases": {"prefill_tokens_per_s": wl.b * wl.s / ((pf_ms + ev_ms) * 1e-3),
                   "decode_tokens_per_s": (wl.b * wl.n_decode / (dec_ms * 1e-3)
                                           if wl.n_decode else None)},
        "workload": wl,
    }


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--config", default="c2", choices=["c1", "c2", "c3", "c4"])
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--hbm-probe", action="store_true",
                    help="only run the plain copy used to calibrate HBM byte counters")
    args = ap.parse_args()
    if args.hbm_probe:
        hbm_probe()
        return
    if args.gpus != 1:
        print(f"bench.py: this build measures one GPU only (--gpus {args.gpus} requested); "
              "the path shards with no communication and is not run across GPUs here.",
              file=sys.stderr)
        sys.exit(2)

    overrides = {}
    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(args.config, overrides, args.cpu_seconds)
    res = gpu_bench(args.config, overrides, args.steps, args.warmup)
    wl = res["workload"]
    line = {
        "metric": "P&D tokens/s (prefill+decode)",
        "value": round(res["value"], 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(res["ms_per_step"], 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": wl.dtype,
        "data": "synthetic",
        "config": {"workload": wl.name, "b": wl.b, "n_heads": wl.n_heads,
                   "n_kv_heads": wl.n_kv_heads, "head_dim": wl.head_dim, "s": wl.s,
                   "kv_max": wl.kv_max, "block": wl.block, "decode_steps": wl.n_decode,
                   "parallelism": "single GPU"},
        "roofline": res["roofline"],
        "cpu_baseline": cpu,
        "kernels": res["kernels"],
        "phases": res["phases"],
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
