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

    python bench.py [--config c5] [--steps K] [--warmup W] [--gpus 1] [--batch B]

Default workload: c5, the 32-layer Llama-3-8B-shaped attention stack (GQA
32/8, d 128, s 8192, bound 512, block 256, 256 decode steps) at the largest
batch whose bounded caches and block buffers fit the device's free memory; its
prompt inputs are evaluated per (layer, block) on the device by the
counter-based generator (bm_synth.h), whose time is measured and excluded from
the throughput.  c1-c4 are the single-layer workloads with resident inputs.
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


def counters_apply(wl) -> bool:
    """The committed counter records describe Batch-Max's prefill launches with
    score sums and no padding (the ranking rule does not change them, except
    TOVA's extra per-entry writes)."""
    return wl.accumulate and wl.pad_max == 0 and wl.rule in ("ave", "sum") and \
        wl.decode_bound == 0


def measured_traffic(workload: str, units: int = 0):
    """HBM bytes per prefill launch from a committed counter record
    (`traffic-record:` line under profiles/), or None when there is none for
    this workload or the kernel sources changed since it was taken.  A record
    given per unit is scaled by the launch's unit count."""
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
                    if "bytes_per_launch" in kv:
                        return int(kv["bytes_per_launch"])
                    if "bytes_per_unit" in kv and units:
                        return int(kv["bytes_per_unit"]) * units
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


def peak_probe():
    """What the box achieves against the published peaks: the device's compute
    units; the library's own probes (bm_probe.h) -- a streaming read of 4 GiB
    (plain and non-temporal loads) and a loop of independent bf16 MFMAs with no
    memory traffic; a large bf16 GEMM through the vendor BLAS and a plain
    device copy.  Context for the roofline fractions, not a target."""
    import torch

    from paper_2412_05693_amd import batchmax as bmx

    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    props = torch.cuda.get_device_properties(dev)
    cus = props.multi_processor_count
    out = {"device": props.name, "compute_units": cus, "memory_bytes": props.total_memory}
    stream = torch.cuda.current_stream(dev)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)

    def timed(fn, reps):
        fn()
        torch.cuda.synchronize()
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps * 1e-3     # seconds per call

    nbytes = 4 << 30
    buf = torch.ones(nbytes, dtype=torch.uint8, device=dev)
    sink = torch.empty(cus * 16, dtype=torch.int32, device=dev)
    # one workgroup per compute unit sweeping the buffer together, and 16 per
    # compute unit (more than can be resident at once)
    for per_cu in (1, 16):
        for nt in (False, True):
            t = timed(lambda: bmx.bm_probe_stream_read(buf.data_ptr(), nbytes, sink.data_ptr(),
                                                       cus * per_cu, nt, stream.cuda_stream), 10)
            key = f"stream_read{'_nt' if nt else ''}_{per_cu}wg_per_cu_gb_per_s"
            out[key] = nbytes / t / 1e9
    del buf
    for waves_per_cu in (8, 16):
        blocks_m, iters = cus * waves_per_cu // 4, 20000
        fsink = torch.empty(blocks_m * 4, dtype=torch.float32, device=dev)
        t = timed(lambda: bmx.bm_probe_mfma(iters, fsink.data_ptr(), blocks_m, stream.cuda_stream), 5)
        flops = blocks_m * 4 * iters * 4 * 32768
        out[f"mfma_loop_tflops_{waves_per_cu}_waves_per_cu"] = flops / t / 1e12
    n = 8192
    a = torch.randn(n, n, device=dev, dtype=torch.bfloat16)
    b = torch.randn(n, n, device=dev, dtype=torch.bfloat16)
    c = torch.empty(n, n, device=dev, dtype=torch.bfloat16)
    t = timed(lambda: torch.matmul(a, b, out=c), 20)
    out["bf16_gemm_tflops"] = 2 * n ** 3 / t / 1e12
    x = torch.ones(HBM_PROBE_BYTES, dtype=torch.uint8, device=dev)
    y = torch.empty_like(x)
    t = timed(lambda: y.copy_(x), 20)
    out["copy_gb_per_s"] = 2 * HBM_PROBE_BYTES / t / 1e9     # read + write
    for k in list(out):
        if k.endswith("_tflops") or "tflops_" in k:
            out[k + "_frac_of_peak"] = out[k] / (PEAK_BF16_MFMA / 1e12)
        elif k.endswith("_gb_per_s"):
            out[k + "_frac_of_peak"] = out[k] / (PEAK_HBM / 1e9)
    print(json.dumps({"peak_probe": out}), flush=True)


# ---------------------------------------------------------------------------
# CPU baseline: the oracle as it stands, one unit per worker process
# ---------------------------------------------------------------------------
def _oracle_unit(args):
    name, overrides, layer, bi, hk = args
    from threadpoolctl import threadpool_limits

    from oracle import pd as opd
    from paper_2412_05693_amd import synth

    wl = synth.WORKLOADS[name].with_(**overrides)
    if wl.n_layers > 1:
        q, k, v = synth.stack_unit_inputs(wl, layer, bi, hk)
    else:
        q, k, v = synth.unit_inputs(wl, layer, bi, hk)
    with threadpool_limits(1):     # one unit per process, one BLAS thread each
        t = time.perf_counter()
        opd.run_unit(q, k, v, s=wl.s, kv_max=wl.kv_max, block=wl.block, n_decode=wl.n_decode,
                     sm_scale=wl.sm_scale, p_dec=wl.decode_p, rule=wl.rule,
                     kv_dec=wl.decode_bound or None, pad=int(synth.sample_pads(wl)[bi]))
        return time.perf_counter() - t


def cpu_baseline(name, overrides, budget_s, method="bm"):
    """Time the oracle on a sample of units (one per process).  Returns the
    measurement; ``cpu_baseline_line`` scales it to the workload that ran."""
    from paper_2412_05693_amd import synth

    wl = method_workload(synth.WORKLOADS[name].with_(**overrides), method)
    overrides = dict(overrides, kv_max=wl.kv_max, rule=wl.rule, decode_bound=wl.decode_bound,
                     decode_p=wl.decode_p, accumulate=wl.accumulate)
    if wl.b == 0:                     # the stack's batch is planned on the GPU later;
        wl = wl.with_(b=64)           # a unit's oracle cost does not depend on b
    cores = len(os.sched_getaffinity(0))
    cores = max(1, min(cores, 16))
    for var in ("OMP_NUM_THREADS", "OPENBLAS_NUM_THREADS", "MKL_NUM_THREADS"):
        os.environ[var] = "1"
    ctx = mp.get_context("fork")     # forked before any GPU initialisation
    units = synth.checked_units(wl, min(wl.units, 100000), seed=7)
    if wl.n_layers > 1:               # spread the sample over the layers too
        units = [((i * 7919) % wl.n_layers, bi, hk) for i, (bi, hk) in enumerate(units)]
    else:
        units = [(0, bi, hk) for (bi, hk) in units]
    ov = dict(overrides, b=wl.b)
    t0 = time.perf_counter()
    with ctx.Pool(cores) as pool:
        # first wave sizes the sample: keep to about budget_s of wall time
        first = pool.map(_oracle_unit, [(name, ov) + u for u in units[:cores]])
        per_unit = sum(first) / len(first)
        want = max(cores, int(budget_s * cores / max(per_unit, 1e-6)))
        want = min(want, len(units))
        rest = units[cores:want]
        more = pool.map(_oracle_unit, [(name, ov) + u for u in rest]) if rest else []
    done = cores + len(rest)
    unit_s = sum(first) + sum(more)
    return {"per_unit_s": unit_s / done, "cores": cores, "done": done, "unit_s": unit_s,
            "wall": time.perf_counter() - t0, "n_layers": wl.n_layers}


def cpu_baseline_line(m, wl):
    """The oracle's throughput on the workload that ran: units are independent
    and equal in cost, so its time is the sampled units' mean oracle time times
    all units, spread over the same number of processes."""
    total_units = wl.units * wl.n_layers
    t_full = m["per_unit_s"] * total_units / m["cores"]
    from paper_2412_05693_amd import synth

    tok = wl.b * (wl.s + wl.n_decode) - int(synth.sample_pads(wl).sum())
    what = "(layer, sample, KV head)" if wl.n_layers > 1 else "(sample, KV head)"
    return {"value": tok / t_full, "unit": "tokens/s", "cores": m["cores"], "kind": "oracle",
            "cpu": cpu_model(),
            "sample": f"{m['done']} {what} units of {wl.name}, full P&D each, float64 numpy, "
                      f"one unit per process and one BLAS thread; {m['unit_s']:.1f} s of oracle "
                      f"time in {m['wall']:.1f} s wall, scaled (extrapolated: units are "
                      f"independent and equal in cost) to all {total_units} units of "
                      f"b={wl.b} over {m['cores']} processes"}


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


# ---------------------------------------------------------------------------
# GPU run
# ---------------------------------------------------------------------------
METHODS = {
    # Batch-Max: bounded cache in prefill and decode (Algorithm 1, Sec. 3.2 rule)
    "bm": {},
    # extreme decoding-only eviction (Algorithm 3): full prompt cache, no score
    # sums, then keep only the most recent pair at every decode step
    "ed": {"rule": "recent", "decode_bound": 2, "decode_p": 1, "accumulate": False},
    # full KV cache: nothing is ever removed, no score sums
    "fkv": {"accumulate": False},
}


def method_workload(wl, method):
    """The workload as the named method runs it (ED and FKV keep the whole
    prompt in the cache; FKV also every generated token)."""
    if method == "ed":
        return wl.with_(kv_max=max(wl.s, 2), **METHODS["ed"])
    if method == "fkv":
        return wl.with_(kv_max=wl.s + wl.n_decode, **METHODS["fkv"])
    return wl


def apply_method(pd, wl):
    pd.set_decode_removal(wl.decode_p)
    pd.set_rank_rule(wl.rule)
    if wl.decode_bound:
        pd.set_decode_bound(wl.decode_bound)
    pd.set_score_accumulation(wl.accumulate)


def decode_bytes(bmx, wl, b):
    """Algorithmic HBM bytes of all decode launches of one layer: each step at
    the cache length its attention reads (the removal launches of the p > 0
    schedule run inside the timed decode phase but add no bytes here)."""
    es = 4 if wl.dtype == "f32" else 2
    lens = bmx.decode_cache_lengths(s=wl.s, kv_max=wl.kv_max, n_decode=wl.n_decode,
                                    p=wl.decode_p, bound=wl.decode_bound or None)
    total = 0
    for n in lens:
        if n + 1 > bmx.MAX_DECODE_LEN:       # outputs-only split path (no score traffic)
            total += bmx.decode_bytes_outputs_only(b=b, n_kv_heads=wl.n_kv_heads,
                                                   group=wl.group, head_dim=wl.head_dim, n=n,
                                                   elem_bytes=es)
        else:
            total += bmx.decode_bytes_per_step(b=b, n_kv_heads=wl.n_kv_heads, group=wl.group,
                                               head_dim=wl.head_dim, kv_max=n, elem_bytes=es)
    return total


def cut_kernel_entry(ms, launches, fused_cut):
    """Timing of the launches that follow each block's attention kernel: the
    fused fold/select/compaction kernel, or the score fold plus the separate
    select and compaction kernels."""
    return {"kernel": "fold_cut" if fused_cut else "score_reduce+select+compact",
            "ms_per_step": ms, "launches_per_step": launches}


def gpu_bench(name, overrides, steps, warmup, method="bm", graph=False, fused_cut=True):
    import torch

    from paper_2412_05693_amd import batchmax as bmx
    from paper_2412_05693_amd import synth

    wl = method_workload(synth.WORKLOADS[name].with_(**overrides), method)
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    q, k, v = synth.batch_inputs(wl, dev)
    o = torch.zeros_like(q)
    pd = bmx.PDAttention(b=wl.b, s=wl.s, kv_max=wl.kv_max, block=wl.block, max_gen=wl.n_decode,
                         n_heads=wl.n_heads, n_kv_heads=wl.n_kv_heads, head_dim=wl.head_dim,
                         dtype=wl.dtype, sm_scale=wl.sm_scale, device=dev)
    apply_method(pd, wl)
    pads = synth.sample_pads(wl)
    if wl.pad_max > 0:
        pd.set_left_padding(torch.from_numpy(pads).to(dev))
    stream = torch.cuda.current_stream(dev)
    blocks = [(t0, min(wl.block, wl.s - t0)) for t0 in range(0, wl.s, wl.block)]
    mk = lambda: torch.cuda.Event(enable_timing=True)

    def one_step(ev=None):
        # per block: [start] attention [split] fold/cut [end]; the split event
        # is recorded by the library between its launches
        pd.reset()
        for bi_, (t0, n) in enumerate(blocks):
            if ev is not None:
                pd.set_split_event(ev["split"][bi_])
                ev["start"][bi_].record(stream)
            if fused_cut:
                pd.prefill_block_cut(t0, n, q, k, v, o)
            else:
                pd.prefill_block(t0, n, q, k, v, o)
                pd.evict_compact(t0 + n - 1)
            if ev is not None:
                ev["end"][bi_].record(stream)
        pd.set_split_event(None)
        if ev is not None:
            ev["dec"][0].record(stream)
        run_decode_loop()
        if ev is not None:
            ev["dec"][1].record(stream)

    def new_events():
        return {"start": [mk() for _ in blocks], "split": [mk() for _ in blocks],
                "end": [mk() for _ in blocks], "dec": (mk(), mk())}

    def run_decode_loop():
        for t in range(wl.n_decode):
            pd.decode_step(wl.s + t, q, k, v, o, row=wl.s + t)

    for _ in range(warmup):
        one_step()
    torch.cuda.synchronize()
    if graph and wl.n_decode:
        # the decode loop as one HIP graph, recorded where the decode starts
        pd.reset()
        pd.run_prefill(q, k, v, o, fused_cut=fused_cut)
        dec_graph = pd.capture_decode(q, k, v, o)
        torch.cuda.synchronize()
        run_decode_loop = dec_graph.replay
    evs = [new_events() for _ in range(steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(steps):
        one_step(evs[i])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0

    nb = len(blocks)
    pf_ms = sum(e["start"][i].elapsed_time(e["split"][i]) for e in evs for i in range(nb)) / steps
    ev_ms = sum(e["split"][i].elapsed_time(e["end"][i]) for e in evs for i in range(nb)) / steps
    dec_ms = sum(e["dec"][0].elapsed_time(e["dec"][1]) for e in evs) / steps
    ms_step = wall * 1e3 / steps

    G = wl.group
    if wl.pad_max > 0:
        flops = bmx.prefill_flops_padded(pads=pads, n_kv_heads=wl.n_kv_heads, group=G,
                                         head_dim=wl.head_dim, s=wl.s, kv_max=wl.kv_max,
                                         block=wl.block)
    else:
        flops = bmx.prefill_flops(b=wl.b, n_kv_heads=wl.n_kv_heads, group=G,
                                  head_dim=wl.head_dim, s=wl.s, kv_max=wl.kv_max, block=wl.block)
    dbytes = decode_bytes(bmx, wl, wl.b)
    peak_f = PEAK_F32_MFMA if wl.dtype == "f32" else PEAK_BF16_MFMA
    prefill_tflops = flops / (pf_ms * 1e-3) / 1e12
    decode_gbs = dbytes / (dec_ms * 1e-3) / 1e9 if wl.n_decode else 0.0
    cut_bytes = cut_fixed_bytes(wl, wl.b) if fused_cut else None
    kernels = {
        "prefill_attention": {"bound": "mfma", "achieved": prefill_tflops,
                              "peak": peak_f / 1e12, "unit": "TFLOP/s",
                              "frac": prefill_tflops / (peak_f / 1e12),
                              "ms_per_step": pf_ms, "launches_per_step": nb,
                              "algorithmic_per_launch": flops / nb},
        "evict_compact": cut_kernel_entry(ev_ms, nb, fused_cut),
        "decode_step": {"bound": "hbm", "achieved": decode_gbs, "peak": PEAK_HBM / 1e9,
                        "unit": "GB/s", "frac": decode_gbs / (PEAK_HBM / 1e9),
                        "ms_per_step": dec_ms, "launches_per_step": wl.n_decode,
                        "algorithmic_per_launch": dbytes / max(wl.n_decode, 1)},
    }
    if cut_bytes is not None:
        kernels["evict_compact"].update(cut_roofline(cut_bytes, ev_ms))
    dom = "prefill_attention" if pf_ms >= dec_ms else "decode_step"
    kd = kernels[dom]
    traffic = (measured_traffic(wl.name)
               if dom == "prefill_attention" and counters_apply(wl) else None)
    roofline = {"bound": kd["bound"], "achieved": round(kd["achieved"], 3), "peak": kd["peak"],
                "unit": kd["unit"], "frac": round(kd["frac"], 5), "traffic": traffic,
                "kernel": dom}
    prompt_tokens = int(wl.b * wl.s - pads.sum())        # real tokens only (Sec. 3 padding)
    tokens = prompt_tokens + wl.b * wl.n_decode
    return {
        "value": tokens / (ms_step * 1e-3),
        "ms_per_step": ms_step,
        "steps": steps,
        "warmup": warmup,
        "roofline": roofline,
        "kernels": kernels,
        "phases": {"prefill_tokens_per_s": prompt_tokens / ((pf_ms + ev_ms) * 1e-3),
                   "decode_tokens_per_s": (wl.b * wl.n_decode / (dec_ms * 1e-3)
                                           if wl.n_decode else None)},
        "workload": wl,
    }


FUSED_CUT_MAX_ENTRIES = 4096   # bm_prefill_block_cut's one-workgroup cut (include/batchmax.h)


def cut_fixed_bytes(wl, b) -> int:
    """HBM bytes of one prefill step's cut launches that do not depend on the
    data.  Up to 4096 live entries one fold/cut kernel per block reads every
    live slot's partial column sums (one row per attention workgroup that saw
    the slot, and only when scores accumulate), reads and writes its score,
    reads its position, and under TOVA its last-query weight.  Above 4096 the
    call folds with the score-reduce kernel (cached scores read, every score
    written, the partials) and, if the block overflows the bound, cuts with
    the select kernel (scores and positions read).  The moved K/V rows come on
    top (their number depends on which entries the rule removes)."""
    from paper_2412_05693_amd import batchmax as bmx

    ppw = bmx.bm_prefill_positions_per_workgroup(bmx.make_dims(
        b=1, s=wl.s, kv_max=wl.kv_max, block=wl.block, max_gen=wl.n_decode,
        n_heads=wl.n_heads, n_kv_heads=wl.n_kv_heads, head_dim=wl.head_dim, dtype=wl.dtype))
    total = 0
    length = 0
    for t0 in range(0, wl.s, wl.block):
        n = min(wl.block, wl.s - t0)
        npt = -(-n // ppw)
        part = length * npt + sum(npt - r // ppw for r in range(n)) if wl.accumulate else 0
        live = length + n
        if live <= FUSED_CUT_MAX_ENTRIES:
            total += 4 * part + 12 * live + (4 * live if wl.rule == "tova" else 0)
        else:
            total += 4 * part + 4 * length + 4 * live + (8 * live if live > wl.kv_max else 0)
        length = min(wl.kv_max, live)
    return total * b * wl.n_kv_heads


def cut_roofline(nbytes, ms):
    gbs = nbytes / (ms * 1e-3) / 1e9 if ms > 0 else 0.0
    return {"bound": "hbm", "achieved": gbs, "peak": PEAK_HBM / 1e9, "unit": "GB/s",
            "frac": gbs / (PEAK_HBM / 1e9), "algorithmic_bytes_per_step": nbytes,
            "algorithmic_basis": "partial sums (when scores accumulate), scores and positions only (moved rows excluded)"}


STACK_RESERVE = 3 << 30      # device bytes left to the runtime when planning the batch
STACK_TIMED_BUDGET_S = 90.0  # wall seconds of timed layer-stack passes (default)


def profiler_attached() -> bool:
    """rocprofv3 exports ROCPROF_* variables to the program it profiles."""
    return any(k.startswith("ROCPROF_") for k in os.environ)


def stack_warmup(requested: int) -> int:
    """Untimed layer-stack passes actually run: at most one (a pass is tens of
    seconds and the first one already warms every kernel and the allocator)."""
    return min(max(requested, 0), 1)


def more_stack_passes(done: int, requested: int, elapsed_s: float, last_pass_s: float,
                      budget_s: float) -> bool:
    """Time another layer-stack pass?  Always at least one; never more than
    requested; otherwise only while the next pass (taken to last as long as the
    previous one) still ends inside the wall budget."""
    if done < 1:
        return True
    if done >= requested:
        return False
    return elapsed_s + last_pass_s <= budget_s


def gpu_bench_stack(name, overrides, steps, warmup, batch=None, method="bm", fused_cut=True,
                    budget_s=STACK_TIMED_BUDGET_S):
    """The layer stack at the largest batch that fits: per (layer, block) the
    device generator writes the block's Q/K/V, then prefill and the cut; then
    the decode steps, layer by layer.  Generator time is measured and left out
    of the throughput (the inputs of a resident workload are not generated).
    Timed passes stop at ``steps`` or when the next one would end past
    ``budget_s`` seconds of timed wall time, whichever comes first."""
    import torch

    from paper_2412_05693_amd import batchmax as bmx
    from paper_2412_05693_amd import synth

    wl = method_workload(synth.WORKLOADS[name].with_(**overrides), method)
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    shape = dict(n_layers=wl.n_layers, s=wl.s, kv_max=wl.kv_max, block=wl.block,
                 max_gen=wl.n_decode, n_heads=wl.n_heads, n_kv_heads=wl.n_kv_heads,
                 head_dim=wl.head_dim, dtype=wl.dtype)
    free, total = torch.cuda.mem_get_info(dev)
    budget = free - STACK_RESERVE
    b_plan = bmx.plan_stack_batch(budget, **shape)
    es = 4 if wl.dtype == "f32" else 2
    io_per_sample = (wl.block + 1) * (2 * wl.n_heads + 2 * wl.n_kv_heads) * wl.head_dim * es
    b_do = int(budget // (bmx.full_cache_bytes_per_sample(
        n_layers=wl.n_layers, s=wl.s, n_kv_heads=wl.n_kv_heads, head_dim=wl.head_dim,
        dtype=wl.dtype) + io_per_sample))
    b = batch if batch else b_plan
    wl = wl.with_(b=b)
    print(f"[bench] {wl.name}: device free {free / 1e9:.1f} GB of {total / 1e9:.1f} GB; "
          f"max batch {b_plan} (decoding-only compression: {b_do}); running b={b}", flush=True)
    stack = bmx.PDStack(n_layers=wl.n_layers, b=b, s=wl.s, kv_max=wl.kv_max, block=wl.block,
                        max_gen=wl.n_decode, n_heads=wl.n_heads, n_kv_heads=wl.n_kv_heads,
                        head_dim=wl.head_dim, dtype=wl.dtype, sm_scale=wl.sm_scale, device=dev)
    for pd_ in stack.layers:
        apply_method(pd_, wl)
    tdt = torch.float32 if wl.dtype == "f32" else torch.bfloat16
    H, Hk, d, B = wl.n_heads, wl.n_kv_heads, wl.head_dim, wl.block
    q = torch.empty((b, H, B, d), dtype=tdt, device=dev)
    k = torch.empty((b, Hk, B, d), dtype=tdt, device=dev)
    v = torch.empty_like(k)
    o = torch.empty_like(q)
    qd = torch.empty((b, H, 1, d), dtype=tdt, device=dev)
    kd = torch.empty((b, Hk, 1, d), dtype=tdt, device=dev)
    vd = torch.empty_like(kd)
    od = torch.empty_like(qd)
    params = [bmx.synth_params(b=b, n_heads=H, n_kv_heads=Hk, head_dim=d, dtype=wl.dtype,
                               seed=wl.seed, layer=layer, s=wl.s, hh_frac=wl.hh_frac,
                               hh_scale=wl.hh_scale, n_sinks=wl.n_sinks,
                               sink_scale=wl.sink_scale, heavy=wl.hh_mode != "none")
              for layer in range(wl.n_layers)]
    stream = torch.cuda.current_stream(dev)
    blocks = [(t0, min(B, wl.s - t0)) for t0 in range(0, wl.s, B)]
    L = wl.n_layers
    mk = lambda: torch.cuda.Event(enable_timing=True)

    def one_step(timed):
        ev = {"gen": [], "pf": [], "cut": [], "dec": []} if timed else None

        def rec(kind, fn):
            if ev is None:
                fn()
                return
            a, z = mk(), mk()
            a.record(stream)
            fn()
            z.record(stream)
            ev[kind].append((a, z))

        stack.reset()
        for (t0, n) in blocks:
            for layer in range(L):
                pd = stack.layers[layer]
                rec("gen", lambda: bmx.synth_qkv(params[layer], t0, q, k, v))
                if ev is None:
                    if fused_cut:
                        pd.prefill_block_cut(t0, n, q, k, v, o, row=0)
                    else:
                        pd.prefill_block(t0, n, q, k, v, o, row=0)
                        pd.evict_compact(t0 + n - 1)
                    continue
                # [start] attention [split] fold/cut [end]
                a, sp, z = mk(), mk(), mk()
                pd.set_split_event(sp)
                a.record(stream)
                if fused_cut:
                    pd.prefill_block_cut(t0, n, q, k, v, o, row=0)
                else:
                    pd.prefill_block(t0, n, q, k, v, o, row=0)
                    pd.evict_compact(t0 + n - 1)
                z.record(stream)
                pd.set_split_event(None)
                ev["pf"].append((a, sp))
                ev["cut"].append((sp, z))
        for t in range(wl.n_decode):
            p = wl.s + t
            for layer in range(L):
                pd = stack.layers[layer]
                rec("gen", lambda: bmx.synth_qkv(params[layer], p, qd, kd, vd))
                rec("dec", lambda: pd.decode_step(p, qd, kd, vd, od, row=0))
        return ev

    warm = stack_warmup(warmup)
    for i in range(warm):
        t0w = time.perf_counter()
        one_step(False)
        torch.cuda.synchronize()
        print(f"[bench] warm-up pass {i + 1}/{warm}: {time.perf_counter() - t0w:.1f} s", flush=True)
    evs, walls = [], []
    while more_stack_passes(len(walls), steps, sum(walls), walls[-1] if walls else 0.0, budget_s):
        torch.cuda.synchronize()
        t0w = time.perf_counter()
        evs.append(one_step(True))
        torch.cuda.synchronize()
        walls.append(time.perf_counter() - t0w)
        print(f"[bench] timed pass {len(walls)}: {walls[-1]:.1f} s", flush=True)
    done = len(walls)

    def ms(kind):
        return sum(a.elapsed_time(z) for e in evs for (a, z) in e[kind]) / done

    gen_ms, pf_ms, ev_ms, dec_ms = ms("gen"), ms("pf"), ms("cut"), ms("dec")
    wall_ms = sum(walls) * 1e3 / done
    ms_step = wall_ms - gen_ms
    G = wl.group
    flops = L * bmx.prefill_flops(b=b, n_kv_heads=Hk, group=G, head_dim=d, s=wl.s,
                                  kv_max=wl.kv_max, block=B)
    dbytes = L * decode_bytes(bmx, wl, b)
    peak_f = PEAK_F32_MFMA if wl.dtype == "f32" else PEAK_BF16_MFMA
    prefill_tflops = flops / (pf_ms * 1e-3) / 1e12
    decode_gbs = dbytes / (dec_ms * 1e-3) / 1e9
    n_pf = L * len(blocks)
    kernels = {
        "prefill_attention": {"bound": "mfma", "achieved": prefill_tflops,
                              "peak": peak_f / 1e12, "unit": "TFLOP/s",
                              "frac": prefill_tflops / (peak_f / 1e12),
                              "ms_per_step": pf_ms, "launches_per_step": n_pf,
                              "algorithmic_per_launch": flops / n_pf},
        "evict_compact": cut_kernel_entry(ev_ms, n_pf, fused_cut),
        "decode_step": {"bound": "hbm", "achieved": decode_gbs, "peak": PEAK_HBM / 1e9,
                        "unit": "GB/s", "frac": decode_gbs / (PEAK_HBM / 1e9),
                        "ms_per_step": dec_ms, "launches_per_step": L * wl.n_decode,
                        "algorithmic_per_launch": dbytes / (L * max(wl.n_decode, 1))},
    }
    if fused_cut:
        kernels["evict_compact"].update(cut_roofline(L * cut_fixed_bytes(wl, b), ev_ms))
    dom = "prefill_attention" if pf_ms >= dec_ms else "decode_step"
    kd_ = kernels[dom]
    traffic = (measured_traffic(wl.name, b * Hk)
               if dom == "prefill_attention" and counters_apply(wl) else None)
    roofline = {"bound": kd_["bound"], "achieved": round(kd_["achieved"], 3), "peak": kd_["peak"],
                "unit": kd_["unit"], "frac": round(kd_["frac"], 5), "traffic": traffic,
                "kernel": dom}
    if traffic is not None:
        roofline["traffic_basis"] = ("FETCH_SIZE/WRITE_SIZE per unit of the same launches "
                                     "measured on c2, scaled to this launch's units")
    tokens = b * (wl.s + wl.n_decode)
    return {
        "value": tokens / (ms_step * 1e-3),
        "ms_per_step": ms_step,
        "steps": done,
        "warmup": warm,
        "roofline": roofline,
        "kernels": kernels,
        "phases": {"prefill_tokens_per_s": b * wl.s / ((pf_ms + ev_ms) * 1e-3),
                   "decode_tokens_per_s": b * wl.n_decode / (dec_ms * 1e-3),
                   "generated_tokens_per_s": b * wl.n_decode / (ms_step * 1e-3),
                   "input_generation_ms_per_step": gen_ms,
                   "wall_ms_per_step_with_generation": wall_ms,
                   "timed_wall_s": sum(walls), "timed_wall_budget_s": budget_s},
        "stack": {"n_layers": L, "max_batch": b_plan, "max_batch_decoding_only": b_do,
                  "device_free_bytes": free, "arena_bytes": stack.arena_bytes},
        "workload": wl,
        "close": stack.close,
    }


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None,
                    help="timed steps (default 10; for the layer stack at most this many, "
                         "within --time-budget)")
    ap.add_argument("--warmup", type=int, default=None,
                    help="untimed steps first (default 2; the layer stack runs at most 1)")
    ap.add_argument("--time-budget", type=float, default=STACK_TIMED_BUDGET_S,
                    help="layer stack: wall seconds of timed passes; no pass starts that "
                         "would end past it (at least one always runs)")
    ap.add_argument("--config", default="c5", choices=["c1", "c2", "c3", "c4", "c5"],
                    help="workload (default c5: the 32-layer stack at the largest batch that "
                         "fits, the configuration the metric is quoted at)")
    ap.add_argument("--batch", type=int, default=0,
                    help="layer stack only: run this batch instead of the largest that fits")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--decode-p", type=int, default=0,
                    help="decode removal schedule: 0 = one removal per step (default); p > 0 = "
                         "Algorithm 1's decoding loop, p removals when a step starts full")
    ap.add_argument("--method", default="bm", choices=sorted(METHODS),
                    help="bm: Batch-Max (default); ed: Algorithm 3's extreme decoding-only "
                         "eviction; fkv: full KV cache (the comparators of Sec. 4, run with the "
                         "same kernels at the largest batch their caches allow)")
    ap.add_argument("--rule", default="ave", choices=["ave", "sum", "tova"],
                    help="ranking key of Batch-Max's cuts: ave (Sec. 3.2, default), sum (the "
                         "cumulative rule it corrects) or tova (the last query's weights)")
    ap.add_argument("--pad-max", type=int, default=0,
                    help="single-layer workloads: left-pad sample j by pad_j in [0, N] tokens "
                         "(per-sample prompt lengths s - pad_j, Sec. 3); value counts real tokens")
    ap.add_argument("--separate-cut", action="store_true",
                    help="cut each block with the score fold, select and compaction kernels "
                         "(three launches) instead of the fused fold/cut kernel (the default)")
    ap.add_argument("--graph", action="store_true",
                    help="single-layer workloads: replay the decode loop as one HIP graph")
    ap.add_argument("--peak-probe", action="store_true",
                    help="only report what this box achieves: bf16 GEMM TFLOP/s, copy GB/s")
    ap.add_argument("--hbm-probe", action="store_true",
                    help="only run the plain copy used to calibrate HBM byte counters")
    args = ap.parse_args()
    stack = args.config == "c5"
    if args.steps is None:
        args.steps = 1 if stack else 10
    if args.warmup is None:
        args.warmup = 1 if stack else 2
    if args.hbm_probe:
        hbm_probe()
        return
    if args.peak_probe:
        peak_probe()
        return
    if args.gpus != 1:
        print(f"bench.py: measures one GPU only (--gpus {args.gpus} requested); "
              "the path shards with no communication and is not run across GPUs here.",
              file=sys.stderr)
        sys.exit(2)
    if stack and not args.batch and profiler_attached():
        # Three profiler runs of the full-batch stack ended in a host-side crash
        # inside the profiler's launch interception; profile a given --batch.
        print("bench.py: the layer stack at the largest batch that fits is not run under a "
              "profiler; pass --batch N", file=sys.stderr)
        sys.exit(2)

    overrides = {"decode_p": args.decode_p} if args.decode_p else {}
    if args.rule != "ave":
        if args.method != "bm":
            print("bench.py: --rule applies to Batch-Max (--method bm)", file=sys.stderr)
            sys.exit(2)
        overrides["rule"] = args.rule
    if args.pad_max:
        if args.config == "c5":
            print("bench.py: --pad-max applies to the single-layer workloads", file=sys.stderr)
            sys.exit(2)
        overrides["pad_max"] = args.pad_max
    fused_cut = not args.separate_cut
    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(args.config, overrides, args.cpu_seconds, args.method)
    if stack:
        res = gpu_bench_stack(args.config, overrides, args.steps, args.warmup, args.batch,
                              method=args.method, fused_cut=fused_cut,
                              budget_s=args.time_budget)
    else:
        res = gpu_bench(args.config, overrides, args.steps, args.warmup, method=args.method,
                        graph=args.graph, fused_cut=fused_cut)
    wl = res["workload"]
    line = {
        "metric": ("P&D tokens/s (prefill+decode) at max batch; prefill MFMA %, decode HBM GB/s"
                   if "stack" in res else "P&D tokens/s (prefill+decode)"),
        "value": round(res["value"], 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": res["steps"],
        "warmup": res["warmup"],
        "steps_requested": args.steps,
        "warmup_requested": args.warmup,
        "ms_per_step": round(res["ms_per_step"], 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": wl.dtype,
        "data": "synthetic",
        "config": {"workload": wl.name, "b": wl.b, "n_heads": wl.n_heads,
                   "n_kv_heads": wl.n_kv_heads, "head_dim": wl.head_dim, "s": wl.s,
                   "kv_max": wl.kv_max, "block": wl.block, "decode_steps": wl.n_decode,
                   "decode_removal": (f"{wl.decode_p} at once when full" if wl.decode_p
                                      else "one per step"),
                   "left_pad_max": wl.pad_max,
                   "rank_rule": wl.rule,
                   "decode_graph": bool(args.graph and not stack),
                   "fused_cut": fused_cut,
                   "method": {"bm": "Batch-Max (Algorithm 1)",
                              "ed": "extreme decoding-only (Algorithm 3)",
                              "fkv": "full KV cache"}[args.method],
                   "parallelism": "single GPU"},
        "roofline": res["roofline"],
        "cpu_baseline": cpu_baseline_line(cpu, wl) if cpu else None,
        "kernels": res["kernels"],
        "phases": res["phases"],
    }
    if "stack" in res:
        line["config"]["n_layers"] = res["stack"]["n_layers"]
        line["config"]["max_batch_decoding_only"] = res["stack"]["max_batch_decoding_only"]
        line["stack"] = res["stack"]
    print(json.dumps(line), flush=True)
    if "close" in res:
        res["close"]()


if __name__ == "__main__":
    main()
