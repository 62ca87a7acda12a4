"""Host logic of bench.py (no GPU): the comparators' workloads, the byte and
flop models behind the roofline figures, which counter records apply, the
CPU-baseline scaling, and the one-GPU guard."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_2412_05693_amd import batchmax as bmx  # noqa: E402
from paper_2412_05693_amd import synth  # noqa: E402


def test_method_workloads():
    c5 = synth.WORKLOADS["c5"]
    ed = bench.method_workload(c5, "ed")
    assert ed.kv_max == c5.s and ed.rule == "recent" and ed.decode_bound == 2
    assert ed.decode_p == 1 and not ed.accumulate
    fkv = bench.method_workload(c5, "fkv")
    assert fkv.kv_max == c5.s + c5.n_decode and not fkv.accumulate and fkv.rule == "ave"
    assert bench.method_workload(c5, "bm") == c5


def test_counter_records_apply_only_to_their_launches():
    c2 = synth.WORKLOADS["c2"]
    assert bench.counters_apply(c2)
    assert bench.counters_apply(c2.with_(rule="sum"))
    assert not bench.counters_apply(c2.with_(rule="tova"))
    assert not bench.counters_apply(c2.with_(pad_max=100))
    for m in ("ed", "fkv"):
        assert not bench.counters_apply(bench.method_workload(c2, m))


def test_decode_bytes_follow_the_schedule():
    c2 = synth.WORKLOADS["c2"]
    per = bmx.decode_bytes_per_step(b=c2.b, n_kv_heads=c2.n_kv_heads, group=c2.group,
                                    head_dim=c2.head_dim, kv_max=c2.kv_max, elem_bytes=2)
    assert bench.decode_bytes(bmx, c2, c2.b) == per * c2.n_decode
    # ED: every step reads one cached entry
    ed = bench.method_workload(c2, "ed")
    one = bmx.decode_bytes_per_step(b=c2.b, n_kv_heads=c2.n_kv_heads, group=c2.group,
                                    head_dim=c2.head_dim, kv_max=1, elem_bytes=2)
    assert bench.decode_bytes(bmx, ed, c2.b) == one * c2.n_decode
    # FKV past 4097 entries: the outputs-only byte model (no score traffic)
    fkv = bench.method_workload(c2, "fkv")
    lens = bmx.decode_cache_lengths(s=fkv.s, kv_max=fkv.kv_max, n_decode=fkv.n_decode)
    assert lens[0] == c2.s and lens[-1] == c2.s + c2.n_decode - 1
    want = sum(bmx.decode_bytes_outputs_only(b=c2.b, n_kv_heads=8, group=4, head_dim=128, n=n,
                                             elem_bytes=2) if n + 1 > bmx.MAX_DECODE_LEN
               else bmx.decode_bytes_per_step(b=c2.b, n_kv_heads=8, group=4, head_dim=128,
                                              kv_max=n, elem_bytes=2) for n in lens)
    assert bench.decode_bytes(bmx, fkv, c2.b) == want


def test_cpu_baseline_scaling():
    wl = synth.WORKLOADS["c2"]
    m = {"per_unit_s": 0.5, "cores": 8, "done": 16, "unit_s": 8.0, "wall": 1.2}
    line = bench.cpu_baseline_line(m, wl)
    t_full = 0.5 * wl.units / 8
    assert abs(line["value"] - wl.b * (wl.s + wl.n_decode) / t_full) < 1e-6
    assert line["kind"] == "oracle" and line["cores"] == 8 and line["cpu"]
    # padded workloads count real tokens only
    wp = wl.with_(pad_max=1000)
    lp = bench.cpu_baseline_line(m, wp)
    real = wp.b * (wp.s + wp.n_decode) - int(synth.sample_pads(wp).sum())
    assert abs(lp["value"] - real / t_full) < 1e-6


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2 and "one GPU" in r.stderr


def test_stack_pass_budget():
    # at most one untimed pass, whatever is requested
    assert bench.stack_warmup(5) == 1 and bench.stack_warmup(1) == 1 and bench.stack_warmup(0) == 0
    # the driver's request (--steps 20) with 35 s passes and a 90 s budget: 2 passes
    done, walls = 0, []
    while bench.more_stack_passes(done, 20, sum(walls), walls[-1] if walls else 0.0, 90.0):
        walls.append(35.0)
        done += 1
    assert done == 2 and sum(walls) <= 90.0
    # one pass always runs, even past the budget
    assert bench.more_stack_passes(0, 20, 0.0, 0.0, 1.0)
    assert not bench.more_stack_passes(1, 20, 500.0, 500.0, 1.0)
    # never more than requested
    assert not bench.more_stack_passes(3, 3, 1.0, 0.1, 1e9)
    assert bench.more_stack_passes(2, 3, 1.0, 0.1, 1e9)


def test_driver_command_fits_its_limit():
    """The driver's `--steps 20 --warmup 5` on the stack: one warm-up pass and
    the timed passes the budget allows, worst case (one timed pass of any
    length is still taken) the pass time twice plus the budget."""
    pass_s = 40.0                        # measured c5 pass with input generation: about 35 s
    warm = bench.stack_warmup(5)
    done, walls = 0, []
    while bench.more_stack_passes(done, 20, sum(walls), walls[-1] if walls else 0.0,
                                  bench.STACK_TIMED_BUDGET_S):
        walls.append(pass_s)
        done += 1
    gpu_s = warm * pass_s + sum(walls)
    assert gpu_s <= 300.0


def test_profiler_guard(monkeypatch):
    monkeypatch.delenv("ROCPROF_OUTPUT_PATH", raising=False)
    for k in list(os.environ):
        if k.startswith("ROCPROF_"):
            monkeypatch.delenv(k)
    assert not bench.profiler_attached()
    monkeypatch.setenv("ROCPROF_OUTPUT_PATH", "/tmp/x")
    assert bench.profiler_attached()


def test_full_batch_stack_refused_under_a_profiler():
    env = dict(os.environ, ROCPROF_OUTPUT_PATH="/tmp/none")
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--no-cpu-baseline"],
                       capture_output=True, text=True, timeout=120, env=env)
    assert r.returncode == 2 and "--batch" in r.stderr


def test_cut_fixed_bytes():
    """Fused fold/cut bytes per step: per block, each live slot's partial rows
    (one per attention workgroup that saw it) plus score read/write and
    position read, checked by hand on a two-block case."""
    wl = synth.WORKLOADS["c2"].with_(b=1, s=512, kv_max=256, block=256)
    d = bmx.make_dims(b=1, s=512, kv_max=256, block=256, max_gen=wl.n_decode, n_heads=32,
                      n_kv_heads=8, head_dim=128, dtype="bf16")
    ppw = bmx.bm_prefill_positions_per_workgroup(d)
    assert ppw == 128 // wl.group
    npt = 256 // ppw
    # block 0: no cache; block row r is seen by the workgroups pt >= r // ppw
    b0 = sum(npt - r // ppw for r in range(256))
    # block 1: 256 cached slots seen by every workgroup, then the block rows
    b1 = 256 * npt + b0
    want = (4 * b0 + 12 * 256) + (4 * b1 + 12 * 512)
    assert bench.cut_fixed_bytes(wl, 1) == want * wl.n_kv_heads


def test_cut_fixed_bytes_without_accumulation_tova_and_long_caches():
    """No partial sums when scores do not accumulate (the comparators); the
    last-query weight under TOVA; above 4096 live entries the score-reduce fold
    (cached scores read, every score written) with no position reads."""
    wl = synth.WORKLOADS["c2"].with_(b=1, s=512, kv_max=256, block=256)
    d = bmx.make_dims(b=1, s=512, kv_max=256, block=256, max_gen=wl.n_decode, n_heads=32,
                      n_kv_heads=8, head_dim=128, dtype="bf16")
    ppw = bmx.bm_prefill_positions_per_workgroup(d)
    npt = 256 // ppw
    b0 = sum(npt - r // ppw for r in range(256))
    b1 = 256 * npt + b0
    assert bench.cut_fixed_bytes(wl.with_(accumulate=False), 1) == (12 * 256 + 12 * 512) * 8
    want_tova = (4 * b0 + 16 * 256) + (4 * b1 + 16 * 512)
    assert bench.cut_fixed_bytes(wl.with_(rule="tova"), 1) == want_tova * 8
    # a full-cache prompt of 8192 tokens in blocks of 4096: the second block
    # holds 8192 live entries, past the fused cut's 4096
    big = synth.WORKLOADS["c2"].with_(b=1, s=8192, kv_max=8192, block=4096, accumulate=False)
    assert bench.cut_fixed_bytes(big, 1) == (12 * 4096 + (4 * 4096 + 4 * 8192)) * 8
