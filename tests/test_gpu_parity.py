"""GPU parity: the HIP path through the C ABI against the float64 oracle.

Sizes: every unit of the small float32 workload and of reduced bf16 shapes
(several tiles, ragged tails, every group size), seeded samples of units at the
full benchmark shapes, the sharp supplementary distribution, degenerate cases
(no eviction, bound larger than the prompt, one-token blocks), determinism and
sub-batch independence.
"""
import sys

import numpy as np
import pytest
import torch

from paper_2412_05693_amd import synth

pytestmark = pytest.mark.gpu


def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _run(wl, checked, **kw):
    _need_gpu()
    from pd_harness import run_parity

    _say(f"[parity] {wl.name} dtype={wl.dtype} b={wl.b} H={wl.n_heads}/{wl.n_kv_heads} "
         f"d={wl.head_dim} s={wl.s} kv={wl.kv_max} B={wl.block} D={wl.n_decode} "
         f"units={len(checked)} {kw}")
    st = run_parity(wl, checked, **kw)
    _say(f"[parity] -> {st.summary()}")
    assert not st.failures, "\n".join(st.failures)
    return st


C1 = synth.WORKLOADS["c1"]
C2 = synth.WORKLOADS["c2"]


def test_c1_all_units_fp32():
    st = _run(C1, synth.checked_units(C1, C1.units))
    assert st.cuts > 0


def test_c2_shape_reduced_batch_all_units():
    wl = C2.with_(b=2, s=1024, n_decode=24)
    st = _run(wl, synth.checked_units(wl, wl.units))
    assert st.cuts > 0


@pytest.mark.parametrize("case", [
    # ragged: prompt not a multiple of the block, bound not a multiple of 64,
    # partial workgroup tiles, group sizes 1, 2, 4, head dims 64 and 128
    dict(dtype="bf16", b=3, n_heads=8, n_kv_heads=4, head_dim=64, s=300, kv_max=100, block=48,
         n_decode=20),
    dict(dtype="bf16", b=2, n_heads=4, n_kv_heads=4, head_dim=128, s=333, kv_max=77, block=100,
         n_decode=9),
    dict(dtype="f32", b=2, n_heads=8, n_kv_heads=2, head_dim=128, s=200, kv_max=70, block=33,
         n_decode=7),
    dict(dtype="f32", b=1, n_heads=4, n_kv_heads=2, head_dim=64, s=129, kv_max=64, block=64,
         n_decode=5),
    # one-token blocks and a bound below the block
    dict(dtype="bf16", b=1, n_heads=4, n_kv_heads=1, head_dim=128, s=40, kv_max=8, block=1,
         n_decode=6),
    dict(dtype="bf16", b=2, n_heads=4, n_kv_heads=1, head_dim=128, s=260, kv_max=16, block=128,
         n_decode=6),
], ids=lambda c: f"{c['dtype']}-G{c['n_heads'] // c['n_kv_heads']}-d{c['head_dim']}-s{c['s']}-kv{c['kv_max']}-B{c['block']}")
def test_ragged_shapes_all_units(case):
    wl = C2.with_(name="ragged", hh_mode="scatter", n_sinks=4, **case)
    _run(wl, synth.checked_units(wl, wl.units))


@pytest.mark.parametrize("case", [
    # the smallest bound: every cut keeps one entry
    dict(dtype="bf16", b=2, n_heads=4, n_kv_heads=4, head_dim=64, s=37, kv_max=1, block=3,
         n_decode=5),
    dict(dtype="f32", b=1, n_heads=2, n_kv_heads=1, head_dim=128, s=20, kv_max=1, block=1,
         n_decode=3),
    # one sample, one KV head, a prompt shorter than one block
    dict(dtype="bf16", b=1, n_heads=4, n_kv_heads=1, head_dim=128, s=5, kv_max=3, block=64,
         n_decode=4),
], ids=lambda c: f"{c['dtype']}-s{c['s']}-kv{c['kv_max']}-B{c['block']}")
def test_degenerate_bounds(case):
    wl = C2.with_(name="degenerate", hh_mode="scatter", n_sinks=0, **case)
    st = _run(wl, synth.checked_units(wl, wl.units))
    assert st.cuts > 0


@pytest.mark.parametrize("case", [
    # the largest block the library takes (1024 tokens: 32 position tiles per
    # unit at G = 4), a ragged last block, both cut paths
    dict(name="maxblock", b=1, n_heads=4, n_kv_heads=1, s=2300, kv_max=1000, block=1024,
         n_decode=3, fused_cut=False),
    dict(name="maxblock", b=1, n_heads=4, n_kv_heads=1, s=2300, kv_max=1000, block=1024,
         n_decode=3, fused_cut=True),
    # the same at G = 1 in fp32 with d = 64 (128 positions per workgroup)
    dict(name="maxblock", dtype="f32", b=1, n_heads=2, n_kv_heads=2, head_dim=64, s=1500,
         kv_max=600, block=1024, n_decode=2, fused_cut=True),
    # decode steps over exactly 4097 entries, the most the fused decode kernel
    # attends to in one workgroup (4096 cached, full, plus the step's own pair)
    dict(name="decode4097", b=1, n_heads=4, n_kv_heads=1, s=4096, kv_max=4096, block=512,
         n_decode=3, fused_cut=True),
], ids=lambda c: f"{c['name']}-{c.get('dtype', 'bf16')}-B{c['block']}-kv{c['kv_max']}-"
                 f"{'fused' if c['fused_cut'] else 'separate'}")
def test_maximum_sizes(case):
    case = dict(case)
    fused = case.pop("fused_cut")
    wl = C2.with_(hh_mode="scatter", n_sinks=4, **case)
    st = _run(wl, synth.checked_units(wl, wl.units), fused_cut=fused)
    assert st.cuts > 0


def test_no_eviction_dense_fixed_point():
    # bound >= s + D: nothing is ever evicted, every output is dense causal attention
    wl = C2.with_(b=2, s=600, kv_max=700, block=256, n_decode=10)
    st = _run(wl, synth.checked_units(wl, wl.units))
    assert st.cuts == 0


def test_bound_larger_than_prompt_then_decode_cuts():
    # decode appends without eviction until the bound is reached, then cuts one per step
    wl = C2.with_(b=1, s=300, kv_max=310, block=128, n_decode=20)
    st = _run(wl, synth.checked_units(wl, wl.units))
    assert st.cuts == wl.units * (300 + 20 - 310)


@pytest.mark.parametrize("p", [1, 8, 512])
def test_alg1_decode_removal_c2_shape(p):
    # Algorithm 1's decoding loop taken literally: p removals whenever a step
    # starts with a full cache (p = kv_max empties it); the prompt leaves it full
    wl = C2.with_(b=2, s=1024, n_decode=24)
    st = _run(wl, synth.checked_units(wl, wl.units), decode_p=p)
    assert st.cuts == wl.units * (1024 // 256 - 512 // 256 + -(-24 // p))


def test_alg1_decode_removal_ragged_fp32_bound_above_prompt():
    # cache first fills during decode (step kv_max - s), then p = 4 at a time
    wl = C2.with_(name="ragged", hh_mode="scatter", n_sinks=4, dtype="f32", b=2, n_heads=8,
                  n_kv_heads=2, head_dim=64, s=300, kv_max=310, block=48, n_decode=20)
    st = _run(wl, synth.checked_units(wl, wl.units), decode_p=4)
    assert st.cuts == wl.units * 3


def test_sharp_distribution():
    wl = C2.with_(b=2, s=2048, n_decode=32)
    st = _run(wl, synth.checked_units(wl, wl.units), sharp=True)
    assert st.cuts > 0


def test_c2_full_shape_sampled_units():
    # 64 of the 512 units (units are independent; the kernels do not depend on
    # which unit they process)
    st = _run(C2, synth.checked_units(C2, 64))
    assert st.cuts > 0


def test_uniform_attention_closed_form():
    """All-zero keys: every softmax is uniform, so with one-hot values each
    output is the indicator of the entries the query sees divided by their
    count, and every prefill cut keeps exactly positions 0..bound-1."""
    _need_gpu()
    from pd_harness import make_pd

    wl = C2.with_(b=1, n_heads=4, n_kv_heads=1, head_dim=128, s=96, kv_max=32, block=32,
                  n_decode=0)
    dev = "cuda"
    T = wl.s
    q = torch.randn((1, 4, T, 128), device=dev).to(torch.bfloat16)
    k = torch.zeros((1, 1, T, 128), device=dev, dtype=torch.bfloat16)
    v = torch.zeros((1, 1, T, 128), device=dev, dtype=torch.bfloat16)
    v[0, 0, torch.arange(T), torch.arange(T)] = 1.0
    o = torch.zeros_like(q)
    pd = make_pd(wl, dev)
    for t0 in range(0, wl.s, wl.block):
        pd.prefill_block(t0, wl.block, q, k, v, o)
        torch.cuda.synchronize()
        got = o[0, :, t0:t0 + wl.block].float().cpu().numpy()
        live = list(range(min(t0, wl.kv_max)))
        for r in range(wl.block):
            vis = live + list(range(t0, t0 + r + 1))
            want = np.zeros(128)
            want[vis] = 1.0 / len(vis)
            assert np.max(np.abs(got[:, r] - want)) < 2e-3, (t0, r)
        pd.evict_compact(t0 + wl.block - 1)
        torch.cuda.synchronize()
        if t0 + wl.block > wl.kv_max:
            kept = sorted(pd.pos[0, 0, :pd.length].cpu().tolist())
            assert kept == list(range(wl.kv_max))


def test_determinism_and_subbatch_independence():
    """Two runs give bit-identical caches and outputs; a unit's results do not
    depend on the other units in the batch."""
    _need_gpu()
    from pd_harness import make_pd

    wl = C2.with_(b=4, s=768, n_decode=16)
    q, k, v = synth.batch_inputs(wl, "cuda")
    outs = []
    for rep in range(2):
        o = torch.zeros_like(q)
        pd = make_pd(wl)
        pd.run_prefill(q, k, v, o)
        pd.run_decode(q, k, v, o)
        torch.cuda.synchronize()
        outs.append((o.clone(), pd.k.clone(), pd.v.clone(), pd.score.clone(), pd.pos.clone()))
    for a, b in zip(outs[0], outs[1]):
        assert torch.equal(a, b)
    sub = wl.with_(b=2)
    o2 = torch.zeros_like(q[1:3])
    pd2 = make_pd(sub)
    q2, k2, v2 = q[1:3].contiguous(), k[1:3].contiguous(), v[1:3].contiguous()
    pd2.run_prefill(q2, k2, v2, o2)
    pd2.run_decode(q2, k2, v2, o2)
    torch.cuda.synchronize()
    assert torch.equal(o2, outs[0][0][1:3])
    assert torch.equal(pd2.score, outs[0][3][1:3])
    assert torch.equal(pd2.pos, outs[0][4][1:3])


def test_snapshot_resume_bit_exact():
    """Checkpoint/resume: snapshot the cache mid-decode, continue, restore the
    snapshot into fresh buffers via bm_resume, continue again: identical."""
    _need_gpu()
    from pd_harness import make_pd

    wl = C2.with_(b=2, s=512, n_decode=24)
    q, k, v = synth.batch_inputs(wl, "cuda")
    o = torch.zeros_like(q)
    pd = make_pd(wl)
    pd.run_prefill(q, k, v, o)
    pd.run_decode(q, k, v, o, steps=10)
    snap = [x.clone() for x in (pd.k, pd.v, pd.score, pd.pos, pd.len)]
    length, nxt = pd.length, pd.next_pos
    for t in range(10, 24):
        pd.decode_step(wl.s + t, q, k, v, o, row=wl.s + t)
    torch.cuda.synchronize()
    pd2 = make_pd(wl)
    for dst, src in zip((pd2.k, pd2.v, pd2.score, pd2.pos, pd2.len), snap):
        dst.copy_(src)
    pd2.resume(length, nxt)
    o2 = o.clone()
    o2[:, :, wl.s + 10:] = 0
    for t in range(10, 24):
        pd2.decode_step(wl.s + t, q, k, v, o2, row=wl.s + t)
    torch.cuda.synchronize()
    assert torch.equal(o2, o)
    assert torch.equal(pd2.score, pd.score) and torch.equal(pd2.pos, pd.pos)


@pytest.mark.parametrize("sample_seed", [0, 1])
def test_c3_full_shape_sampled_units(sample_seed):
    # 2 x 16 seeded units (first and last unit in both)
    wl = synth.WORKLOADS["c3"]
    st = _run(wl, synth.checked_units(wl, 16, seed=sample_seed))
    assert st.cuts > 0


def test_c4_full_shape_sampled_units():
    # decode-heavy: 512 steps with one eviction each per unit
    wl = synth.WORKLOADS["c4"]
    st = _run(wl, synth.checked_units(wl, 32))
    assert st.cuts > 0


@pytest.mark.parametrize("decode_p", [0, 8])
def test_decode_graph_replays_match_eager(decode_p):
    # the decode loop captured once, replayed three times, each after a fresh
    # eager prefill: outputs, scores, positions and lengths equal the eager run
    _need_gpu()
    from pd_harness import make_pd

    wl = C2.with_(b=2, s=1024, n_decode=24)
    q, k, v = synth.batch_inputs(wl, "cuda")
    o = torch.zeros_like(q)
    pd = make_pd(wl)
    pd.set_decode_removal(decode_p)
    pd.run_prefill(q, k, v, o)
    pd.run_decode(q, k, v, o)
    torch.cuda.synchronize()
    ref = (o.clone(), pd.score.clone(), pd.pos.clone(), pd.len.clone())

    pd.reset()
    pd.run_prefill(q, k, v, o)
    g = pd.capture_decode(q, k, v, o)
    for rep in range(3):
        pd.reset()
        o.zero_()
        pd.run_prefill(q, k, v, o)
        g.replay()
        torch.cuda.synchronize()
        _say(f"[graph] replay {rep} decode_p={decode_p}")
        assert torch.equal(o, ref[0])
        L = int(ref[3][0, 0])
        assert torch.equal(pd.len, ref[3])
        assert torch.equal(pd.pos[..., :L], ref[2][..., :L])
        assert torch.equal(pd.score[..., :L], ref[1][..., :L])
