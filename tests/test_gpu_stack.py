"""GPU: the counter-based input generator and the 32-layer stack.

The generator is checked word for word (raw Philox outputs) and element for
element (Q/K/V rows, bf16 and float32) against the host evaluation of the same
stream; the stack is checked against the float64 oracle on units spread over
its first, middle and last layers, at the full per-unit shape (s = 8192, bound
512, block 256, 256 decode steps), at a reduced batch and at the largest batch
that fits the device (the benchmark's).
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


def test_philox_device_matches_host():
    _need_gpu()
    from paper_2412_05693_amd import batchmax as bmx

    rng = np.random.default_rng(11)
    n = 1 << 14
    inp = rng.integers(0, 2 ** 32, size=(n, 6), dtype=np.uint64).astype(np.uint32)
    inp[:3] = [[0, 0, 0, 0, 0, 0], [0xFFFFFFFF] * 6,
               [0x243F6A88, 0x85A308D3, 0x13198A2E, 0x03707344, 0xA4093822, 0x299F31D0]]
    _say(f"[stack] philox words n={n}")
    d_in = torch.from_numpy(inp.view(np.int32)).cuda()
    d_out = torch.empty((n, 4), dtype=torch.int32, device="cuda")
    bmx.bm_philox4x32_10(d_in.data_ptr(), d_out.data_ptr(), n, torch.cuda.current_stream().cuda_stream)
    got = d_out.cpu().numpy().view(np.uint32)
    want = synth.philox4x32_10(inp[:, :4], inp[:, 4:])
    assert np.array_equal(got, want)


@pytest.mark.parametrize("dtype,d,G,t0,rows", [("bf16", 128, 4, 0, 40), ("bf16", 128, 4, 490, 40),
                                               ("f32", 64, 2, 7, 33)])
def test_synth_qkv_device_matches_host(dtype, d, G, t0, rows):
    _need_gpu()
    from paper_2412_05693_amd import batchmax as bmx

    Hk = 2
    wl = synth.WORKLOADS["c5"].with_(dtype=dtype, b=3, n_heads=G * Hk, n_kv_heads=Hk, head_dim=d,
                                     s=512, n_decode=32, n_layers=4)
    layer = 2
    _say(f"[stack] synth {dtype} d={d} G={G} rows [{t0}, {t0 + rows})")
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    q = torch.empty((wl.b, wl.n_heads, rows, d), dtype=tdt, device="cuda")
    k = torch.empty((wl.b, Hk, rows, d), dtype=tdt, device="cuda")
    v = torch.empty_like(k)
    p = bmx.synth_params(b=wl.b, n_heads=wl.n_heads, n_kv_heads=Hk, head_dim=d, dtype=dtype,
                         seed=wl.seed, layer=layer, s=wl.s, hh_frac=wl.hh_frac, hh_scale=wl.hh_scale,
                         n_sinks=wl.n_sinks, sink_scale=wl.sink_scale)
    bmx.synth_qkv(p, t0, q, k, v)
    gq, gk, gv = (x.float().cpu().numpy() for x in (q, k, v))
    for bi in range(wl.b):
        for hk in range(Hk):
            uq, uk, uv = synth.stack_unit_inputs(wl, layer, bi, hk)
            assert np.array_equal(gk[bi, hk], uk[t0:t0 + rows])
            assert np.array_equal(gv[bi, hk], uv[t0:t0 + rows])
            assert np.array_equal(gq[bi, hk * G:(hk + 1) * G], uq[:, t0:t0 + rows])


@pytest.mark.parametrize("fused_cut", [False, True])
def test_c5_stack_parity_reduced_batch(fused_cut):
    _need_gpu()
    from pd_harness import run_stack_parity

    wl = synth.WORKLOADS["c5"].with_(b=2)
    L = wl.n_layers
    # 16 (layer, sample, KV head) units over the first, middle and last layers
    checked = [(0, 0, 0), (0, 1, 7), (0, 0, 2), (0, 1, 5), (1, 0, 1),
               (L // 2, 0, 3), (L // 2, 1, 4), (L // 2, 0, 6), (L // 2 + 1, 1, 2),
               (L - 1, 0, 5), (L - 1, 1, 0), (L - 1, 0, 7), (L - 1, 1, 3), (L - 2, 0, 4),
               (L - 2, 1, 6), (L // 4, 1, 1)]
    _say(f"[stack] {wl.name} b={wl.b} layers={L} s={wl.s} kv={wl.kv_max} B={wl.block} "
         f"D={wl.n_decode} fused_cut={fused_cut} units={checked}")
    st = run_stack_parity(wl, checked, fused_cut=fused_cut)
    _say(f"[stack] -> {st.summary()}")
    assert not st.failures, "\n".join(st.failures)
    assert st.cuts == len(checked) * (wl.s // wl.block - wl.kv_max // wl.block + wl.n_decode)


def test_c5_stack_parity_full_batch():
    """The 32-layer stack at the batch the benchmark runs (the largest that fits
    the device) and on its path (each block and its cut in one call: attention,
    then the fused fold/select/compaction kernel), checked on sampled units of
    the first, middle and last layers and of the first, middle and last
    samples."""
    _need_gpu()
    import gc

    from paper_2412_05693_amd import batchmax as bmx
    from pd_harness import run_stack_parity

    gc.collect()
    torch.cuda.empty_cache()
    wl = synth.WORKLOADS["c5"]
    shape = dict(n_layers=wl.n_layers, s=wl.s, kv_max=wl.kv_max, block=wl.block,
                 max_gen=wl.n_decode, n_heads=wl.n_heads, n_kv_heads=wl.n_kv_heads,
                 head_dim=wl.head_dim, dtype=wl.dtype)
    free, _ = torch.cuda.mem_get_info()
    b = bmx.plan_stack_batch(free - (3 << 30), **shape)
    assert b >= 2, f"only {free / 1e9:.1f} GB free"
    wl = wl.with_(b=b)
    L = wl.n_layers
    checked = [(0, 0, 0), (0, b - 1, 7), (L // 2, b // 2, 3), (L // 2, b - 1, 4),
               (L - 1, 0, 5), (L - 1, b - 1, 2)]
    _say(f"[stack] {wl.name} full batch b={b} layers={L} s={wl.s} fused_cut=True units={checked}")
    st = run_stack_parity(wl, checked, fused_cut=True)
    _say(f"[stack] -> {st.summary()}")
    assert not st.failures, "\n".join(st.failures)
    assert st.cuts == len(checked) * (wl.s // wl.block - wl.kv_max // wl.block + wl.n_decode)
