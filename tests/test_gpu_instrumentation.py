"""GPU checks of the measurement hooks the benchmark relies on.

* The split event (bm_set_split_event) is recorded after a block's attention
  kernel and before its cut: with a host-side event before and after the call,
  both intervals are positive and add up to the whole; it changes no result.
* The roofline probes (bm_probe.h) run and their sinks hold what the host
  predicts: the XOR of every 32-bit word each workgroup read, and finite
  MFMA sums.
* The prefill timeline build (a separate library, so a separate process)
  records one ordered set of timestamps per workgroup of the last launch.
"""
import numpy as np
import pytest
import torch

from paper_2412_05693_amd import batchmax as bmx
from paper_2412_05693_amd import synth

pytestmark = pytest.mark.gpu


def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def test_split_event_between_attention_and_cut():
    _need_gpu()
    from pd_harness import make_pd

    wl = synth.WORKLOADS["c2"].with_(b=4, s=1024, n_decode=4)
    q, k, v = synth.batch_inputs(wl, "cuda")
    outs = []
    for with_events in (False, True):
        o = torch.zeros_like(q)
        pd = make_pd(wl)
        stream = torch.cuda.current_stream()
        for t0 in range(0, wl.s, wl.block):
            if with_events:
                a, sp, z = (torch.cuda.Event(enable_timing=True) for _ in range(3))
                pd.set_split_event(sp)
                a.record(stream)
            pd.prefill_block_cut(t0, wl.block, q, k, v, o)
            if with_events:
                z.record(stream)
                torch.cuda.synchronize()
                t_att, t_cut, t_all = a.elapsed_time(sp), sp.elapsed_time(z), a.elapsed_time(z)
                print(f"[split] block {t0}: attention {t_att:.4f} ms, cut {t_cut:.4f} ms", flush=True)
                assert t_att > 0 and t_cut > 0
                assert abs(t_att + t_cut - t_all) < 1e-3 + 1e-3 * t_all
        pd.set_split_event(None)
        pd.run_decode(q, k, v, o)
        torch.cuda.synchronize()
        outs.append((o.clone(), pd.score.clone(), pd.pos.clone()))
    for x, y in zip(*outs):
        assert torch.equal(x, y)


def test_probe_stream_read_sink():
    _need_gpu()
    blocks = 64
    n_words = 1 << 20
    rng = np.random.default_rng(3)
    host = rng.integers(0, 2 ** 32, size=n_words, dtype=np.uint64).astype(np.uint32)
    buf = torch.from_numpy(host.view(np.int32)).cuda()
    sink = torch.zeros(blocks, dtype=torch.int32, device="cuda")
    for nt in (False, True):
        bmx.bm_probe_stream_read(buf.data_ptr(), n_words * 4, sink.data_ptr(), blocks, nt,
                                 torch.cuda.current_stream().cuda_stream)
        torch.cuda.synchronize()
        got = sink.cpu().numpy().view(np.uint32)
        # workgroup w reads the 16-byte chunks w*256 + t + i*blocks*256
        chunks = host.reshape(-1, 4)
        want = np.zeros(blocks, dtype=np.uint32)
        for w in range(blocks):
            idx = (np.arange(len(chunks)) // 256) % blocks == w
            want[w] = np.bitwise_xor.reduce(chunks[idx].reshape(-1))
        assert np.array_equal(got, want)


def test_probe_mfma_runs():
    _need_gpu()
    blocks = 8
    sink = torch.full((blocks * 4,), float("nan"), dtype=torch.float32, device="cuda")
    bmx.bm_probe_mfma(16, sink.data_ptr(), blocks, torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    s = sink.cpu().numpy()
    assert np.all(np.isfinite(s)) and np.all(s == s[0])


def test_prefill_timeline_records():
    _need_gpu()
    import os
    import subprocess
    import sys

    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    lib = os.path.join(root, "paper_2412_05693_amd", "libbatchmax_timeline.so")
    if not os.path.exists(lib):
        pytest.skip("timeline build not present")
    code = (
        "import numpy as np, torch\n"
        "from paper_2412_05693_amd import batchmax as bmx, synth\n"
        "wl = synth.WORKLOADS['c2'].with_(b=2, s=768, n_decode=1)\n"
        "q, k, v = synth.batch_inputs(wl, 'cuda'); o = torch.zeros_like(q)\n"
        "pd = bmx.PDAttention(b=wl.b, s=wl.s, kv_max=wl.kv_max, block=wl.block, max_gen=1,\n"
        "    n_heads=wl.n_heads, n_kv_heads=wl.n_kv_heads, head_dim=wl.head_dim, dtype=wl.dtype,\n"
        "    sm_scale=wl.sm_scale, device='cuda')\n"
        "for t0 in range(0, wl.s, wl.block): pd.prefill_block_cut(t0, wl.block, q, k, v, o)\n"
        "torch.cuda.synchronize()\n"
        "nwg = wl.b * wl.n_kv_heads * (wl.block // 32)\n"
        "r = bmx.bm_prefill_timeline(nwg).astype(np.int64)\n"
        "mono = np.all(np.diff(r[:, :8], axis=1) >= 0)\n"
        "units = sorted(set((r[:, 14] >> 32).tolist()))\n"
        "print(int(mono), int(np.all(r[:, 0] > 0)), len(units), int(r[:, 15].min()), int(r[:, 15].max()))\n")
    env = dict(os.environ, BATCHMAX_LIB=lib, PYTHONPATH=root)
    print("[timeline] c2 shape b=2 s=768, last block", flush=True)
    res = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, env=env,
                         timeout=240)
    assert res.returncode == 0, res.stderr[-2000:]
    mono, positive, n_units, tmin, tmax = map(int, res.stdout.split()[-5:])
    assert mono == 1 and positive == 1
    assert n_units == 2 * 8
    # last block: 512 cached keys (8 tiles) + 1..4 block tiles of 64 positions
    assert tmin == 8 + 1 and tmax == 8 + 4
