"""The seeded workload generator: determinism, bf16 rounding, heavy hitters."""
import numpy as np
import torch

from paper_2412_05693_amd import synth


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(0)
    x = (rng.standard_normal(100000) * 10.0 ** rng.integers(-6, 6, 100000)).astype(np.float32)
    x[:4] = [0.0, -0.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8]      # exact ties round to even
    ours = synth.f32_to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)


def test_unit_stream_deterministic_and_representable():
    wl = synth.WORKLOADS["c2"].with_(s=512, n_decode=8)
    a = synth.unit_inputs(wl, 0, 3, 5)
    b = synth.unit_inputs(wl, 0, 3, 5)
    c = synth.unit_inputs(wl, 0, 3, 6)
    for x, y in zip(a, b):
        assert np.array_equal(x, y)
    assert not np.array_equal(a[1], c[1])
    for x in a:
        assert np.array_equal(synth.round_to_dtype(x, "bf16"), x)
    q, k, v = a
    assert q.shape == (4, 520, 128) and k.shape == (520, 128) and v.shape == (520, 128)


def test_heavy_hitters_and_sinks():
    wl = synth.WORKLOADS["c2"]
    hh = synth.heavy_positions(wl, 0, 0)
    assert len(hh) == round(0.02 * wl.s) and hh.min() >= 4 and len(set(hh)) == len(hh)
    prof = synth.key_scale_profile(wl, 0, 0)
    assert np.all(prof[:4] == 6.0) and np.all(prof[hh] == 4.0)
    assert np.all(prof[wl.s:] == 1.0)
    wl3 = synth.WORKLOADS["c3"]
    sp = synth.heavy_positions(wl3, 0, 1)
    assert len(sp) == 512 and len(set(sp)) == 512
    c1 = synth.WORKLOADS["c1"]
    assert len(synth.heavy_positions(c1, 0, 0)) == round(0.02 * 512)


def test_batch_inputs_overwrite_checked_units():
    wl = synth.WORKLOADS["c2"].with_(b=2, s=64, n_decode=4)
    q, k, v = synth.batch_inputs(wl, "cpu", checked=[(1, 2)])
    uq, uk, uv = synth.unit_inputs(wl, 0, 1, 2)
    assert torch.equal(k[1, 2].float(), torch.from_numpy(uk))
    assert torch.equal(q[1, 8:12].float(), torch.from_numpy(uq))
    assert q.dtype == torch.bfloat16 and q.shape == (2, 32, 68, 128)
