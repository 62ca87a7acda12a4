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


# --- the counter-based stream of the layer stack -------------------------------
# Known-answer vectors of Philox4x32-10 (counter, key -> output), as published
# with the generator's reference implementation (Random123).
PHILOX_KAT = [
    ((0, 0, 0, 0), (0, 0), (0x6627E8D5, 0xE169C58D, 0xBC57AC4C, 0x9B00DBD8)),
    ((0xFFFFFFFF,) * 4, (0xFFFFFFFF,) * 2, (0x408F276D, 0x41C83B0E, 0xA20BC7C6, 0x6D5451FD)),
    ((0x243F6A88, 0x85A308D3, 0x13198A2E, 0x03707344), (0xA4093822, 0x299F31D0),
     (0xD16CFE09, 0x94FDCCEB, 0x5001E420, 0x24126EA1)),
]


def test_philox_known_answers():
    for ctr, key, want in PHILOX_KAT:
        got = synth.philox4x32_10(np.array(ctr, dtype=np.uint32), np.array(key, dtype=np.uint32))
        assert tuple(int(x) for x in got) == want
    # vectorised evaluation equals one call per element
    ctr = np.array([c for c, _, _ in PHILOX_KAT], dtype=np.uint32)
    key = np.array([k for _, k, _ in PHILOX_KAT], dtype=np.uint32)
    assert [tuple(int(x) for x in r) for r in synth.philox4x32_10(ctr, key)] == [w for _, _, w in PHILOX_KAT]


def test_stack_stream_element_layout():
    wl = synth.WORKLOADS["c5"].with_(b=2, s=64, n_decode=4)
    q, k, v = synth.stack_unit_inputs(wl, 3, 1, 2)
    # element (pos 5, dims 6 and 7) of V head 2: one Philox call, words 0-1 and 2-3
    w = synth.philox4x32_10(np.array([5 * 64 + 3, (synth.T_V << 8) | 2, 1, 3], dtype=np.uint32),
                            np.array([wl.seed, 0], dtype=np.uint32)).astype(np.int64)
    h = lambda x: (x & 0xFFFF) + (x >> 16)
    c = synth.stack_value_scale(128)
    z = [(np.float32(h(w[0]) + h(w[1])) - np.float32(131070)) * c,
         (np.float32(h(w[2]) + h(w[3])) - np.float32(131070)) * c]
    assert np.array_equal(v[5, 6:8], synth.round_to_dtype(np.array(z, dtype=np.float32), "bf16"))
    # Q head of query head 2 * 4 + 1 uses tensor 0
    q2 = synth._stack_values(wl, 3, 1, synth.T_Q, 2 * 4 + 1, np.arange(wl.total))
    assert np.array_equal(q[1], synth.round_to_dtype(q2, "bf16"))
    # every coordinate of the counter matters
    for args in ((4, 1, 2), (3, 0, 2), (3, 1, 3)):
        assert not np.array_equal(synth.stack_unit_inputs(wl, *args)[2], v)


def test_stack_stream_statistics():
    wl = synth.WORKLOADS["c5"].with_(b=2)
    q, k, v = synth.stack_unit_inputs(wl, 0, 0, 0)
    d = wl.head_dim
    for x in (q, v):
        assert abs(float(x.mean())) < 3e-3 / np.sqrt(d) * 10
        assert abs(float(x.std()) * np.sqrt(d) - 1.0) < 0.01
        assert float(np.abs(x).max()) <= 2 * np.sqrt(3) / np.sqrt(d) * 1.01   # Irwin-Hall bound
        assert np.array_equal(synth.round_to_dtype(x, "bf16"), x)
    f = synth.stack_key_factor(wl, 0, 0, np.arange(wl.total))
    assert np.all(f[:4] == 6.0) and np.all(f[wl.s:] == 1.0)
    n_heavy = int(np.sum(f == 4.0))
    expect = wl.hh_frac * (wl.s - 4)
    assert abs(n_heavy - expect) < 4 * np.sqrt(expect)
    # the heavy rows are exactly 4x the plain stream
    plain = synth._stack_values(wl, 0, 0, synth.T_K, 0, np.arange(wl.total))
    assert np.array_equal(k, synth.round_to_dtype(plain * f[:, None], "bf16"))


def test_stack_planner():
    from paper_2412_05693_amd import batchmax as bmx

    sh = dict(n_layers=32, s=8192, kv_max=512, block=256, max_gen=256, n_heads=32, n_kv_heads=8,
              head_dim=128, dtype="bf16")
    per = bmx.stack_layer_bytes(b=1, kv_max=512, block=256, n_kv_heads=8, head_dim=128,
                                dtype="bf16")
    assert per * 32 == 102_244_352          # K, V, scores, positions and lengths of 32 layers
    budget = 285 * 10 ** 9
    b = bmx.plan_stack_batch(budget, **sh)
    assert bmx.stack_bytes(b=b, **sh) <= budget < bmx.stack_bytes(b=b + 1, **sh)
    full = bmx.full_cache_bytes_per_sample(n_layers=32, s=8192, n_kv_heads=8, head_dim=128,
                                           dtype="bf16")
    assert full == 32 * 8 * 8192 * 128 * 2 * 2
    assert b > 9 * (budget // full)          # the bounded caches hold ~10x the samples


def test_sample_pads():
    wl = synth.WORKLOADS["c2"].with_(pad_max=2048)
    p = synth.sample_pads(wl)
    assert p.dtype == np.int32 and p.shape == (wl.b,)
    assert p[0] == 0 and p[-1] == 2048 and p.min() >= 0 and p.max() <= 2048
    assert np.array_equal(p, synth.sample_pads(wl))          # seeded
    assert not synth.sample_pads(synth.WORKLOADS["c2"]).any()  # no padding by default
