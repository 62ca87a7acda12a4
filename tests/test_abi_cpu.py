"""The C ABI without a GPU: the library loads, exports every declared symbol,
and every argument, capacity and order error is reported before any device
work.  Contexts here come from bm_resume with placeholder addresses, which no
call below ever dereferences: each call is one the host checks reject."""
import ctypes
import os
import re

import pytest

from paper_2412_05693_amd import batchmax as bmx

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "batchmax.h")

FAKE = 0x7F0000000000  # placeholder device address, 4 KiB aligned, never touched


def dims(**kw):
    base = dict(b=2, s=512, kv_max=128, block=64, max_gen=32, n_heads=8, n_kv_heads=2,
                head_dim=128, dtype="bf16")
    base.update(kw)
    return bmx.make_dims(**base)


def fake_cache(d):
    return bmx.bm_cache(FAKE, FAKE + 0x1000000, FAKE + 0x2000000, FAKE + 0x3000000,
                        FAKE + 0x4000000, FAKE + 0x5000000, bmx.bm_workspace_bytes(d))


def status_of(fn, *args):
    try:
        fn(*args)
    except bmx.BatchMaxError as e:
        return e.status
    return bmx.BM_OK


def test_header_symbols_exported():
    inc = os.path.join(ROOT, "include")
    text = "".join(open(os.path.join(inc, f)).read() for f in sorted(os.listdir(inc))
                   if f.endswith(".h"))
    declared = sorted(set(re.findall(r"\b(bm_[a-z0-9_]+)\s*\(", text)))
    assert declared, "no declarations found"
    lib = ctypes.CDLL(bmx.LIB_PATH)
    for name in declared:
        assert hasattr(lib, name), f"{name} declared but not exported"
    assert sorted(bmx.EXPORTED) == declared


def test_version_matches_header():
    m = re.search(r"#define BM_ABI_VERSION (\d+)", open(HEADER).read())
    assert bmx.bm_abi_version() == int(m.group(1))


def test_slots_and_workspace():
    d = dims()
    assert bmx.bm_cache_slots(d) == 128 + 64
    ws = bmx.bm_workspace_bytes(d)
    # partial sums: units x ceil(block / (128 / G)) x cap floats, plus lists
    U, cap, npt = 4, 192, 2
    assert ws >= U * npt * cap * 4 + 2 * U * cap * 4 + U * 4
    assert bmx.bm_cache_slots(dims(b=0)) == -1
    assert bmx.bm_prefill_positions_per_workgroup(d) == 128 // 4
    assert bmx.bm_prefill_positions_per_workgroup(dims(n_heads=2, n_kv_heads=2)) == 128
    assert bmx.bm_prefill_positions_per_workgroup(dims(b=0)) == -1
    assert bmx.bm_workspace_bytes(dims(head_dim=96)) == 0


@pytest.mark.parametrize("kw,status", [
    (dict(b=0), bmx.BM_ERR_INVALID_ARG),
    (dict(s=-1), bmx.BM_ERR_INVALID_ARG),
    (dict(kv_max=0), bmx.BM_ERR_INVALID_ARG),
    (dict(block=0), bmx.BM_ERR_INVALID_ARG),
    (dict(max_gen=-1), bmx.BM_ERR_INVALID_ARG),
    (dict(n_heads=6, n_kv_heads=4), bmx.BM_ERR_INVALID_ARG),
    (dict(sm_scale=float("nan")), bmx.BM_ERR_INVALID_ARG),
    (dict(sm_scale=-1.0), bmx.BM_ERR_INVALID_ARG),
    (dict(head_dim=96), bmx.BM_ERR_UNSUPPORTED),
    (dict(dtype=7), bmx.BM_ERR_UNSUPPORTED),
    (dict(n_heads=16, n_kv_heads=2), bmx.BM_ERR_UNSUPPORTED),
    (dict(n_heads=6, n_kv_heads=2), bmx.BM_ERR_UNSUPPORTED),
    (dict(block=2048), bmx.BM_ERR_UNSUPPORTED),
    (dict(kv_max=65100, block=512), bmx.BM_ERR_UNSUPPORTED),
])
def test_validate_dims_errors(kw, status):
    assert status_of(bmx.bm_validate_dims, dims(**kw)) == status
    assert bmx.bm_last_error() != ""


def test_validate_dims_ok():
    bmx.bm_validate_dims(dims())
    bmx.bm_validate_dims(dims(dtype="f32", head_dim=64, n_heads=4, n_kv_heads=4))
    assert bmx.bm_last_error() == ""


def test_cache_pointer_checks():
    d = dims()
    for field in ("k", "v", "score", "pos", "len", "work"):
        c = fake_cache(d)
        setattr(c, field, 0)
        assert status_of(bmx.bm_resume, d, c, 0, 0) == bmx.BM_ERR_INVALID_ARG
    c = fake_cache(d)
    c.k = FAKE + 8
    assert status_of(bmx.bm_resume, d, c, 0, 0) == bmx.BM_ERR_INVALID_ARG
    c = fake_cache(d)
    c.work_bytes = 16
    assert status_of(bmx.bm_resume, d, c, 0, 0) == bmx.BM_ERR_INVALID_ARG
    c = fake_cache(d)
    assert status_of(bmx.bm_resume, d, c, 200, 300) == bmx.BM_ERR_INVALID_ARG   # len > cap
    assert status_of(bmx.bm_resume, d, c, 10, 5) == bmx.BM_ERR_INVALID_ARG      # len > next_pos


def _ctx(d, length, next_pos):
    return bmx.bm_resume(d, fake_cache(d), length, next_pos)


def test_prefill_order_and_capacity_errors():
    d = dims()
    ctx = _ctx(d, 128, 192)
    P = FAKE
    try:
        assert status_of(bmx.bm_prefill_block, ctx, 100, 64, P, P, P, P, 64, 0) == bmx.BM_ERR_ORDER
        assert status_of(bmx.bm_prefill_block, ctx, 192, 0, P, P, P, P, 64, 0) == bmx.BM_ERR_INVALID_ARG
        assert status_of(bmx.bm_prefill_block, ctx, 192, 65, P, P, P, P, 65, 0) == bmx.BM_ERR_INVALID_ARG
        assert status_of(bmx.bm_prefill_block, ctx, 192, 64, P, P, P, P, 32, 0) == bmx.BM_ERR_INVALID_ARG
        assert status_of(bmx.bm_prefill_block, ctx, 192, 64, 0, P, P, P, 64, 0) == bmx.BM_ERR_INVALID_ARG
        assert status_of(bmx.bm_prefill_block, ctx, 192, 64, P + 2, P, P, P, 64, 0) == bmx.BM_ERR_INVALID_ARG
        # the fused block-and-cut call runs the same checks before any launch
        cut = bmx.bm_prefill_block_cut
        assert status_of(cut, ctx, 100, 64, P, P, P, P, 64, 0) == bmx.BM_ERR_ORDER
        assert status_of(cut, ctx, 192, 0, P, P, P, P, 64, 0) == bmx.BM_ERR_INVALID_ARG
        assert status_of(cut, ctx, 192, 65, P, P, P, P, 65, 0) == bmx.BM_ERR_INVALID_ARG
        assert status_of(cut, ctx, 192, 64, 0, P, P, P, 64, 0) == bmx.BM_ERR_INVALID_ARG
        assert bmx.bm_ctx_next_pos(ctx) == 192 and bmx.bm_ctx_len(ctx) == 128
    finally:
        bmx.bm_destroy(ctx)
    # past the prompt
    ctx = _ctx(d, 128, 480)
    try:
        assert status_of(bmx.bm_prefill_block, ctx, 480, 64, P, P, P, P, 64, 0) == bmx.BM_ERR_ORDER
    finally:
        bmx.bm_destroy(ctx)
    # cache over the bound: must evict first
    ctx = _ctx(d, 192, 192)
    try:
        assert status_of(bmx.bm_prefill_block, ctx, 192, 64, P, P, P, P, 64, 0) == bmx.BM_ERR_ORDER
        assert status_of(bmx.bm_prefill_block_cut, ctx, 192, 64, P, P, P, P, 64, 0) == bmx.BM_ERR_ORDER
        assert status_of(bmx.bm_evict_compact, ctx, 190, 0) == bmx.BM_ERR_ORDER
    finally:
        bmx.bm_destroy(ctx)


def test_evict_noop_when_within_bound():
    d = dims()
    ctx = _ctx(d, 100, 100)
    try:
        bmx.bm_evict_compact(ctx, 99, 0)          # nothing to cut: no device work
        assert bmx.bm_ctx_len(ctx) == 100
        assert status_of(bmx.bm_evict_compact, ctx, 98, 0) == bmx.BM_ERR_ORDER
    finally:
        bmx.bm_destroy(ctx)


def test_decode_order_and_capacity_errors():
    d = dims()
    P = FAKE
    ctx = _ctx(d, 128, 448)           # prefill not finished
    try:
        assert status_of(bmx.bm_decode_step, ctx, 448, P, P, P, P, 1, 0) == bmx.BM_ERR_ORDER
    finally:
        bmx.bm_destroy(ctx)
    ctx = _ctx(d, 192, 512)           # last block not evicted
    try:
        assert status_of(bmx.bm_decode_step, ctx, 512, P, P, P, P, 1, 0) == bmx.BM_ERR_CAPACITY
    finally:
        bmx.bm_destroy(ctx)
    ctx = _ctx(d, 128, 544)           # past s + max_gen
    try:
        assert status_of(bmx.bm_decode_step, ctx, 544, P, P, P, P, 1, 0) == bmx.BM_ERR_ORDER
    finally:
        bmx.bm_destroy(ctx)
    ctx = _ctx(d, 128, 520)
    try:
        assert status_of(bmx.bm_decode_step, ctx, 519, P, P, P, P, 1, 0) == bmx.BM_ERR_ORDER
        assert status_of(bmx.bm_decode_step, ctx, 520, P, P, P, P, 0, 0) == bmx.BM_ERR_INVALID_ARG
        assert status_of(bmx.bm_decode_step, ctx, 520, P, 0, P, P, 1, 0) == bmx.BM_ERR_INVALID_ARG
    finally:
        bmx.bm_destroy(ctx)


def test_decode_removal_range():
    d = dims()
    ctx = _ctx(d, 128, 520)
    try:
        for p in (0, 1, d.kv_max):
            bmx.bm_set_decode_removal(ctx, p)
        assert status_of(bmx.bm_set_decode_removal, ctx, -1) == bmx.BM_ERR_INVALID_ARG
        assert status_of(bmx.bm_set_decode_removal, ctx, d.kv_max + 1) == bmx.BM_ERR_INVALID_ARG
        assert bmx.bm_ctx_len(ctx) == 128            # choosing the schedule does no work
    finally:
        bmx.bm_destroy(ctx)
    assert status_of(bmx.bm_set_decode_removal, None, 1) == bmx.BM_ERR_INVALID_ARG


def test_rule_bound_and_accumulation_setters():
    d = dims()
    ctx = _ctx(d, 128, 520)
    try:
        for r in (bmx.BM_RANK_AVE, bmx.BM_RANK_SUM, bmx.BM_RANK_RECENT, bmx.BM_RANK_TOVA):
            bmx.bm_set_rank_rule(ctx, r)
        assert status_of(bmx.bm_set_rank_rule, ctx, 4) == bmx.BM_ERR_INVALID_ARG
        assert status_of(bmx.bm_set_rank_rule, ctx, -1) == bmx.BM_ERR_INVALID_ARG
        for bnd in (1, 2, d.kv_max):
            bmx.bm_set_decode_bound(ctx, bnd)
        assert status_of(bmx.bm_set_decode_bound, ctx, 0) == bmx.BM_ERR_INVALID_ARG
        assert status_of(bmx.bm_set_decode_bound, ctx, d.kv_max + 1) == bmx.BM_ERR_INVALID_ARG
        bmx.bm_set_score_accumulation(ctx, 0)
        bmx.bm_set_score_accumulation(ctx, 1)
        assert status_of(bmx.bm_set_score_accumulation, ctx, 2) == bmx.BM_ERR_INVALID_ARG
        assert bmx.bm_ctx_len(ctx) == 128
    finally:
        bmx.bm_destroy(ctx)
    for fn, arg in ((bmx.bm_set_rank_rule, 0), (bmx.bm_set_decode_bound, 1),
                    (bmx.bm_set_score_accumulation, 1)):
        assert status_of(fn, None, arg) == bmx.BM_ERR_INVALID_ARG


def test_decode_removal_beyond_the_decode_bound_is_rejected_before_launch():
    d = dims()
    P = FAKE
    ctx = _ctx(d, 128, 520)
    try:
        bmx.bm_set_decode_bound(ctx, 4)
        bmx.bm_set_decode_removal(ctx, 5)
        assert status_of(bmx.bm_decode_step, ctx, 520, P, P, P, P, 1, 0) == bmx.BM_ERR_INVALID_ARG
        assert bmx.bm_ctx_len(ctx) == 128
    finally:
        bmx.bm_destroy(ctx)


def test_null_context():
    P = FAKE
    assert status_of(bmx.bm_prefill_block, None, 0, 1, P, P, P, P, 1, 0) == bmx.BM_ERR_INVALID_ARG
    assert status_of(bmx.bm_prefill_block_cut, None, 0, 1, P, P, P, P, 1, 0) == bmx.BM_ERR_INVALID_ARG
    assert status_of(bmx.bm_evict_compact, None, 0, 0) == bmx.BM_ERR_INVALID_ARG
    assert status_of(bmx.bm_decode_step, None, 0, P, P, P, P, 1, 0) == bmx.BM_ERR_INVALID_ARG
    assert bmx.bm_ctx_len(None) == -1 and bmx.bm_ctx_next_pos(None) == -1


def test_algorithmic_work_figures():
    # c2: b=64, GQA 32/8, d=128, s=4096, |kv|=512, block=256
    f = bmx.prefill_flops(b=64, n_kv_heads=8, group=4, head_dim=128, s=4096, kv_max=512, block=256)
    assert abs(f - 2.545e12) / 2.545e12 < 1e-3
    by = bmx.decode_bytes_per_step(b=64, n_kv_heads=8, group=4, head_dim=128, kv_max=512,
                                   elem_bytes=2)
    assert by == 512 * 271368


def test_synth_argument_checks():
    # every check runs on the host before a launch, so fake pointers are safe
    mk = lambda **kw: bmx.synth_params(**{**dict(b=2, n_heads=8, n_kv_heads=2, head_dim=64,
                                                 dtype="bf16", seed=1, layer=0, s=64), **kw})
    p = mk()
    call = lambda prm, t0, n, q, k, v, ld: status_of(bmx.bm_synth_qkv, prm, t0, n, q, k, v, ld, 0)
    bad = bmx.BM_ERR_INVALID_ARG
    assert call(p, 0, 0, FAKE, FAKE, FAKE, 1) == bad          # no rows
    assert call(p, -1, 4, FAKE, FAKE, FAKE, 4) == bad         # negative position
    assert call(p, 0, 4, FAKE, FAKE, FAKE, 3) == bad          # seq_ld < rows
    assert call(p, 0, 4, 0, FAKE, FAKE, 4) == bad             # null q
    assert call(p, 0, 4, FAKE + 2, FAKE, FAKE, 4) == bad      # misaligned q
    assert call(mk(head_dim=63), 0, 4, FAKE, FAKE, FAKE, 4) == bad
    assert call(mk(dtype=7), 0, 4, FAKE, FAKE, FAKE, 4) == bad
    assert call(mk(b=0), 0, 4, FAKE, FAKE, FAKE, 4) == bad
    assert status_of(bmx.bm_philox4x32_10, FAKE, FAKE, 0, 0) == bad
    assert status_of(bmx.bm_philox4x32_10, 0, FAKE, 4, 0) == bad


@pytest.mark.parametrize("p", [0, 1, 3, 8])
def test_decode_cache_lengths_follow_the_oracle(p):
    # the host's schedule model (used for the decode roofline) against the
    # oracle stepping the same schedule: entries each step's attention reads
    import numpy as np

    from oracle import pd as opd

    s, kv_max, block, n_decode, d = 20, 8, 4, 15, 4
    rng = np.random.default_rng(3)
    unit = opd.UnitOracle(head_dim=d, group=1, kv_max=kv_max, sm_scale=0.5)
    for t0 in range(0, s, block):
        unit.prefill_block(t0, rng.standard_normal((1, block, d)),
                           rng.standard_normal((block, d)), rng.standard_normal((block, d)))
        unit.evict(t0 + block - 1, "prefill")
    seen = []
    for t in range(n_decode):
        pos = s + t
        q, k, v = rng.standard_normal((1, d)), rng.standard_normal(d), rng.standard_normal(d)
        if p:
            if unit.n == kv_max:
                unit.evict(pos - 1, "decode", target=kv_max - p)
            seen.append(unit.n)
            unit.append(pos, k[None], v[None])
            unit.attend(q[:, None, :], pos)
        else:
            seen.append(unit.n)
            unit.decode_step(pos, q, k, v)
    assert bmx.decode_cache_lengths(s=s, kv_max=kv_max, n_decode=n_decode, p=p) == seen
    # prompt shorter than the bound: the cache first fills during decode
    assert bmx.decode_cache_lengths(s=5, kv_max=8, n_decode=6, p=2) == [5, 6, 7, 6, 7, 6]


def test_padded_prefill_flops():
    # no padding: the plain count; a pad of whole blocks: the unpadded count of
    # the shorter prompt (pads leave before any real entry, so the real cache
    # evolves as without them); the count never grows with padding
    kw = dict(n_kv_heads=2, group=4, head_dim=64, kv_max=96, block=32)
    assert bmx.prefill_flops_padded(pads=[0, 0, 0], s=300, **kw) == \
        bmx.prefill_flops(b=3, s=300, **kw)
    for k in (1, 3, 5):
        assert bmx.prefill_flops_padded(pads=[32 * k], s=320, **kw) == \
            bmx.prefill_flops(b=1, s=320 - 32 * k, **kw)
    f = [bmx.prefill_flops_padded(pads=[p], s=300, **kw) for p in range(0, 300, 7)]
    assert all(a >= b for a, b in zip(f, f[1:]))


def test_fused_cut_refuses_an_unscored_cut():
    # outputs-only prefill leaves no scores to rank by: a block whose cut is due
    # is refused before any launch unless the rule ignores scores
    d = dims()
    ctx = _ctx(d, 128, 192)
    P = FAKE
    try:
        bmx.bm_set_score_accumulation(ctx, 0)
        assert status_of(bmx.bm_prefill_block_cut, ctx, 192, 64, P, P, P, P, 64, 0) == bmx.BM_ERR_ORDER
        assert bmx.bm_ctx_len(ctx) == 128 and bmx.bm_ctx_next_pos(ctx) == 192
    finally:
        bmx.bm_destroy(ctx)


def test_split_event_hook():
    d = dims()
    assert status_of(bmx.bm_set_split_event, 0, 0) == bmx.BM_ERR_INVALID_ARG
    ctx = _ctx(d, 0, 0)
    try:
        bmx.bm_set_split_event(ctx, FAKE)       # stored only; never recorded here
        bmx.bm_set_split_event(ctx, None)
    finally:
        bmx.bm_destroy(ctx)


def test_static_workspace_refuses_oversized_dims_before_device_work():
    # c4's shape needs about 200 MB of workspace, more than the static array
    d = dims(b=1024, s=2048, kv_max=512, block=256, n_heads=32, n_kv_heads=8)
    assert bmx.bm_workspace_bytes(d) > (64 << 20)
    assert status_of(bmx.bm_init_static_workspace, d, fake_cache(d), 0) == bmx.BM_ERR_UNSUPPORTED
    assert "static workspace" in bmx.bm_last_error()
    assert status_of(bmx.bm_init_static_workspace, dims(b=0), fake_cache(d), 0) == \
        bmx.BM_ERR_INVALID_ARG


def test_probe_argument_errors():
    P = FAKE
    assert status_of(bmx.bm_probe_stream_read, 0, 1024, P, 4, False, 0) == bmx.BM_ERR_INVALID_ARG
    assert status_of(bmx.bm_probe_stream_read, P + 8, 1024, P, 4, False, 0) == bmx.BM_ERR_INVALID_ARG
    assert status_of(bmx.bm_probe_stream_read, P, 1000, P, 4, False, 0) == bmx.BM_ERR_INVALID_ARG
    assert status_of(bmx.bm_probe_stream_read, P, 1024, P, 0, False, 0) == bmx.BM_ERR_INVALID_ARG
    assert status_of(bmx.bm_probe_mfma, 0, P, 4, 0) == bmx.BM_ERR_INVALID_ARG
    assert status_of(bmx.bm_probe_mfma, 10, 0, 4, 0) == bmx.BM_ERR_INVALID_ARG
    assert status_of(bmx.bm_probe_mfma, 10, P, 0, 0) == bmx.BM_ERR_INVALID_ARG


def test_prefill_timeline_only_in_timeline_build():
    """The ordinary library records no timeline and says so; the timestamp
    build checks its arguments (neither call touches a GPU)."""
    import subprocess
    import sys

    with pytest.raises(bmx.BatchMaxError) as e:
        bmx.bm_prefill_timeline(4)
    assert e.value.status == bmx.BM_ERR_UNSUPPORTED
    tl_lib = os.path.join(ROOT, "paper_2412_05693_amd", "libbatchmax_timeline.so")
    if not os.path.exists(tl_lib):
        pytest.skip("timeline build not present (python -m paper_2412_05693_amd.build --timeline)")
    code = (
        "import ctypes\n"
        "from paper_2412_05693_amd import batchmax as bmx\n"
        "f = bmx._lib.bm_prefill_timeline\n"
        "print(f(None, 4), f(ctypes.c_void_p(1), 0), f(ctypes.c_void_p(1), bmx.TIMELINE_MAX_RECORDS + 1))\n")
    env = dict(os.environ, BATCHMAX_LIB=tl_lib, PYTHONPATH=ROOT)
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, env=env,
                       timeout=300)
    assert r.returncode == 0, r.stderr
    assert r.stdout.split() == [str(bmx.BM_ERR_INVALID_ARG)] * 3
