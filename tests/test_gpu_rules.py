"""GPU parity of the other ranking rules and of the comparators of Sec. 4.

* the cumulative sum_weights rule that Sec. 3.2 corrects (BM_RANK_SUM);
* Algorithm 3, extreme decoding-only eviction (ED): the prompt is processed
  with no removal and no score sums, then every decode step keeps only the
  most recent pair (decode bound 2, p = 1, BM_RANK_RECENT) -- at a ragged
  shape and at the 8192-token prompt of the layer-stack workload, whose first
  decode cut streams 8192 keys through the select kernel;
* the full-cache comparator (FKV): bound above s + D, outputs only, also
  with decode steps over more than 4097 entries (the split decode path);
* a cut of more than 4096 live entries (streaming select) under the paper's
  rule;
* the host-side guard against ranking by scores that a block did not add to.
"""
import sys

import pytest
import torch

from paper_2412_05693_amd import synth

pytestmark = pytest.mark.gpu

C2 = synth.WORKLOADS["c2"]


def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _run(wl, checked, **kw):
    _need_gpu()
    from pd_harness import run_parity

    print(f"[parity] {wl.name} dtype={wl.dtype} b={wl.b} H={wl.n_heads}/{wl.n_kv_heads} "
          f"d={wl.head_dim} s={wl.s} kv={wl.kv_max} B={wl.block} D={wl.n_decode} "
          f"units={len(checked)} {kw}", flush=True)
    st = run_parity(wl, checked, **kw)
    print(f"[parity] -> {st.summary()}", flush=True)
    sys.stdout.flush()
    assert not st.failures, "\n".join(st.failures)
    return st


def test_sum_rule_c2_shape():
    wl = C2.with_(b=2, s=1024, n_decode=24)
    st = _run(wl, synth.checked_units(wl, wl.units), rule="sum")
    assert st.cuts == wl.units * (1024 // 256 - 512 // 256 + 24)


def test_sum_rule_ragged_fp32_literal_decode():
    wl = C2.with_(name="ragged", hh_mode="scatter", n_sinks=4, dtype="f32", b=2, n_heads=8,
                  n_kv_heads=2, head_dim=128, s=200, kv_max=70, block=33, n_decode=9)
    _run(wl, synth.checked_units(wl, wl.units), rule="sum", decode_p=4)


def test_ed_algorithm_3_ragged():
    wl = C2.with_(name="ragged", hh_mode="scatter", n_sinks=4, b=2, n_heads=8, n_kv_heads=4,
                  head_dim=64, s=300, kv_max=300, block=48, n_decode=10)
    st = _run(wl, synth.checked_units(wl, wl.units), rule="recent", decode_bound=2, decode_p=1,
              accumulate=False)
    assert st.cuts == wl.units * wl.n_decode


def test_ed_algorithm_3_long_prompt():
    wl = C2.with_(b=1, s=8192, kv_max=8192, block=256, n_decode=4)
    st = _run(wl, synth.checked_units(wl, 2), rule="recent", decode_bound=2, decode_p=1,
              accumulate=False)
    assert st.cuts == 2 * wl.n_decode


def test_fkv_outputs_only():
    wl = C2.with_(b=2, s=600, kv_max=700, block=256, n_decode=10)
    st = _run(wl, synth.checked_units(wl, wl.units), accumulate=False)
    assert st.cuts == 0


def test_fkv_long_decode_bf16():
    # decode steps over 4201..4208 entries: the split outputs-only path
    wl = C2.with_(b=1, s=4200, kv_max=4208, block=256, n_decode=8)
    st = _run(wl, synth.checked_units(wl, 2), accumulate=False)
    assert st.cuts == 0


def test_fkv_long_decode_fp32_d64_g2():
    wl = C2.with_(name="ragged", hh_mode="scatter", n_sinks=4, dtype="f32", b=1, n_heads=4,
                  n_kv_heads=2, head_dim=64, s=4500, kv_max=4505, block=300, n_decode=5)
    st = _run(wl, synth.checked_units(wl, wl.units), accumulate=False)
    assert st.cuts == 0


def test_long_decode_needs_outputs_only():
    _need_gpu()
    from pd_harness import make_pd
    from paper_2412_05693_amd.batchmax import BM_ERR_UNSUPPORTED, BatchMaxError

    wl = C2.with_(b=1, s=4200, kv_max=4208, block=512, n_decode=2)
    q, k, v = synth.batch_inputs(wl, "cuda")
    o = torch.zeros_like(q)
    pd = make_pd(wl)
    for t0 in range(0, wl.s, wl.block):
        n = min(wl.block, wl.s - t0)
        pd.prefill_block(t0, n, q, k, v, o)
        pd.evict_compact(t0 + n - 1)
    with pytest.raises(BatchMaxError) as e:      # scores on: refused before any launch
        pd.decode_step(wl.s, q, k, v, o, row=wl.s)
    assert e.value.status == BM_ERR_UNSUPPORTED
    torch.cuda.synchronize()
    assert pd.length == wl.s


def test_streaming_select_large_cache():
    # cap = 4512 > 4096 slots: every prefill cut streams its keys
    wl = C2.with_(b=1, n_heads=4, n_kv_heads=1, s=6000, kv_max=4000, block=512, n_decode=4)
    st = _run(wl, synth.checked_units(wl, wl.units))
    assert st.cuts == 5 + 4     # after blocks 7..11 (4096 > 4000 first), then every step


def test_unaccumulated_scores_reject_score_ranked_cut():
    _need_gpu()
    from pd_harness import make_pd
    from paper_2412_05693_amd.batchmax import BM_ERR_ORDER, BatchMaxError

    wl = C2.with_(b=1, s=256, kv_max=64, block=128, n_decode=0)
    q, k, v = synth.batch_inputs(wl, "cuda")
    o = torch.zeros_like(q)
    pd = make_pd(wl)
    pd.set_score_accumulation(False)
    pd.reset()                      # settings survive a new context
    pd.prefill_block(0, 128, q, k, v, o)
    with pytest.raises(BatchMaxError) as e:
        pd.evict_compact(127)
    assert e.value.status == BM_ERR_ORDER
    assert pd.length == 128
    pd.set_rank_rule("recent")
    pd.evict_compact(127)
    torch.cuda.synchronize()
    assert pd.length == 64
    assert sorted(pd.pos[0, 0, :64].tolist()) == list(range(64, 128))
    # both settings again after a reset: accumulation still off, rule still recent
    pd.reset()
    pd.prefill_block(0, 128, q, k, v, o)
    pd.evict_compact(127)
    torch.cuda.synchronize()
    assert sorted(pd.pos[0, 0, :64].tolist()) == list(range(64, 128))


# --- left padding (Sec. 3): per-sample prompt lengths s_j = s - pad_j -------------
@pytest.mark.parametrize("case", [
    # pads below, across and beyond the first cut; one sample unpadded, one by pad_max
    dict(dtype="bf16", b=4, n_heads=32, n_kv_heads=8, head_dim=128, s=1024, kv_max=512,
         block=256, n_decode=16, pad_max=700),
    dict(dtype="bf16", b=3, n_heads=8, n_kv_heads=4, head_dim=64, s=300, kv_max=100, block=48,
         n_decode=12, pad_max=250),
    dict(dtype="f32", b=3, n_heads=8, n_kv_heads=2, head_dim=128, s=200, kv_max=70, block=33,
         n_decode=7, pad_max=150),
], ids=lambda c: f"{c['dtype']}-d{c['head_dim']}-s{c['s']}-kv{c['kv_max']}-pad{c['pad_max']}")
def test_left_padding_all_units(case):
    wl = C2.with_(name="padded", hh_mode="scatter", n_sinks=4, **case)
    st = _run(wl, synth.checked_units(wl, wl.units))
    assert st.cuts > 0


def test_left_padding_with_literal_decode_and_long_prompt_pad():
    # a sample padded for most of the prompt: pads fill whole cache tiles
    wl = C2.with_(name="padded", b=3, s=2048, kv_max=512, block=256, n_decode=70, pad_max=1900)
    _run(wl, synth.checked_units(wl, wl.units), decode_p=64)


def test_left_padding_full_cache_long_decode():
    # FKV with padding: K6 masks pad entries too (decode over 4201+ entries)
    wl = C2.with_(name="padded", b=2, n_heads=8, n_kv_heads=2, s=4200, kv_max=4208, block=256,
                  n_decode=6, pad_max=3000)
    st = _run(wl, synth.checked_units(wl, wl.units), accumulate=False)
    assert st.cuts == 0


# --- TOVA: the last processed query alone ranks the entries -----------------------
def test_tova_rule_c2_shape():
    wl = C2.with_(b=2, s=1024, n_decode=24)
    st = _run(wl, synth.checked_units(wl, wl.units), rule="tova")
    assert st.cuts == wl.units * (1024 // 256 - 512 // 256 + 24)


@pytest.mark.parametrize("case", [
    dict(dtype="f32", b=2, n_heads=8, n_kv_heads=2, head_dim=128, s=200, kv_max=70, block=33,
         n_decode=9),
    dict(dtype="bf16", b=3, n_heads=8, n_kv_heads=4, head_dim=64, s=300, kv_max=100, block=48,
         n_decode=12, pad_max=250),
], ids=lambda c: f"{c['dtype']}-d{c['head_dim']}-pad{c.get('pad_max', 0)}")
def test_tova_rule_ragged_literal_decode(case):
    # the literal schedule's pre-cut ranks by the previous step's weights
    wl = C2.with_(name="ragged", hh_mode="scatter", n_sinks=4, **case)
    _run(wl, synth.checked_units(wl, wl.units), rule="tova", decode_p=4)


def test_decode_bound_below_prefill_bound_one_removal_per_step():
    # the first decode step cuts 512 -> 300 at the last processed position (seen
    # only through the end state, so the sharp inputs keep near-ties away), then
    # one removal per step keeps 300
    wl = C2.with_(b=2, s=1024, n_decode=12)
    st = _run(wl, synth.checked_units(wl, wl.units), sharp=True, decode_bound=300)
    assert st.cuts == wl.units * (1024 // 256 - 512 // 256 + 12)


def test_ed_algorithm_3_with_left_padding():
    wl = C2.with_(name="padded", hh_mode="scatter", n_sinks=4, b=3, n_heads=8, n_kv_heads=4,
                  head_dim=64, s=300, kv_max=300, block=48, n_decode=8, pad_max=200)
    st = _run(wl, synth.checked_units(wl, wl.units), rule="recent", decode_bound=2, decode_p=1,
              accumulate=False)
    assert st.cuts == wl.units * wl.n_decode


# --- a block and its cut in one call (fold + select + compaction fused) -----------
@pytest.mark.parametrize("case", [
    dict(name="c2-reduced", b=2, s=1024, n_decode=8),
    dict(name="ragged", hh_mode="scatter", n_sinks=4, dtype="f32", b=2, n_heads=8, n_kv_heads=2,
         head_dim=128, s=200, kv_max=70, block=33, n_decode=5),
    dict(name="ragged", hh_mode="scatter", n_sinks=4, dtype="bf16", b=3, n_heads=8,
         n_kv_heads=4, head_dim=64, s=300, kv_max=100, block=48, n_decode=5, pad_max=250),
    # exactly 4096 live entries before each cut: the fused kernel's largest LDS
    # footprint (80 KB of slot arrays)
    dict(name="edge", b=2, n_heads=8, n_kv_heads=2, s=4352, kv_max=3840, block=256, n_decode=3),
    # more than 4096 live entries: the call falls back to the separate kernels
    dict(name="large", b=1, n_heads=4, n_kv_heads=1, s=6000, kv_max=4000, block=512, n_decode=2),
], ids=lambda c: f"{c['name']}-{c.get('dtype', 'bf16')}-kv{c.get('kv_max', 512)}")
def test_fused_block_cut(case):
    wl = C2.with_(**case)
    st = _run(wl, synth.checked_units(wl, wl.units), fused_cut=True)
    assert st.cuts > 0


@pytest.mark.parametrize("rule", ["sum", "tova"])
def test_fused_block_cut_other_rules(rule):
    wl = C2.with_(b=2, s=1024, n_decode=8)
    _run(wl, synth.checked_units(wl, wl.units), fused_cut=True, rule=rule)


def test_fused_block_cut_outputs_only_recent_rule():
    # outputs-only prefill (no score sums) with cuts by recency inside the
    # fused call: the kernel folds nothing and keeps the newest entries
    wl = C2.with_(name="ragged", hh_mode="scatter", n_sinks=4, b=2, n_heads=8, n_kv_heads=2,
                  head_dim=128, s=300, kv_max=100, block=48, n_decode=4)
    st = _run(wl, synth.checked_units(wl, wl.units), fused_cut=True, rule="recent",
              accumulate=False)
    assert st.cuts > 0


def test_fused_block_cut_c3_shape():
    # block 512 and bound 1024: 16 workgroups per unit fold into each cut
    wl = synth.WORKLOADS["c3"].with_(b=2, s=2048, n_decode=4)
    st = _run(wl, synth.checked_units(wl, wl.units), fused_cut=True)
    assert st.cuts > 0
