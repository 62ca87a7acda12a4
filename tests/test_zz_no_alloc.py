"""bm_init_static_workspace: a context whose workspace is the library's static
device array instead of a caller-allocated buffer gives exactly the results of
bm_init's context on the same inputs -- on two runs in a row, the second with a
smaller batch and prompt (the array keeps the first run's contents) -- and a
workspace beyond the static size is refused before any device work."""
import pytest
import torch

from paper_2412_05693_amd import batchmax as bmx
from paper_2412_05693_amd import synth

pytestmark = pytest.mark.gpu


def _pd_run(wl, inputs, static, fused_cut):
    q, k, v = inputs
    o = torch.zeros_like(q)
    pd = bmx.PDAttention(b=wl.b, s=wl.s, kv_max=wl.kv_max, block=wl.block, max_gen=wl.n_decode,
                         n_heads=wl.n_heads, n_kv_heads=wl.n_kv_heads, head_dim=wl.head_dim,
                         dtype=wl.dtype, sm_scale=wl.sm_scale, device="cuda",
                         static_workspace=static)
    assert (pd.work is None) == static
    pd.run_prefill(q, k, v, o, fused_cut=fused_cut)
    pd.run_decode(q, k, v, o)
    torch.cuda.synchronize()
    L = pd.length
    out = (o.clone(), pd.len.clone(), pd.pos[..., :L].clone(), pd.score[..., :L].clone(),
           pd.k[..., :L, :].clone(), pd.v[..., :L, :].clone())
    pd.close()
    return out


@pytest.mark.parametrize("fused_cut", [False, True])
def test_static_workspace_matches_caller_workspace(fused_cut):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(0)
    c2 = synth.WORKLOADS["c2"]
    # the larger run first, then a smaller one over the array it left behind
    for wl in (c2.with_(b=6, s=1536, n_decode=40), c2.with_(b=2, s=700, kv_max=300, n_decode=24)):
        print(f"[no-alloc] b={wl.b} s={wl.s} kv={wl.kv_max} B={wl.block} D={wl.n_decode} "
              f"fused_cut={fused_cut} workspace={bmx.bm_workspace_bytes(bmx.make_dims(b=wl.b, s=wl.s, kv_max=wl.kv_max, block=wl.block, max_gen=wl.n_decode, n_heads=wl.n_heads, n_kv_heads=wl.n_kv_heads, head_dim=wl.head_dim, dtype=wl.dtype))}",
              flush=True)
        inputs = synth.batch_inputs(wl, "cuda")
        ref = _pd_run(wl, inputs, static=False, fused_cut=fused_cut)
        got = _pd_run(wl, inputs, static=True, fused_cut=fused_cut)
        names = ("o", "len", "pos", "score", "k", "v")
        for nm, a, b in zip(names, ref, got):
            assert torch.equal(a, b), f"{nm} differs (b={wl.b})"


def test_static_workspace_refuses_large_dims():
    d = bmx.make_dims(b=1024, s=2048, kv_max=512, block=256, max_gen=8, n_heads=32,
                      n_kv_heads=8, head_dim=128, dtype="bf16")
    assert bmx.bm_workspace_bytes(d) > (64 << 20)
    c = bmx.bm_cache(1 << 40, 1 << 40, 1 << 40, 1 << 40, 1 << 40, 0, 0)
    with pytest.raises(bmx.BatchMaxError) as e:
        bmx.bm_init_static_workspace(d, c, 0)
    assert e.value.status == bmx.BM_ERR_UNSUPPORTED
    assert "static workspace" in bmx.bm_last_error()
