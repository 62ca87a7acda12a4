"""GPU: a seeded sweep of small random shapes against the float64 oracle.

Each case draws the dtype, head size, group size, batch, block, bound, prompt
length, decode steps, ranking rule, decode removal, left padding and whether
each block is cut in the same call, and checks every unit of the run.
"""
import sys

import numpy as np
import pytest
import torch

from paper_2412_05693_amd import synth

pytestmark = pytest.mark.gpu

RULES = ("ave", "sum", "recent", "tova")


def _cases(n=64, seed=2412):
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n):
        g = int(rng.choice([1, 2, 4]))
        hk = int(rng.integers(1, 3))
        s = int(rng.integers(1, 521))
        kv = int(rng.integers(1, 261))
        block = int(min(s, max(1, round(float(np.exp(rng.uniform(0, np.log(160))))))))
        n_decode = int(rng.integers(0, 7))
        p = int(rng.integers(1, kv + 1)) if rng.random() < 0.3 else 0
        pad = int(rng.integers(1, s // 2 + 1)) if s >= 4 and rng.random() < 0.3 else 0
        out.append(dict(
            id=i, dtype=str(rng.choice(["bf16", "f32"])), head_dim=int(rng.choice([64, 128])),
            n_heads=g * hk, n_kv_heads=hk, b=int(rng.integers(1, 4)), s=s, kv_max=kv,
            block=block, n_decode=n_decode, pad_max=pad, rule=str(rng.choice(RULES)),
            decode_p=p, fused_cut=bool(rng.random() < 0.5)))
    return out


@pytest.mark.parametrize("case", _cases(), ids=lambda c: f"case{c['id']}")
def test_random_shape(case):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from pd_harness import run_parity

    c = dict(case)
    kw = dict(rule=c.pop("rule"), decode_p=c.pop("decode_p"), fused_cut=c.pop("fused_cut"))
    c.pop("id")
    wl = synth.WORKLOADS["c2"].with_(name="sweep", **c)
    print(f"[sweep] {c} {kw}", flush=True)
    sys.stdout.flush()
    st = run_parity(wl, synth.checked_units(wl, wl.units), **kw)
    print(f"[sweep] -> {st.summary()}", flush=True)
    assert not st.failures, "\n".join(st.failures)
