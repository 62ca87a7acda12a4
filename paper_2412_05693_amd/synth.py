"""Seeded synthetic workloads for P&D KV-compressed attention.

This module only draws inputs; it holds none of the method's arithmetic, and it
is the one piece that both the HIP path's harness and the CPU oracle's tests
use.  It never imports the oracle or the native library.

Recipe (stand-in for the long-input, short-output tasks of Sec. 4 -- CNN/DM,
NarrativeQA, GSM8K -- whose data and model weights are not used here):

* Q, K, V elements are N(0, 1) / sqrt(d), drawn in float64 by numpy's PCG64 and
  rounded once to float32.
* Heavy hitters: a share of the *prompt* key positions has its K rows scaled
  (x4) in float32; "sink" positions 0..3 are scaled x6.  Decode-step inputs
  are never scaled.  The positions are shared by every KV head of a sample.
* bf16 workloads round the float32 values to bf16 (round to nearest even)
  once, on the host; both sides then see exactly those values.

Per-unit streams: the unit (layer, sample, kv_head) draws, in this order,
K[s+D, d], V[s+D, d], Q[G, s+D, d] from
``PCG64(SeedSequence([seed, 0, layer, sample, kv_head]))``; heavy-hitter
positions come from ``SeedSequence([seed, 1, layer, sample])``.  Bulk units of
large configurations are drawn on the device with ``torch.randn`` (timing
only, same distributions and the same heavy-hitter positions); checked units
are overwritten with the host stream so the oracle can reproduce them.

The 32-layer stack (c5) cannot hold its prompt inputs (3.2 GB per sample), so
its Q/K/V come from a counter-based stream that the device evaluates per block
and this module evaluates for checked units: Philox4x32-10 (Salmon, Moraes,
Dror and Shaw, "Parallel random numbers: as easy as 1, 2, 3", SC 2011).  Each
call yields two elements; an element is the Irwin-Hall sum S of four 16-bit
uniforms, z = (S - 131070) * c with c = float32(sqrt(3) / sqrt(d) / 65536)
(mean 0, variance 1/d; every step but the final multiply is exact in float32,
and that multiply is correctly rounded on both sides).  A prompt position
p >= n_sinks carries heavy-hitter keys when its selector word is below
hh_frac * 2^32 (a Bernoulli draw per position, shared by the sample's KV
heads); sinks and heavy hitters scale K as above.  Counter words: (pos * d/2 +
pair, tensor << 8 | head, sample, layer) with tensor 0 = Q, 1 = K, 2 = V, 3 =
selector; key (seed, 0).
"""
from __future__ import annotations

from dataclasses import dataclass, replace

import numpy as np


@dataclass(frozen=True)
class Workload:
    name: str
    dtype: str            # "f32" or "bf16"
    b: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    s: int                # prompt length
    kv_max: int           # cache bound |kv|-bar
    block: int            # prefill block (the paper's p)
    n_decode: int         # decode steps
    hh_mode: str          # "scatter", "spans" or "none"
    hh_frac: float = 0.02
    hh_scale: float = 4.0
    n_sinks: int = 0
    sink_scale: float = 6.0
    n_spans: int = 8
    span_len: int = 64
    n_layers: int = 1
    seed: int = 1
    decode_p: int = 0     # 0: one removal per decode step; p > 0: Algorithm 1's p at once
    rule: str = "ave"     # ranking rule of a cut: "ave", "sum" or "recent"
    decode_bound: int = 0  # cache bound during decode (0: kv_max)
    accumulate: bool = True  # score sums during prefill
    pad_max: int = 0      # left padding: sample j has pads[j] in [0, pad_max] pad tokens

    @property
    def group(self) -> int:
        return self.n_heads // self.n_kv_heads

    @property
    def units(self) -> int:
        return self.b * self.n_kv_heads

    @property
    def total(self) -> int:
        return self.s + self.n_decode

    @property
    def sm_scale(self) -> float:
        return 1.0 / float(np.sqrt(self.head_dim))

    def with_(self, **kw) -> "Workload":
        return replace(self, **kw)


# The five workloads of the benchmark suite.  c4's prefill block is not given
# by the workload statement; 256 (as in c2 and c5) is used.
WORKLOADS = {
    "c1": Workload("c1-fp32-mha-b2-s512", "f32", b=2, n_heads=4, n_kv_heads=4, head_dim=64,
                   s=512, kv_max=128, block=64, n_decode=32, hh_mode="scatter", seed=1),
    "c2": Workload("c2-llama3-8b-layer-b64-s4096", "bf16", b=64, n_heads=32, n_kv_heads=8,
                   head_dim=128, s=4096, kv_max=512, block=256, n_decode=128,
                   hh_mode="scatter", n_sinks=4, seed=2),
    "c3": Workload("c3-long-prefill-b128-s16384", "bf16", b=128, n_heads=32, n_kv_heads=8,
                   head_dim=128, s=16384, kv_max=1024, block=512, n_decode=64,
                   hh_mode="spans", n_sinks=4, seed=3),
    "c4": Workload("c4-decode-heavy-b1024-s2048", "bf16", b=1024, n_heads=32, n_kv_heads=8,
                   head_dim=128, s=2048, kv_max=512, block=256, n_decode=512,
                   hh_mode="scatter", n_sinks=4, seed=4),
    "c5": Workload("c5-llama3-8b-32layer-s8192", "bf16", b=0, n_heads=32, n_kv_heads=8,
                   head_dim=128, s=8192, kv_max=512, block=256, n_decode=256,
                   hh_mode="scatter", n_sinks=4, n_layers=32, seed=5),
}

# A supplementary "sharp" distribution: Q, K ~ N(0, 1) per element (no 1/sqrt(d)),
# which spreads the averages apart so kept-set comparisons are discriminating.
SHARP_SEED = 101


# ---------------------------------------------------------------------------
# bf16 helpers (input preparation only)
# ---------------------------------------------------------------------------
def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 (nearest, ties to even); return uint16 bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    rounded = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return rounded.astype(np.uint16)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def round_to_dtype(x: np.ndarray, dtype: str) -> np.ndarray:
    """float32 values exactly representable in the workload's element type."""
    x = np.asarray(x, dtype=np.float32)
    if dtype == "f32":
        return x
    if dtype == "bf16":
        return bf16_bits_to_f32(f32_to_bf16_bits(x))
    raise ValueError(dtype)


# ---------------------------------------------------------------------------
# heavy hitters and sinks
# ---------------------------------------------------------------------------
def heavy_positions(wl: Workload, layer: int, sample: int) -> np.ndarray:
    """Prompt positions whose keys are scaled by ``hh_scale`` (sorted, unique)."""
    if wl.hh_mode == "none":
        return np.zeros(0, dtype=np.int64)
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([wl.seed, 1, layer, sample])))
    lo = wl.n_sinks
    if wl.hh_mode == "scatter":
        count = int(round(wl.hh_frac * wl.s))
        pos = rng.choice(np.arange(lo, wl.s), size=count, replace=False)
        return np.sort(pos).astype(np.int64)
    if wl.hh_mode == "spans":
        # n_spans non-overlapping spans: one random span per equal segment of [lo, s)
        seg = (wl.s - lo) // wl.n_spans
        if seg < wl.span_len:
            raise ValueError("prompt too short for the requested spans")
        out = []
        for i in range(wl.n_spans):
            start = lo + i * seg + int(rng.integers(0, seg - wl.span_len + 1))
            out.append(np.arange(start, start + wl.span_len))
        return np.concatenate(out).astype(np.int64)
    raise ValueError(wl.hh_mode)


def key_scale_profile(wl: Workload, layer: int, sample: int) -> np.ndarray:
    """Per-position multiplier of K rows: 1, hh_scale or sink_scale ([s + D])."""
    prof = np.ones(wl.total, dtype=np.float32)
    prof[heavy_positions(wl, layer, sample)] = np.float32(wl.hh_scale)
    prof[: wl.n_sinks] = np.float32(wl.sink_scale)
    return prof


# ---------------------------------------------------------------------------
# per-unit host streams (checked units)
# ---------------------------------------------------------------------------
def unit_inputs(wl: Workload, layer: int, sample: int, kv_head: int, sharp: bool = False):
    """Inputs of one unit as float32 arrays exactly representable in wl.dtype.

    Returns q [G, s+D, d], k [s+D, d], v [s+D, d].
    """
    d, T, G = wl.head_dim, wl.total, wl.group
    seed = SHARP_SEED if sharp else wl.seed
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 0, layer, sample, kv_head])))
    k = rng.standard_normal((T, d))
    v = rng.standard_normal((T, d))
    q = rng.standard_normal((G, T, d))
    scale = 1.0 / np.sqrt(d)
    v = (v * scale).astype(np.float32)
    if sharp:
        k = k.astype(np.float32)
        q = q.astype(np.float32)
    else:
        k = (k * scale).astype(np.float32)
        q = (q * scale).astype(np.float32)
        k = k * key_scale_profile(wl, layer, sample)[:, None]
    return (round_to_dtype(q, wl.dtype), round_to_dtype(k, wl.dtype), round_to_dtype(v, wl.dtype))


def sample_pads(wl: Workload) -> np.ndarray:
    """Left pad tokens per sample (Sec. 3: sample j's prompt is s_j = s - pad_j
    tokens long): uniform on [0, pad_max], sample 0 unpadded and the last
    sample padded by exactly pad_max; zeros without padding."""
    pads = np.zeros(wl.b, dtype=np.int32)
    if wl.pad_max <= 0:
        return pads
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([wl.seed, 5])))
    pads[:] = rng.integers(0, wl.pad_max + 1, size=wl.b)
    pads[0] = 0
    if wl.b > 1:
        pads[-1] = wl.pad_max
    return pads


def checked_units(wl: Workload, count: int, seed: int = 0) -> list:
    """A seeded sample of (sample, kv_head) units that always holds the first and
    the last unit; all units when ``count`` covers them."""
    U = wl.units
    if count >= U:
        return [(u // wl.n_kv_heads, u % wl.n_kv_heads) for u in range(U)]
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([wl.seed, 2, seed])))
    pick = set([0, U - 1])
    rest = rng.choice(np.arange(1, U - 1), size=count - 2, replace=False)
    pick.update(int(x) for x in rest)
    return [(u // wl.n_kv_heads, u % wl.n_kv_heads) for u in sorted(pick)]


# ---------------------------------------------------------------------------
# full-batch tensors (torch; device or CPU)
# ---------------------------------------------------------------------------
def batch_inputs(wl: Workload, device, layer: int = 0, checked=(), sharp: bool = False,
                 gen_seed: int | None = None):
    """q [b, H, s+D, d], k/v [b, Hk, s+D, d] in the workload's dtype.

    Bulk values come from ``torch.randn`` under a seeded generator on
    ``device``; units listed in ``checked`` (pairs (sample, kv_head)) are
    overwritten with their host stream (``unit_inputs``).
    """
    import torch

    tdt = torch.float32 if wl.dtype == "f32" else torch.bfloat16
    b, H, Hk, d, T, G = wl.b, wl.n_heads, wl.n_kv_heads, wl.head_dim, wl.total, wl.group
    g = torch.Generator(device=device)
    g.manual_seed((gen_seed if gen_seed is not None else wl.seed) * 1000003 + layer)
    scale = 1.0 if sharp else 1.0 / float(np.sqrt(d))

    def draw(shape, s):
        x = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
        if s != 1.0:
            x.mul_(s)
        return x

    k = draw((b, Hk, T, d), scale)
    if not sharp:
        prof = np.stack([key_scale_profile(wl, layer, i) for i in range(b)])     # [b, T]
        k.mul_(torch.from_numpy(prof).to(device)[:, None, :, None])
    k = k.to(tdt)
    v = draw((b, Hk, T, d), 1.0 / float(np.sqrt(d))).to(tdt)
    q = draw((b, H, T, d), scale).to(tdt)
    for (bi, hk) in checked:
        uq, uk, uv = unit_inputs(wl, layer, bi, hk, sharp=sharp)
        q[bi, hk * G:(hk + 1) * G] = torch.from_numpy(uq).to(device=device, dtype=tdt)
        k[bi, hk] = torch.from_numpy(uk).to(device=device, dtype=tdt)
        v[bi, hk] = torch.from_numpy(uv).to(device=device, dtype=tdt)
    return q, k, v


# ---------------------------------------------------------------------------
# counter-based stream (Philox4x32-10) for the layer stack
# ---------------------------------------------------------------------------
PHILOX_M0, PHILOX_M1 = 0xD2511F53, 0xCD9E8D57      # round multipliers
PHILOX_W0, PHILOX_W1 = 0x9E3779B9, 0xBB67AE85      # key schedule (Weyl) increments
T_Q, T_K, T_V, T_SEL = 0, 1, 2, 3


def philox4x32_10(ctr: np.ndarray, key: np.ndarray) -> np.ndarray:
    """Philox4x32 with 10 rounds.  ctr [..., 4] and key [..., 2] (uint32,
    broadcastable) -> [..., 4] uint32.  A round maps (c0, c1, c2, c3) with
    (hi0, lo0) = M0 * c0 and (hi1, lo1) = M1 * c2 (64-bit products) to
    (hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0); the key grows by (W0, W1)
    between rounds."""
    ctr = np.asarray(ctr, dtype=np.uint32)
    key = np.asarray(key, dtype=np.uint32)
    mask = np.uint64(0xFFFFFFFF)
    c0, c1, c2, c3 = (ctr[..., i].astype(np.uint64) for i in range(4))
    k0 = key[..., 0].astype(np.uint64)
    k1 = key[..., 1].astype(np.uint64)
    for _ in range(10):
        p0 = c0 * np.uint64(PHILOX_M0)
        p1 = c2 * np.uint64(PHILOX_M1)
        c0, c1, c2, c3 = ((p1 >> np.uint64(32)) ^ c1 ^ k0, p1 & mask,
                          (p0 >> np.uint64(32)) ^ c3 ^ k1, p0 & mask)
        k0 = (k0 + np.uint64(PHILOX_W0)) & mask
        k1 = (k1 + np.uint64(PHILOX_W1)) & mask
    return np.stack([c0, c1, c2, c3], axis=-1).astype(np.uint32)


def stack_value_scale(head_dim: int) -> np.float32:
    """c = float32(sqrt(3) / sqrt(d) / 65536): the Irwin-Hall sum of four 16-bit
    uniforms has variance 4 * 65536^2 / 12, so (S - mean) * c has variance 1/d."""
    return np.float32(np.sqrt(3.0) / np.sqrt(head_dim) / 65536.0)


def stack_hh_threshold(wl: Workload) -> int:
    return int(round(wl.hh_frac * 2.0 ** 32)) if wl.hh_mode != "none" else 0


def _stack_values(wl: Workload, layer: int, sample: int, tensor: int, head: int,
                  positions: np.ndarray) -> np.ndarray:
    """float32 [len(positions), d] elements of one (tensor, head) row range."""
    d = wl.head_dim
    pair = np.arange(d // 2, dtype=np.uint64)
    j = (positions.astype(np.uint64)[:, None] * np.uint64(d // 2) + pair[None, :])
    ctr = np.zeros(j.shape + (4,), dtype=np.uint32)
    ctr[..., 0] = j.astype(np.uint32)
    ctr[..., 1] = (tensor << 8) | head
    ctr[..., 2] = sample
    ctr[..., 3] = layer
    w = philox4x32_10(ctr, np.array([wl.seed, 0], dtype=np.uint32)).astype(np.uint32)  # [T, d/2, 4]
    lo, hi = w & np.uint32(0xFFFF), w >> np.uint32(16)
    s0 = lo[..., 0] + hi[..., 0] + lo[..., 1] + hi[..., 1]      # element 2 * pair
    s1 = lo[..., 2] + hi[..., 2] + lo[..., 3] + hi[..., 3]      # element 2 * pair + 1
    S = np.stack([s0, s1], axis=-1).reshape(len(positions), d)
    c = stack_value_scale(d)
    return (S.astype(np.float32) - np.float32(131070.0)) * c


def stack_key_factor(wl: Workload, layer: int, sample: int, positions: np.ndarray) -> np.ndarray:
    """float32 multiplier of the K row at each position (1, hh_scale or sink_scale)."""
    positions = np.asarray(positions, dtype=np.int64)
    ctr = np.zeros(positions.shape + (4,), dtype=np.uint32)
    ctr[..., 0] = positions.astype(np.uint32)
    ctr[..., 1] = T_SEL << 8
    ctr[..., 2] = sample
    ctr[..., 3] = layer
    sel = philox4x32_10(ctr, np.array([wl.seed, 0], dtype=np.uint32))[..., 0]
    f = np.ones(positions.shape, dtype=np.float32)
    prompt = positions < wl.s
    heavy = prompt & (positions >= wl.n_sinks) & (sel.astype(np.uint64) < np.uint64(stack_hh_threshold(wl)))
    f[heavy] = np.float32(wl.hh_scale)
    f[prompt & (positions < wl.n_sinks)] = np.float32(wl.sink_scale)
    return f


def stack_unit_inputs(wl: Workload, layer: int, sample: int, kv_head: int):
    """Counter-stream inputs of one unit of the layer stack, float32 arrays exactly
    representable in wl.dtype: q [G, s+D, d], k [s+D, d], v [s+D, d]."""
    pos = np.arange(wl.total, dtype=np.int64)
    G = wl.group
    k = _stack_values(wl, layer, sample, T_K, kv_head, pos)
    k = k * stack_key_factor(wl, layer, sample, pos)[:, None]
    v = _stack_values(wl, layer, sample, T_V, kv_head, pos)
    q = np.stack([_stack_values(wl, layer, sample, T_Q, kv_head * G + g, pos) for g in range(G)])
    return (round_to_dtype(q, wl.dtype), round_to_dtype(k, wl.dtype), round_to_dtype(v, wl.dtype))
