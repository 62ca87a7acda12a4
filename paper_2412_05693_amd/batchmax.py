"""Thin ctypes binding of ``libbatchmax.so`` (include/batchmax.h).

The functions named ``bm_*`` mirror the C ABI one to one: they marshal
arguments (integers, pointers as Python ints, ctypes structs) and raise
``BatchMaxError`` on a non-OK status.  Every step of the path runs in the HIP
kernels behind the library; nothing here computes.

``PDAttention`` is a convenience owner of the cache tensors (torch allocates the
device memory; the library never does) that checks dtype, device, shape and
contiguity before handing raw pointers and the current HIP stream to the ABI.

Importing this module loads the library and fails loudly if it is missing:
there is no fallback path.
"""
from __future__ import annotations

import ctypes
import math
import os

HERE = os.path.dirname(os.path.abspath(__file__))
# BATCHMAX_LIB selects another build of the same library (the host-sanitizer
# build of build.py --sanitize, for CPU tests); the default is the in-tree one
LIB_PATH = os.environ.get("BATCHMAX_LIB") or os.path.join(HERE, "libbatchmax.so")

BM_OK, BM_ERR_INVALID_ARG, BM_ERR_UNSUPPORTED, BM_ERR_CAPACITY, BM_ERR_ORDER, BM_ERR_HIP = range(6)
BM_F32, BM_BF16 = 0, 1
BM_RANK_AVE, BM_RANK_SUM, BM_RANK_RECENT, BM_RANK_TOVA = 0, 1, 2, 3
RANK_RULES = {"ave": BM_RANK_AVE, "sum": BM_RANK_SUM, "recent": BM_RANK_RECENT,
              "tova": BM_RANK_TOVA}
STATUS_NAMES = {0: "BM_OK", 1: "BM_ERR_INVALID_ARG", 2: "BM_ERR_UNSUPPORTED",
                3: "BM_ERR_CAPACITY", 4: "BM_ERR_ORDER", 5: "BM_ERR_HIP"}


class BatchMaxError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {message}")
        self.status = status


class bm_dims(ctypes.Structure):
    _fields_ = [("b", ctypes.c_int32), ("s", ctypes.c_int32), ("kv_max", ctypes.c_int32),
                ("block", ctypes.c_int32), ("max_gen", ctypes.c_int32),
                ("n_heads", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("dtype", ctypes.c_int32),
                ("sm_scale", ctypes.c_float)]


class bm_synth(ctypes.Structure):
    _fields_ = [("b", ctypes.c_int32), ("n_heads", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("dtype", ctypes.c_int32), ("seed", ctypes.c_uint32),
                ("layer", ctypes.c_int32), ("s", ctypes.c_int32), ("hh_threshold", ctypes.c_uint32),
                ("hh_scale", ctypes.c_float), ("n_sinks", ctypes.c_int32),
                ("sink_scale", ctypes.c_float), ("value_scale", ctypes.c_float)]


class bm_cache(ctypes.Structure):
    _fields_ = [("k", ctypes.c_void_p), ("v", ctypes.c_void_p), ("score", ctypes.c_void_p),
                ("pos", ctypes.c_void_p), ("len", ctypes.c_void_p), ("work", ctypes.c_void_p),
                ("work_bytes", ctypes.c_size_t)]


def _load() -> ctypes.CDLL:
    # torch ships its own HIP runtime under the same soname as ROCm's; load it
    # first so this library binds to that single runtime instead of a second copy
    import torch  # noqa: F401

    if not os.path.exists(LIB_PATH):
        raise ImportError(
            f"{LIB_PATH} is not built; run `python -m paper_2412_05693_amd.build` "
            "(there is no non-HIP fallback)")
    lib = ctypes.CDLL(LIB_PATH)
    P, I32, SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
    dims_p, cache_p = ctypes.POINTER(bm_dims), ctypes.POINTER(bm_cache)
    sig = {
        "bm_abi_version": (ctypes.c_int, []),
        "bm_last_error": (ctypes.c_char_p, []),
        "bm_cache_slots": (I32, [dims_p]),
        "bm_workspace_bytes": (SZ, [dims_p]),
        "bm_prefill_positions_per_workgroup": (I32, [dims_p]),
        "bm_validate_dims": (ctypes.c_int, [dims_p]),
        "bm_init": (ctypes.c_int, [dims_p, cache_p, P, ctypes.POINTER(P)]),
        "bm_init_static_workspace": (ctypes.c_int, [dims_p, cache_p, P, ctypes.POINTER(P)]),
        "bm_resume": (ctypes.c_int, [dims_p, cache_p, I32, I32, ctypes.POINTER(P)]),
        "bm_prefill_block": (ctypes.c_int, [P, I32, I32, P, P, P, P, I32, P]),
        "bm_prefill_block_cut": (ctypes.c_int, [P, I32, I32, P, P, P, P, I32, P]),
        "bm_evict_compact": (ctypes.c_int, [P, I32, P]),
        "bm_set_decode_removal": (ctypes.c_int, [P, I32]),
        "bm_set_rank_rule": (ctypes.c_int, [P, I32]),
        "bm_set_decode_bound": (ctypes.c_int, [P, I32]),
        "bm_set_score_accumulation": (ctypes.c_int, [P, I32]),
        "bm_set_left_padding": (ctypes.c_int, [P, P]),
        "bm_set_split_event": (ctypes.c_int, [P, P]),
        "bm_decode_step": (ctypes.c_int, [P, I32, P, P, P, P, I32, P]),
        "bm_ctx_len": (I32, [P]),
        "bm_ctx_next_pos": (I32, [P]),
        "bm_destroy": (None, [P]),
        "bm_synth_qkv": (ctypes.c_int, [ctypes.POINTER(bm_synth), I32, I32, P, P, P, I32, P]),
        "bm_philox4x32_10": (ctypes.c_int, [P, P, ctypes.c_int64, P]),
        "bm_probe_stream_read": (ctypes.c_int, [P, SZ, P, I32, I32, P]),
        "bm_probe_mfma": (ctypes.c_int, [I32, P, I32, P]),
        "bm_prefill_timeline": (ctypes.c_int, [P, I32]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    return lib


_lib = _load()
EXPORTED = ("bm_abi_version", "bm_last_error", "bm_cache_slots", "bm_workspace_bytes",
            "bm_prefill_positions_per_workgroup",
            "bm_validate_dims", "bm_init", "bm_init_static_workspace", "bm_resume", "bm_prefill_block",
            "bm_prefill_block_cut", "bm_evict_compact",
            "bm_set_decode_removal", "bm_set_rank_rule", "bm_set_decode_bound",
            "bm_set_score_accumulation", "bm_set_left_padding", "bm_set_split_event",
            "bm_decode_step", "bm_ctx_len", "bm_ctx_next_pos", "bm_destroy", "bm_synth_qkv",
            "bm_philox4x32_10", "bm_probe_stream_read", "bm_probe_mfma",
            "bm_prefill_timeline")


def _check(status: int) -> None:
    if status != BM_OK:
        raise BatchMaxError(status, _lib.bm_last_error().decode())


# ---------------------------------------------------------------------------
# one-to-one ABI wrappers
# ---------------------------------------------------------------------------
def bm_abi_version() -> int:
    return _lib.bm_abi_version()


def bm_last_error() -> str:
    return _lib.bm_last_error().decode()


def bm_cache_slots(dims: bm_dims) -> int:
    return _lib.bm_cache_slots(ctypes.byref(dims))


def bm_workspace_bytes(dims: bm_dims) -> int:
    return _lib.bm_workspace_bytes(ctypes.byref(dims))


def bm_prefill_positions_per_workgroup(dims: bm_dims) -> int:
    return _lib.bm_prefill_positions_per_workgroup(ctypes.byref(dims))


def bm_validate_dims(dims: bm_dims) -> None:
    _check(_lib.bm_validate_dims(ctypes.byref(dims)))


def bm_init(dims: bm_dims, cache: bm_cache, stream: int) -> int:
    out = ctypes.c_void_p()
    _check(_lib.bm_init(ctypes.byref(dims), ctypes.byref(cache), stream, ctypes.byref(out)))
    return out.value


def bm_init_static_workspace(dims: bm_dims, cache: bm_cache, stream: int) -> int:
    out = ctypes.c_void_p()
    _check(_lib.bm_init_static_workspace(ctypes.byref(dims), ctypes.byref(cache), stream,
                                         ctypes.byref(out)))
    return out.value


def bm_resume(dims: bm_dims, cache: bm_cache, length: int, next_pos: int) -> int:
    out = ctypes.c_void_p()
    _check(_lib.bm_resume(ctypes.byref(dims), ctypes.byref(cache), length, next_pos,
                          ctypes.byref(out)))
    return out.value


def bm_prefill_block(ctx: int, t0: int, n_tok: int, q: int, k: int, v: int, o: int,
                     seq_ld: int, stream: int) -> None:
    _check(_lib.bm_prefill_block(ctx, t0, n_tok, q, k, v, o, seq_ld, stream))


def bm_prefill_block_cut(ctx: int, t0: int, n_tok: int, q: int, k: int, v: int, o: int,
                         seq_ld: int, stream: int) -> None:
    _check(_lib.bm_prefill_block_cut(ctx, t0, n_tok, q, k, v, o, seq_ld, stream))


def bm_evict_compact(ctx: int, curr_id: int, stream: int) -> None:
    _check(_lib.bm_evict_compact(ctx, curr_id, stream))


def bm_set_decode_removal(ctx: int, p: int) -> None:
    _check(_lib.bm_set_decode_removal(ctx, p))


def bm_set_rank_rule(ctx: int, rule: int) -> None:
    _check(_lib.bm_set_rank_rule(ctx, rule))


def bm_set_decode_bound(ctx: int, bound: int) -> None:
    _check(_lib.bm_set_decode_bound(ctx, bound))


def bm_set_score_accumulation(ctx: int, on: int) -> None:
    _check(_lib.bm_set_score_accumulation(ctx, on))


def bm_set_left_padding(ctx: int, pad_ptr: int) -> None:
    _check(_lib.bm_set_left_padding(ctx, pad_ptr))


def bm_set_split_event(ctx: int, event: int) -> None:
    _check(_lib.bm_set_split_event(ctx, event))


def bm_decode_step(ctx: int, pos: int, q: int, k: int, v: int, o: int, seq_ld: int,
                   stream: int) -> None:
    _check(_lib.bm_decode_step(ctx, pos, q, k, v, o, seq_ld, stream))


def bm_ctx_len(ctx: int) -> int:
    return _lib.bm_ctx_len(ctx)


def bm_ctx_next_pos(ctx: int) -> int:
    return _lib.bm_ctx_next_pos(ctx)


def bm_destroy(ctx: int) -> None:
    _lib.bm_destroy(ctx)


def bm_synth_qkv(params: bm_synth, t0: int, n_rows: int, q: int, k: int, v: int, seq_ld: int,
                 stream: int) -> None:
    _check(_lib.bm_synth_qkv(ctypes.byref(params), t0, n_rows, q, k, v, seq_ld, stream))


def bm_philox4x32_10(inp: int, out: int, n: int, stream: int) -> None:
    _check(_lib.bm_philox4x32_10(inp, out, n, stream))


def bm_probe_stream_read(src: int, nbytes: int, sink: int, blocks: int, nontemporal: bool,
                         stream: int) -> None:
    _check(_lib.bm_probe_stream_read(src, nbytes, sink, blocks, 1 if nontemporal else 0, stream))


def bm_probe_mfma(iters: int, sink: int, blocks: int, stream: int) -> None:
    _check(_lib.bm_probe_mfma(iters, sink, blocks, stream))


TIMELINE_FIELDS = 16
TIMELINE_MAX_RECORDS = 65536


def bm_prefill_timeline(n_records: int):
    """The last prefill launch's per-workgroup timeline records (a library
    built with BM_PREFILL_TIMELINE): uint64 array [n_records, 16]."""
    import numpy as np

    out = np.zeros((n_records, TIMELINE_FIELDS), dtype=np.uint64)
    _check(_lib.bm_prefill_timeline(out.ctypes.data_as(ctypes.c_void_p), n_records))
    return out


def make_dims(*, b, s, kv_max, block, max_gen, n_heads, n_kv_heads, head_dim, dtype,
              sm_scale=0.0) -> bm_dims:
    dt = {"f32": BM_F32, "bf16": BM_BF16}.get(dtype, dtype)
    return bm_dims(b, s, kv_max, block, max_gen, n_heads, n_kv_heads, head_dim, dt, sm_scale)


# ---------------------------------------------------------------------------
# tensor-owning convenience wrapper
# ---------------------------------------------------------------------------
class PDAttention:
    """Owns one layer's bounded cache (torch tensors on a GPU) and drives the ABI.

    Tensors passed to the calls have the sequence as dimension 2:
    q, o ``[b, n_heads, T, d]`` and k, v ``[b, n_kv_heads, T, d]``, contiguous,
    of the configured dtype, on the cache's device.  ``row`` selects the first
    row of the block (prefill) or the step's row (decode) inside them.
    """

    def __init__(self, *, b, s, kv_max, block, max_gen, n_heads, n_kv_heads, head_dim,
                 dtype="bf16", sm_scale=0.0, device="cuda", init=True, buffers=None,
                 static_workspace=False):
        """``static_workspace``: no workspace tensor; contexts come from
        bm_init_static_workspace and use the library's static device array."""
        import torch

        self.torch = torch
        self.dims = make_dims(b=b, s=s, kv_max=kv_max, block=block, max_gen=max_gen,
                              n_heads=n_heads, n_kv_heads=n_kv_heads, head_dim=head_dim,
                              dtype=dtype, sm_scale=sm_scale)
        bm_validate_dims(self.dims)
        self.tdtype = torch.float32 if self.dims.dtype == BM_F32 else torch.bfloat16
        dev = torch.device(device)
        if dev.type == "cuda" and dev.index is None:
            dev = torch.device("cuda", torch.cuda.current_device())
        self.device = dev
        self.cap = bm_cache_slots(self.dims)
        self.group = n_heads // n_kv_heads
        U = b * n_kv_heads
        self.work_bytes = bm_workspace_bytes(self.dims)
        self.static_workspace = static_workspace
        if static_workspace and buffers is not None:
            raise ValueError("static_workspace takes no caller buffers")
        if buffers is None:
            self.k = torch.empty((b, n_kv_heads, self.cap, head_dim), dtype=self.tdtype, device=self.device)
            self.v = torch.empty_like(self.k)
            self.score = torch.empty((b, n_kv_heads, self.cap), dtype=torch.float32, device=self.device)
            self.pos = torch.zeros((b, n_kv_heads, self.cap), dtype=torch.int32, device=self.device)
            self.len = torch.empty((b, n_kv_heads), dtype=torch.int32, device=self.device)
            self.work = (None if static_workspace else
                         torch.empty(self.work_bytes, dtype=torch.uint8, device=self.device))
        else:
            # caller-provided views (for example slices of one arena); shapes checked
            self.k, self.v, self.score, self.pos, self.len, self.work = buffers
            want = {"k": (b, n_kv_heads, self.cap, head_dim), "v": (b, n_kv_heads, self.cap, head_dim),
                    "score": (b, n_kv_heads, self.cap), "pos": (b, n_kv_heads, self.cap),
                    "len": (b, n_kv_heads)}
            for nm, shp in want.items():
                x = getattr(self, nm)
                if tuple(x.shape) != shp or not x.is_contiguous() or x.device != self.device:
                    raise ValueError(f"buffer {nm}: need a contiguous {shp} tensor on {self.device}")
            if self.work.numel() * self.work.element_size() < self.work_bytes:
                raise ValueError("work buffer is smaller than bm_workspace_bytes")
        self.cache = bm_cache(self.k.data_ptr(), self.v.data_ptr(), self.score.data_ptr(),
                              self.pos.data_ptr(), self.len.data_ptr(),
                              0 if self.work is None else self.work.data_ptr(),
                              0 if self.work is None else self.work_bytes)
        self.units = U
        self.ctx = None
        # schedule settings (bm_set_*): kept here and applied again to every new
        # context, so they survive reset() and resume()
        self._settings = {}
        if init:
            self.reset()

    # -- helpers ----------------------------------------------------------------
    def _stream(self) -> int:
        return self.torch.cuda.current_stream(self.device).cuda_stream

    def _check_tensor(self, x, heads, name):
        t = self.torch
        if x.device != self.device or x.dtype != self.tdtype or not x.is_contiguous():
            raise ValueError(f"{name}: need a contiguous {self.tdtype} tensor on {self.device}")
        if x.dim() != 4 or x.shape[0] != self.dims.b or x.shape[1] != heads or \
                x.shape[3] != self.dims.head_dim:
            raise ValueError(f"{name}: shape {tuple(x.shape)} is not [b, {heads}, T, d]")
        return x

    def _row_ptr(self, x, row):
        if not 0 <= row < x.shape[2]:
            raise ValueError(f"row {row} outside the tensor's {x.shape[2]} rows")
        return x.data_ptr() + row * x.shape[3] * x.element_size()

    # -- schedule ---------------------------------------------------------------
    _SETTERS = {"removal": bm_set_decode_removal, "rule": bm_set_rank_rule,
                "bound": bm_set_decode_bound, "accumulate": bm_set_score_accumulation,
                "pad": bm_set_left_padding, "split": bm_set_split_event}

    def _apply_settings(self) -> None:
        for key, val in self._settings.items():
            self._SETTERS[key](self.ctx, val)

    def _set(self, key, val) -> None:
        if self.ctx is not None:
            self._SETTERS[key](self.ctx, val)   # raises before anything is stored
        self._settings[key] = val

    def reset(self) -> None:
        if self.ctx is not None:
            bm_destroy(self.ctx)
            self.ctx = None
        init = bm_init_static_workspace if self.static_workspace else bm_init
        self.ctx = init(self.dims, self.cache, self._stream())
        self._apply_settings()

    def resume(self, length: int, next_pos: int) -> None:
        if self.static_workspace:
            raise ValueError("resume needs a caller-allocated workspace")
        if self.ctx is not None:
            bm_destroy(self.ctx)
            self.ctx = None
        self.ctx = bm_resume(self.dims, self.cache, length, next_pos)
        self._apply_settings()

    def _block_args(self, t0, n_tok, q, k, v, o, row):
        row = t0 if row is None else row
        H, Hk = self.dims.n_heads, self.dims.n_kv_heads
        for x, hh, nm in ((q, H, "q"), (k, Hk, "k"), (v, Hk, "v"), (o, H, "o")):
            self._check_tensor(x, hh, nm)
            if row + n_tok > x.shape[2]:
                raise ValueError(f"{nm}: rows [{row}, {row + n_tok}) exceed {x.shape[2]}")
        T = q.shape[2]
        if not (k.shape[2] == v.shape[2] == o.shape[2] == T):
            raise ValueError("q, k, v and o need the same number of rows")
        return (self.ctx, t0, n_tok, self._row_ptr(q, row), self._row_ptr(k, row),
                self._row_ptr(v, row), self._row_ptr(o, row), T, self._stream())

    def prefill_block(self, t0, n_tok, q, k, v, o, row=None) -> None:
        bm_prefill_block(*self._block_args(t0, n_tok, q, k, v, o, row))

    def prefill_block_cut(self, t0, n_tok, q, k, v, o, row=None) -> None:
        """prefill_block then evict_compact(t0 + n_tok - 1), fused where possible."""
        bm_prefill_block_cut(*self._block_args(t0, n_tok, q, k, v, o, row))

    def evict_compact(self, curr_id) -> None:
        bm_evict_compact(self.ctx, curr_id, self._stream())

    # settings persist across reset() and resume()
    def set_decode_removal(self, p: int) -> None:
        """0: one removal per decode step after appending (default); p > 0:
        Algorithm 1's decoding loop, p removals when a step starts full."""
        self._set("removal", p)

    def set_rank_rule(self, rule) -> None:
        """"ave" (default, Sec. 3.2), "sum", "recent" or "tova" (or a BM_RANK_* value)."""
        self._set("rule", RANK_RULES.get(rule, rule))

    def set_decode_bound(self, bound: int) -> None:
        self._set("bound", bound)

    def set_score_accumulation(self, on: bool) -> None:
        self._set("accumulate", 1 if on else 0)

    def set_left_padding(self, pads) -> None:
        """Left pad tokens per sample: a contiguous int32 tensor of b values on
        the device (kept referenced here), or None for no padding."""
        if pads is None:
            self._pads = None
            self._set("pad", None)
            return
        t = self.torch
        if pads.dtype != t.int32 or pads.device != self.device or not pads.is_contiguous() or \
                tuple(pads.shape) != (self.dims.b,):
            raise ValueError(f"pads: need a contiguous int32 [{self.dims.b}] tensor on {self.device}")
        self._pads = pads
        self._set("pad", pads.data_ptr())

    def set_split_event(self, event) -> None:
        """Record ``event`` (a torch.cuda.Event, or None to stop) between each
        later prefill block's attention kernel and its fold/cut launches, so the
        two can be timed separately on one stream.  The event is recorded once
        here on the current stream so that it exists."""
        if event is None:
            self._split = None
            self._set("split", None)
            return
        event.record(self.torch.cuda.current_stream(self.device))
        self._split = event
        self._set("split", event.cuda_event)

    def decode_step(self, pos, q, k, v, o, row=0) -> None:
        H, Hk = self.dims.n_heads, self.dims.n_kv_heads
        for x, hh, nm in ((q, H, "q"), (k, Hk, "k"), (v, Hk, "v"), (o, H, "o")):
            self._check_tensor(x, hh, nm)
        T = q.shape[2]
        if not (k.shape[2] == v.shape[2] == o.shape[2] == T):
            raise ValueError("q, k, v and o need the same number of rows")
        bm_decode_step(self.ctx, pos, self._row_ptr(q, row), self._row_ptr(k, row),
                       self._row_ptr(v, row), self._row_ptr(o, row), T, self._stream())

    def run_prefill(self, q, k, v, o, fused_cut=False) -> None:
        """Algorithm 1 prefill under the block loop: every block, then a cut
        (with ``fused_cut`` through prefill_block_cut)."""
        s, B = self.dims.s, self.dims.block
        for t0 in range(0, s, B):
            n = min(B, s - t0)
            if fused_cut:
                self.prefill_block_cut(t0, n, q, k, v, o)
            else:
                self.prefill_block(t0, n, q, k, v, o)
                self.evict_compact(t0 + n - 1)

    def run_decode(self, q, k, v, o, steps=None, first_row=None) -> None:
        """Decode steps at positions s, s+1, ... using rows first_row.. (default s)."""
        s = self.dims.s
        steps = self.dims.max_gen if steps is None else steps
        r0 = s if first_row is None else first_row
        for t in range(steps):
            self.decode_step(s + t, q, k, v, o, row=r0 + t)

    def capture_decode(self, q, k, v, o, steps=None, first_row=None):
        """Record run_decode's launches into one HIP graph (the decode loop of
        Algorithm 1 without host work between steps) and return it.

        Call it where the decode would start (right after the prefill).  Nothing
        runs during the capture; the context then describes the state after the
        decode steps.  Every position, length and pointer is fixed inside the
        graph, so ``graph.replay()`` is valid whenever the device state equals
        the one at capture time, e.g. after the same prefill has run again.  The
        decode path enqueues kernels only (no memset nodes)."""
        t = self.torch
        g = t.cuda.CUDAGraph()
        side = t.cuda.Stream(device=self.device)          # default priority
        side.wait_stream(t.cuda.current_stream(self.device))
        with t.cuda.graph(g, stream=side):
            self.run_decode(q, k, v, o, steps, first_row)
        t.cuda.current_stream(self.device).wait_stream(side)
        return g

    @property
    def length(self) -> int:
        return bm_ctx_len(self.ctx)

    @property
    def next_pos(self) -> int:
        return bm_ctx_next_pos(self.ctx)

    def close(self) -> None:
        if self.ctx is not None:
            bm_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


# ---------------------------------------------------------------------------
# synthetic inputs of the layer stack (bm_synth.h)
# ---------------------------------------------------------------------------
def synth_params(*, b, n_heads, n_kv_heads, head_dim, dtype, seed, layer, s, hh_frac=0.02,
                 hh_scale=4.0, n_sinks=0, sink_scale=6.0, heavy=True) -> bm_synth:
    """Generator parameters: value_scale = float32(sqrt(3) / sqrt(d) / 65536) and
    hh_threshold = round(hh_frac * 2^32) (0 when there are no heavy hitters)."""
    dt = {"f32": BM_F32, "bf16": BM_BF16}.get(dtype, dtype)
    thr = int(round(hh_frac * 2.0 ** 32)) if heavy else 0
    vs = ctypes.c_float(math.sqrt(3.0) / math.sqrt(head_dim) / 65536.0).value
    return bm_synth(b, n_heads, n_kv_heads, head_dim, dt, seed, layer, s, thr, hh_scale, n_sinks,
                    sink_scale, vs)


def synth_qkv(params: bm_synth, t0: int, q, k, v) -> None:
    """Fill every row of q [b, H, T, d], k/v [b, Hk, T, d] (torch, contiguous, on one
    GPU) with the stream's rows for positions t0 .. t0+T-1, on the current stream."""
    import torch

    tdt = torch.float32 if params.dtype == BM_F32 else torch.bfloat16
    T = q.shape[2]
    for x, hh, nm in ((q, params.n_heads, "q"), (k, params.n_kv_heads, "k"), (v, params.n_kv_heads, "v")):
        if x.dtype != tdt or not x.is_contiguous() or x.device.type != "cuda" or \
                tuple(x.shape) != (params.b, hh, T, params.head_dim):
            raise ValueError(f"{nm}: need a contiguous {tdt} [b, {hh}, {T}, d] tensor on the GPU")
    stream = torch.cuda.current_stream(q.device).cuda_stream
    bm_synth_qkv(params, t0, T, q.data_ptr(), k.data_ptr(), v.data_ptr(), T, stream)


# ---------------------------------------------------------------------------
# a stack of layers: one bounded cache per layer in a single device arena
# ---------------------------------------------------------------------------
def _align(n: int, a: int = 256) -> int:
    return (n + a - 1) // a * a


def stack_layer_bytes(*, b, kv_max, block, n_kv_heads, head_dim, dtype) -> int:
    """Device bytes of one layer's cache (K, V, score, pos, len), 256-byte aligned."""
    cap = kv_max + block
    es = 4 if dtype in ("f32", BM_F32) else 2
    rows = b * n_kv_heads * cap
    return (2 * _align(rows * head_dim * es) + 2 * _align(rows * 4) + _align(b * n_kv_heads * 4))


class PDStack:
    """``n_layers`` independent bounded caches (the attention layers of one
    model, each with its own scores and evictions) carved from one device
    arena, sharing one workspace (its contents never outlive a call).  Layer
    ``l`` is driven through ``self.layers[l]``, a ``PDAttention``."""

    def __init__(self, *, n_layers, b, s, kv_max, block, max_gen, n_heads, n_kv_heads, head_dim,
                 dtype="bf16", sm_scale=0.0, device="cuda"):
        import torch

        dims = make_dims(b=b, s=s, kv_max=kv_max, block=block, max_gen=max_gen, n_heads=n_heads,
                         n_kv_heads=n_kv_heads, head_dim=head_dim, dtype=dtype, sm_scale=sm_scale)
        bm_validate_dims(dims)
        dev = torch.device(device)
        if dev.type == "cuda" and dev.index is None:
            dev = torch.device("cuda", torch.cuda.current_device())
        tdt = torch.float32 if dims.dtype == BM_F32 else torch.bfloat16
        es = 4 if dims.dtype == BM_F32 else 2
        cap = kv_max + block
        per_layer = stack_layer_bytes(b=b, kv_max=kv_max, block=block, n_kv_heads=n_kv_heads,
                                      head_dim=head_dim, dtype=dims.dtype)
        work_bytes = bm_workspace_bytes(dims)
        self.arena_bytes = n_layers * per_layer + _align(work_bytes)
        self.arena = torch.empty(self.arena_bytes, dtype=torch.uint8, device=dev)
        work = self.arena[n_layers * per_layer:n_layers * per_layer + work_bytes]
        rows = b * n_kv_heads * cap
        self.layers = []
        for layer in range(n_layers):
            off = layer * per_layer

            def take(nbytes, dt, shape):
                nonlocal off
                x = self.arena[off:off + nbytes].view(dt).view(shape)
                off += _align(nbytes)
                return x

            kk = take(rows * head_dim * es, tdt, (b, n_kv_heads, cap, head_dim))
            vv = take(rows * head_dim * es, tdt, (b, n_kv_heads, cap, head_dim))
            sc = take(rows * 4, torch.float32, (b, n_kv_heads, cap))
            ps = take(rows * 4, torch.int32, (b, n_kv_heads, cap))
            ln = take(b * n_kv_heads * 4, torch.int32, (b, n_kv_heads))
            self.layers.append(PDAttention(b=b, s=s, kv_max=kv_max, block=block, max_gen=max_gen,
                                           n_heads=n_heads, n_kv_heads=n_kv_heads,
                                           head_dim=head_dim, dtype=dtype, sm_scale=sm_scale,
                                           device=dev, init=False,
                                           buffers=(kk, vv, sc, ps, ln, work)))
        self.n_layers = n_layers
        self.device = dev

    def reset(self) -> None:
        for layer in self.layers:
            layer.reset()

    def close(self) -> None:
        for layer in self.layers:
            layer.close()


def stack_bytes(*, b, n_layers, s, kv_max, block, max_gen, n_heads, n_kv_heads, head_dim,
                dtype) -> int:
    """Device bytes a P&D run of the layer stack needs at batch b: every layer's
    bounded cache, the shared workspace, and the reusable input/output buffers
    of one prefill block and one decode row."""
    es = 4 if dtype in ("f32", BM_F32) else 2
    dims = make_dims(b=b, s=s, kv_max=kv_max, block=block, max_gen=max_gen, n_heads=n_heads,
                     n_kv_heads=n_kv_heads, head_dim=head_dim, dtype=dtype)
    caches = n_layers * stack_layer_bytes(b=b, kv_max=kv_max, block=block, n_kv_heads=n_kv_heads,
                                          head_dim=head_dim, dtype=dtype)
    work = _align(bm_workspace_bytes(dims))
    rows = block + 1
    io = rows * b * (2 * n_heads + 2 * n_kv_heads) * head_dim * es
    return caches + work + io


def full_cache_bytes_per_sample(*, n_layers, s, n_kv_heads, head_dim, dtype) -> int:
    """K and V of every prompt position of every layer: the memory a
    decoding-only compression scheme holds before its first decode step."""
    es = 4 if dtype in ("f32", BM_F32) else 2
    return n_layers * n_kv_heads * s * head_dim * es * 2


def plan_stack_batch(budget_bytes: int, **shape) -> int:
    """Largest b with stack_bytes(b, **shape) <= budget_bytes (0 if none)."""
    lo, hi = 0, 1
    while stack_bytes(b=hi, **shape) <= budget_bytes:
        lo, hi = hi, hi * 2
    while hi - lo > 1:
        mid = (lo + hi) // 2
        if stack_bytes(b=mid, **shape) <= budget_bytes:
            lo = mid
        else:
            hi = mid
    return lo


# ---------------------------------------------------------------------------
# algorithmic work (used by the benchmark's roofline figures)
# ---------------------------------------------------------------------------
def prefill_flops_padded(*, pads, n_kv_heads, group, head_dim, s, kv_max, block) -> int:
    """prefill_flops with left padding (Sec. 3): only real queries and the real
    keys they see count.  Pads are removed before any real entry, so after a
    cut the cache holds min(real so far, kv_max) real entries."""
    total = 0
    for p in (int(x) for x in pads):
        real = pad = 0                     # entries in the cache
        for t0 in range(0, s, block):
            t1 = min(s, t0 + block)
            r0 = max(p, t0)                # first real row of the block
            n = max(0, t1 - r0)
            total += n * real + n * (n + 1) // 2
            real += n
            pad += (t1 - t0) - n
            excess = real + pad - kv_max
            if excess > 0:
                drop = min(pad, excess)
                pad -= drop
                real -= excess - drop
    return total * 4 * head_dim * group * n_kv_heads


def prefill_flops(*, b, n_kv_heads, group, head_dim, s, kv_max, block) -> int:
    """QK^T + PV flops the method must do: 4 d G per visible (query, key) pair."""
    total = 0
    length = 0
    for t0 in range(0, s, block):
        n = min(block, s - t0)
        # row r of the block sees length + r + 1 entries
        total += n * length + n * (n + 1) // 2
        length = min(kv_max, length + n)
    return 4 * head_dim * group * total * b * n_kv_heads


def decode_cache_lengths(*, s, kv_max, n_decode, p=0, bound=None) -> list:
    """Cached entries each decode step's attention reads (before its own pair),
    under the removal schedule chosen with ``bm_set_decode_removal`` and the
    decode bound of ``bm_set_decode_bound`` (default kv_max): the prompt leaves
    min(s, kv_max); with p = 0 a cache above the bound is cut to it, and a step
    appends then removes one when over the bound; with p > 0 a step that starts
    at or above the bound first drops to bound - p."""
    kd = kv_max if bound is None else bound
    n = min(s, kv_max)
    out = []
    for _ in range(n_decode):
        if p > 0 and n >= kd:
            n = kd - p
        elif p == 0 and n > kd:
            n = kd
        out.append(n)
        n = min(n + 1, kd)
    return out


MAX_DECODE_LEN = 4097   # entries one step of the scoring decode kernel attends to


def decode_bytes_outputs_only(*, b, n_kv_heads, group, head_dim, n, elem_bytes) -> int:
    """HBM bytes of one outputs-only decode step over n cached entries (the
    split path past MAX_DECODE_LEN): read n K and V rows, q, the new k and v;
    write o and append the new K, V row, score and position."""
    d, G, es = head_dim, group, elem_bytes
    per_unit = 2 * n * d * es + (G + 2) * d * es + G * d * es + 2 * d * es + 8
    return per_unit * b * n_kv_heads


def decode_bytes_per_step(*, b, n_kv_heads, group, head_dim, kv_max, elem_bytes) -> int:
    """HBM bytes one decode step must move per the fused design: read the K̄
    cached K and V rows, scores and positions; write K̄ scores, one K/V row,
    one score and position; read q (G rows), k and v of the step; write o."""
    d, G, es = head_dim, group, elem_bytes
    per_unit = (2 * kv_max * d * es          # cached K and V
                + kv_max * 4 * 2             # scores read and written
                + kv_max * 4                 # positions
                + (G + 2) * d * es           # q, new k, new v
                + G * d * es                 # o
                + 2 * d * es + 8)            # evicted slot overwrite (K, V, score, pos)
    return per_unit * b * n_kv_heads
