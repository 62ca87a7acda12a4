"""Compile the HIP kernels and the C ABI into ``libbatchmax.so`` (gfx950, in-tree).

    python -m paper_2412_05693_amd.build              # the library
    python -m paper_2412_05693_amd.build --sanitize   # host-side ASan + UBSan build
    python -m paper_2412_05693_amd.build --timeline   # prefill timestamp build

Every call recompiles.  Objects go to ``paper_2412_05693_amd/_build/``; the
library lands next to this file, where ``batchmax.py`` loads it.

``--timeline`` builds ``libbatchmax_timeline.so`` with BM_PREFILL_TIMELINE
defined: its prefill attention kernel records per-workgroup timestamps
(include/bm_probe.h; read with ``python -m paper_2412_05693_amd.timeline``).
Measurement only; the ordinary library is compiled without it.

``--sanitize`` builds ``libbatchmax_san.so`` with AddressSanitizer and
UndefinedBehaviorSanitizer on the host code only (argument checks, context
handling, launch setup; the gfx950 device code is built as usual).  It is for
the CPU tests of the C ABI: load it with ``BATCHMAX_LIB`` pointing at it and the
sanitizer runtime preloaded (``sanitizer_env()`` gives both).
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(HERE, "_build")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "libbatchmax.so")
SOURCES = ["bm_abi.hip", "k_prefill.hip", "k_evict.hip", "k_decode.hip", "k_decode_long.hip",
           "k_synth.hip", "k_probe.hip"]
ARCH = "gfx950"


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build libbatchmax.so)")


COMMON = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-fvisibility=hidden",
    # packed fp32 VALU ops stay off: only scalar and plain vector fp32 code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", INCLUDE, "-I", CSRC,
]


# host-only instrumentation: every -fsanitize= applies to the host pass alone
SANITIZE = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host", "-fno-omit-frame-pointer",
            "-Xarch_host", "-g"]
LIB_SAN = os.path.join(HERE, "libbatchmax_san.so")
LIB_TIMELINE = os.path.join(HERE, "libbatchmax_timeline.so")
TIMELINE = ["-DBM_PREFILL_TIMELINE"]


def _compile(src: str, extra=(), tag: str = "") -> str:
    obj = os.path.join(BUILD, os.path.splitext(src)[0] + tag + ".o")
    cmd = [hipcc(), *COMMON, *extra, "-c", os.path.join(CSRC, src), "-o", obj]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n{res.stderr}")
    return obj


def build(jobs: int = 4, sanitize: bool = False, timeline: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    if sanitize:
        extra, tag, lib = SANITIZE, "_san", LIB_SAN
    elif timeline:
        extra, tag, lib = TIMELINE, "_tl", LIB_TIMELINE
    else:
        extra, tag, lib = (), "", LIB
    with cf.ThreadPoolExecutor(max_workers=jobs) as ex:
        objs = list(ex.map(lambda src: _compile(src, extra, tag), SOURCES))
    tmp = lib + ".tmp"
    link = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-shared-libsan"] if sanitize else []
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", *link, *objs, "-o", tmp]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"link failed:\n{res.stderr}")
    os.replace(tmp, lib)
    return lib


def sanitizer_env() -> dict:
    """Environment for a CPU process that loads the sanitizer build: the ASan
    runtime preloaded (the interpreter itself is not instrumented), leak
    checking off (the interpreter's own allocations are not ours to judge),
    and BATCHMAX_LIB pointing the binding at libbatchmax_san.so."""
    res = subprocess.run([hipcc(), "-print-file-name=libclang_rt.asan-x86_64.so"],
                         capture_output=True, text=True)
    rt = res.stdout.strip()
    if not os.path.isabs(rt):
        raise RuntimeError("ASan runtime not found")
    env = dict(os.environ)
    env["LD_PRELOAD"] = rt
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=1"
    env["UBSAN_OPTIONS"] = "print_stacktrace=1:halt_on_error=1"
    env["BATCHMAX_LIB"] = LIB_SAN
    return env


if __name__ == "__main__":
    print(build(sanitize="--sanitize" in sys.argv[1:], timeline="--timeline" in sys.argv[1:]))
    sys.exit(0)
