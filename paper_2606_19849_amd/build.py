"""Compile libvico.so (HIP kernels + C ABI) and the measurement helper
libvico_bench.so for gfx950, in-tree.

Usage: python -m paper_2606_19849_amd.build   (or build() from Python)
"""
from __future__ import annotations

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libvico.so")
SOURCES = ["attn_fwd.hip", "attn_merge.hip", "attn_gather.hip", "retrieve.hip", "token_drop.hip", "kv_append.hip", "vico_api.hip", "noalloc.hip"]
BENCH_LIB = os.path.join(PKG, "libvico_bench.so")
BENCH_SOURCES = ["mfma_peak.hip"]

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

FLAGS = [
    "--offload-arch=gfx950",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-shared",
    "-mcode-object-version=5",
    # keep hipcc from emitting packed fp32 VALU ops (v_pk_*_f32)
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall",
    "-Wno-unused-result",
]


def build(verbose: bool = False, extra_flags=()) -> str:
    """Compile libvico.so and libvico_bench.so; return the path of libvico.so."""
    _compile(SOURCES, LIB, verbose, extra_flags)
    _compile(BENCH_SOURCES, BENCH_LIB, verbose, extra_flags)
    return LIB


def _compile(sources, lib, verbose, extra_flags) -> None:
    srcs = [os.path.join(CSRC, s) for s in sources]
    tmp = lib + ".tmp"
    cmd = [HIPCC, *FLAGS, *extra_flags, "-I", INCLUDE, "-I", CSRC, *srcs, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    # the host pass does not know the packed-fp32 feature and says so; that is expected
    noise = "'-packed-fp32-ops' is not a recognized feature"
    err = "\n".join(l for l in res.stderr.splitlines() if noise not in l)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed ({res.returncode}):\n{err}")
    if verbose and err.strip():
        print(err, file=sys.stderr)
    # A kernel whose host-side launch stub was not emitted links into an
    # unloadable library; refuse it here instead of at load time.
    nm = subprocess.run(["nm", "-u", tmp], capture_output=True, text=True)
    missing = [l.split()[-1] for l in nm.stdout.splitlines() if "__device_stub__" in l]
    if missing:
        raise RuntimeError(f"{os.path.basename(lib)} references kernel stubs that were not emitted: {missing}")
    os.replace(tmp, lib)


if __name__ == "__main__":
    print(build(verbose=True))
