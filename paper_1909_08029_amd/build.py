"""Build librip.so (the P-Reduce library) and libseedgen.so (input generator)
in-tree with hipcc for gfx950.

    python paper_1909_08029_amd/build.py        # or __graft_entry__.build()

Always recompiles.  Flags: -O3, fp contraction off (the kernels' arithmetic
order is part of their contract), packed-fp32 instructions disabled.
"""
from __future__ import annotations

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

COMMON = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-shared",
    "-ffp-contract=off", "-Wall",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]

LIBRIP = os.path.join(PKG, "librip.so")
LIBSEEDGEN = os.path.join(ROOT, "seedgen", "libseedgen.so")


def _run(cmd):
    print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    # hipcc's host pass does not know the (device-only) packed-fp32 feature
    out = "\n".join(l for l in res.stdout.splitlines() if "packed-fp32-ops" not in l)
    if out.strip():
        print(out, flush=True)
    if res.returncode != 0:
        raise subprocess.CalledProcessError(res.returncode, cmd)


def build_librip(out: str = LIBRIP, extra=()):
    csrc = os.path.join(PKG, "csrc")
    srcs = [os.path.join(csrc, f) for f in ("rip_api.hip", "rip_kernels.hip", "rip_sched.cpp")]
    tmp = out + ".tmp"
    _run([HIPCC, *COMMON, *extra, "-I", os.path.join(ROOT, "include"), "-I", csrc,
          "-x", "hip", *srcs, "-o", tmp])
    os.replace(tmp, out)


def build_seedgen(out: str = LIBSEEDGEN):
    tmp = out + ".tmp"
    _run([HIPCC, *COMMON, os.path.join(ROOT, "seedgen", "csrc", "seedgen.hip"), "-o", tmp])
    os.replace(tmp, out)


NATIVE_SMOKE = os.path.join(ROOT, "tests", "native", "cabi_smoke")


def build_native_smoke(out: str = NATIVE_SMOKE):
    """A plain C++ program that uses librip through include/rip.h only."""
    tmp = out + ".tmp"
    _run([HIPCC, f"--offload-arch={ARCH}", "-O2", "-std=c++17", "-Wall",
          "-I", os.path.join(ROOT, "include"), os.path.join(ROOT, "tests", "native", "cabi_smoke.cpp"),
          "-L", PKG, "-lrip", "-Wl,-rpath,$ORIGIN/../../paper_1909_08029_amd", "-o", tmp])
    os.replace(tmp, out)


STREAM_CEILING = os.path.join(PKG, "stream_ceiling")


def build_stream_ceiling(out: str = STREAM_CEILING):
    """The bare-stream HBM ceiling program run by `bench.py --ceiling`."""
    tmp = out + ".tmp"
    flags = [f for f in COMMON if f not in ("-fPIC", "-shared")]
    _run([HIPCC, *flags, os.path.join(PKG, "csrc", "stream_ceiling.hip"), "-o", tmp])
    os.replace(tmp, out)


NATIVE_BENCH = os.path.join(PKG, "rip_bench_native")


def build_native_bench(out: str = NATIVE_BENCH):
    """The C-ABI-only throughput program run by `bench.py --native`."""
    tmp = out + ".tmp"
    _run([HIPCC, f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-Wall",
          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          "-I", os.path.join(ROOT, "include"), os.path.join(PKG, "csrc", "rip_bench_native.hip"),
          "-L", PKG, "-lrip", "-Wl,-rpath,$ORIGIN", "-o", tmp])
    os.replace(tmp, out)


def build_all():
    build_librip()
    build_seedgen()
    build_native_smoke()
    build_stream_ceiling()
    build_native_bench()


if __name__ == "__main__":
    build_all()
    sys.exit(0)
