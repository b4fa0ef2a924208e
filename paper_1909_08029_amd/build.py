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


# Measurement programs beside bench.py (not part of the library): built on
# demand by `bench.py --ceiling` / `bench.py --native`, into _build/.
BENCH_BUILD = os.path.join(ROOT, "_build")


def build_bench_program(name: str) -> str:
    """Builds bench_ceiling (bare HBM streams) or bench_native (the C ABI
    from a C++ loop) from the source beside bench.py; returns the path."""
    if name not in ("bench_ceiling", "bench_native"):
        raise ValueError(name)
    os.makedirs(BENCH_BUILD, exist_ok=True)
    out = os.path.join(BENCH_BUILD, name)
    tmp = out + ".tmp"
    src = os.path.join(ROOT, name + ".hip")
    flags = [f for f in COMMON if f not in ("-fPIC", "-shared")]
    if name == "bench_native":
        flags += ["-I", os.path.join(ROOT, "include"), "-L", PKG, "-lrip",
                  "-Wl,-rpath," + PKG]
    _run([HIPCC, *flags, src, "-o", tmp])
    os.replace(tmp, out)
    return out


BF16_CHECK = os.path.join(ROOT, "tests", "native", "libbf16check.so")


def build_bf16_check(out: str = BF16_CHECK):
    """Test helper: the bf16 store conversion against its definition."""
    tmp = out + ".tmp"
    _run([HIPCC, *COMMON, os.path.join(ROOT, "tests", "native", "bf16_cvt_check.hip"), "-o", tmp])
    os.replace(tmp, out)


def build_all():
    build_librip()
    build_seedgen()
    build_native_smoke()
    build_bf16_check()


if __name__ == "__main__":
    build_all()
    sys.exit(0)
