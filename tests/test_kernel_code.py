"""Properties of the fused kernel's gfx950 device code (CPU only: compiles
rip_kernels.hip to AMDGPU assembly with the library's own flags).

* bf16 results are stored through v_cvt_pk_bf16_f32 (the conversion that
  tests/test_gpu_ieee_edges.py checks on all 2^32 inputs against
  round-to-nearest-even), and no software rounding sequence stands in for it;
* fp32 subnormals are kept, not flushed (the kernel descriptors' fp32 denorm
  mode is 3: inputs and outputs preserved), as the exact group mean needs;
* no fused multiply-add or multiply-accumulate is emitted: every product and
  sum rounds on its own, in the order the oracle follows;
* no packed fp32 arithmetic is emitted (the library is built without it).
"""
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def asm(tmp_path_factory):
    import importlib.util
    spec = importlib.util.spec_from_file_location(
        "rip_build", os.path.join(ROOT, "paper_1909_08029_amd", "build.py"))
    b = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(b)
    out = str(tmp_path_factory.mktemp("asm") / "rip_kernels.s")
    flags = [f for f in b.COMMON if f not in ("-fPIC", "-shared")]
    csrc = os.path.join(ROOT, "paper_1909_08029_amd", "csrc")
    subprocess.run([b.HIPCC, *flags, "--cuda-device-only", "-S", "-I",
                    os.path.join(ROOT, "include"), "-I", csrc, "-x", "hip",
                    os.path.join(csrc, "rip_kernels.hip"), "-o", out],
                   check=True, capture_output=True, text=True, timeout=600)
    return open(out).read()


def instructions(text):
    return re.findall(r"^\s+(v_[a-z0-9_]+)", text, flags=re.M)


def test_bf16_stores_use_the_hardware_conversion(asm):
    ins = instructions(asm)
    assert "v_cvt_pk_bf16_f32" in ins
    # a software round-to-nearest-even would add 0x7fff plus the lsb with
    # 32-bit integer adds and extract bit 16
    assert not re.search(r"0x7fff\b", asm)


def test_fp32_subnormals_are_preserved(asm):
    modes = re.findall(r"\.amdhsa_float_denorm_mode_32\s+(\d+)", asm)
    assert modes and set(modes) == {"3"}


def test_no_fused_multiply_add(asm):
    ins = set(instructions(asm))
    fused = {i for i in ins if re.match(r"v_(pk_)?(fma|fmac|mac|mad|fmamk|fmaak|madmk|madak)", i)
             and "f32" in i}
    assert not fused, fused


def test_no_packed_fp32_arithmetic(asm):
    ins = set(instructions(asm))
    assert not {i for i in ins if i.startswith("v_pk_") and i.endswith("_f32")}
