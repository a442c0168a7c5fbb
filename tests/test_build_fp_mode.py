"""The stage kernel's convert is the IEEE cast only in the default FP mode.

`v_cvt_pk_bf16_f32` keeps fp32 subnormals and NaN/Inf when the kernel runs with
denormals preserved and no fast-math assumptions.  These CPU checks keep the
build honest: the library flags carry no fast-math or denormal-flush option,
stage.hip refuses to compile under -ffast-math, and the kernel descriptors in
the assembly built with the library's own flags preserve fp32 denormals.
"""
import os
import re
import shutil
import subprocess

import pytest

from paper_2607_22614_amd import build

HIPCC = shutil.which("hipcc") or ("/opt/rocm/bin/hipcc" if os.path.exists("/opt/rocm/bin/hipcc") else None)
needs_hipcc = pytest.mark.skipif(HIPCC is None, reason="hipcc not installed")
KERNEL_SOURCES = ["stage.hip", "reshard.hip"]

_BAD_FLAGS = ("fast-math", "fast_math", "flush-denormals", "denormal-fp-math", "finite-math", "unsafe-math",
              "-Ofast", "no-honor-nans", "no-honor-infinities")


def test_library_flags_keep_the_default_fp_mode():
    for flag in build.HIP_FLAGS:
        assert not any(b in flag for b in _BAD_FLAGS), flag


def _device_asm(src, extra=()):
    cmd = [HIPCC, *build.HIP_FLAGS, *extra, "-I", build.INCLUDE, "-I", build.CSRC, "-x", "hip", "--cuda-device-only",
           "-S", os.path.join(build.CSRC, src), "-o", "-"]
    return subprocess.run(cmd, capture_output=True, text=True)


@needs_hipcc
def test_fast_math_build_is_refused():
    r = _device_asm("stage.hip", ["-ffast-math"])
    assert r.returncode != 0 and "default FP mode" in r.stderr


@needs_hipcc
@pytest.mark.parametrize("src", KERNEL_SOURCES)
def test_kernels_preserve_fp32_denormals(src):
    r = _device_asm(src)
    assert r.returncode == 0, r.stderr
    kernels = re.findall(r"^\s*\.amdhsa_kernel\s+(\S+)", r.stdout, re.M)
    modes = re.findall(r"^\s*\.amdhsa_float_denorm_mode_32\s+(\d+)", r.stdout, re.M)
    assert kernels and len(modes) == len(kernels)
    # 3: denormal inputs and outputs both preserved (no flush)
    assert set(modes) == {"3"}, dict(zip(kernels, modes))
