"""The library's build flags on the device pass (CPU only, hipcc
cross-compiles for gfx950): packed fp32 instructions are switched off --
a probe kernel of paired float multiply-adds compiles to v_pk_fma_f32
without the flag and to none with the library's flags (hipcc's host pass
warns that it does not know the feature; the device pass applies it) -- and
FMA contraction is off: the table kernel's device code holds no fused
multiply-add on fp64 values."""
import os
import re
import shutil
import subprocess

import pytest

from paper_2111_05426_amd import build

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
pytestmark = pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc is not installed")

PROBE = r'''
#include <hip/hip_runtime.h>
__global__ void probe(float2 *a, const float2 *b, int n)
{
    int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) {
        float2 x = a[i], y = b[i];
        x.x = x.x * y.x + 1.0f;
        x.y = x.y * y.y + 1.0f;
        a[i] = x;
    }
}
'''


def device_asm(tmp_path, src_text, flags, name="k.hip"):
    src = tmp_path / name
    src.write_text(src_text)
    out = tmp_path / (name + ".s")
    cmd = [HIPCC, "--offload-arch=gfx950", "-O3", "--cuda-device-only", "-S", "-o", str(out), str(src)] + flags
    p = subprocess.run(cmd, capture_output=True, text=True, timeout=600)
    assert p.returncode == 0, p.stderr
    return out.read_text()


def lib_flags():
    keep = []
    skip = {"-shared", "-fPIC", "-fvisibility=hidden", "-Wall", "-Wno-unused-function"}
    f = build.FLAGS
    i = 0
    while i < len(f):
        if f[i].startswith("--offload-arch") or f[i] in skip:
            i += 1
            continue
        keep.append(f[i])
        i += 1
    return keep


PK = re.compile(r"\bv_pk_(add|mul|fma)_f32\b")


def test_packed_fp32_off_on_the_device_pass(tmp_path):
    plain = device_asm(tmp_path, PROBE, ["-ffp-contract=off"])
    assert PK.search(plain), "the probe no longer compiles to packed fp32 without the flag"
    lib = device_asm(tmp_path, PROBE, lib_flags())
    assert not PK.search(lib)


def test_table_kernel_has_no_packed_fp32_and_no_fp64_fma(tmp_path):
    src = os.path.join(build.CSRC, "sim_tables.hip")
    asm = device_asm(tmp_path, open(src).read(), lib_flags() + ["-I", build.CSRC], name="sim_tables.hip")
    assert not PK.search(asm)
    assert not re.search(r"\bv_fma_f64\b", asm)
