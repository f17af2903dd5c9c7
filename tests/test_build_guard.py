"""The packed-FP32 guard of the HIP build (CPU only).

The library's device code must hold no packed FP32 arithmetic
(v_pk_add_f32, v_pk_mul_f32, v_pk_fma_f32): the build switches the target
feature off in the device pass and scans the linked library.  These tests
re-run the scan on the built library, and show on a tiny kernel that the
scan finds such instructions when the feature is left on and that the build's
device flags remove them.
"""
import os
import subprocess

import pytest

from paper_2509_01083_amd import build_lib

KERNEL = r"""
#include <hip/hip_runtime.h>
__global__ void axpy2(float2 *a, const float2 *b, int n) {
  int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) {
    float2 x = a[i], y = b[i];
    x.x = x.x * y.x + 1.0f;
    x.y = x.y * y.y + 1.0f;
    a[i] = x;
  }
}
"""


@pytest.fixture(scope="module")
def built_lib():
    if not os.path.exists(build_lib.LIB):
        build_lib.build()
    return build_lib.LIB


def test_library_has_no_packed_fp32(built_lib):
    bad = build_lib.packed_fp32_instructions(built_lib)
    assert not bad, bad[:5]


def test_library_disassembly_covers_every_source(built_lib):
    text = build_lib.device_disassembly(built_lib)
    for kernel in ("stats_kernel_bf16", "seq_kernel", "next_sl_kernel", "kld_signal_kernel",
                   "shard_accept_kernel", "stream_read_kernel"):
        assert kernel in text, kernel


def _tiny_lib(tmp_path, device_flags):
    src = tmp_path / "axpy2.hip"
    src.write_text(KERNEL)
    dev, obj, so = tmp_path / "axpy2.dev", tmp_path / "axpy2.o", tmp_path / "libaxpy2.so"
    flags = [f"--offload-arch={build_lib.ARCH}", "-O3", "-fPIC", "-cuid=axpy2"]
    subprocess.run([build_lib.HIPCC, *flags, *device_flags, "--cuda-device-only", "-c", str(src), "-o", str(dev)],
                   check=True, capture_output=True)
    subprocess.run([build_lib.HIPCC, *flags, "--cuda-host-only", "-Xclang", "-fcuda-include-gpubinary",
                    "-Xclang", str(dev), "-c", str(src), "-o", str(obj)], check=True, capture_output=True)
    subprocess.run([build_lib.HIPCC, f"--offload-arch={build_lib.ARCH}", "-shared", "-fPIC", "-o", str(so),
                    str(obj)], check=True, capture_output=True)
    return str(so)


def test_scan_finds_packed_fp32_and_the_flags_remove_it(tmp_path):
    on, off = tmp_path / "on", tmp_path / "off"
    on.mkdir()
    off.mkdir()
    assert build_lib.packed_fp32_instructions(_tiny_lib(on, [])), "the compiler no longer packs this kernel"
    assert not build_lib.packed_fp32_instructions(_tiny_lib(off, build_lib.DEVICE_FLAGS))


def test_build_prints_no_ignored_feature_warning(tmp_path):
    src = tmp_path / "axpy2.hip"
    src.write_text(KERNEL)
    flags = [f"--offload-arch={build_lib.ARCH}", "-O3", "-fPIC", "-cuid=axpy2"]
    r = subprocess.run([build_lib.HIPCC, *flags, *build_lib.DEVICE_FLAGS, "--cuda-device-only", "-c", str(src),
                        "-o", str(tmp_path / "a.dev")], capture_output=True, text=True, check=True)
    assert "not a recognized feature" not in r.stdout + r.stderr
