"""Build step of libdsde.so (gfx950) from the HIP sources in csrc/.

Each source is compiled in two passes and linked into one shared library
beside this file:

1. the device pass (``--cuda-device-only``) for gfx950 with the packed-FP32
   target feature switched off, so that the compiler emits no
   ``v_pk_add_f32`` / ``v_pk_mul_f32`` / ``v_pk_fma_f32`` (some of their
   forms have given wrong results on this part without any error);
2. the host pass (``--cuda-host-only``), which embeds the device bundle of
   pass 1.  Giving the feature to a single combined compile would hand it to
   the x86 host pass as well, which does not know it and says so.

After linking, the device code in the library is disassembled and the build
fails if any packed FP32 arithmetic instruction is found
(``packed_fp32_instructions``; a CPU test runs the same check).
"""
import os
import re
import subprocess
import tempfile

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libdsde.so")
BUILD = os.path.join(ROOT, "_build")
SOURCES = ["api.hip", "stats.hip", "verify.hip", "shard.hip", "signal.hip", "probe.hip"]

ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
HIPCC = os.environ.get("HIPCC", os.path.join(ROCM, "bin", "hipcc"))
BUNDLER = os.path.join(ROCM, "llvm", "bin", "clang-offload-bundler")
OBJDUMP = os.path.join(ROCM, "llvm", "bin", "llvm-objdump")
ARCH = "gfx950"
DEVICE_TARGET = f"hipv4-amdgcn-amd-amdhsa--{ARCH}"
FLAGS = [f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-Wall",
         "-I", os.path.join(ROOT, "include"), "-I", CSRC]
DEVICE_FLAGS = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
PACKED_FP32 = re.compile(r"\bv_pk_(add|mul|fma)_f32\b")


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    objs = []
    for src in SOURCES:
        stem = src.replace(".hip", "")
        path = os.path.join(CSRC, src)
        dev = os.path.join(BUILD, stem + ".dev")
        obj = os.path.join(BUILD, stem + ".o")
        cuid = [f"-cuid=dsde_{stem}"]  # the same id in both passes of one source
        _run([HIPCC, *FLAGS, *cuid, *DEVICE_FLAGS, "--cuda-device-only", "-c", path, "-o", dev], verbose)
        _run([HIPCC, *FLAGS, *cuid, "--cuda-host-only", "-Xclang", "-fcuda-include-gpubinary", "-Xclang", dev,
              "-c", path, "-o", obj], verbose)
        objs.append(obj)
    tmp = LIB + ".tmp"
    _run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs], verbose)
    bad = packed_fp32_instructions(tmp)
    if bad:
        os.remove(tmp)
        raise RuntimeError("packed FP32 instructions in the device code: " + "; ".join(bad[:5]))
    os.replace(tmp, LIB)
    return LIB


def _fatbin_section(path):
    """Bytes of the .hip_fatbin section of an ELF shared object or object file."""
    with tempfile.TemporaryDirectory() as d:
        out = os.path.join(d, "fatbin")
        subprocess.run(["objcopy", "-O", "binary", "--only-section=.hip_fatbin", path, out], check=True)
        with open(out, "rb") as f:
            return f.read()


def device_disassembly(path: str = LIB) -> str:
    """Disassembly of every gfx950 code object embedded in a library built
    here (one offload bundle per source file)."""
    data = _fatbin_section(path)
    magic = b"__CLANG_OFFLOAD_BUNDLE__"
    starts = [m.start() for m in re.finditer(re.escape(magic), data)]
    if not starts:
        raise RuntimeError(f"no offload bundle in {path}")
    text = []
    with tempfile.TemporaryDirectory() as d:
        for i, s in enumerate(starts):
            e = starts[i + 1] if i + 1 < len(starts) else len(data)
            bundle, co = os.path.join(d, f"b{i}"), os.path.join(d, f"co{i}")
            with open(bundle, "wb") as f:
                f.write(data[s:e])
            subprocess.run([BUNDLER, "--unbundle", "--type=o", f"--input={bundle}", f"--targets={DEVICE_TARGET}",
                            f"--output={co}"], check=True)
            text.append(subprocess.run([OBJDUMP, "-d", co], check=True, capture_output=True, text=True).stdout)
    return "\n".join(text)


def packed_fp32_instructions(path: str = LIB):
    """Lines of the library's device code that use packed FP32 arithmetic."""
    return [ln.strip() for ln in device_disassembly(path).splitlines() if PACKED_FP32.search(ln)]


if __name__ == "__main__":
    print(build(verbose=True))
