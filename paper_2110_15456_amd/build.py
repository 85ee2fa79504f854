"""Build libfastbfp.so (the C ABI of include/fastbfp.h) for gfx950, in-tree.

Every HIP source is compiled with hipcc for gfx950 only.  The shared library
is linked against the HIP runtime that PyTorch ships (same SONAME), so that a
process which imported torch runs our kernels in torch's runtime instance and
can launch on torch's streams; the rpath also lists /opt/rocm/lib for use
without torch.
"""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libfastbfp.so")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
ARCH = "gfx950"
SOURCES = ["quantize.hip", "packed.hip", "repack.hip", "gemm_mx.hip", "gemm_general.hip", "api.cpp"] + [
    "gemm_mx_%s%s.hip" % (p, g) for g in ("", "_g32") for p in ("11", "12", "21", "22")] + [
    "gemm_mx_11n_%d%d.hip" % (fa, fb) for fa in (0, 1) for fb in (0, 1)]
# Per-source extra flags: the quantizers align values with ldexp and rely on
# FP32 denormal flushing to read subnormal inputs as zero.
SOURCE_FLAGS = {"quantize.hip": ["-fgpu-flush-denormals-to-zero"], "packed.hip": ["-fgpu-flush-denormals-to-zero"]}
HIPFLAGS = [
    "-O3", "-std=c++17", "-fPIC", "--offload-arch=" + ARCH,
    # CDNA packed-FP32 instructions stay off: ordinary float code only.
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-result",
]


def _torch_lib_dir() -> str | None:
    try:
        import importlib.util
        spec = importlib.util.find_spec("torch")
        if spec and spec.origin:
            d = os.path.join(os.path.dirname(spec.origin), "lib")
            if os.path.exists(os.path.join(d, "libamdhip64.so")):
                return d
    except Exception:
        pass
    return None


def _compile(src: str, build_dir: str = BUILD, defines=()) -> str:
    obj = os.path.join(build_dir, os.path.splitext(src)[0] + ".o")
    cmd = [os.path.join(ROCM, "bin", "hipcc"), *HIPFLAGS, *SOURCE_FLAGS.get(src, []), *["-D" + d for d in defines], "-c",
           os.path.join(CSRC, src), "-o", obj]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError("hipcc failed for %s:\n%s\n%s" % (src, " ".join(cmd), res.stderr))
    return obj


def build(verbose: bool = False, out: str = LIB, defines=()) -> str:
    """Compile every source and link the library (default: libfastbfp.so next
    to this file).  ``defines``: extra preprocessor definitions (NAME=VALUE)
    that select kernel tile shapes."""
    build_dir = BUILD if not defines else BUILD + "_" + "_".join(d.replace("=", "") for d in defines)
    os.makedirs(build_dir, exist_ok=True)
    with ThreadPoolExecutor(max_workers=min(len(SOURCES), os.cpu_count() or 1)) as ex:
        objs = list(ex.map(lambda src: _compile(src, build_dir, defines), SOURCES))
    tlib = _torch_lib_dir()
    rpath = ":".join([p for p in (tlib, os.path.join(ROCM, "lib")) if p])
    link = [os.path.join(ROCM, "llvm", "bin", "clang++"), "-shared", "-fPIC", "-o", out + ".tmp", *objs]
    if tlib:
        link += ["-L" + tlib]
    else:
        link += ["-L" + os.path.join(ROCM, "lib")]
    link += ["-lamdhip64", "-Wl,-rpath," + rpath, "-Wl,--no-undefined"]
    res = subprocess.run(link, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError("link failed:\n%s\n%s" % (" ".join(link), res.stderr))
    os.replace(out + ".tmp", out)
    if verbose:
        print("built", out)
    return out


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
