"""Build libcl.so (the C-ABI library of HIP kernels) in-tree for gfx950.

    python -m paper_2605_05819_amd.build

Every source is compiled with hipcc for gfx950 only.  Packed fp32 VALU
instructions are disabled for all device code; the quantizer, the
compensation builder and the rank allocator are built with floating-point
contraction off so their fp64 arithmetic is exactly the stated sequence of
IEEE operations.

    python -m paper_2605_05819_amd.build --ubsan DIR

builds a second copy, DIR/libcl.so, whose host code (argument validation,
workspace sizing, the rank allocator, the compensation driver) carries
clang's undefined-behaviour checks and stops at the first report.  Its
device code is compiled without optimisation, to build quickly: it is for
checking the host side, not for timing.  Load it by naming it in the
CL_LIBRARY environment variable.
"""

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(os.path.dirname(HERE), "_build")
LIB = os.path.join(HERE, "libcl.so")

SOURCES = ["api.hip", "quant.hip", "decode.hip", "prefill.hip", "moe.hip", "comp.hip", "ranks.hip"]
EXTRA = {"quant.hip": ["-ffp-contract=off"], "comp.hip": ["-ffp-contract=off"], "ranks.hip": ["-ffp-contract=off"]}
ARCH = "gfx950"
FLAGS = ["-O3", "-std=c++17", "-fPIC", "--offload-arch=" + ARCH,
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-Wall", "-Wno-unused-function"]


def hipcc():
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    return os.path.join(rocm, "bin", "hipcc")


def _compile(src):
    obj = os.path.join(BUILD, src.replace(".hip", ".o"))
    cmd = [hipcc(), "-c", os.path.join(CSRC, src), "-o", obj] + FLAGS + EXTRA.get(src, [])
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode:
        raise RuntimeError("hipcc failed on %s:\n%s\n%s" % (src, " ".join(cmd), r.stderr))
    return obj


def build(verbose=False):
    """Compile every source and link ``libcl.so``; always rebuilds."""
    os.makedirs(BUILD, exist_ok=True)
    with ThreadPoolExecutor(max_workers=min(8, len(SOURCES))) as ex:
        objs = list(ex.map(_compile, SOURCES))
    tmp = LIB + ".tmp"
    cmd = [hipcc(), "-shared", "-o", tmp, "--offload-arch=" + ARCH] + objs
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode:
        raise RuntimeError("link failed:\n%s\n%s" % (" ".join(cmd), r.stderr))
    os.replace(tmp, LIB)
    if verbose:
        print("built", LIB)
    return LIB


def sanitizer_runtime_dir():
    """Directory of clang's shared sanitizer runtimes in the ROCm toolchain."""
    base = os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "llvm", "lib", "clang")
    for ver in sorted(os.listdir(base), reverse=True):
        d = os.path.join(base, ver, "lib", "linux")
        if os.path.exists(os.path.join(d, "libclang_rt.ubsan_standalone-x86_64.so")):
            return d
    raise RuntimeError("no shared UBSan runtime under " + base)


def build_ubsan(out_dir, verbose=False):
    """Build ``out_dir/libcl.so`` with undefined-behaviour checks on the host
    code (every check fatal) and unoptimised device code."""
    os.makedirs(out_dir, exist_ok=True)
    rt = sanitizer_runtime_dir()
    host = ["-Xarch_host", "-fsanitize=undefined", "-Xarch_host", "-fno-sanitize-recover=undefined",
            "-Xarch_host", "-fno-omit-frame-pointer"]
    flags = ["-O1", "-g", "-std=c++17", "-fPIC", "--offload-arch=" + ARCH,
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", "-Xarch_device", "-O0"] + host

    def one(src):
        obj = os.path.join(out_dir, src.replace(".hip", ".o"))
        cmd = [hipcc(), "-c", os.path.join(CSRC, src), "-o", obj] + flags + EXTRA.get(src, [])
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode:
            raise RuntimeError("hipcc failed on %s:\n%s\n%s" % (src, " ".join(cmd), r.stderr))
        return obj

    with ThreadPoolExecutor(max_workers=min(8, len(SOURCES))) as ex:
        objs = list(ex.map(one, SOURCES))
    lib = os.path.join(out_dir, "libcl.so")
    cmd = [hipcc(), "-shared", "-o", lib, "--offload-arch=" + ARCH] + objs + \
          ["-fsanitize=undefined", "-shared-libsan", "-Wl,-rpath," + rt]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode:
        raise RuntimeError("link failed:\n%s\n%s" % (" ".join(cmd), r.stderr))
    if verbose:
        print("built", lib)
    return lib


if __name__ == "__main__":
    if len(sys.argv) == 3 and sys.argv[1] == "--ubsan":
        build_ubsan(sys.argv[2], verbose=True)
    else:
        build(verbose=True)
    sys.exit(0)
