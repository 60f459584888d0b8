"""Builds libgvc.so (the HIP library behind include/gvc.h) for gfx950 in-tree.

    python -m paper_2608_10824_amd.build            # libgvc.so
    python -m paper_2608_10824_amd.build --asan     # libgvc_asan.so: host code under AddressSanitizer

Every source is compiled with hipcc for gfx950 only, with the packed-fp32
target feature turned off, into paper_2608_10824_amd/_build/, then linked into
paper_2608_10824_amd/libgvc.so.
"""
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libgvc.so")
SOURCES = ["k_gemm.hip", "k_select.hip", "k_misc.hip", "k_attn.hip", "k_decode.hip", "gvc_api.hip"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-Wall", "-Wno-unused-function",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-I", os.path.join(ROOT, "include"), "-I", CSRC]


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        out = "\n".join(l for l in (r.stdout + r.stderr).splitlines() if "packed-fp32-ops" not in l)
        raise RuntimeError("command failed: %s\n%s" % (" ".join(cmd), out))


# Host-code AddressSanitizer build (device code is compiled as usual): the
# sanitizer flags apply to the host pass only, and the runtime is the ROCm
# clang one, preloaded by whoever loads this library (see asan_runtime()).
ASAN_LIB = os.path.join(PKG, "libgvc_asan.so")
ASAN_BUILD = os.path.join(PKG, "_build_asan")
ASAN_FLAGS = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fno-omit-frame-pointer",
              "-Xarch_host", "-shared-libasan"]


def asan_runtime() -> str:
    """Path of the clang AddressSanitizer runtime matching hipcc's host compiler."""
    import glob
    hits = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    if not hits:
        raise FileNotFoundError("libclang_rt.asan-x86_64.so not found under /opt/rocm/llvm")
    return hits[-1]


def build(jobs: int = 5, asan: bool = False) -> str:
    out_dir, lib, extra = (ASAN_BUILD, ASAN_LIB, ASAN_FLAGS) if asan else (BUILD, LIB, [])
    os.makedirs(out_dir, exist_ok=True)
    objs = [os.path.join(out_dir, s.replace(".hip", ".o")) for s in SOURCES]
    cmds = [[HIPCC] + FLAGS + extra + ["-c", os.path.join(CSRC, s), "-o", o] for s, o in zip(SOURCES, objs)]
    with ThreadPoolExecutor(max_workers=jobs) as ex:
        list(ex.map(_run, cmds))
    tmp = lib + ".tmp"
    _run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC"] + extra + ["-o", tmp] + objs)
    os.replace(tmp, lib)
    return lib


if __name__ == "__main__":
    print(build(asan="--asan" in sys.argv[1:]))
    sys.exit(0)
