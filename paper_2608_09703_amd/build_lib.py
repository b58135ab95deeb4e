"""Builds ``libmls.so`` (HIP kernels for gfx950 + the C-ABI host code) in-tree.

Usage: ``python -m paper_2608_09703_amd.build_lib`` (or ``__graft_entry__.build()``).
Every call recompiles all sources.
"""

from __future__ import annotations

import concurrent.futures
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libmls.so")

SOURCES = ["mls_api.cpp", "mls_fused.hip", "mls_gemm.hip", "mls_rows.hip", "mls_diag.hip", "mls_junction.hip", "mls_decode.hip", "mls_static.hip",
           "mls_probe.hip"]
ARCH = "gfx950"


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def common_flags():
    return [
        f"--offload-arch={ARCH}",
        "-O3",
        "-std=c++17",
        "-fPIC",
        "-Wall",
        "-Wno-unused-function",
        # keep the compiler from forming packed fp32 VALU ops
        "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
        f"-I{INCLUDE}",
        f"-I{CSRC}",
    ]


# Host-side sanitizers (device code is built as usual): each -fsanitize= applies
# to the host compilation only.
SANITIZE_FLAGS = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                  "-Xarch_host", "-fno-omit-frame-pointer", "-Xarch_host", "-fno-sanitize-recover=all",
                  "-shared-libsan"]
SAN_BUILD = os.path.join(ROOT, "_build_san")
SAN_LIB = os.path.join(SAN_BUILD, "libmls_san.so")


def _compile(src: str, sanitize: bool = False) -> str:
    out = SAN_BUILD if sanitize else BUILD
    obj = os.path.join(out, os.path.splitext(src)[0] + ".o")
    cmd = [hipcc(), "-x", "hip", "-c", os.path.join(CSRC, src), "-o", obj] + common_flags()
    if sanitize:
        cmd += SANITIZE_FLAGS
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"compile of {src} failed:\n{' '.join(cmd)}\n{res.stdout}\n{res.stderr}")
    return obj


def build(verbose: bool = False, sanitize: bool = False) -> str:
    """Compiles every source and links libmls.so; with sanitize=True, a copy
    whose host code is built with AddressSanitizer and UndefinedBehaviorSanitizer
    (_build_san/libmls_san.so; load it with MLS_LIBRARY and the sanitizer
    runtime preloaded, for CPU-only host tests)."""
    out_dir = SAN_BUILD if sanitize else BUILD
    os.makedirs(out_dir, exist_ok=True)
    with concurrent.futures.ThreadPoolExecutor(max_workers=min(4, len(SOURCES))) as ex:
        objs = list(ex.map(lambda f: _compile(f, sanitize), SOURCES))
    target = SAN_LIB if sanitize else LIB
    tmp = target + ".tmp"
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp] + objs
    if sanitize:
        cmd += SANITIZE_FLAGS
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"link failed:\n{' '.join(cmd)}\n{res.stdout}\n{res.stderr}")
    os.replace(tmp, target)
    if verbose:
        print(f"built {target}")
    return target


def sanitizer_runtime() -> str:
    """Path of the compiler's AddressSanitizer runtime (to LD_PRELOAD into python)."""
    clang = os.path.join(os.path.dirname(os.path.realpath(hipcc())), "..", "lib", "llvm", "bin", "clang++")
    for cand in (clang, "/opt/rocm/llvm/bin/clang++"):
        if os.path.exists(cand):
            r = subprocess.run([cand, "-print-file-name=libclang_rt.asan-x86_64.so"], capture_output=True,
                               text=True)
            if r.returncode == 0 and os.path.exists(r.stdout.strip()):
                return r.stdout.strip()
    raise RuntimeError("AddressSanitizer runtime not found")


if __name__ == "__main__":
    if "--sanitize" in sys.argv:
        build(verbose=True, sanitize=True)
        print(f"LD_PRELOAD={sanitizer_runtime()} MLS_LIBRARY={SAN_LIB} "
              f"ASAN_OPTIONS=detect_leaks=0 python -m pytest tests/test_abi_host.py")
    else:
        build(verbose=True)
    sys.exit(0)
