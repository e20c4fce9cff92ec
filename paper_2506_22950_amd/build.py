"""Build libinfs.so (HIP kernels + host runtime + scheduler) for gfx950 with hipcc,
and libinfs_calib.so (a streaming-read kernel that bench.py uses as the
one-launch read-bandwidth reference; not part of the decode path).

Usage: python -m paper_2506_22950_amd.build   (or call build()).
The libraries are written next to this file so that they travel with the source tree.
"""

import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "libinfs.so")
CALIB_LIB = os.path.join(HERE, "libinfs_calib.so")
BUILD_DIR = os.path.join(HERE, "_build")

# Decode kernel instantiations are spread over several translation units
# (inst_*.hip) that compile in parallel; the device code is in decode.h.
SOURCES = ["kernels.hip", "inst_wave_f32_d64.hip", "inst_wave_f32_d128.hip", "inst_wave_bf16_d64.hip",
           "inst_wave_bf16_d128.hip", "inst_mfma_d64.hip", "inst_mfma_d128a.hip", "inst_mfma_d128b.hip",
           "inst_kv8a.hip", "inst_kv8b.hip", "scratch.hip", "runtime.cpp", "sched.cpp"]
CALIB_SOURCES = ["calib.hip"]


def _hipcc():
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("hipcc not found (ROCm is required to build libinfs.so)")


def _flags():
    return [
        "--offload-arch=gfx950",
        "-O3",
        "-std=c++17",
        "-fPIC",
        "-Wall",
        "-Wno-unused-function",
        "-I" + INCLUDE,
        "-I" + CSRC,
        # Packed fp32 VALU ops are kept out of every kernel.
        "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    ]


def build(verbose: bool = False) -> str:
    """Compile every source and link libinfs.so; returns the library path."""
    hipcc = _hipcc()
    os.makedirs(BUILD_DIR, exist_ok=True)

    def compile_one(src):
        obj = os.path.join(BUILD_DIR, src + ".o")
        cmd = [hipcc, *_flags(), "-c", os.path.join(CSRC, src), "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        r = subprocess.run(cmd, capture_output=True, text=True)
        msgs = [ln for ln in (r.stderr or "").splitlines() if "packed-fp32-ops" not in ln]
        if r.returncode != 0:
            raise RuntimeError(f"compiling {src} failed:\n" + "\n".join(msgs))
        if verbose and msgs:
            print("\n".join(msgs))
        return obj

    with ThreadPoolExecutor(max_workers=min(os.cpu_count() or 8, 16, len(SOURCES) + len(CALIB_SOURCES))) as ex:
        objs = list(ex.map(compile_one, SOURCES + CALIB_SOURCES))
    for lib, part in ((LIB, objs[:len(SOURCES)]), (CALIB_LIB, objs[len(SOURCES):])):
        tmp = lib + ".tmp"
        cmd = [hipcc, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp, *part]
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"linking {os.path.basename(lib)} failed:\n" + r.stderr)
        os.replace(tmp, lib)
    return LIB


# Host-only sanitizer build: the host runtime (runtime.cpp, sched.cpp) with
# AddressSanitizer and UndefinedBehaviorSanitizer, the kernel objects as built
# by build().  Sanitizers apply to host code only: each -fsanitize= follows
# -Xarch_host, so no device code is instrumented.  The library is written as
# _san/libinfs.so (select it with INFS_LIBRARY); a process that loads it
# needs the sanitizer runtime preloaded (sanitizer_runtime()).
SAN_DIR = os.path.join(HERE, "_san")
SAN_LIB = os.path.join(SAN_DIR, "libinfs.so")
SAN_SOURCES = ["runtime.cpp", "sched.cpp"]


def sanitizer_runtime() -> str:
    """Path of the clang AddressSanitizer runtime (it also carries the
    UndefinedBehaviorSanitizer handlers) that matches hipcc's compiler."""
    import glob

    clang = os.path.join(os.path.dirname(os.path.realpath(_hipcc())), "..", "lib", "llvm", "bin", "clang++")
    if not os.path.exists(clang):
        clang = shutil.which("amdclang++") or "/opt/rocm/llvm/bin/clang++"
    res = subprocess.run([clang, "-print-resource-dir"], capture_output=True, text=True).stdout.strip()
    for pat in ("lib/linux/libclang_rt.asan-x86_64.so", "lib/x86_64-unknown-linux-gnu/libclang_rt.asan.so"):
        hits = glob.glob(os.path.join(res, pat))
        if hits:
            return hits[0]
    raise RuntimeError(f"no AddressSanitizer runtime under {res}")


def build_sanitized(verbose: bool = False) -> str:
    """Build _san/libinfs.so (after build()); returns its path."""
    hipcc = _hipcc()
    objdir = os.path.join(BUILD_DIR, "san")
    os.makedirs(objdir, exist_ok=True)
    os.makedirs(SAN_DIR, exist_ok=True)
    san = ["-O1", "-g", "-fno-omit-frame-pointer",
           "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=undefined"]
    flags = [f for f in _flags() if f != "-O3"] + san
    objs = []
    for src in SAN_SOURCES:
        obj = os.path.join(objdir, src + ".o")
        cmd = [hipcc, *flags, "-c", os.path.join(CSRC, src), "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"compiling {src} (sanitized) failed:\n" + r.stderr)
        objs.append(obj)
    kernels = [os.path.join(BUILD_DIR, src + ".o") for src in SOURCES if src not in SAN_SOURCES]
    missing = [o for o in kernels if not os.path.exists(o)]
    if missing:
        raise RuntimeError("build() first: missing " + ", ".join(os.path.basename(o) for o in missing))
    # a host link: the kernel objects already carry their device code; the library
    # records the sanitizer runtime as a dependency so that plain programs link to it
    rt = sanitizer_runtime()
    tmp = SAN_LIB + ".tmp"
    cmd = [hipcc, "-shared", "-fPIC", "-o", tmp, *kernels, *objs, rt, "-Wl,-rpath," + os.path.dirname(rt)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("linking the sanitized library failed:\n" + r.stderr)
    os.replace(tmp, SAN_LIB)
    return SAN_LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
    if "--sanitized" in sys.argv:
        print(build_sanitized(verbose="-v" in sys.argv))
