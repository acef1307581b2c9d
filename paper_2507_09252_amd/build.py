"""Builds libtppsd.so in-tree for gfx950.

Device and host sources are compiled with hipcc; the shared library is
linked against the HIP runtime that torch ships (found next to torch's own
libraries and recorded as the library's run path), so that streams and
device pointers handed over from torch belong to the same runtime instance.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libtppsd.so")
ARCH = "gfx950"

HIPCC_FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    # no packed-fp32 instructions in device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # device code reinterprets bf16 storage as MFMA vector operands (also in LDS)
    "-fno-strict-aliasing",
    "-Wall", "-Wno-unused-function", "-Wno-unused-variable",
]


# Kernels take their leading scalar arguments preloaded into registers
# (gfx950 kernel-argument preloading, as many as fit the user SGPRs; a code
# object prologue loads them where the firmware does not), so that their
# first loads need no kernel-argument load.
PRELOAD = ["-mllvm", "-amdgpu-kernarg-preload-count=16"]
FILE_FLAGS = {"tppsd_draft_rows.hip": PRELOAD, "tppsd_kernels.hip": PRELOAD, "tppsd_attention.hip": PRELOAD,
              "tppsd_poisson.hip": PRELOAD}


def source_flags(src: str) -> list:
    """hipcc flags for one source file of the library."""
    return HIPCC_FLAGS + FILE_FLAGS.get(os.path.basename(src), [])


def _torch_lib_dir() -> str:
    import importlib.util
    spec = importlib.util.find_spec("torch")
    if spec is None or not spec.origin:
        raise RuntimeError("torch is not importable; it provides the HIP runtime this library links to")
    return os.path.join(os.path.dirname(spec.origin), "lib")


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(l for l in r.stdout.splitlines() if "packed-fp32-ops" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"build step failed ({r.returncode}): {' '.join(cmd)}\n{out}")
    if verbose and out.strip():
        print(out)


def build(verbose: bool = False) -> str:
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    os.makedirs(BUILD, exist_ok=True)
    inc = ["-I", os.path.join(ROOT, "include"), "-I", CSRC]
    from concurrent.futures import ThreadPoolExecutor
    srcs = ("tppsd_kernels.hip", "tppsd_attention.hip", "tppsd_poisson.hip", "tppsd_draft_rows.hip", "tppsd.cpp")
    objs = [os.path.join(BUILD, src + ".o") for src in srcs]
    cmds = [[hipcc] + source_flags(src) + inc + ["-x", "hip", "-c", os.path.join(CSRC, src), "-o", obj]
            for src, obj in zip(srcs, objs)]
    with ThreadPoolExecutor(len(cmds)) as ex:
        for f in [ex.submit(_run, c, verbose) for c in cmds]:
            f.result()
    tlib = _torch_lib_dir()
    tmp = LIB + ".tmp"
    _run(["g++", "-shared", "-o", tmp] + objs +
         [f"-L{tlib}", "-l:libamdhip64.so", f"-Wl,-rpath,{tlib}", "-Wl,--no-undefined"], verbose)
    os.replace(tmp, LIB)
    return LIB


def build_host_sanitized(out_dir: str, verbose: bool = False) -> str:
    """The library with its host source (tppsd.cpp) built under
    AddressSanitizer and UndefinedBehaviorSanitizer and the device sources as
    in build(), whose objects it reuses (built first if missing), for CPU
    tests of the host-side paths. Load it with the sanitizer runtime
    preloaded (sanitizer_runtime())."""
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    dev = ("tppsd_kernels.hip", "tppsd_attention.hip", "tppsd_poisson.hip", "tppsd_draft_rows.hip")
    objs = [os.path.join(BUILD, src + ".o") for src in dev]
    if not all(os.path.exists(o) for o in objs):
        build(verbose)
    os.makedirs(out_dir, exist_ok=True)
    inc = ["-I", os.path.join(ROOT, "include"), "-I", CSRC]
    san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer"]
    flags = [f for f in HIPCC_FLAGS if f != "-O3"] + ["-O1", "-g"]
    host_obj = os.path.join(out_dir, "tppsd_san.cpp.o")
    _run([hipcc] + flags + san + inc + ["-x", "hip", "-c", os.path.join(CSRC, "tppsd.cpp"), "-o", host_obj], verbose)
    tlib = _torch_lib_dir()
    out = os.path.join(out_dir, "libtppsd_san.so")
    _run([_clangxx(), "-shared", "-fsanitize=address,undefined", "-shared-libasan", "-o", out] + objs + [host_obj] +
         [f"-L{tlib}", "-l:libamdhip64.so", f"-Wl,-rpath,{tlib}"], verbose)
    return out


def _clangxx() -> str:
    for c in ("/opt/rocm/llvm/bin/clang++", shutil.which("amdclang++") or ""):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("clang++ of the ROCm toolchain not found")


def sanitizer_runtime() -> str:
    """Path of the AddressSanitizer runtime the sanitized library links to."""
    r = subprocess.run([_clangxx(), "-print-file-name=libclang_rt.asan-x86_64.so"], stdout=subprocess.PIPE, text=True)
    return r.stdout.strip()


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
