"""Builds libsparseattn.so (gfx950) in-tree with hipcc.

Every source is compiled for gfx950 only; packed-fp32 instructions are
disabled for the device code (the host pass warns that it does not know the
feature, which is harmless)."""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
OUT_DIR = os.path.join(ROOT, "_build")
LIB = os.path.join(HERE, "libsparseattn.so")

SOURCES = ["api.hip", "select.hip", "sched.hip", "fwd_bf16.hip", "fwd_fp8.hip", "quant_fp8.hip",
           "comp.hip", "linear_fp8.hip", "bwd.hip"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-Wall", "-Wno-unused-command-line-argument",
         "-I", INCLUDE, "-I", CSRC]


def _run(cmd):
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    # drop the host pass's notice about the device-only target feature
    out = "\n".join(l for l in r.stdout.splitlines()
                    if "packed-fp32-ops" not in l and l.strip() != "1 warning generated.")
    if r.returncode != 0:
        raise RuntimeError(f"command failed ({r.returncode}): {' '.join(cmd)}\n{r.stdout}")
    return out


def build(verbose: bool = False, jobs: int = 8) -> str:
    """Compile every source and link the shared library; returns its path."""
    os.makedirs(OUT_DIR, exist_ok=True)

    def compile_one(src):
        obj = os.path.join(OUT_DIR, src.replace(".hip", ".o"))
        out = _run([HIPCC, *FLAGS, "-c", os.path.join(CSRC, src), "-o", obj])
        if verbose and out.strip():
            print(out)
        return obj

    with ThreadPoolExecutor(max_workers=jobs) as ex:
        objs = list(ex.map(compile_one, SOURCES))
    tmp = LIB + ".tmp"
    _run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", tmp])
    os.replace(tmp, LIB)
    return LIB


SANITIZED_LIB = os.path.join(OUT_DIR, "asan", "libsparseattn_host_asan.so")


def asan_runtime() -> str:
    """The compiler's shared AddressSanitizer runtime (preloaded into the
    Python process that loads the sanitized library)."""
    res = _run([HIPCC, "-print-file-name=libclang_rt.asan-x86_64.so"]).strip().splitlines()
    path = res[-1].strip() if res else ""
    if not os.path.exists(path):
        import glob
        hits = glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so")
        path = hits[0] if hits else ""
    if not path:
        raise RuntimeError("no shared AddressSanitizer runtime found")
    return path


def build_host_sanitized(jobs: int = 8) -> str:
    """Build of every source with AddressSanitizer and
    UndefinedBehaviorSanitizer on the host code only (the gfx950 device code
    is built as usual, without them): the CPU build under which the
    argument-check tests of the C ABI run."""
    out = os.path.dirname(SANITIZED_LIB)
    os.makedirs(out, exist_ok=True)
    san = ["-Xarch_host", "-fsanitize=address,undefined",
           "-Xarch_host", "-fno-sanitize-recover=undefined",
           "-Xarch_host", "-fno-omit-frame-pointer", "-shared-libsan"]
    flags = [f for f in FLAGS if f != "-O3"] + ["-O1", "-g"]

    def compile_one(src):
        obj = os.path.join(out, src.replace(".hip", ".o"))
        _run([HIPCC, *flags, *san, "-c", os.path.join(CSRC, src), "-o", obj])
        return obj

    with ThreadPoolExecutor(max_workers=jobs) as ex:
        objs = list(ex.map(compile_one, SOURCES))
    tmp = SANITIZED_LIB + ".tmp"
    _run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", *san, *objs, "-o", tmp])
    os.replace(tmp, SANITIZED_LIB)
    return SANITIZED_LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
