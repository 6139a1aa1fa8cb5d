"""Build libragged.so (the HIP kernels and the C interface) for gfx950 with hipcc.

Each source compiles to its own object in parallel; the objects link into one
shared library placed next to this file, where the binding loads it.
"""
from __future__ import annotations

import concurrent.futures
import os
import shutil
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "libragged.so")
OBJ_DIR = os.path.join(ROOT, "_build", "ragged")

SOURCES = ["api.cpp", "offsets.hip", "attention.hip", "gemm.hip", "layernorm.hip", "noalloc.hip"]
ARCH = "gfx950"

COMMON = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}", "-I", INCLUDE, "-I", CSRC,
          "-Wall", "-Wno-unused-function"]
# packed fp32 instructions stay off for all device code
DEVICE = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
# host-side AddressSanitizer + UndefinedBehaviorSanitizer (device code unchanged)
SANITIZE = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-omit-frame-pointer", "-g"]


def hipcc() -> str:
    for cand in (shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build the HIP library)")


def _compile(src: str, defines=(), obj_dir: str = OBJ_DIR, sanitize: bool = False) -> str:
    path = os.path.join(CSRC, src)
    obj = os.path.join(obj_dir, src + ".o")
    cmd = ([hipcc()] + COMMON + list(defines) + (DEVICE if src.endswith(".hip") else []) +
           (SANITIZE if sanitize else []) + ["-c", path, "-o", obj])
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"compiling {src} failed:\n{' '.join(cmd)}\n{res.stdout}\n{res.stderr}")
    return obj


def build(jobs: int | None = None, out: str = LIB, defines=(), sanitize: bool = False) -> str:
    """Compile and link; `out` and `defines` (extra -D flags) serve alternate builds;
    `sanitize` instruments the host code with AddressSanitizer and
    UndefinedBehaviorSanitizer (the loading process must preload clang's ASan
    runtime; CPU checks only)."""
    obj_dir = os.path.join(OBJ_DIR, "sanitize") if sanitize else OBJ_DIR
    if out != LIB:
        obj_dir = os.path.join(obj_dir, os.path.basename(out) + ".objs")
    os.makedirs(obj_dir, exist_ok=True)
    jobs = jobs or min(len(SOURCES), os.cpu_count() or 4)
    with concurrent.futures.ThreadPoolExecutor(jobs) as ex:
        objs = list(ex.map(lambda src: _compile(src, defines, obj_dir, sanitize), SOURCES))
    tmp = out + ".tmp"
    cmd = [hipcc(), "-shared", "-fPIC", f"--offload-arch={ARCH}", "-o", tmp] + (SANITIZE if sanitize else []) + objs
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"linking failed:\n{' '.join(cmd)}\n{res.stdout}\n{res.stderr}")
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    import argparse

    ap = argparse.ArgumentParser()
    ap.add_argument("--out", default=LIB)
    ap.add_argument("-D", dest="defines", action="append", default=[])
    ap.add_argument("--sanitize", action="store_true", help="host-side ASan + UBSan build (CPU checks)")
    a = ap.parse_args()
    print(build(out=os.path.abspath(a.out), defines=[f"-D{d}" for d in a.defines], sanitize=a.sanitize))
