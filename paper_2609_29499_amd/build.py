"""Builds libtasp.so (the C-ABI library with every gfx950 kernel) in-tree with hipcc.

Usage: ``python -m paper_2609_29499_amd.build`` (or ``build()`` from Python). Every call
recompiles; objects go to ``paper_2609_29499_amd/_build/``.
"""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
OBJ = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libtasp.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

SOURCES = ["plan_kernels.hip", "gemv_kernels.hip", "mfma_kernels.hip", "attn_kernels.hip",
           "prefill_kernels.hip", "prefill_attn.hip", "mask_kernels.hip", "token_kernels.hip",
           "router_kernels.hip", "shared_kernels.hip", "runtime.hip"]
FLAGS = [
    "--offload-arch=gfx950", "-O3", "-fPIC", "-std=c++17", "-Wall", "-Wno-unused-function",
    # packed FP32 instructions stay off: ordinary float code only
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", os.path.join(ROOT, "include"), "-I", CSRC,
]


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    noise = "is not a recognized feature for this target"
    err = "\n".join(l for l in r.stderr.splitlines() if noise not in l)
    if r.returncode != 0:
        raise RuntimeError(f"command failed ({r.returncode}): {' '.join(cmd)}\n{err}")
    return err


def build(verbose: bool = False, jobs: int = 4) -> str:
    os.makedirs(OBJ, exist_ok=True)

    def compile_one(src):
        obj = os.path.join(OBJ, os.path.splitext(src)[0] + ".o")
        msg = _run([HIPCC, *FLAGS, "-c", os.path.join(CSRC, src), "-o", obj])
        return obj, msg

    with ThreadPoolExecutor(max_workers=jobs) as ex:
        results = list(ex.map(compile_one, SOURCES))
    for obj, msg in results:
        if verbose and msg.strip():
            print(msg, file=sys.stderr)
    tmp = LIB + ".tmp"
    _run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp, *[o for o, _ in results]])
    os.replace(tmp, LIB)
    return LIB


# Host-side sanitizers for the argument checks (device code is built as usual): each -fsanitize
# goes to the host compilation only.
SAN_FLAGS = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined"]


def build_sanitized(out_dir: str) -> str:
    """libtasp_san.so in out_dir: runtime.hip (every host-side check of the C ABI) rebuilt with
    AddressSanitizer and UndefinedBehaviorSanitizer, linked with the kernel objects of the last
    build(). Load it with the sanitizer runtime preloaded (asan_runtime())."""
    others = [os.path.join(OBJ, os.path.splitext(s)[0] + ".o") for s in SOURCES if s != "runtime.hip"]
    missing = [o for o in others if not os.path.exists(o)]
    if missing:
        raise RuntimeError(f"kernel objects missing (run build() first): {missing}")
    os.makedirs(out_dir, exist_ok=True)
    obj = os.path.join(out_dir, "runtime_san.o")
    flags = [f for f in FLAGS if f != "-O3"] + ["-O1", "-g", "-fno-omit-frame-pointer"]
    _run([HIPCC, *flags, *SAN_FLAGS, "-c", os.path.join(CSRC, "runtime.hip"), "-o", obj])
    lib = os.path.join(out_dir, "libtasp_san.so")
    _run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", *SAN_FLAGS, "-shared-libsan", "-o", lib,
          *others, obj])
    return lib


def asan_runtime() -> str:
    """Path of the compiler's shared AddressSanitizer runtime."""
    r = subprocess.run([HIPCC, "-print-file-name=libclang_rt.asan-x86_64.so"], capture_output=True,
                       text=True, check=True)
    return r.stdout.strip()


if __name__ == "__main__":
    print(build(verbose=True))
