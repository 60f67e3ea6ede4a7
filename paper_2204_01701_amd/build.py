"""Build the gfx950 HIP library ``libqlayer.so`` in-tree with hipcc.

Each translation unit (the C ABI and one launcher file per kernel family)
is compiled to an object in ``_build/`` in parallel, then the objects are
linked into ``libqlayer.so`` next to this file.

Usage: ``python -m paper_2204_01701_amd.build`` (or ``build()`` from Python).
"""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "libqlayer.so")
BUILD_DIR = os.path.join(PKG, "_build")
SOURCES = [os.path.join(CSRC, f) for f in sorted(os.listdir(CSRC)) if f.endswith(".hip")]
HEADERS = [os.path.join(ROOT, "include", f) for f in ("qlayer.h", "qnet.h")] + [
    os.path.join(CSRC, f) for f in sorted(os.listdir(CSRC)) if f.endswith(".h")
]

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    "-I" + os.path.join(ROOT, "include"), "-I" + CSRC,
    # no packed-fp32 instructions in device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


def _obj(src: str) -> str:
    return os.path.join(BUILD_DIR, os.path.basename(src)[:-4] + ".o")


# Per-file flags: the small-output forward keeps its MFMA accumulators in VGPRs
# (in the AGPR form, at one workgroup per CU, the compiler moved them between
# registers on every K step).
FILE_FLAGS = {"qlaunch_fwd_ksplit.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"]}


def compile_command(src: str, obj: str) -> list[str]:
    return [HIPCC, *FLAGS, *FILE_FLAGS.get(os.path.basename(src), []), "-c", "-o", obj, src]


def link_command(objs: list[str], out: str = LIB) -> list[str]:
    return [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", out, *objs]


def _run(cmd: list[str]) -> subprocess.CompletedProcess:
    return subprocess.run(cmd, capture_output=True, text=True)


def build(verbose: bool = False, jobs: int | None = None) -> str:
    """Compile every translation unit and link libqlayer.so (always recompiles); return its path."""
    os.makedirs(BUILD_DIR, exist_ok=True)
    objs = [_obj(s) for s in SOURCES]
    jobs = jobs or min(len(SOURCES), max(1, min(8, os.cpu_count() or 1)))
    with ThreadPoolExecutor(max_workers=jobs) as ex:
        results = list(ex.map(_run, [compile_command(s, o) for s, o in zip(SOURCES, objs)]))
    failed = [(s, r) for s, r in zip(SOURCES, results) if r.returncode != 0]
    for s, r in zip(SOURCES, results):
        if verbose or r.returncode != 0:
            sys.stderr.write(r.stdout + r.stderr)
    if failed:
        raise RuntimeError("hipcc failed on " + ", ".join(os.path.basename(s) for s, _ in failed))
    tmp = LIB + ".tmp"
    res = _run(link_command(objs, tmp))
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError("linking libqlayer.so failed")
    os.replace(tmp, LIB)
    return LIB


def is_stale() -> bool:
    if not os.path.exists(LIB):
        return True
    t = os.path.getmtime(LIB)
    return any(os.path.getmtime(f) > t for f in SOURCES + HEADERS)


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
