"""Compile ``libsalt.so`` (HIP kernels + C ABI runtime) for gfx950, in-tree.

    python -m paper_2608_03579_amd.build

The library lands next to this file; ``salt.py`` loads it from there.
"""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libsalt.so")
SOURCES = [os.path.join(CSRC, f) for f in ("salt_plan.hip", "salt_apply.hip", "salt_fuse_gram.hip", "salt_swap.hip", "salt_runtime.cpp")]
ARCH = "gfx950"

BUILD_DIR = os.path.join(HERE, "_build")

HIPCC_FLAGS = [
    f"--offload-arch={ARCH}",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-Wall",
    "-fvisibility=hidden",
    "-fvisibility-inlines-hidden",
    # no packed-fp32 instructions in device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    f"-I{os.path.join(ROOT, 'include')}",
]


def hipcc() -> str:
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    return os.path.join(rocm, "bin", "hipcc")


def _filtered(stderr: str):
    return [l for l in (stderr or "").splitlines() if "packed-fp32-ops" not in l and l.strip()]


def build(verbose: bool = False) -> str:
    """Compile every source into ``libsalt.so``; always recompiles (one hipcc
    process per source, in parallel, then one link)."""
    os.makedirs(BUILD_DIR, exist_ok=True)
    objs, procs = [], []
    for src in SOURCES:
        obj = os.path.join(BUILD_DIR, os.path.basename(src) + ".o")
        cmd = [hipcc(), *HIPCC_FLAGS, "-c", src, "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        procs.append((src, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.PIPE, text=True)))
        objs.append(obj)
    failed = []
    for src, p in procs:
        _, err = p.communicate()
        errs = _filtered(err)
        if p.returncode != 0:
            failed.append(f"{os.path.basename(src)}:\n" + "\n".join(errs))
        elif verbose and errs:
            print("\n".join(errs), file=sys.stderr)
    if failed:
        raise RuntimeError("hipcc failed:\n" + "\n".join(failed))
    tmp = LIB + ".tmp"
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError("hipcc link failed:\n" + "\n".join(_filtered(res.stderr)))
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
