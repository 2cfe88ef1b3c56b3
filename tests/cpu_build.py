"""A host build of libsalt (its own runtime and kernel sources, compiled for the
CPU against ``tests/cpu_kernels/hip``), run under AddressSanitizer.

``build()`` compiles the sources with the host clang of ROCm, once per source
hash, into ``tests/cpu_kernels/_build/harness``.  The only change made to a
source is the declaration of the dynamic LDS array, which becomes a pointer to
the exact-size buffer the host runtime allocates for each launch.  ``run()``
writes a run description (context, pinned centroids, residual loads, batches),
runs the harness and parses what the C ABI returned.

Test infrastructure only.
"""
from __future__ import annotations

import fcntl
import hashlib
import os
import shutil
import struct
import subprocess
from typing import Dict, List, Optional, Sequence

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(ROOT, "paper_2608_03579_amd", "csrc")
SHIM = os.path.join(HERE, "cpu_kernels")
BUILD = os.path.join(SHIM, "_build")
SOURCES = ("salt_plan.hip", "salt_apply.hip", "salt_fuse_gram.hip", "salt_swap.hip", "salt_runtime.cpp")
HEADERS = ("salt_device.h", "salt_internal.h", "salt_layout.h", "salt_launch.h")
DYN_LDS = "extern __shared__ __attribute__((aligned(16))) char lds[];"
CLANG = "/opt/rocm/llvm/bin/clang++"


def available() -> bool:
    return os.path.exists(CLANG)


def _digest() -> str:
    h = hashlib.sha256()
    for d, names in ((CSRC, SOURCES + HEADERS), (SHIM, ("harness.cpp", "hip/hip_runtime.h", "hip/hip_ext.h"))):
        for n in names:
            h.update(n.encode())
            h.update(open(os.path.join(d, n), "rb").read())
    h.update(open(os.path.join(ROOT, "include", "salt.h"), "rb").read())
    return h.hexdigest()[:16]


def build() -> str:
    """The harness for the current sources, built once; concurrent test
    processes wait on a lock file while one of them builds."""
    exe = os.path.join(BUILD, "harness-" + _digest())
    if os.path.exists(exe):
        return exe
    os.makedirs(BUILD, exist_ok=True)
    with open(os.path.join(BUILD, ".lock"), "w") as lk:
        fcntl.flock(lk, fcntl.LOCK_EX)
        try:
            return exe if os.path.exists(exe) else _build(exe)
        finally:
            fcntl.flock(lk, fcntl.LOCK_UN)


def _build(exe: str) -> str:
    src = os.path.join(BUILD, "src")
    shutil.rmtree(src, ignore_errors=True)
    os.makedirs(src)
    for n in SOURCES + HEADERS:
        text = open(os.path.join(CSRC, n)).read()
        text = text.replace(DYN_LDS, "char* lds = salt_cpu::g_dyn_lds;")
        with open(os.path.join(src, n), "w") as f:
            f.write(text)
    srcs = [os.path.join(src, n) for n in SOURCES] + [os.path.join(SHIM, "harness.cpp")]
    flags = ["-std=c++17", "-O1", "-g", "-fsanitize=address", "-fno-omit-frame-pointer", "-w"]
    for old in os.listdir(BUILD):
        if old.startswith("harness-") and old != os.path.basename(exe):
            os.remove(os.path.join(BUILD, old))
    # one compiler process per source, then one link
    objs = [os.path.join(src, os.path.basename(s) + ".o") for s in srcs]
    procs = [subprocess.Popen([CLANG, *flags, f"-I{SHIM}", f"-I{os.path.join(ROOT, 'include')}", f"-I{CSRC}",
                               "-x", "c++", "-c", s, "-o", o], stdout=subprocess.PIPE, stderr=subprocess.PIPE,
                              text=True) for s, o in zip(srcs, objs)]
    errs = [(p.communicate()[1], p.returncode) for p in procs]
    res = subprocess.run([CLANG, *flags, *objs, "-o", exe + ".tmp"], capture_output=True, text=True)
    if any(rc for _, rc in errs) or res.returncode != 0:
        msg = "".join(e for e, rc in errs if rc) + res.stderr
        raise RuntimeError("host build of libsalt failed:\n" + msg[-6000:])
    os.replace(exe + ".tmp", exe)
    return exe


class Batch:
    def __init__(self, tok_c, tok_u, gamma, tables: Sequence[int], xs: Sequence[np.ndarray],
                 y0s: Sequence[np.ndarray], mode: int = 0, plan: int = 0):
        self.tok_c = np.ascontiguousarray(tok_c, np.int32)
        self.tok_u = np.ascontiguousarray(tok_u, np.int32)
        self.gamma = None if gamma is None else np.ascontiguousarray(gamma, np.float32)
        self.tables = list(tables)
        self.xs = [np.ascontiguousarray(x) for x in xs]
        self.y0s = [np.ascontiguousarray(y) for y in y0s]
        self.mode = mode
        self.plan = plan


def run(dtype: str, shapes: Sequence, n_centroids: int, r_c: int, n_slots: int, r_u_max: int, max_tokens: int,
        centroids: Sequence, loads: Sequence, batches: Sequence[Batch], workdir: str, n_cu: int = 256) -> List[Dict]:
    """centroids: per table (At [C][r_c][in], B [C][r_c][out]) storage arrays (C > 0);
    loads: (slot, rank, blob) triples.  Returns per batch the statuses, the plan
    and the y arrays (storage form)."""
    exe = build()
    esize = 4 if dtype == "f32" else 2
    sdt = np.float32 if dtype == "f32" else np.uint16
    inp, outp = os.path.join(workdir, "in.bin"), os.path.join(workdir, "out.bin")
    with open(inp, "wb") as f:
        w = lambda *v: f.write(struct.pack(f"<{len(v)}i", *v))
        w(0x53414C54, 0 if dtype == "f32" else 1, len(shapes), n_centroids, r_c, n_slots, r_u_max, max_tokens, n_cu)
        for i, o in shapes:
            w(int(i), int(o))
        if n_centroids:
            for at, b in centroids:
                f.write(np.ascontiguousarray(at, sdt).tobytes())
                f.write(np.ascontiguousarray(b, sdt).tobytes())
        w(len(loads))
        for slot, rank, blob in loads:
            w(int(slot), int(rank))
            if rank:
                f.write(np.ascontiguousarray(blob, sdt).tobytes())
        w(len(batches))
        for bt in batches:
            T = len(bt.tok_c)
            w(bt.mode, bt.plan, T, 0 if bt.gamma is None else 1)
            f.write(bt.tok_c.tobytes())
            f.write(bt.tok_u.tobytes())
            if bt.gamma is not None:
                f.write(bt.gamma.tobytes())
            w(len(bt.tables))
            f.write(np.asarray(bt.tables, np.int32).tobytes())
            for x, y in zip(bt.xs, bt.y0s):
                f.write(np.ascontiguousarray(x, sdt).tobytes())
                f.write(np.ascontiguousarray(y, sdt).tobytes())
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=0")
    res = subprocess.run([exe, inp, outp], capture_output=True, text=True, env=env, timeout=1800)
    if res.returncode != 0:
        raise RuntimeError(f"host build of libsalt exited with {res.returncode}:\n{res.stderr[-6000:]}")
    data = open(outp, "rb").read()
    pos = 0

    def ints(n):
        nonlocal pos
        a = np.frombuffer(data, np.int32, count=n, offset=pos).copy()
        pos += 4 * n
        return a

    out = []
    for bt in batches:
        T = len(bt.tok_c)
        s_set, s_build, s_apply, s_err, n_err, n_seg, n_grp, tile_m, n_tiles = ints(9)
        r = dict(status=(int(s_set), int(s_build), int(s_apply), int(s_err)), n_errors=int(n_err),
                 tile_tokens=int(tile_m), n_tiles=int(n_tiles))
        r["perm"] = ints(T)
        r["seg_off"] = ints(n_seg + 1)
        r["seg_c"] = ints(n_seg)
        r["seg_u"] = ints(n_seg)
        r["grp_off"] = ints(n_grp + 1)
        ys = []
        for t, y0 in zip(bt.tables, bt.y0s):
            n = y0.size
            ys.append(np.frombuffer(data, sdt, count=n, offset=pos).reshape(y0.shape).copy())
            pos += n * esize
        r["ys"] = ys
        r["stderr"] = res.stderr
        out.append(r)
    return out
