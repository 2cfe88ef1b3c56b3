"""Test-side driver: runs a synthetic workload through libsalt and through the oracle.

GPU side: the C ABI via ``paper_2608_03579_amd.salt``; device memory and the stream
come from ``paper_2608_03579_amd.hip`` (the HIP runtime libsalt links).  CPU side: ``oracle`` on the same seeded inputs.
"""
from __future__ import annotations

import numpy as np

import oracle
from paper_2608_03579_amd import synth

TOL_BF16 = 1e-2      # |y - ref| <= 1e-2 * (1 + |ref|) for bf16 outputs
TOL_F32 = 1e-5             # fp32 Tiny config: fp32 accumulation of K <= 256 terms


def hipmod():
    from paper_2608_03579_amd import hip
    return hip


def to_dev(a: np.ndarray):
    return hipmod().DeviceArray.from_host(np.ascontiguousarray(a))


def to_host(d, dtype: str) -> np.ndarray:
    return d.to_host()


def close_enough(got: np.ndarray, ref: np.ndarray, tol: float):
    """Element-wise |got - ref| <= tol * (1 + |ref|); returns (ok, worst ratio, n_bad)."""
    err = np.abs(got - ref)
    bound = tol * (1.0 + np.abs(ref))
    ratio = err / bound
    return bool(np.all(err <= bound)), float(ratio.max(initial=0.0)), int(np.sum(err > bound))


def fuse_within_bound(got: np.ndarray, ref: np.ndarray, w0: np.ndarray, a: np.ndarray, b: np.ndarray,
                      gamma: float, dtype: str):
    """Bound of a fused weight (rne of W + gamma * A B with an fp32 contraction):
    one rounding of the result, 2^-8 |ref| for bf16 (2^-22 for fp32), plus the
    fp32 accumulation error, 2^-16 (|W| + |gamma| sum_r |A_ir B_ro|).  Returns
    (ok, worst ratio, n_bad)."""
    rel = 2.0 ** -8 if dtype == "bf16" else 2.0 ** -22
    bound = rel * np.abs(ref) + 2.0 ** -16 * (np.abs(w0) + abs(gamma) * (np.abs(a).T @ np.abs(b)))
    err = np.abs(got - ref)
    return bool(np.all(err <= bound)), float(np.max(err / bound, initial=0.0)), int(np.sum(err > bound))


class Run:
    """One context + one plan for workload ``w``; residual generations per slot."""

    def __init__(self, w: synth.Workload, max_tokens: int = None, pin_tables=None):
        from paper_2608_03579_amd import salt
        self.salt = salt
        self.w = w
        self.gen = {}
        tables = [(i, o) for _, i, o in w.tables]
        self.ctx = salt.Context(w.dtype, tables, w.n_centroids, w.r_c, w.n_slots, w.r_u_max,
                                max_tokens or max(1, w.T))
        if w.n_centroids:
            for t in (range(len(tables)) if pin_tables is None else pin_tables):
                at, b = w.centroids(t)
                self.ctx.pin_centroids(t, at, b)
        for s in w.referenced_slots():
            self.load(int(s), 0)
        self.ctx.wait_loads()
        self.plan = self.ctx.plan()
        self._stream = hipmod().Stream()
        self.stream = self._stream.h

    def load(self, slot: int, gen: int):
        r = int(self.w.slot_rank[slot])
        self.ctx.load_residual(slot, r, self.w.residual_blob(slot, gen) if r else None)
        self.gen[slot] = gen

    def set_and_build(self, tok_c=None, tok_u=None, gamma="w"):
        w = self.w
        tok_c = w.tok_c if tok_c is None else tok_c
        tok_u = w.tok_u if tok_u is None else tok_u
        g = w.gamma if isinstance(gamma, str) else gamma
        self.maps = (np.asarray(tok_c, np.int32), np.asarray(tok_u, np.int32), g)
        self.plan.set_maps(tok_c, tok_u, g, self.stream)
        self.plan.build(self.stream)

    def apply(self, table: int, x=None, y0=None):
        w = self.w
        xd = to_dev(w.x(table) if x is None else x)
        yd = to_dev(w.y0(table) if y0 is None else y0)
        self.ctx.apply(table, self.plan, xd.ptr, yd.ptr, self.stream)
        self._stream.synchronize()
        out = yd.to_host()
        xd.free()
        yd.free()
        return out

    def apply_batch(self, tables, xs=None, y0s=None):
        """salt_apply_batch of several tables in one call; returns their y arrays."""
        w = self.w
        xd = [to_dev(w.x(t) if xs is None else xs[i]) for i, t in enumerate(tables)]
        yd = [to_dev(w.y0(t) if y0s is None else y0s[i]) for i, t in enumerate(tables)]
        self.ctx.apply_batch(tables, self.plan, [d.ptr for d in xd], [d.ptr for d in yd], self.stream)
        self._stream.synchronize()
        out = [d.to_host() for d in yd]
        for d in xd + yd:
            d.free()
        return out

    # ---- oracle side ----------------------------------------------------------
    def oracle_table(self, table: int, rows=None):
        w = self.w
        d = w.dtype
        tok_c, tok_u, g = self.maps
        need = range(len(tok_c)) if rows is None else rows
        used_rows = sorted(set(int(r) for r in need))
        pos = {r: i for i, r in enumerate(used_rows)}
        x = oracle.decode(w.x(table, rows=used_rows), d)
        y0 = oracle.decode(w.y0(table, rows=used_rows), d)
        if w.n_centroids:
            cat, cb = (oracle.decode(a, d) for a in w.centroids(table))
        else:
            _, i, o = w.tables[table]
            cat, cb = np.zeros((0, 0, i)), np.zeros((0, 0, o))
        res = {}
        for s in set(int(tok_u[r]) for r in used_rows if tok_u[r] >= 0):
            res[s] = tuple(oracle.decode(a, d) for a in w.residual(s, table, self.gen.get(s, 0)))
        sub_c = np.asarray([tok_c[r] for r in used_rows], np.int32)
        sub_u = np.asarray([tok_u[r] for r in used_rows], np.int32)
        sub_g = None if g is None else np.asarray([g[r] for r in used_rows], np.float32)
        ref = oracle.apply(x, y0, cat, cb, res, sub_c, sub_u, sub_g)
        return ref[[pos[int(r)] for r in need]]

    def close(self):
        self.plan.close()
        self.ctx.close()
        self._stream.destroy()
