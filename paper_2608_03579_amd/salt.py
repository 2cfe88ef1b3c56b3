"""ctypes binding of the libsalt C ABI (``include/salt.h``).

Argument marshalling only: every step of the apply runs in libsalt's HIP kernels.
Device buffers are passed as raw device addresses (``hip.DeviceArray.ptr``, or any
allocation of the HIP runtime libsalt links) and streams as ``hipStream_t`` values;
host arrays are numpy arrays.  There is no fallback: if ``libsalt.so`` is missing
the import of this module fails.
"""
from __future__ import annotations

import ctypes as C
import os
from typing import Dict, Optional, Sequence, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libsalt.so")

OK, ERR_INVALID_ARG, ERR_OUT_OF_RANGE, ERR_OUT_OF_MEMORY, ERR_NOT_PINNED, ERR_SLOT_EMPTY, \
    ERR_HIP, ERR_BAD_STATE = range(8)
F32, BF16 = 0, 1

# every entry point declared in include/salt.h
EXPORTS = (
    "salt_create", "salt_destroy", "salt_pin_centroids", "salt_residual_bytes",
    "salt_residual_bytes_for", "salt_load_residual", "salt_load_residuals", "salt_wait_loads",
    "salt_host_alloc", "salt_host_free", "salt_plan_create", "salt_plan_destroy", "salt_plan_set_maps",
    "salt_plan_build", "salt_plan_download", "salt_plan_errors", "salt_plan_tiling", "salt_apply",
    "salt_apply_batch", "salt_apply_batch_noalloc", "salt_apply_batch_timed", "salt_apply_map", "salt_fuse_centroid",
    "salt_fuse_centroid_timed", "salt_adapter_gram", "salt_route",
    "salt_status_str",
    "salt_last_error", "salt_version",
)


class Shape(C.Structure):
    _fields_ = [("in_dim", C.c_int32), ("out_dim", C.c_int32)]


class Config(C.Structure):
    _fields_ = [("dtype", C.c_int), ("n_tables", C.c_int32), ("tables", C.POINTER(Shape)),
                ("n_centroids", C.c_int32), ("r_c", C.c_int32), ("n_slots", C.c_int32),
                ("r_u_max", C.c_int32), ("max_tokens", C.c_int32), ("device", C.c_int32),
                ("flags", C.c_int32)]



class RouteResult(C.Structure):
    _fields_ = [("k_star", C.c_int32), ("ood", C.c_int32), ("blended", C.c_int32), ("z_n_min", C.c_double),
                ("z_r_min", C.c_double)]


def _load() -> C.CDLL:
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run `python -m paper_2608_03579_amd.build`")
    lib = C.CDLL(LIB_PATH)
    P, I32, SZ, VP = C.c_void_p, C.c_int32, C.c_size_t, C.c_void_p
    IP = C.POINTER(C.c_int32)
    sig = {
        "salt_create": (C.c_int, [C.POINTER(Config), C.POINTER(P)]),
        "salt_destroy": (None, [P]),
        "salt_pin_centroids": (C.c_int, [P, I32, I32, I32, VP, VP]),
        "salt_residual_bytes": (SZ, [P, I32]),
        "salt_residual_bytes_for": (SZ, [C.c_int, I32, C.POINTER(Shape), I32]),
        "salt_load_residual": (C.c_int, [P, I32, I32, VP, SZ]),
        "salt_load_residuals": (C.c_int, [P, I32, IP, IP, C.POINTER(VP), C.POINTER(SZ)]),
        "salt_wait_loads": (C.c_int, [P]),
        "salt_host_alloc": (C.c_int, [SZ, C.POINTER(VP)]),
        "salt_host_free": (None, [VP]),
        "salt_plan_create": (C.c_int, [P, C.POINTER(P)]),
        "salt_plan_destroy": (None, [P, P]),
        "salt_plan_set_maps": (C.c_int, [P, P, I32, IP, IP, C.POINTER(C.c_float), VP]),
        "salt_plan_build": (C.c_int, [P, P, VP]),
        "salt_plan_download": (C.c_int, [P, P, VP, IP, IP, IP, IP, IP, IP, IP]),
        "salt_plan_errors": (C.c_int, [P, P, VP, IP]),
        "salt_plan_tiling": (C.c_int, [P, P, IP, IP, IP]),
        "salt_apply": (C.c_int, [P, I32, P, VP, VP, VP]),
        "salt_apply_batch": (C.c_int, [P, I32, IP, P, C.POINTER(VP), C.POINTER(VP), VP]),
        "salt_apply_batch_noalloc": (C.c_int, [P, I32, IP, P, C.POINTER(VP), C.POINTER(VP), VP]),
        "salt_apply_batch_timed": (C.c_int, [P, I32, IP, P, C.POINTER(VP), C.POINTER(VP), VP, C.POINTER(VP)]),
        "salt_apply_map": (C.c_int, [P, I32, I32, IP, IP, C.POINTER(C.c_float), VP, VP, VP]),
        "salt_fuse_centroid": (C.c_int, [P, I32, I32, C.c_float, VP, C.c_int64, VP]),
        "salt_fuse_centroid_timed": (C.c_int, [P, I32, I32, C.c_float, VP, C.c_int64, VP, VP, VP]),
        "salt_adapter_gram": (C.c_int, [P, VP, I32, VP, I32, C.POINTER(C.c_double), VP]),
        "salt_route": (C.c_int, [I32] + [C.POINTER(C.c_double)] * 5 + [C.c_double, C.c_double] +
                       [C.POINTER(C.c_double)] * 2 + [C.POINTER(RouteResult)]),
        "salt_status_str": (C.c_char_p, [C.c_int]),
        "salt_last_error": (C.c_char_p, [P]),
        "salt_version": (I32, []),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    return lib


lib = _load()


def route(n, mu_n, sigma_n, mu_r, sigma_r, tau_n: float = 2.0, tau_r: float = 2.0):
    """salt_route (Sec. 3.2, host only): returns (status, result dict)."""
    K = len(n)
    arrs = [np.ascontiguousarray(a, dtype=np.float64) for a in (n, mu_n, sigma_n, mu_r, sigma_r)]
    z_n = np.zeros(K, np.float64)
    z_r = np.zeros(K, np.float64)
    res = RouteResult()
    dp = C.POINTER(C.c_double)
    st = lib.salt_route(K, *[a.ctypes.data_as(dp) for a in arrs], tau_n, tau_r, z_n.ctypes.data_as(dp),
                        z_r.ctypes.data_as(dp), C.byref(res))
    return st, {"k_star": res.k_star, "ood": bool(res.ood), "blended": bool(res.blended), "z_n_min": res.z_n_min,
                "z_r_min": res.z_r_min, "z_n": z_n, "z_r": z_r}


class SaltError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{lib.salt_status_str(status).decode()} ({status}): {msg}")
        self.status = status


def _i32p(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(C.POINTER(C.c_int32))


def residual_bytes_for(dtype: int, tables: Sequence[Tuple[int, int]], r_u: int) -> int:
    arr = (Shape * len(tables))(*[Shape(int(i), int(o)) for i, o in tables])
    return int(lib.salt_residual_bytes_for(dtype, len(tables), arr, r_u))


class HostBuffer:
    """Page-locked host memory from salt_host_alloc, viewed as a numpy array."""

    def __init__(self, nbytes: int):
        p = C.c_void_p()
        st = lib.salt_host_alloc(max(16, int(nbytes)), C.byref(p))
        if st != OK:
            raise SaltError(st, f"salt_host_alloc({nbytes})")
        self.ptr = p.value
        self.nbytes = int(nbytes)

    def view(self, dtype) -> np.ndarray:
        buf = (C.c_char * max(16, self.nbytes)).from_address(self.ptr)
        return np.frombuffer(buf, dtype=np.uint8, count=self.nbytes).view(dtype)

    def free(self):
        if self.ptr:
            lib.salt_host_free(self.ptr)
            self.ptr = None

    def __del__(self):
        try:
            self.free()
        except Exception:
            pass


class Context:
    """One libsalt context: centroid store, residual slot pool, side stream."""

    _N_STAGE = 8

    def __init__(self, dtype: str, tables: Sequence[Tuple[int, int]], n_centroids: int, r_c: int,
                 n_slots: int, r_u_max: int, max_tokens: int, device: int = 0):
        self.dtype = dtype
        self._shapes = (Shape * len(tables))(*[Shape(int(i), int(o)) for i, o in tables])
        cfg = Config(F32 if dtype == "f32" else BF16, len(tables), self._shapes, n_centroids, r_c,
                     n_slots, r_u_max, max_tokens, device, 0)
        h = C.c_void_p()
        st = lib.salt_create(C.byref(cfg), C.byref(h))
        if st != OK:
            raise SaltError(st, "salt_create: " + lib.salt_last_error(None).decode())
        self.h = h.value
        self.tables = [tuple(t) for t in tables]
        self._blobs: Dict[int, HostBuffer] = {}
        self._stage_next = 0

    def _check(self, st: int, what: str):
        if st != OK:
            raise SaltError(st, f"{what}: {lib.salt_last_error(self.h).decode()}")

    def close(self):
        if getattr(self, "h", None):
            lib.salt_destroy(self.h)
            self.h = None
        for b in self._blobs.values():
            b.free()
        self._blobs.clear()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def pin_centroids(self, table: int, at: np.ndarray, b: np.ndarray, c0: int = 0):
        at = np.ascontiguousarray(at)
        b = np.ascontiguousarray(b)
        self._check(lib.salt_pin_centroids(self.h, table, c0, at.shape[0], at.ctypes.data,
                                           b.ctypes.data), "salt_pin_centroids")

    def residual_bytes(self, r_u: int) -> int:
        return int(lib.salt_residual_bytes(self.h, r_u))

    def load_residual(self, slot: int, r_u: int, blob: Optional[np.ndarray]):
        """Swap ``blob`` (any host array) into ``slot``.

        The blob is first copied into one of a few page-locked staging buffers that
        the binding reuses round-robin; before a buffer is reused the earlier swaps
        are waited for, so an asynchronous copy never reads a recycled buffer."""
        nbytes = self.residual_bytes(r_u)
        if r_u == 0:
            self._check(lib.salt_load_residual(self.h, slot, 0, None, 0), "salt_load_residual")
            return
        src = np.ascontiguousarray(blob).view(np.uint8).reshape(-1)
        if src.nbytes != nbytes:
            raise SaltError(ERR_INVALID_ARG, f"blob has {src.nbytes} bytes, rank {r_u} needs {nbytes}")
        k = self._stage_next % self._N_STAGE
        if self._stage_next >= self._N_STAGE and k == 0:
            self.wait_loads()
        self._stage_next += 1
        buf = self._blobs.get(k)
        if buf is None or buf.nbytes < nbytes:
            if buf is not None:
                self.wait_loads()
                buf.free()
            buf = HostBuffer(nbytes)
            self._blobs[k] = buf
        buf.view(np.uint8)[:nbytes] = src
        self._check(lib.salt_load_residual(self.h, slot, r_u, buf.ptr, nbytes), "salt_load_residual")

    def load_residual_ptr(self, slot: int, r_u: int, ptr: int, nbytes: int) -> int:
        """Raw call: ``ptr`` must be page-locked host memory.  Returns the status."""
        return lib.salt_load_residual(self.h, slot, r_u, ptr, nbytes)

    def wait_loads(self):
        self._check(lib.salt_wait_loads(self.h), "salt_wait_loads")

    def plan(self) -> "Plan":
        return Plan(self)

    def apply(self, table: int, plan: "Plan", x_ptr: int, y_ptr: int, stream: int = 0):
        self._check(lib.salt_apply(self.h, table, plan.h, x_ptr, y_ptr, stream), "salt_apply")

    def apply_status(self, table: int, plan: "Plan", x_ptr: int, y_ptr: int, stream: int = 0) -> int:
        return lib.salt_apply(self.h, table, plan.h, x_ptr, y_ptr, stream)

    @staticmethod
    def _ptrs(ptrs):
        return (C.c_void_p * len(ptrs))(*[C.c_void_p(int(p)) for p in ptrs])

    def apply_batch(self, tables: Sequence[int], plan: "Plan", x_ptrs: Sequence[int], y_ptrs: Sequence[int],
                    stream: int = 0):
        """salt_apply_batch: tables[i] with x_ptrs[i] -> y_ptrs[i], one plan."""
        n = len(tables)
        tabs = np.ascontiguousarray(tables, dtype=np.int32)
        self._check(lib.salt_apply_batch(self.h, n, _i32p(tabs), plan.h, self._ptrs(x_ptrs), self._ptrs(y_ptrs),
                                         stream), "salt_apply_batch")

    def apply_batch_noalloc(self, tables: Sequence[int], plan: "Plan", x_ptrs: Sequence[int],
                            y_ptrs: Sequence[int], stream: int = 0):
        """salt_apply_batch_noalloc: salt_apply_batch with the partials in the
        library's static device scratch (no allocation)."""
        self._check(self.apply_batch_noalloc_status(tables, plan, x_ptrs, y_ptrs, stream), "salt_apply_batch_noalloc")

    def apply_batch_noalloc_status(self, tables, plan, x_ptrs, y_ptrs, stream: int = 0) -> int:
        tabs = np.ascontiguousarray(tables, dtype=np.int32)
        return lib.salt_apply_batch_noalloc(self.h, len(tables), _i32p(tabs), plan.h, self._ptrs(x_ptrs),
                                            self._ptrs(y_ptrs), stream)

    def apply_batch_status(self, tables, plan, x_ptrs, y_ptrs, stream: int = 0) -> int:
        tabs = np.ascontiguousarray(tables, dtype=np.int32)
        return lib.salt_apply_batch(self.h, len(tables), _i32p(tabs), plan.h, self._ptrs(x_ptrs),
                                    self._ptrs(y_ptrs), stream)

    def apply_batch_timed(self, tables, plan, x_ptrs, y_ptrs, stream: int, events: Sequence[int]):
        """``apply_batch`` (one launch) whose four HIP events record the start and end
        of the shrink kernel and of the expand kernel."""
        tabs = np.ascontiguousarray(tables, dtype=np.int32)
        self._check(lib.salt_apply_batch_timed(self.h, len(tables), _i32p(tabs), plan.h, self._ptrs(x_ptrs),
                                               self._ptrs(y_ptrs), stream, self._ptrs(events)),
                    "salt_apply_batch_timed")

    def apply_map(self, table: int, tok_c, tok_u, gamma, x_ptr: int, y_ptr: int, stream: int = 0):
        """salt_apply_map: build + apply on host maps with the context's own plan."""
        st = self.apply_map_status(table, tok_c, tok_u, gamma, x_ptr, y_ptr, stream)
        self._check(st, "salt_apply_map")

    def apply_map_status(self, table: int, tok_c, tok_u, gamma, x_ptr: int, y_ptr: int, stream: int = 0) -> int:
        tok_c = np.ascontiguousarray(tok_c, dtype=np.int32)
        tok_u = np.ascontiguousarray(tok_u, dtype=np.int32)
        g = None if gamma is None else np.ascontiguousarray(gamma, dtype=np.float32)
        gp = None if g is None else g.ctypes.data_as(C.POINTER(C.c_float))
        return lib.salt_apply_map(self.h, table, int(tok_c.shape[0]), _i32p(tok_c), _i32p(tok_u), gp, x_ptr, y_ptr,
                                  stream)

    def load_residuals_ptr(self, slots: Sequence[int], ranks: Sequence[int], ptrs: Sequence[int],
                           nbytes: Sequence[int]) -> int:
        """salt_load_residuals on page-locked blobs; returns the status."""
        sl = np.ascontiguousarray(slots, dtype=np.int32)
        rk = np.ascontiguousarray(ranks, dtype=np.int32)
        sz = (C.c_size_t * len(nbytes))(*[int(n) for n in nbytes])
        return lib.salt_load_residuals(self.h, len(sl), _i32p(sl), _i32p(rk), self._ptrs(ptrs), sz)

    def fuse_centroid(self, table: int, c: int, gamma: float, w_ptr: int, ldw: int, stream: int = 0):
        """Fold gamma * centroid c of `table` into the base weight at w_ptr ([in][ldw], device)."""
        self._check(lib.salt_fuse_centroid(self.h, table, c, gamma, w_ptr, ldw, stream), "salt_fuse_centroid")

    def fuse_centroid_status(self, table: int, c: int, gamma: float, w_ptr: int, ldw: int, stream: int = 0) -> int:
        return lib.salt_fuse_centroid(self.h, table, c, gamma, w_ptr, ldw, stream)

    def adapter_gram(self, blob1_ptr: int, r1: int, blob2_ptr: int, r2: int, stream: int = 0) -> np.ndarray:
        """Per table (Tr(dW1^T dW2), ||dW1||^2, ||dW2||^2) of two adapter blobs in device memory."""
        out = np.zeros((len(self.tables), 3), dtype=np.float64)
        self._check(lib.salt_adapter_gram(self.h, blob1_ptr, r1, blob2_ptr, r2,
                                          out.ctypes.data_as(C.POINTER(C.c_double)), stream), "salt_adapter_gram")
        return out

    def adapter_gram_status(self, blob1_ptr: int, r1: int, blob2_ptr: int, r2: int, stream: int = 0) -> int:
        out = np.zeros((len(self.tables), 3), dtype=np.float64)
        return lib.salt_adapter_gram(self.h, blob1_ptr, r1, blob2_ptr, r2,
                                     out.ctypes.data_as(C.POINTER(C.c_double)), stream)

    def fuse_centroid_timed(self, table: int, c: int, gamma: float, w_ptr: int, ldw: int, stream: int,
                            start_event: int, stop_event: int):
        """``fuse_centroid`` whose two HIP events record the kernel's own start and end."""
        self._check(lib.salt_fuse_centroid_timed(self.h, table, c, gamma, w_ptr, ldw, stream, start_event,
                                                 stop_event), "salt_fuse_centroid_timed")


class Plan:
    def __init__(self, ctx: Context):
        self.ctx = ctx
        h = C.c_void_p()
        ctx._check(lib.salt_plan_create(ctx.h, C.byref(h)), "salt_plan_create")
        self.h = h.value
        self.T = 0

    def close(self):
        if self.h and self.ctx.h:
            lib.salt_plan_destroy(self.ctx.h, self.h)
        self.h = None

    def set_maps(self, tok_c: np.ndarray, tok_u: np.ndarray, gamma: Optional[np.ndarray] = None,
                 stream: int = 0):
        tok_c = np.ascontiguousarray(tok_c, dtype=np.int32)
        tok_u = np.ascontiguousarray(tok_u, dtype=np.int32)
        g = None if gamma is None else np.ascontiguousarray(gamma, dtype=np.float32)
        gp = None if g is None else g.ctypes.data_as(C.POINTER(C.c_float))
        self.ctx._check(lib.salt_plan_set_maps(self.ctx.h, self.h, int(tok_c.shape[0]), _i32p(tok_c),
                                               _i32p(tok_u), gp, stream), "salt_plan_set_maps")
        self.T = int(tok_c.shape[0])

    def set_maps_status(self, tok_c, tok_u, gamma=None, stream: int = 0) -> int:
        tok_c = np.ascontiguousarray(tok_c, dtype=np.int32)
        tok_u = np.ascontiguousarray(tok_u, dtype=np.int32)
        g = None if gamma is None else np.ascontiguousarray(gamma, dtype=np.float32)
        gp = None if g is None else g.ctypes.data_as(C.POINTER(C.c_float))
        return lib.salt_plan_set_maps(self.ctx.h, self.h, int(tok_c.shape[0]), _i32p(tok_c), _i32p(tok_u),
                                      gp, stream)

    def build(self, stream: int = 0):
        self.ctx._check(lib.salt_plan_build(self.ctx.h, self.h, stream), "salt_plan_build")

    def errors(self, stream: int = 0) -> int:
        n = C.c_int32()
        self.ctx._check(lib.salt_plan_errors(self.ctx.h, self.h, stream, C.byref(n)), "salt_plan_errors")
        return int(n.value)

    def tiling(self) -> Tuple[int, int, int]:
        """(tokens per tile, tiles, kernel launches per apply) of the staged maps."""
        m, n, l = C.c_int32(), C.c_int32(), C.c_int32()
        self.ctx._check(lib.salt_plan_tiling(self.ctx.h, self.h, C.byref(m), C.byref(n), C.byref(l)),
                        "salt_plan_tiling")
        return int(m.value), int(n.value), int(l.value)

    def download(self, stream: int = 0) -> Dict[str, np.ndarray]:
        T = self.T
        perm = np.zeros(T + 1, np.int32)
        seg_off = np.zeros(T + 1, np.int32)
        seg_c = np.zeros(T + 1, np.int32)
        seg_u = np.zeros(T + 1, np.int32)
        grp_off = np.zeros(T + 1, np.int32)
        ns, ng = C.c_int32(), C.c_int32()
        self.ctx._check(lib.salt_plan_download(self.ctx.h, self.h, stream, _i32p(perm), _i32p(seg_off),
                                               _i32p(seg_c), _i32p(seg_u), _i32p(grp_off),
                                               C.byref(ns), C.byref(ng)), "salt_plan_download")
        n_seg, n_grp = ns.value, ng.value
        return dict(perm=perm[:T], seg_off=seg_off[:n_seg + 1], seg_c=seg_c[:n_seg],
                    seg_u=seg_u[:n_seg], grp_off=grp_off[:n_grp + 1])
