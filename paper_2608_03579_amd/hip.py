"""Device memory, streams and events through the HIP runtime that libsalt links.

Plumbing only (allocation, copies, streams, timing events).  It binds the same
``libamdhip64.so.7`` instance that ``libsalt.so`` loads, so pointers and streams
created here are valid for libsalt.  PyTorch wheels bundle a second HIP runtime;
two runtimes in one process do not share a device, so processes that drive
libsalt use this module and do not initialise torch's GPU support.
"""
from __future__ import annotations

import ctypes as C
import os
from typing import Optional, Sequence

import numpy as np

from . import salt as _salt  # noqa: F401  (loads libsalt first, which pulls in its HIP runtime)

_ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
_hip = C.CDLL(os.path.join(_ROCM, "lib", "libamdhip64.so.7"))

_H2D, _D2H, _D2D = 1, 2, 3
_hip.hipGetErrorString.restype = C.c_char_p
_hip.hipGetErrorString.argtypes = [C.c_int]
for _n, _a in {
    "hipMalloc": [C.POINTER(C.c_void_p), C.c_size_t],
    "hipFree": [C.c_void_p],
    "hipMemcpy": [C.c_void_p, C.c_void_p, C.c_size_t, C.c_int],
    "hipMemcpyAsync": [C.c_void_p, C.c_void_p, C.c_size_t, C.c_int, C.c_void_p],
    "hipMemsetAsync": [C.c_void_p, C.c_int, C.c_size_t, C.c_void_p],
    "hipDeviceSynchronize": [],
    "hipSetDevice": [C.c_int],
    "hipGetDeviceCount": [C.POINTER(C.c_int)],
    "hipStreamCreateWithFlags": [C.POINTER(C.c_void_p), C.c_uint],
    "hipStreamDestroy": [C.c_void_p],
    "hipStreamSynchronize": [C.c_void_p],
    "hipEventCreate": [C.POINTER(C.c_void_p)],
    "hipEventDestroy": [C.c_void_p],
    "hipEventRecord": [C.c_void_p, C.c_void_p],
    "hipEventSynchronize": [C.c_void_p],
    "hipEventElapsedTime": [C.POINTER(C.c_float), C.c_void_p, C.c_void_p],
    "hipMemGetInfo": [C.POINTER(C.c_size_t), C.POINTER(C.c_size_t)],
}.items():
    getattr(_hip, _n).restype = C.c_int
    getattr(_hip, _n).argtypes = _a


class HipError(RuntimeError):
    pass


def check(err: int, what: str = ""):
    if err != 0:
        raise HipError(f"{what}: {_hip.hipGetErrorString(err).decode()} ({err})")


def device_count() -> int:
    n = C.c_int(0)
    err = _hip.hipGetDeviceCount(C.byref(n))
    return n.value if err == 0 else 0


def set_device(d: int = 0):
    check(_hip.hipSetDevice(d), "hipSetDevice")


def synchronize():
    check(_hip.hipDeviceSynchronize(), "hipDeviceSynchronize")


def mem_info():
    free, total = C.c_size_t(), C.c_size_t()
    check(_hip.hipMemGetInfo(C.byref(free), C.byref(total)), "hipMemGetInfo")
    return free.value, total.value


class DeviceArray:
    """A device allocation with a numpy dtype and shape (row-major)."""

    def __init__(self, shape: Sequence[int], dtype):
        self.shape = tuple(int(s) for s in shape)
        self.dtype = np.dtype(dtype)
        self.nbytes = int(np.prod(self.shape, dtype=np.int64)) * self.dtype.itemsize
        p = C.c_void_p()
        check(_hip.hipMalloc(C.byref(p), max(self.nbytes, 256)), f"hipMalloc({self.nbytes})")
        self.ptr = p.value

    @classmethod
    def from_host(cls, a: np.ndarray) -> "DeviceArray":
        a = np.ascontiguousarray(a)
        d = cls(a.shape, a.dtype)
        d.upload(a)
        return d

    def upload(self, a: np.ndarray):
        a = np.ascontiguousarray(a, dtype=self.dtype)
        assert a.nbytes == self.nbytes
        check(_hip.hipMemcpy(self.ptr, a.ctypes.data, self.nbytes, _H2D), "hipMemcpy H2D")

    def to_host(self) -> np.ndarray:
        out = np.empty(self.shape, self.dtype)
        check(_hip.hipMemcpy(out.ctypes.data, self.ptr, self.nbytes, _D2H), "hipMemcpy D2H")
        return out

    def copy_from(self, other: "DeviceArray", stream: Optional["Stream"] = None):
        assert other.nbytes == self.nbytes
        check(_hip.hipMemcpyAsync(self.ptr, other.ptr, self.nbytes, _D2D, stream.h if stream else None),
              "hipMemcpyAsync D2D")

    def free(self):
        if self.ptr:
            _hip.hipFree(self.ptr)
            self.ptr = None

    def __del__(self):
        try:
            self.free()
        except Exception:
            pass


class Stream:
    def __init__(self, non_blocking: bool = True):
        h = C.c_void_p()
        check(_hip.hipStreamCreateWithFlags(C.byref(h), 1 if non_blocking else 0), "hipStreamCreate")
        self.h = h.value

    def synchronize(self):
        check(_hip.hipStreamSynchronize(self.h), "hipStreamSynchronize")

    def destroy(self):
        if self.h:
            _hip.hipStreamDestroy(self.h)
            self.h = None


class Event:
    def __init__(self):
        h = C.c_void_p()
        check(_hip.hipEventCreate(C.byref(h)), "hipEventCreate")
        self.h = h.value

    def record(self, stream: Optional[Stream] = None):
        check(_hip.hipEventRecord(self.h, stream.h if stream else None), "hipEventRecord")

    def synchronize(self):
        check(_hip.hipEventSynchronize(self.h), "hipEventSynchronize")

    def elapsed_ms(self, later: "Event") -> float:
        ms = C.c_float()
        check(_hip.hipEventElapsedTime(C.byref(ms), self.h, later.h), "hipEventElapsedTime")
        return float(ms.value)

    def destroy(self):
        if self.h:
            _hip.hipEventDestroy(self.h)
            self.h = None
