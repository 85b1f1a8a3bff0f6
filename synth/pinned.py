"""Exact-size pinned host buffers (hipHostMalloc / hipHostFree).

torch's pinned allocator rounds requests up to a power of two and caches
freed blocks, which wastes tens of GB for the largest workload's host
buffers; these buffers are allocated at their exact size and freed when
closed.  `.tensor` is a CPU uint8 view of the same memory.
"""
from __future__ import annotations

import ctypes as C

import torch

_hip = None


def _lib():
    global _hip
    if _hip is None:
        _hip = C.CDLL("libamdhip64.so")
        _hip.hipHostMalloc.argtypes = [C.POINTER(C.c_void_p), C.c_size_t, C.c_uint]
        _hip.hipHostMalloc.restype = C.c_int
        _hip.hipHostFree.argtypes = [C.c_void_p]
        _hip.hipHostFree.restype = C.c_int
        _hip.hipGetLastError.argtypes = []
        _hip.hipGetLastError.restype = C.c_int
    return _hip


class Pinned:
    def __init__(self, nbytes: int, fill: int | None = None):
        self.nbytes = max(int(nbytes), 1)
        p = C.c_void_p()
        rc = _lib().hipHostMalloc(C.byref(p), self.nbytes, 0)
        if rc != 0 or not p.value:
            # a failed call also leaves its error as the thread's last HIP
            # error, which torch's next kernel launch check would report as
            # its own: clear it
            _lib().hipGetLastError()
            raise MemoryError(f"hipHostMalloc({self.nbytes}) failed with HIP error {rc}")
        self.ptr = p.value
        arr = (C.c_uint8 * self.nbytes).from_address(self.ptr)
        self.tensor = torch.frombuffer(arr, dtype=torch.uint8)
        if fill is not None:
            self.tensor.fill_(fill)

    def close(self):
        if self.ptr:
            self.tensor = None
            _lib().hipHostFree(C.c_void_p(self.ptr))
            self.ptr = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
