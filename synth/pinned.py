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


class Pageable:
    """Ordinary (pageable) host memory, 256-byte aligned, with the interface
    of Pinned."""

    def __init__(self, nbytes: int, fill: int | None = None):
        self.nbytes = max(int(nbytes), 1)
        self._raw = torch.empty(self.nbytes + 256, dtype=torch.uint8)
        off = (-self._raw.data_ptr()) % 256
        self.tensor = self._raw[off:off + self.nbytes]
        self.ptr = self.tensor.data_ptr()
        if fill is not None:
            self.tensor.fill_(fill)

    def close(self):
        self.tensor = self._raw = None


def host_buffers(sizes, force_pageable: bool = False):
    """Host buffers of one reshard, from `sizes` = [(bytes, fill, dma_only)].

    Every buffer is pinned if the host can pin them all at once (about 69 GB
    for the 80-layer TP 8->7 share).  Otherwise the buffers that only DMA
    copies touch (`dma_only`: the in-place KV inflow, which lands through the
    landing ring) are taken as ordinary memory and the rest pinned; the copy
    kernel itself reads or writes the others, so they must be pinned.
    Returns (buffers, pageable bytes); raises MemoryError, having freed what
    it took, when even that fails."""
    err = None
    for pageable_dma in ((True,) if force_pageable else (False, True)):
        if pageable_dma and not any(d for _, _, d in sizes):
            break
        bufs = []
        try:
            for nbytes, f, dma_only in sizes:
                bufs.append((Pageable if pageable_dma and dma_only else Pinned)(nbytes, fill=f))
            return bufs, sum(int(n) for n, _, d in sizes if d) if pageable_dma else 0
        except MemoryError as e:
            err = e
            for b in bufs:
                b.close()
    need = sum(int(n) for n, _, d in sizes if not (force_pageable and d))
    raise MemoryError(f"this host cannot pin the reshard's host buffers ({need / 1e9:.1f} GB): {err}")
