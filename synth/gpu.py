"""GPU filling of synthetic inputs (binding of synth/libatp_synth.so).

Input generation only: writes the words of synth.content into device
buffers.  Every region is bounds-checked on the host before launch.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

from .content import IH_STD, KIND_BF16, KIND_FP16

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libatp_synth.so")


class Region(C.Structure):
    _fields_ = [("key", C.c_uint64), ("kind", C.c_int32), ("scale", C.c_float),
                ("dst_off", C.c_uint64), ("n0", C.c_int64), ("n1", C.c_int64), ("n2", C.c_int64),
                ("ds0", C.c_int64), ("ds1", C.c_int64), ("idx0", C.c_int64), ("is0", C.c_int64),
                ("is1", C.c_int64), ("is2", C.c_int64)]


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise ImportError(f"{_LIB_PATH} missing: run `python -m paper_2511_11617_amd.build`")
        # torch's own HIP runtime must be mapped before this library, or the
        # process would hold two HIP runtimes (they share a soname)
        import torch  # noqa: F401
        L = C.CDLL(_LIB_PATH)
        L.synth_fill.argtypes = [C.c_void_p, C.POINTER(Region), C.c_int, C.c_void_p]
        L.synth_fill_kv.argtypes = [C.c_void_p, C.c_uint64, C.c_void_p, C.c_void_p, C.c_void_p,
                                    C.c_int64, C.c_int64, C.c_int32, C.c_int32, C.c_int32, C.c_int32,
                                    C.c_int64, C.c_int32, C.c_int32, C.c_uint64, C.c_int32, C.c_float,
                                    C.c_void_p]
        _lib = L
    return _lib


def _scale(kind, sigma):
    return float(np.float32(sigma / IH_STD)) if kind in (KIND_BF16, KIND_FP16) else 0.0


def shard_region(key, kind, sigma, dst_off, rows, cols, sharded_rows: bool, unit, a, b) -> Region:
    """Units [a, b) of a full [rows, cols] tensor, packed row-major at dst_off."""
    if sharded_rows:
        r0, r1 = a * unit, b * unit
        return Region(key, kind, _scale(kind, sigma), dst_off, 1, r1 - r0, cols,
                      0, cols * 2, r0 * cols, 0, cols, 1)
    c0, c1 = a * unit, b * unit
    return Region(key, kind, _scale(kind, sigma), dst_off, 1, rows, c1 - c0,
                  0, (c1 - c0) * 2, c0, 0, cols, 1)


def _extent(r: Region):
    if r.n0 * r.n1 * r.n2 == 0:
        return 0
    return r.dst_off + (r.n0 - 1) * r.ds0 + (r.n1 - 1) * r.ds1 + (r.n2 - 1) * 2 + 2


def fill(buf, regions, stream=0):
    """buf: torch uint8 CUDA tensor."""
    if not regions:
        return
    size = buf.numel()
    for r in regions:
        if _extent(r) > size:
            raise ValueError("synthetic region past the end of the buffer")
    arr = (Region * len(regions))(*regions)
    rc = lib().synth_fill(buf.data_ptr(), arr, len(regions), stream)
    if rc:
        raise RuntimeError(f"synth_fill: HIP error {rc}")


def fill_kv(buf, base, seq, blk, pos, block_stride, layout, h0, h1, n_kv, seq_tokens, bt, hd,
            key, kind, sigma, stream=0):
    """seq/blk/pos: torch int32/int32/int64 CUDA tensors of the same length."""
    n = int(seq.numel())
    if n == 0 or h1 <= h0:
        return
    per = (h1 - h0) * bt * hd * 2
    pmax = int(pos.max().item())
    if base + pmax * block_stride + per > buf.numel() or per > block_stride:
        raise ValueError("synthetic KV items past the end of the buffer")
    rc = lib().synth_fill_kv(buf.data_ptr(), base, seq.data_ptr(), blk.data_ptr(), pos.data_ptr(), n,
                             block_stride, layout, h0, h1, n_kv, seq_tokens, bt, hd, key, kind,
                             _scale(kind, sigma), stream)
    if rc:
        raise RuntimeError(f"synth_fill_kv: HIP error {rc}")
