"""Synthetic safetensors checkpoints (input generation only).

A checkpoint holds the full, unsharded weight tensors of a workload with the
seeded content of synth.content, one 2-D tensor per (layer, name), named
`layers.{layer}.{name}` (experts stacked as the workload's tensor list
states them).  Two writers:
  * `write_package` uses the safetensors package itself (small files, tests):
    the library's reader is then checked against an independent writer;
  * `write_stream` writes the same format with its own header and can leave
    holes: only the element ranges it is given are written, the rest of each
    tensor stays a hole of the file (full-size benchmarks, where only the
    ranges a reload reads are needed).
"""
from __future__ import annotations

import json
import os

import numpy as np

from .content import TAGS, Content

DTYPES = {"bf16": "BF16", "fp16": "F16"}


def name(tensor: str, layer: int) -> str:
    return f"layers.{layer}.{tensor}"


def full_words(content: Content, tensor: str, layer: int, rows: int, cols: int) -> np.ndarray:
    """[rows, cols] uint16 words of the full tensor."""
    idx = np.arange(rows * cols, dtype=np.int64)
    return content(TAGS[tensor], layer, idx).reshape(rows, cols)


def write_package(path: str, content: Content, tensors, dtype: str = "bf16", metadata=None):
    """tensors: [(name, layer, rows, cols)]."""
    import torch
    from safetensors.torch import save_file

    tdt = torch.bfloat16 if dtype == "bf16" else torch.float16
    d = {}
    for t, layer, rows, cols in tensors:
        w = full_words(content, t, layer, rows, cols)
        d[name(t, layer)] = torch.from_numpy(w.view(np.int16)).view(tdt)
    save_file(d, path, metadata=metadata)


def header(tensors, dtype: str = "bf16"):
    """(header bytes padded to 8, {name: absolute data offset}) in list order."""
    meta, at = {}, 0
    for t, layer, rows, cols in tensors:
        n = rows * cols * 2
        meta[name(t, layer)] = {"dtype": DTYPES[dtype], "shape": [rows, cols], "data_offsets": [at, at + n]}
        at += n
    h = json.dumps(meta, separators=(",", ":")).encode()
    h += b" " * (-len(h) % 8)
    base = 8 + len(h)
    offs = {k: base + v["data_offsets"][0] for k, v in meta.items()}
    return len(h).to_bytes(8, "little") + h, offs, base + at


def write_stream(path: str, tensors, regions, dtype: str = "bf16"):
    """Write a checkpoint whose data holds only `regions`.

    regions: iterable of (name, layer, cols, row0, row1, col0, col1, words),
    words a uint16 array of shape [row1 - row0, col1 - col0] placed at rows
    [row0, row1) and columns [col0, col1) of that tensor.  Tensors with no
    region are left as holes (reading as zero bytes); within a tensor whose
    regions are column ranges, the rows they span are written whole.
    Written with pwrite, so a full disk raises OSError."""
    head, offs, total = header(tensors, dtype)
    # regions of one tensor that are not whole rows are assembled into the
    # row span they cover (zeros elsewhere) and written at once
    whole, strided = [], {}
    for r in regions:
        t, layer, cols, r0, r1, c0, c1, words = r
        (whole.append(r) if c0 == 0 and c1 == cols else strided.setdefault((t, layer, cols), []).append(r))
    fd = os.open(path, os.O_WRONLY | os.O_CREAT | os.O_TRUNC, 0o644)
    try:
        os.pwrite(fd, head, 0)
        os.ftruncate(fd, total)
        for t, layer, cols, r0, r1, c0, c1, words in whole:
            w = np.ascontiguousarray(words, dtype=np.uint16)
            _pwrite_all(fd, memoryview(w.reshape(-1)).cast("B"), offs[name(t, layer)] + r0 * cols * 2)
        for (t, layer, cols), rs in strided.items():
            lo, hi = min(r[3] for r in rs), max(r[4] for r in rs)
            span = np.zeros((hi - lo, cols), np.uint16)
            for _, _, _, r0, r1, c0, c1, words in rs:
                span[r0 - lo:r1 - lo, c0:c1] = words
            _pwrite_all(fd, memoryview(span.reshape(-1)).cast("B"), offs[name(t, layer)] + lo * cols * 2)
    finally:
        os.close(fd)
    return total


def _pwrite_all(fd: int, buf: memoryview, off: int):
    while len(buf):
        n = os.pwrite(fd, buf, off)
        buf, off = buf[n:], off + n
