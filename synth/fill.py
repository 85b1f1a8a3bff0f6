"""Fill full-size workload buffers on the GPU (input generation only).

Callers describe what goes where; this module only writes the seeded
content there:
  * weight shards / packed weight inflow: (tag, layer, sharded_rows, rows,
    cols, unit, unit_begin, unit_end, dst_off) = units [a, b) of the full
    [rows, cols] tensor, row-major at dst_off;
  * a KV arena: every live block of the block table, heads [h0, h1);
  * packed KV inflow: per (layer, K|V, heads [a, b), host offset), the live
    blocks in ascending id order.
"""
from __future__ import annotations

import numpy as np
import torch

from . import gpu, pagetable
from .content import TAGS, Content


def weights(buf, content: Content, shards, stream=0):
    regions = []
    for tag, layer, sharded_rows, rows, cols, unit, a, b, dst_off in shards:
        kind, sigma = content.kind_sigma(tag)
        regions.append(gpu.shard_region(content.key(tag, layer), kind, sigma, dst_off, rows, cols,
                                        sharded_rows, unit, a, b))
    gpu.fill(buf, regions, stream)


def _dev(a, dtype):
    return torch.from_numpy(np.ascontiguousarray(a).astype(dtype)).cuda()


def kv_arena(buf, content: Content, table: np.ndarray, pool: int, n_layers: int, heads, n_kv: int,
             seq_tokens: int, bt: int, hd: int, layout: int, stream=0):
    h0, h1 = heads
    block = (h1 - h0) * bt * hd * 2
    s_idx, b_idx = np.nonzero(table >= 0)
    pos = table[s_idx, b_idx].astype(np.int64)
    seq, blk, pos_d = _dev(s_idx, np.int32), _dev(b_idx, np.int32), _dev(pos, np.int64)
    for l in range(n_layers):
        for which in (0, 1):
            tag = TAGS["k_cache"] + which
            kind, sigma = content.kind_sigma(tag)
            base = (l * 2 + which) * pool * block
            gpu.fill_kv(buf, base, seq, blk, pos_d, block, layout, h0, h1, n_kv, seq_tokens, bt, hd,
                        content.key(tag, l), kind, sigma, stream)


def kv_packed(buf, content: Content, table: np.ndarray, pool: int, segments, n_kv: int,
              seq_tokens: int, bt: int, hd: int, layout: int, stream=0):
    """segments: (layer, which, a, b, host_offset) in buffer order."""
    seq_of, blk_of = pagetable.inverse(table, pool)
    live = np.unique(table[table >= 0]).astype(np.int64)
    seq, blk = _dev(seq_of[live], np.int32), _dev(blk_of[live], np.int32)
    pos = _dev(np.arange(len(live)), np.int64)
    for layer, which, a, b, off in segments:
        tag = TAGS["k_cache"] + which
        kind, sigma = content.kind_sigma(tag)
        gpu.fill_kv(buf, off, seq, blk, pos, (b - a) * bt * hd * 2, layout, a, b, n_kv, seq_tokens,
                    bt, hd, content.key(tag, layer), kind, sigma, stream)
