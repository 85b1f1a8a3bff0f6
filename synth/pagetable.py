"""Seeded paged-KV block tables for the synthetic workloads.

A block table is int32 [n_seq][max_blocks]; entry -1 marks an unused slot.
Every sequence is full (its length is a multiple of the block size), so
sequence s uses logical blocks 0 .. seq_tokens/block_tokens - 1.

* sequential: physical id = s * blocks_per_seq + b, pool = live blocks.
* fragmented: pool P = ceil(pool_factor * live); the live ids are the first
  `live` entries of a seeded permutation of range(P) (numpy PCG64), handed
  out in sequence order; the other P - live blocks are free.
"""
from __future__ import annotations

import math

import numpy as np


def make(n_seq: int, seq_tokens: int, block_tokens: int, fragmented: bool,
         pool_factor: float = 1.0, seed: int = 0, extra_slots: int = 0):
    """Returns (table int32 [n_seq, max_blocks], pool size P)."""
    bps = -(-seq_tokens // block_tokens)
    live = n_seq * bps
    max_blocks = bps + extra_slots
    table = np.full((n_seq, max_blocks), -1, dtype=np.int32)
    if fragmented:
        pool = int(math.ceil(pool_factor * live))
        ids = np.random.Generator(np.random.PCG64(seed)).permutation(pool)[:live]
    else:
        pool = live
        ids = np.arange(live)
    table[:, :bps] = ids.reshape(n_seq, bps).astype(np.int32)
    return table, pool


def make_for(cfg: dict, extra_slots: int = 0):
    return make(cfg["n_seq"], cfg["seq_tokens"], cfg["block_tokens"],
                cfg["fragmented"], cfg["pool_factor"], cfg["seed"], extra_slots)


def inverse(table: np.ndarray, pool: int):
    """For each physical block: (seq, logical block) or (-1, -1) if free.

    A block referenced by several slots maps to its first reference in
    (seq, block) order."""
    seq = np.full(pool, -1, dtype=np.int64)
    blk = np.full(pool, -1, dtype=np.int64)
    s_idx, b_idx = np.nonzero(table >= 0)
    ids = table[s_idx, b_idx].astype(np.int64)
    order = np.arange(len(ids))[::-1]  # last write wins -> reverse for first
    seq[ids[order]] = s_idx[order]
    blk[ids[order]] = b_idx[order]
    return seq, blk
