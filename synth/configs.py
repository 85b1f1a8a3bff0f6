"""The five synthetic reshard workloads, as plain shape data.

Each entry restates a decoder shape, the TP change, the failed rank(s) and
the surviving GPU whose share of the reshard is measured.  Nothing here
computes a partition or a plan: widths are either stated explicitly or named
by rule ("ceil_first", "gqa"), and both the oracle and the library derive
ranges from them independently.

Defaults where a workload leaves a choice open:
  * failed old rank 1;
  * FFN sharded in 16-column units (1 column for the tiny model, whose
    230/229/229 split needs it);
  * KV heads of a rank follow its query heads (GQA-consistent split);
  * weights ~N(0, 0.02) and KV ~N(0, 1) in the stated 16-bit type.
"""
from __future__ import annotations

import copy

from .content import KIND_BF16, KIND_FP16

GB = 10 ** 9

_BASE = dict(
    seed=0,
    failed=[1],
    ffn_unit=16,
    kv_rule="gqa",
    block_tokens=16,
    elem_bytes=2,
    w_kind=KIND_BF16,
    kv_kind=KIND_BF16,
    fragmented=False,
    pool_factor=1.0,
    inplace=False,
    staging_cap=None,
    experts=0,
    expert_ffn=0,
    ffn=0,
    new_q_widths=None,
    new_kv_widths=None,
    new_ffn_widths=None,
    new_expert_widths=None,
    kv_layout="head",
)


def _cfg(**kw):
    c = copy.deepcopy(_BASE)
    c.update(kw)
    return c


CONFIGS = {
    1: _cfg(
        name="tiny-dense-2L-h256-tp4to3",
        layers=2, hidden=256, n_q=4, n_kv=2, head_dim=64, ffn=688,
        ffn_unit=1, w_kind=KIND_FP16, kv_kind=KIND_FP16,
        old_tp=4, new_tp=3, failed=[1], self_old=0,
        new_q_widths=[2, 1, 1], new_ffn_widths=[230, 229, 229],
        n_seq=8, seq_tokens=128,
    ),
    2: _cfg(
        name="dense-40L-h5120-tp4to3",
        layers=40, hidden=5120, n_q=40, n_kv=8, head_dim=128, ffn=17408,
        old_tp=4, new_tp=3, failed=[1], self_old=2,
        new_q_widths=[14, 13, 13], new_kv_widths=[3, 3, 2],
        n_seq=32, seq_tokens=4096,
    ),
    3: _cfg(
        name="dense-40L-h5120-tp8to7-fragmented-kv",
        layers=40, hidden=5120, n_q=40, n_kv=8, head_dim=128, ffn=17408,
        old_tp=8, new_tp=7, failed=[1], self_old=3,
        new_q_widths=[6, 6, 6, 6, 6, 5, 5],
        n_seq=64, seq_tokens=8192, fragmented=True, pool_factor=1.125,
    ),
    4: _cfg(
        name="moe-48L-h2048-128e-tp4to3",
        layers=48, hidden=2048, n_q=32, n_kv=4, head_dim=128,
        experts=128, expert_ffn=768,
        old_tp=4, new_tp=3, failed=[1], self_old=2,
        new_q_widths=[11, 11, 10], new_expert_widths=[43, 43, 42],
        n_seq=64, seq_tokens=4096,
    ),
    5: _cfg(
        name="dense-80L-h8192-tp8to7-inplace",
        layers=80, hidden=8192, n_q=64, n_kv=8, head_dim=128, ffn=28672,
        old_tp=8, new_tp=7, failed=[1], self_old=2,
        n_seq=128, seq_tokens=8192, inplace=True, staging_cap=2 * 2 ** 30,
    ),
}


def get(n: int, **overrides) -> dict:
    """A copy of workload `n` with optional field overrides."""
    c = copy.deepcopy(CONFIGS[n])
    c.update(overrides)
    c["id"] = n
    return c


def scaled(n: int, layers: int | None = None, n_seq: int | None = None,
           seq_tokens: int | None = None, **overrides) -> dict:
    """Workload `n` with fewer layers / sequences (same per-layer shapes)."""
    c = get(n, **overrides)
    if layers is not None:
        c["layers"] = layers
    if n_seq is not None:
        c["n_seq"] = n_seq
    if seq_tokens is not None:
        c["seq_tokens"] = seq_tokens
    return c
