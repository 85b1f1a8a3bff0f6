"""Parity at the workloads' full sizes (GPU, through the C ABI).

Inputs are generated on the GPU from the ORACLE's description of the old
layout and of the packed inflow (seeded generator only), the reshard runs
through the same entry points and launch configuration as bench.py, and
the result is compared with the oracle's definition evaluated word by
word: a random sample of every arena, the first and last bytes of every
weight shard, all of layer 0's weights, and whole KV blocks.  The in-place
workload also checks the outbound bytes read out before the overwrite.
"""
import numpy as np
import pytest
import torch

from oracle import model, repack
from paper_2511_11617_amd import atp, problem
from synth import configs, fill, pagetable
from synth.pinned import Pageable, Pinned, host_buffers
from synth.content import Content
from tests.gpu_harness import say

pytestmark = pytest.mark.gpu

SAMPLES = 1 << 20


@pytest.fixture(autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    yield
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def _gather(arena, offs):
    idx = torch.from_numpy((offs // 2).astype(np.int64)).cuda()
    return arena.view(torch.int16)[idx].cpu().numpy().view(np.uint16)


def _check(name, got, want, valid):
    bad = np.flatnonzero((got != want) & valid)
    assert bad.size == 0, f"{name}: {bad.size} of {valid.sum()} sampled words wrong"


def _pin_all(sizes, force_pageable=False):
    """Host buffers of the reshard, taken before any device memory (see
    synth.pinned.host_buffers).  A host that cannot pin even the buffers the
    copy kernel touches is a limit of the machine, not a result: the test is
    skipped, naming the size."""
    try:
        bufs, pageable = host_buffers(sizes, force_pageable)
    except MemoryError as e:
        pytest.skip(str(e))
    if pageable:
        say(f"[fullsize] {pageable / 1e9:.1f} GB of DMA-only inflow in pageable memory")
    return bufs


def run_full(n, inplace=None, pageable_kv_inflow=False):
    c = configs.get(n, **({} if inplace is None else {"inplace": inplace}))
    pb = model.build(c)
    content = Content(c["seed"], c["w_kind"], c["kv_kind"])
    table, pool = pagetable.make_for(c)
    live = repack.live_blocks(table)
    inplace = bool(c["inplace"])
    flags = atp.INPLACE if inplace else 0
    say(f"[fullsize] workload {n} {c['name']} inplace={inplace}")
    b = problem.build(c, n_live=len(live), pool=pool, flags=flags, staging_cap=c["staging_cap"] or 0)
    plan = b.plan()
    st = plan.stats()
    hin_w, hin_k, hout_w, hout_k = _pin_all([(st.inflow_w, None, False), (st.inflow_kv, None, inplace),
                                             (st.outbound_w, 0x3C, False), (st.outbound_kv, 0x3C, False)],
                                            force_pageable=pageable_kv_inflow)
    o_offs, o_size = pb.layout("old")
    n_offs, n_size = pb.layout("new")
    k_old, k_new = pb.kv_arena_bytes("old", pool), pb.kv_arena_bytes("new", pool)
    assert (st.old_arena_bytes, st.new_arena_bytes, st.old_kv_bytes, st.new_kv_bytes) == \
        (o_size, n_size, k_old, k_new)
    dev = torch.device("cuda")
    u8 = torch.uint8

    def arena(old_b, new_b):
        if inplace:
            return torch.empty(max(old_b, new_b), dtype=u8, device=dev), None
        return torch.empty(old_b, dtype=u8, device=dev), torch.full((new_b,), 0xA5, dtype=u8, device=dev)

    aw, nw = arena(o_size, n_size)
    ak, nk = arena(k_old, k_new)
    # ---- inputs from the oracle's description --------------------------------
    shards = []
    for t, off in zip(pb.tensors, o_offs):
        a, bb = pb.old_range(t.space)
        shards.append((t.tag, t.layer, t.kind == model.ROWS, t.rows, t.cols, t.unit, a, bb, off))
    fill.weights(aw, content, shards)
    lay = atp.KV_TOKEN_MAJOR if pb.kv_layout == "token" else atp.KV_HEAD_MAJOR
    fill.kv_arena(ak, content, table, pool, pb.n_layers, pb.kv_heads("old"), pb.n_kv,
                  c["seq_tokens"], pb.block_tokens, pb.head_dim, lay)
    w_in, k_in = repack.inflow_segments(pb, len(live))
    w_bytes, k_bytes = sum(s[-1] for s in w_in), sum(s[-1] for s in k_in)
    assert (w_bytes, k_bytes) == (st.inflow_w, st.inflow_kv)
    tmp = torch.empty(max(w_bytes, k_bytes, 1), dtype=u8, device=dev)
    fill.weights(tmp, content, [(pb.tensors[s[0]].tag, s[1], pb.tensors[s[0]].kind == model.ROWS,
                                 pb.tensors[s[0]].rows, pb.tensors[s[0]].cols, pb.tensors[s[0]].unit,
                                 s[4], s[5], s[6]) for s in w_in])
    hin_w.tensor.copy_(tmp[:hin_w.nbytes])
    fill.kv_packed(tmp, content, table, pool, [(s[1], s[2], s[4], s[5], s[6]) for s in k_in], pb.n_kv,
                   c["seq_tokens"], pb.block_tokens, pb.head_dim, lay)
    hin_k.tensor.copy_(tmp[:hin_k.nbytes])
    del tmp
    w_out, k_out = repack.outbound_segments(pb, len(live))
    stage_w = torch.empty(max(st.staging_w, 256), dtype=u8, device=dev)
    stage_k = torch.empty(max(st.staging_kv, 256), dtype=u8, device=dev)
    table_d = torch.from_numpy(table).to(dev)
    torch.cuda.synchronize()
    # ---- the reshard --------------------------------------------------------------
    compute, copy = torch.cuda.current_stream(), torch.cuda.Stream()
    ptr = lambda t: None if t is None else (t.ptr if isinstance(t, (Pinned, Pageable)) else t.data_ptr())
    plan.reshard_weights(ptr(aw), aw.numel(), ptr(nw), nw.numel() if nw is not None else 0,
                         ptr(hin_w), st.inflow_w, ptr(hout_w), st.outbound_w if inplace else 0,
                         ptr(stage_w), stage_w.numel(), compute.cuda_stream, copy.cuda_stream)
    plan.reshard_kv(ptr(ak), ak.numel(), ptr(nk), nk.numel() if nk is not None else 0, ptr(table_d),
                    table.shape[0], table.shape[1], ptr(hin_k), st.inflow_kv, ptr(hout_k),
                    st.outbound_kv if inplace else 0, ptr(stage_k), stage_k.numel(),
                    compute.cuda_stream, copy.cuda_stream)
    t = plan.sync()
    torch.cuda.synchronize()
    say(f"[fullsize] workload {n}: wall {t.wall_ms:.1f} ms, repack {t.repack_w_ms + t.repack_kv_ms:.3f} ms")
    # ---- checks ---------------------------------------------------------------------
    rng = np.random.default_rng(n)
    w_arena = aw if inplace else nw
    k_arena = ak if inplace else nk
    # weights: random sample, shard edges, all of layer 0
    offs = [rng.integers(0, n_size // 2, SAMPLES) * 2]
    for tt, off in zip(pb.tensors, n_offs):
        r, cc = tt.shard_shape(pb.new_range(tt.space))
        nb = r * cc * pb.eb
        offs.append(off + np.arange(0, min(nb, 256), 2))
        offs.append(off + nb - 2 - np.arange(0, min(nb, 256), 2))
    l0_end = n_offs[[tt.layer for tt in pb.tensors].index(1)] if pb.n_layers > 1 else n_size
    offs.append(np.arange(0, l0_end, 2))
    offs = np.concatenate(offs)
    want, valid = repack.expected_weight_words(pb, content, offs)
    _check("weights", _gather(w_arena, offs), want, valid)
    # KV: random sample and whole blocks at both ends of the pool
    block = pb.kv_block_bytes("new")
    kk = [rng.integers(0, k_new // 2, SAMPLES) * 2]
    for g in (0, 2 * pb.n_layers - 1):
        for p in list(live[:64]) + list(live[-64:]):
            kk.append((g * pool + p) * block + np.arange(0, block, 2))
    kk = np.concatenate(kk)
    kw, kv = repack.expected_kv_words(pb, content, table, pool, kk)
    _check("kv", _gather(k_arena, kk), kw, kv)
    if inplace and st.outbound_w:
        oo = rng.integers(0, st.outbound_w // 2, SAMPLES) * 2
        ow = repack.expected_packed_weight_words(pb, content, w_out, oo)
        _check("outbound", hout_w.tensor.numpy().view(np.uint16)[oo // 2], ow, np.ones(oo.shape, bool))
    assert st.global_reload == st.reload_min
    for h in (hin_w, hin_k, hout_w, hout_k):
        h.close()
    return t


@pytest.mark.parametrize("n", [5, 4, 3, 2])   # the largest pinned buffers first
def test_full_size_workload(n):
    run_full(n)


def test_full_size_workload_2_in_place():
    """The headline shape resharded over its own old shard (what the state
    plane's regions hold)."""
    run_full(2, inplace=True)


def test_full_size_workload_2_in_place_kv_inflow_pageable():
    """In place the KV inflow lands through the landing ring by DMA only,
    so it may sit in ordinary host memory (the fallback of hosts that
    cannot pin every buffer of the 80-layer workload)."""
    run_full(2, inplace=True, pageable_kv_inflow=True)
