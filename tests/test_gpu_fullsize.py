"""Parity at the workloads' full sizes (GPU, through the C ABI).

Inputs are generated on the GPU from the ORACLE's description of the old
layout and of the packed inflow (seeded generator only), the reshard runs
through the same entry points and launch configuration as bench.py, and
the result is compared with the oracle's definition evaluated word by
word: a random sample of every arena, the first and last bytes of every
weight shard, all of layer 0's weights, and whole KV blocks.  The in-place
workload also checks the outbound bytes read out before the overwrite.
Then every byte of the new shard (and of the outbound buffer) is compared
on the device with the content the seeded generator writes from the
oracle's description of the new layout.
"""
import numpy as np
import pytest
import torch

from oracle import model, repack
from paper_2511_11617_amd import atp, problem
from synth import configs, fill, gpu, pagetable
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


def _every_byte(pb, content, table, pool, live, w_arena, k_arena, hout_w, w_out):
    """Every byte of the new shard, compared on the device with the content
    the seeded generator writes from the oracle's description of the new
    layout (weights one layer at a time, KV one (layer, K|V) plane at a
    time, free blocks and alignment padding excepted), and, in place, every
    byte of the outbound buffer against the oracle's outbound segments."""
    dev = torch.device("cuda")
    n_offs, n_size = pb.layout("new")
    starts = [i for i, t in enumerate(pb.tensors) if i == 0 or t.layer != pb.tensors[i - 1].layer]
    bounds = [n_offs[i] for i in starts] + [n_size]
    buf = torch.empty(max(b - a for a, b in zip(bounds, bounds[1:])), dtype=torch.uint8, device=dev)
    checked = 0
    for k, i0 in enumerate(starts):
        i1 = starts[k + 1] if k + 1 < len(starts) else len(pb.tensors)
        base = bounds[k]
        shards = []
        for i in range(i0, i1):
            t = pb.tensors[i]
            a, b = pb.new_range(t.space)
            shards.append((t.tag, t.layer, t.kind == model.ROWS, t.rows, t.cols, t.unit, a, b, n_offs[i] - base))
        fill.weights(buf, content, shards)
        for i in range(i0, i1):
            t = pb.tensors[i]
            r, cc = t.shard_shape(pb.new_range(t.space))
            nb = r * cc * pb.eb
            o = n_offs[i]
            if not torch.equal(w_arena[o:o + nb], buf[o - base:o - base + nb]):
                bad = int((w_arena[o:o + nb] != buf[o - base:o - base + nb]).sum())
                raise AssertionError(f"weights: tensor {t.name} layer {t.layer}: {bad} bytes differ")
            checked += nb
    del buf
    # KV: plane by plane; only live blocks are defined
    h0, h1 = pb.kv_heads("new")
    block = pb.kv_block_bytes("new")
    plane = pool * block
    s_idx, b_idx = np.nonzero(table >= 0)
    first = {}
    for s_, b_ in zip(s_idx, b_idx):
        first.setdefault(int(table[s_, b_]), (s_, b_))
    ids = np.array(sorted(first), np.int64)
    seq = torch.from_numpy(np.array([first[p][0] for p in ids], np.int32)).to(dev)
    blk = torch.from_numpy(np.array([first[p][1] for p in ids], np.int32)).to(dev)
    pos = torch.from_numpy(ids).to(dev)
    live_d = torch.from_numpy(ids).to(dev)
    assert np.array_equal(ids, live)
    kbuf = torch.empty(plane, dtype=torch.uint8, device=dev)
    lay = atp.KV_TOKEN_MAJOR if pb.kv_layout == "token" else atp.KV_HEAD_MAJOR
    for l in range(pb.n_layers):
        for which in (0, 1):
            tag = 10 + which
            kind, sigma = content.kind_sigma(tag)
            kbuf.fill_(0)
            gpu.fill_kv(kbuf, 0, seq, blk, pos, block, lay, h0, h1, pb.n_kv, pb.cfg["seq_tokens"],
                        pb.block_tokens, pb.head_dim, content.key(tag, l), kind, sigma)
            g = 2 * l + which
            got = k_arena[g * plane:(g + 1) * plane].view(pool, block).index_select(0, live_d)
            want = kbuf.view(pool, block).index_select(0, live_d)
            if not torch.equal(got, want):
                raise AssertionError(f"kv: layer {l} {'KV'[which]}: {int((got != want).sum())} bytes differ")
            checked += got.numel()
    del kbuf
    if hout_w is not None and w_out:
        total = sum(sg[-1] for sg in w_out)
        ob = torch.empty(total, dtype=torch.uint8, device=dev)
        fill.weights(ob, content, [(pb.tensors[sg[0]].tag, sg[1], pb.tensors[sg[0]].kind == model.ROWS,
                                    pb.tensors[sg[0]].rows, pb.tensors[sg[0]].cols, pb.tensors[sg[0]].unit,
                                    sg[4], sg[5], sg[6]) for sg in w_out])
        step = 1 << 30
        for a in range(0, total, step):
            b = min(total, a + step)
            got = hout_w.tensor[a:b].to(dev)
            if not torch.equal(got, ob[a:b]):
                raise AssertionError(f"outbound: {int((got != ob[a:b]).sum())} bytes differ in [{a}, {b})")
        checked += total
        del ob
    torch.cuda.synchronize()
    say(f"[fullsize] every byte checked: {checked / 1e9:.2f} GB")
    return checked


def run_full(n, inplace=None, pageable_kv_inflow=False, cfg=None, corrupt=None):
    """`cfg` replaces workload n's shape; `corrupt(w_arena, k_arena, hout_w)`
    changes the result before the every-byte check (to show it is not
    vacuous)."""
    c = cfg if cfg is not None else configs.get(n, **({} if inplace is None else {"inplace": inplace}))
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
    # every byte, on the device (the sampled words above anchor it to the oracle on the CPU)
    del stage_w, stage_k
    torch.cuda.empty_cache()
    try:
        if corrupt is not None:
            corrupt(w_arena, k_arena, hout_w)
            torch.cuda.synchronize()
        _every_byte(pb, content, table, pool, live, w_arena, k_arena, hout_w if inplace else None, w_out)
    finally:
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


@pytest.mark.parametrize("where", ["weights", "kv", "outbound"])
def test_every_byte_check_catches_one_wrong_byte(where):
    """The device-side every-byte comparison fails when one byte of the
    result is changed after the reshard (2 layers of the 80-layer TP 8 -> 7
    shape in place, 4 sequences)."""
    c = configs.scaled(5, layers=2, n_seq=4, seq_tokens=1024)

    def flip(w, k, hout):
        if where == "weights":
            w[12345] ^= 1
        elif where == "kv":
            k[k.numel() // 2 + 4096 + 17] ^= 0x80
        else:
            hout.tensor[777] ^= 4

    run_full(5, cfg=c)  # unchanged: passes
    with pytest.raises(AssertionError, match=where):
        run_full(5, cfg=c, corrupt=flip)
