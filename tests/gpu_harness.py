"""Run one reshard through the C ABI on the GPU and check it against the
oracle (shared helper of the GPU tests).

Inputs and expected bytes come from the oracle (plain CPU definition) and
the seeded generator; the library only sees the old arena, the packed
inflow buffer and the block table.
"""
from __future__ import annotations

import os
import sys

import numpy as np
import torch

from oracle import kvbudget, model, repack
from paper_2511_11617_amd import atp, problem
from synth import pagetable
from synth.content import KIND_FP16, Content

POISON = 0xA5


class CachedContent:
    """Memoises full-tensor requests (idx = arange(n)) of a Content."""

    def __init__(self, content):
        self.c = content
        self.cache = {}

    def __call__(self, tag, layer, idx):
        n = len(idx)
        if n and idx[0] == 0 and idx[-1] == n - 1:
            k = (tag, layer, n)
            if k not in self.cache:
                self.cache[k] = self.c(tag, layer, idx)
            return self.cache[k]
        return self.c(tag, layer, idx)


SQUEEZED_RING_CAP = 24 << 20


def squeezed_ring_cfg():
    """A tiny decoder with 4 KV heads (GQA groups of 2), TP 4 -> 3, old rank 2
    -> new rank 1, whose in-place KV inflow is one head of every live block:
    64 MiB for 64 sessions of 2048 tokens.  Under SQUEEZED_RING_CAP bytes of
    staging the landing ring shrinks to 4 slots of 4 MiB that 16 chunks
    reuse in turn."""
    from synth import configs
    from synth.content import KIND_TAG16
    return configs.get(1, hidden=512, n_q=8, n_kv=4, head_dim=64, new_q_widths=None, new_ffn_widths=None,
                       self_old=2, n_seq=64, seq_tokens=2048, w_kind=KIND_TAG16, kv_kind=KIND_TAG16)


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def run_case(c, flags=0, staging_cap=0, assign="inorder", check_outbound=True, name="", variant="cm",
             ckpt_dir=None, evict=None, pipelined=False, sparse_ckpt=False, kv_first=False, one_stream=False,
             between=None, close_files_early=False):
    return prepare_case(c, flags, staging_cap, assign, check_outbound, name, variant, ckpt_dir, evict, pipelined,
                        sparse_ckpt, kv_first, one_stream, between=between,
                        close_files_early=close_files_early)()()


def prepare_case(c, flags=0, staging_cap=0, assign="inorder", check_outbound=True, name="", variant="cm",
               ckpt_dir=None, evict=None, pipelined=False, sparse_ckpt=False, kv_first=False, one_stream=False,
               streams=None, between=None, close_files_early=False):
    """Reshard one workload on the GPU and compare with the oracle.  With
    `ckpt_dir`, the weight inflow is read from a safetensors checkpoint
    written there by the library's range-read loader instead of being copied
    from the oracle's packed inflow; with `pipelined` too, the reads and the
    weights reshard run together (atp_load_reshard_weights).  A
    `pipelined="async"` the reads run behind atp_load_reshard_weights_async:
    the KV call is issued while they run and atp_sync issues the weight
    pieces as the reads complete.  A
    `sparse_ckpt` holds only the intervals the plan reads (the oracle's
    packed inflow put back at its tensor coordinates), holes elsewhere.
    `kv_first` issues the KV call before the weights call (out of place
    only: in place that order is refused).  `one_stream` passes the same
    stream as compute and copy stream.  `between(bufs, compute)` runs
    between the two calls (bufs: dict of the device buffers), e.g. to queue
    caller work on the compute stream that the second call must follow.

    prepare_case() builds the plan and the device and host buffers and
    returns issue(), which enqueues the reshard and returns finish(), which
    syncs and checks it: several plans can then be pending together, on the
    `streams` (compute, copy) given.  run_case() does all three.  With `evict` = (last_use, budget
    fraction of the new KV demand), the oracle's LRU policy picks the kept
    sessions; the old arena holds every session, the reshard gets the kept
    rows, and with ATP_KV_COMPACT the result is the oracle's compact arena."""
    say(f"[gpu case] {name} cfg={c.get('name', '?')} layers={c['layers']} flags={flags} "
        f"old_tp={c['old_tp']} new_tp={c['new_tp']} failed={c['failed']} self_old={c['self_old']}")
    pb = model.build(c, assign=assign, variant=variant)
    content = CachedContent(Content(c["seed"], c["w_kind"], c["kv_kind"]))
    table, pool = pagetable.make_for(c)
    full_table = table
    if evict is not None:
        last_use, frac = evict
        bb = pb.kv_arena_bytes("new", pool) // pool
        keep = kvbudget.lru_keep(table, last_use, bb, int(frac * len(repack.live_blocks(table)) * bb))
        table = kvbudget.evicted_table(table, keep, compact=False)
    n_live = int(len(repack.live_blocks(table)))
    inplace = bool(flags & atp.INPLACE)
    compact = bool(flags & atp.KV_COMPACT)

    old_w = repack.weight_arena(pb, content, "old")
    want_w = repack.weight_arena(pb, content, "new")
    mask_w = repack.weight_live_mask(pb, "new")
    in_w = repack.packed_weight_inflow(pb, content)
    old_k = repack.kv_arena(pb, content, full_table, pool, "old", poison=0xDEAD)
    if compact:
        want_k = repack.kv_arena_compact(pb, content, table, pool)
        mask_k = np.ones(want_k.size, bool)
    else:
        want_k = repack.kv_arena(pb, content, table, pool, "new")
        mask_k = repack.kv_live_mask(pb, table, pool, "new")
    in_k = repack.packed_kv_inflow(pb, content, table, pool)

    b = problem.build(c, n_live=n_live, pool=pool, flags=flags, staging_cap=staging_cap)
    plan = b.plan()
    st = plan.stats()
    assert st.inflow_w == in_w.size and st.inflow_kv == in_k.size

    dev = torch.device("cuda")
    u8 = torch.uint8

    def device_arena(old, new_size):
        if inplace:
            a = torch.full((max(old.size, new_size, 256),), POISON, dtype=u8, device=dev)
            a[:old.size].copy_(torch.from_numpy(old))
            return a, None
        a = torch.from_numpy(old).to(dev) if old.size else torch.zeros(256, dtype=u8, device=dev)
        n = torch.full((max(new_size, 256),), POISON, dtype=u8, device=dev)
        return a, n

    def pinned(arr):
        if arr.size == 0:
            return None
        t = torch.empty(arr.size, dtype=u8, pin_memory=True)
        t.copy_(torch.from_numpy(arr))
        return t

    aw, nw = device_arena(old_w, want_w.size)
    ak, nk = device_arena(old_k, want_k.size)
    stage_w = torch.full((max(st.staging_w, 256),), 0x5A, dtype=u8, device=dev)
    stage_k = torch.full((max(st.staging_kv, 256),), 0x5A, dtype=u8, device=dev)
    hin_w, hin_k = pinned(in_w), pinned(in_k)
    if ckpt_dir is not None and in_w.size:
        from synth import checkpoint
        tl = problem.tensor_list(c)
        path = os.path.join(str(ckpt_dir), "model.safetensors")
        tens = [(n, l, r, cc) for (n, l, k, sp, r, cc, u) in tl]
        dtype = "fp16" if c["w_kind"] == KIND_FP16 else "bf16"
        if sparse_ckpt:
            regions = []
            for sg in plan.segments(atp.SEG_INFLOW_W):
                n, l, kind, sp, rows, cols, unit = tl[sg.tensor]
                a, b = sg.unit_begin * unit, sg.unit_end * unit
                w = in_w[sg.host_offset:sg.host_offset + sg.bytes].view(np.uint16)
                if kind == atp.ROWS:
                    regions.append((n, l, cols, a, b, 0, cols, w.reshape(b - a, cols)))
                else:
                    regions.append((n, l, cols, 0, rows, a, b, w.reshape(rows, b - a)))
            checkpoint.write_stream(path, tens, regions, dtype)
        else:
            checkpoint.write_package(path, Content(c["seed"], c["w_kind"], c["kv_kind"]), tens, dtype)
        hin_w.fill_(0xA5)  # the loader must write every byte
        files = atp.StFiles([path])
        ckpt_names = [checkpoint.name(n, l) for (n, l, *_) in tl]
        if not pipelined:
            plan.load_weights(files, ckpt_names, hin_w.data_ptr(), in_w.size)
            files.close()
            files = None
    hout_w = torch.full((max(st.outbound_w, 1),), 0x3C, dtype=u8, pin_memory=True)
    hout_k = torch.full((max(st.outbound_kv, 1),), 0x3C, dtype=u8, pin_memory=True)
    table_d = torch.from_numpy(table).to(dev)
    if streams is not None:
        compute, copy = streams
    else:
        compute = torch.cuda.current_stream()
        copy = compute if one_stream else torch.cuda.Stream()
    torch.cuda.synchronize()

    ptr = lambda t: t.data_ptr() if t is not None else None
    w_args = (ptr(aw), aw.numel(), ptr(nw), nw.numel() if nw is not None else 0, ptr(hin_w), in_w.size,
              ptr(hout_w), st.outbound_w, ptr(stage_w), stage_w.numel(), compute.cuda_stream, copy.cuda_stream)

    deferred = ckpt_dir is not None and in_w.size and pipelined == "async"

    def weights_call():
        if deferred:
            plan.load_reshard_weights_async(files, ckpt_names, *w_args)
            if close_files_early:  # the reads keep descriptors of their own
                files.close()
        elif ckpt_dir is not None and in_w.size and pipelined:
            ls = plan.load_reshard_weights(files, ckpt_names, *w_args)
            assert ls.bytes == in_w.size
            files.close()
        else:
            plan.reshard_weights(*w_args)

    def kv_call():
        plan.reshard_kv(ptr(ak), ak.numel(), ptr(nk), nk.numel() if nk is not None else 0,
                        ptr(table_d), table.shape[0], table.shape[1], ptr(hin_k), in_k.size,
                        ptr(hout_k), st.outbound_kv, ptr(stage_k), stage_k.numel(),
                        compute.cuda_stream, copy.cuda_stream)

    def issue():
        first, second = (kv_call, weights_call) if kv_first else (weights_call, kv_call)
        if kv_first:
            assert not inplace, "in place the weights call comes first"
        first()
        if between is not None:
            between(dict(aw=aw, nw=nw, ak=ak, nk=nk, stage_w=stage_w, stage_k=stage_k), compute)
        second()
        return finish

    def finish():
        t = plan.sync()
        torch.cuda.synchronize()
        if deferred:
            assert plan.load_stats().bytes == in_w.size
            if not close_files_early:
                files.close()
        got_w = (aw if inplace else nw).cpu().numpy()[:want_w.size]
        got_k = (ak if inplace else nk).cpu().numpy()[:want_k.size]
        bad_w = np.flatnonzero(got_w[mask_w] != want_w[mask_w])
        bad_k = np.flatnonzero(got_k[mask_k] != want_k[mask_k])
        assert bad_w.size == 0, f"weights: {bad_w.size} wrong bytes, first at live byte {bad_w[:5]}"
        assert bad_k.size == 0, f"kv: {bad_k.size} wrong bytes, first at live byte {bad_k[:5]}"
        if inplace and check_outbound:
            ow = repack.packed_weight_outbound(pb, content)
            ok = repack.packed_kv_outbound(pb, content, table, pool)
            np.testing.assert_array_equal(hout_w.numpy()[:ow.size], ow)
            np.testing.assert_array_equal(hout_k.numpy()[:ok.size], ok)
        return t, plan, st

    # the calls hold raw pointers: every buffer stays referenced until the
    # plan is synced, or the caching allocators would hand its memory to the
    # next case's tensors while this plan still reads and writes it
    finish.keep = (aw, nw, ak, nk, stage_w, stage_k, hin_w, hin_k, hout_w, hout_k, table_d)
    return issue
