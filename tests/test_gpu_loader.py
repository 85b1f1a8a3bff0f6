"""Reload from a checkpoint, end to end on the GPU: the library's range-read
loader fills the pinned weight inflow buffer from a safetensors file, the
reshard lands it, and the new arena equals the oracle's new shard byte for
byte (through the C ABI)."""
import random

import pytest
import torch

from paper_2511_11617_amd import atp
from synth import configs
from synth.content import KIND_TAG16
from tests.gpu_harness import run_case
from tests.test_oracle_repack import tiny_cfg

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    yield
    torch.cuda.synchronize()


@pytest.mark.parametrize("flags", [0, atp.INPLACE])
def test_cfg1_from_checkpoint(tmp_path, flags):
    run_case(configs.get(1, w_kind=KIND_TAG16), flags=flags, ckpt_dir=tmp_path, name="cfg1-ckpt")


@pytest.mark.parametrize("seed,experts", [(3, True), (8, False), (21, True)])
def test_tiny_from_checkpoint(tmp_path, seed, experts):
    run_case(tiny_cfg(random.Random(seed), experts), ckpt_dir=tmp_path, name=f"tiny{seed}-ckpt")


def test_full_reload_from_checkpoint(tmp_path):
    run_case(configs.get(1, w_kind=KIND_TAG16), flags=atp.PLAN_FULL, variant="full", ckpt_dir=tmp_path,
             name="cfg1-full-ckpt")


# ---- the reads pipelined with the weights reshard (atp_load_reshard_weights) ----

@pytest.mark.parametrize("flags", [0, atp.INPLACE])
def test_cfg1_pipelined_from_checkpoint(tmp_path, flags):
    run_case(configs.get(1, w_kind=KIND_TAG16), flags=flags, ckpt_dir=tmp_path, pipelined=True,
             name="cfg1-ckpt-pipelined")


@pytest.mark.parametrize("seed,experts", [(3, True), (8, False)])
def test_tiny_pipelined_from_checkpoint(tmp_path, seed, experts):
    run_case(tiny_cfg(random.Random(seed), experts), ckpt_dir=tmp_path, pipelined=True,
             name=f"tiny{seed}-ckpt-pipelined")


@pytest.mark.parametrize("seed,experts", [(4, False), (9, True)])
def test_tiny_pipelined_after_the_kv_call(tmp_path, seed, experts):
    """Out of place the KV call may come first: its inflow then uses the link
    while the weight reads run."""
    run_case(tiny_cfg(random.Random(seed), experts), ckpt_dir=tmp_path, pipelined=True, kv_first=True,
             name=f"tiny{seed}-ckpt-pipelined-kv-first")


def test_large_layer_pipelined_from_checkpoint(tmp_path):
    """One layer of the 40-layer TP 4->3 shape: 110 MB of weight inflow, so
    the host reads go out in several pieces as the reads complete (the
    checkpoint holds the intervals read, holes elsewhere)."""
    c = configs.scaled(2, layers=1, n_seq=2, seq_tokens=256, w_kind=KIND_TAG16, kv_kind=KIND_TAG16)
    run_case(c, ckpt_dir=tmp_path, pipelined=True, sparse_ckpt=True, name="dense40-1layer-ckpt-pipelined")


def test_large_layer_pipelined_after_the_kv_call(tmp_path):
    c = configs.scaled(2, layers=1, n_seq=2, seq_tokens=256, w_kind=KIND_TAG16, kv_kind=KIND_TAG16)
    run_case(c, ckpt_dir=tmp_path, pipelined=True, sparse_ckpt=True, kv_first=True,
             name="dense40-1layer-ckpt-pipelined-kv-first")


def test_pipelined_read_failure_drains_and_reports(tmp_path):
    """A read that fails after part of the reshard is enqueued (the file is
    cut short after it was opened): the call drains the enqueued work, then
    reports ATP_EINVAL; nothing is left pending and the next reshard works.
    The condition is made on the host: every kernel runs in bounds."""
    import os

    import numpy as np

    from oracle import model, repack
    from paper_2511_11617_amd import problem
    from synth import checkpoint, pagetable
    from synth.content import Content

    c = configs.get(1, w_kind=KIND_TAG16)
    table, pool = pagetable.make_for(c)
    plan = problem.build(c, n_live=len(repack.live_blocks(table)), pool=pool).plan()
    st = plan.stats()
    tl = problem.tensor_list(c)
    path = str(tmp_path / "model.safetensors")
    checkpoint.write_package(path, Content(c["seed"], c["w_kind"], c["kv_kind"]),
                             [(n, l, r, cc) for (n, l, k, sp, r, cc, u) in tl], "bf16")
    files = atp.StFiles([path])
    os.truncate(path, os.path.getsize(path) // 2)  # reads past the middle come back short
    dev = torch.device("cuda")
    u8 = torch.uint8
    aw = torch.zeros(max(st.old_arena_bytes, 256), dtype=u8, device=dev)
    nw = torch.zeros(max(st.new_arena_bytes, 256), dtype=u8, device=dev)
    sw = torch.zeros(max(st.staging_w, 256), dtype=u8, device=dev)
    hw = torch.zeros(max(st.inflow_w, 1), dtype=u8, pin_memory=True)
    s0, s1 = torch.cuda.current_stream(), torch.cuda.Stream()
    with pytest.raises(atp.AtpError) as e:
        plan.load_reshard_weights(files, [checkpoint.name(n, l) for (n, l, *_) in tl], aw.data_ptr(), aw.numel(),
                                  nw.data_ptr(), nw.numel(), hw.data_ptr(), st.inflow_w, None, 0, sw.data_ptr(),
                                  sw.numel(), s0.cuda_stream, s1.cuda_stream)
    assert e.value.code == atp.EINVAL and "range read failed" in str(e.value)
    files.close()
    plan.sync()  # nothing pending: returns at once
    torch.cuda.synchronize()
    del aw, nw, sw, hw
    run_case(configs.get(1, w_kind=KIND_TAG16), name="cfg1-after-a-failed-read")


# ---- the reads behind atp_load_reshard_weights_async: the KV call is issued
# while they run, atp_sync issues the weight pieces as they complete ----

@pytest.mark.parametrize("flags", [0, atp.INPLACE])
def test_cfg1_async_from_checkpoint(tmp_path, flags):
    run_case(configs.get(1, w_kind=KIND_TAG16), flags=flags, ckpt_dir=tmp_path, pipelined="async",
             name="cfg1-ckpt-async")


@pytest.mark.parametrize("seed,experts,flags", [(3, True, 0), (8, False, atp.INPLACE), (12, True, atp.INPLACE)])
def test_tiny_async_from_checkpoint(tmp_path, seed, experts, flags):
    run_case(tiny_cfg(random.Random(seed), experts), flags=flags, ckpt_dir=tmp_path, pipelined="async",
             name=f"tiny{seed}-ckpt-async")


@pytest.mark.parametrize("flags", [0, atp.INPLACE])
def test_large_layer_async_from_checkpoint(tmp_path, flags):
    """One layer of the 40-layer TP 4->3 shape (110 MB of weight inflow, in
    several pieces), out of place and in place."""
    c = configs.scaled(2, layers=1, n_seq=2, seq_tokens=256, w_kind=KIND_TAG16, kv_kind=KIND_TAG16)
    run_case(c, flags=flags, ckpt_dir=tmp_path, pipelined="async", sparse_ckpt=True,
             name="dense40-1layer-ckpt-async")


@pytest.mark.parametrize("flags", [0, atp.INPLACE])
def test_async_reads_outlive_the_closed_files(tmp_path, flags):
    """The files are closed right after the asynchronous call, before any read
    may have run: the reads keep duplicates of the descriptors, so the
    reshard still gets every byte (a closed descriptor's number could
    otherwise name another file by then)."""
    c = configs.scaled(2, layers=1, n_seq=2, seq_tokens=256, w_kind=KIND_TAG16, kv_kind=KIND_TAG16)
    run_case(c, flags=flags, ckpt_dir=tmp_path, pipelined="async", sparse_ckpt=True, close_files_early=True,
             name="dense40-1layer-ckpt-async-closed")


@pytest.mark.parametrize("flags", [0, atp.INPLACE])
def test_async_read_failure_is_reported_by_sync(tmp_path, flags):
    """The file is cut short after it was opened: the async call returns, the
    KV call is issued, and atp_sync drains everything queued before it
    reports ATP_EINVAL; no read statistics are given, nothing is left
    pending, and the next reshard works.  The condition is made on the host:
    every kernel runs in bounds."""
    import os

    from oracle import repack
    from paper_2511_11617_amd import problem
    from synth import checkpoint, pagetable
    from synth.content import Content

    c = configs.get(1, w_kind=KIND_TAG16)
    table, pool = pagetable.make_for(c)
    plan = problem.build(c, n_live=len(repack.live_blocks(table)), pool=pool, flags=flags).plan()
    st = plan.stats()
    tl = problem.tensor_list(c)
    path = str(tmp_path / "model.safetensors")
    checkpoint.write_package(path, Content(c["seed"], c["w_kind"], c["kv_kind"]),
                             [(n, l, r, cc) for (n, l, k, sp, r, cc, u) in tl], "bf16")
    files = atp.StFiles([path])
    os.truncate(path, os.path.getsize(path) // 2)  # reads past the middle come back short
    dev = torch.device("cuda")
    u8 = torch.uint8
    inplace = bool(flags & atp.INPLACE)
    aw = torch.zeros(max(st.old_arena_bytes, st.new_arena_bytes if inplace else 0, 256), dtype=u8, device=dev)
    nw = None if inplace else torch.zeros(max(st.new_arena_bytes, 256), dtype=u8, device=dev)
    ak = torch.zeros(max(st.old_kv_bytes, st.new_kv_bytes if inplace else 0, 256), dtype=u8, device=dev)
    nk = None if inplace else torch.zeros(max(st.new_kv_bytes, 256), dtype=u8, device=dev)
    sw = torch.zeros(max(st.staging_w, 256), dtype=u8, device=dev)
    sk = torch.zeros(max(st.staging_kv, 256), dtype=u8, device=dev)
    hw = torch.zeros(max(st.inflow_w, 1), dtype=u8, pin_memory=True)
    hk = torch.zeros(max(st.inflow_kv, 1), dtype=u8, pin_memory=True)
    ow = torch.zeros(max(st.outbound_w, 1), dtype=u8, pin_memory=True)
    ok = torch.zeros(max(st.outbound_kv, 1), dtype=u8, pin_memory=True)
    table_d = torch.from_numpy(table).to(dev)
    s0, s1 = torch.cuda.current_stream(), torch.cuda.Stream()
    torch.cuda.synchronize()
    ptr = lambda t: t.data_ptr() if t is not None else None
    plan.load_reshard_weights_async(files, [checkpoint.name(n, l) for (n, l, *_) in tl], aw.data_ptr(), aw.numel(),
                                    ptr(nw), nw.numel() if nw is not None else 0, hw.data_ptr(), st.inflow_w,
                                    ow.data_ptr(), st.outbound_w if inplace else 0, sw.data_ptr(), sw.numel(),
                                    s0.cuda_stream, s1.cuda_stream)
    plan.reshard_kv(ak.data_ptr(), ak.numel(), ptr(nk), nk.numel() if nk is not None else 0, table_d.data_ptr(),
                    table.shape[0], table.shape[1], hk.data_ptr(), st.inflow_kv, ok.data_ptr(),
                    st.outbound_kv if inplace else 0, sk.data_ptr(), sk.numel(), s0.cuda_stream, s1.cuda_stream)
    with pytest.raises(atp.AtpError) as e:
        plan.sync()
    assert e.value.code == atp.EINVAL and "range read failed" in str(e.value)
    with pytest.raises(atp.AtpError) as e2:
        plan.load_stats()
    assert e2.value.code == atp.ESTATE
    files.close()
    plan.sync()  # nothing pending: returns at once
    torch.cuda.synchronize()
    del aw, nw, ak, nk, sw, sk, hw, hk, ow, ok, table_d
    run_case(configs.get(1, w_kind=KIND_TAG16), flags=flags, name="cfg1-after-a-failed-async-read")
