"""Successive TP switches and error paths on the GPU (through the C ABI).

* 8 -> 7 -> 6: the second switch starts from the first one's unequal
  layout, reading the arena the first switch produced (in and out of
  place); every byte is compared with the oracle after each switch.
* Kernel-side validation: a block table with an id beyond the pool, or
  with a live-block count different from the plan's, makes atp_sync return
  ATP_EINVAL; nothing is copied and no access leaves its buffer.
* A second reshard call before atp_sync is ATP_ESTATE.
* Fresh in-place plans one after another, with the earlier plans still
  alive (as a benchmark loop holds them), each choose the stream for the
  outbound work and stay bit-exact (outbound buffer included).
* A refused pinned allocation leaves no HIP error behind for the next
  kernel launch to report.
"""
import numpy as np
import pytest
import torch

from oracle import model, repack
from paper_2511_11617_amd import atp, problem
from synth import configs, pagetable
from synth.content import KIND_TAG16, Content
from tests.gpu_harness import CachedContent, run_case, say

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _pinned(arr):
    t = torch.empty(max(arr.size, 1), dtype=torch.uint8, pin_memory=True)
    if arr.size:
        t[:arr.size].copy_(torch.from_numpy(arr))
    return t


def _switch(c, arena_w, arena_k, inplace, table, pool):
    """One reshard of this GPU's share; arenas hold the old layout on entry
    and are returned holding the new one."""
    pb = model.build(c)
    content = CachedContent(Content(c["seed"], c["w_kind"], c["kv_kind"]))
    live = repack.live_blocks(table)
    flags = atp.INPLACE if inplace else 0
    b = problem.build(c, n_live=len(live), pool=pool, flags=flags, staging_cap=1 << 30)
    plan = b.plan()
    st = plan.stats()
    in_w = repack.packed_weight_inflow(pb, content)
    in_k = repack.packed_kv_inflow(pb, content, table, pool)
    dev = torch.device("cuda")
    u8 = torch.uint8
    if inplace:
        w = torch.full((max(st.old_arena_bytes, st.new_arena_bytes),), 0xA5, dtype=u8, device=dev)
        w[:arena_w.numel()].copy_(arena_w[:min(arena_w.numel(), w.numel())])
        k = torch.full((max(st.old_kv_bytes, st.new_kv_bytes),), 0xA5, dtype=u8, device=dev)
        k[:arena_k.numel()].copy_(arena_k[:min(arena_k.numel(), k.numel())])
        nw = nk = None
    else:
        w, k = arena_w, arena_k
        nw = torch.full((st.new_arena_bytes,), 0xA5, dtype=u8, device=dev)
        nk = torch.full((st.new_kv_bytes,), 0xA5, dtype=u8, device=dev)
    sw = torch.empty(max(st.staging_w, 256), dtype=u8, device=dev)
    sk = torch.empty(max(st.staging_kv, 256), dtype=u8, device=dev)
    hw, hk = _pinned(in_w), _pinned(in_k)
    ow = torch.empty(max(st.outbound_w, 1), dtype=u8, pin_memory=True)
    ok = torch.empty(max(st.outbound_kv, 1), dtype=u8, pin_memory=True)
    td = torch.from_numpy(table).to(dev)
    s0, s1 = torch.cuda.current_stream(), torch.cuda.Stream()
    p = lambda t: t.data_ptr() if t is not None else None
    plan.reshard_weights(p(w), w.numel(), p(nw), nw.numel() if nw is not None else 0, p(hw), in_w.size,
                         p(ow), st.outbound_w if inplace else 0, p(sw), sw.numel(), s0.cuda_stream,
                         s1.cuda_stream)
    plan.reshard_kv(p(k), k.numel(), p(nk), nk.numel() if nk is not None else 0, p(td), table.shape[0],
                    table.shape[1], p(hk), in_k.size, p(ok), st.outbound_kv if inplace else 0, p(sk),
                    sk.numel(), s0.cuda_stream, s1.cuda_stream)
    plan.sync()
    torch.cuda.synchronize()
    out_w = w if inplace else nw
    out_k = k if inplace else nk
    want_w = repack.weight_arena(pb, content, "new")
    mask_w = repack.weight_live_mask(pb, "new")
    want_k = repack.kv_arena(pb, content, table, pool, "new")
    mask_k = repack.kv_live_mask(pb, table, pool, "new")
    gw = out_w[:want_w.size].cpu().numpy()
    gk = out_k[:want_k.size].cpu().numpy()
    assert np.array_equal(gw[mask_w], want_w[mask_w])
    assert np.array_equal(gk[mask_k], want_k[mask_k])
    return pb, out_w[:st.new_arena_bytes].clone(), out_k[:st.new_kv_bytes].clone()


@pytest.mark.parametrize("inplace", [False, True])
@pytest.mark.parametrize("layout", ["head", "token"])
def test_successive_switches_8_7_6(inplace, layout):
    # a small dense decoder in TP 8, query heads 16, KV heads 8, FFN 8 x 9 units
    c1 = configs.get(3, layers=2, hidden=64, n_q=16, n_kv=8, head_dim=8, ffn=72 * 16, ffn_unit=16,
                     new_q_widths=None, n_seq=3, seq_tokens=64, w_kind=KIND_TAG16, kv_kind=KIND_TAG16,
                     failed=[1], self_old=3, kv_layout=layout, fragmented=True)
    table, pool = pagetable.make_for(c1)
    pb1 = model.build(c1)
    content = Content(c1["seed"], c1["w_kind"], c1["kv_kind"])
    old_w = torch.from_numpy(repack.weight_arena(pb1, content, "old")).cuda()
    old_k = torch.from_numpy(repack.kv_arena(pb1, content, table, pool, "old")).cuda()
    say(f"[switch] 8->7 inplace={inplace} layout={layout}")
    pb1, w1, k1 = _switch(c1, old_w, old_k, inplace, table, pool)
    # second switch: the new 7-rank layout is the old one; new rank 4 dies
    old_ranges = {name: [tuple(r) for r in pb1.new[name]] for name in pb1.new}
    self_old = pb1.self_new   # this GPU's rank in the 7-rank layout
    c2 = dict(c1, old_tp=7, new_tp=6, failed=[4 if self_old != 4 else 5], self_old=self_old,
              old_ranges=old_ranges, new_q_widths=None, new_kv_widths=None, new_ffn_widths=None)
    say(f"[switch] 7->6 from rank {self_old}")
    _switch(c2, w1, k1, inplace, table, pool)


def _bad_table_case(table_mod, live_override=None):
    c = configs.get(1)
    table, pool = pagetable.make_for(c)
    pb = model.build(c)
    content = Content(0, c["w_kind"], c["kv_kind"])
    live = repack.live_blocks(table)
    b = problem.build(c, n_live=live_override or len(live), pool=pool)
    plan = b.plan()
    st = plan.stats()
    old_k = repack.kv_arena(pb, content, table, pool, "old")
    in_k = np.zeros(st.inflow_kv, np.uint8)
    dev = torch.device("cuda")
    ak = torch.from_numpy(old_k).to(dev)
    nk = torch.full((st.new_kv_bytes,), 0xA5, dtype=torch.uint8, device=dev)
    sk = torch.empty(max(st.staging_kv, 256), dtype=torch.uint8, device=dev)
    bad = table.copy()
    table_mod(bad, pool)
    td = torch.from_numpy(bad).to(dev)
    hk = _pinned(in_k)
    s0, s1 = torch.cuda.current_stream(), torch.cuda.Stream()
    plan.reshard_kv(ak.data_ptr(), ak.numel(), nk.data_ptr(), nk.numel(), td.data_ptr(), bad.shape[0],
                    bad.shape[1], hk.data_ptr() if in_k.size else None, in_k.size, None, 0,
                    sk.data_ptr(), sk.numel(), s0.cuda_stream, s1.cuda_stream)
    with pytest.raises(atp.AtpError) as e:
        plan.sync()
    torch.cuda.synchronize()
    assert e.value.code == atp.EINVAL
    # nothing was copied into the new arena
    assert bool((nk == 0xA5).all())
    return str(e.value)


def test_block_id_beyond_pool_is_einval():
    def mod(t, pool):
        t[0, 0] = pool + 7
    assert "num_blocks" in _bad_table_case(mod)


def test_live_count_mismatch_is_einval():
    def mod(t, pool):
        t[1, :] = -1   # one sequence fewer than the plan declared
    assert "live" in _bad_table_case(mod)


def test_second_call_before_sync_is_estate():
    c = configs.get(1)
    table, pool = pagetable.make_for(c)
    pb = model.build(c)
    content = Content(0, c["w_kind"], c["kv_kind"])
    b = problem.build(c, n_live=len(repack.live_blocks(table)), pool=pool)
    plan = b.plan()
    st = plan.stats()
    dev = torch.device("cuda")
    aw = torch.from_numpy(repack.weight_arena(pb, content, "old")).to(dev)
    nw = torch.empty(st.new_arena_bytes, dtype=torch.uint8, device=dev)
    sw = torch.empty(st.staging_w, dtype=torch.uint8, device=dev)
    hw = _pinned(repack.packed_weight_inflow(pb, content))
    s0, s1 = torch.cuda.current_stream(), torch.cuda.Stream()
    args = (aw.data_ptr(), aw.numel(), nw.data_ptr(), nw.numel(), hw.data_ptr(), st.inflow_w, None, 0,
            sw.data_ptr(), sw.numel(), s0.cuda_stream, s1.cuda_stream)
    plan.reshard_weights(*args)
    with pytest.raises(atp.AtpError) as e:
        plan.reshard_weights(*args)
    assert e.value.code == atp.ESTATE
    plan.sync()
    torch.cuda.synchronize()


def test_fresh_in_place_plans_in_a_row():
    c = configs.scaled(5, layers=2, n_seq=2, seq_tokens=256)
    alive = []
    for i in range(4):
        t, plan, st = run_case(c, flags=atp.INPLACE, staging_cap=c["staging_cap"], name=f"fresh-in-place-{i}")
        assert st.outbound_w > 0 and t.d2h_bytes == st.outbound_w + st.outbound_kv
        alive.append(plan)


def test_warmup_then_reshard():
    """atp_warmup ahead of the first reshard (twice: harmless), on the streams
    the reshard then uses; the reshard stays bit-exact."""
    s0, s1 = torch.cuda.current_stream(), torch.cuda.Stream()
    atp.warmup(s0.cuda_stream, s1.cuda_stream, 64)
    atp.warmup(s0.cuda_stream, s1.cuda_stream, 0)
    torch.cuda.synchronize()
    for flags in (0, atp.INPLACE):
        run_case(configs.get(1), flags=flags, name=f"after-warmup-flags{flags}")


@pytest.mark.parametrize("flags", [0, atp.INPLACE])
def test_one_stream_for_compute_and_copy(flags):
    """The caller may pass one stream as both: the landings then queue behind
    the repack on it, the side stream still comes from another hardware
    queue, and the result is the same."""
    run_case(configs.get(1), flags=flags, one_stream=True, name=f"one-stream-flags{flags}")
    c = configs.scaled(2, layers=1, n_seq=2, seq_tokens=256)
    run_case(c, flags=flags, one_stream=True, name=f"one-stream-dense40-flags{flags}")


def test_failed_pin_leaves_no_hip_error_behind():
    """A pinned allocation the host refuses raises MemoryError, and the
    next kernel launch (torch's fill here) does not report that stale
    error as its own."""
    from synth.pinned import Pinned
    with pytest.raises(MemoryError):
        Pinned(1 << 60)
    x = torch.full((1 << 20,), 7, dtype=torch.uint8, device="cuda")
    torch.cuda.synchronize()
    assert int(x[-1]) == 7


def _direct_landing_cfg():
    """2 layers, hidden 8192, TP 2 -> 1: the one target takes every tensor
    whole, and the dead rank's half of W_gate / W_up (2048 rows x 8192, 32 MiB
    each) lands by DMA straight into place."""
    from synth.content import KIND_TAG16
    return configs.get(1, layers=2, hidden=8192, n_q=16, n_kv=4, head_dim=128, ffn=4096, ffn_unit=16,
                       old_tp=2, new_tp=1, failed=[1], self_old=0, new_q_widths=None, new_ffn_widths=None,
                       n_seq=2, seq_tokens=256, w_kind=KIND_TAG16, kv_kind=KIND_TAG16)


def test_caller_work_between_the_calls_comes_first():
    """Each call starts after what the caller queued on the compute stream
    before it, also when the other call of the plan is pending: the caller
    fills the weights' new arena between the KV call and the weights call,
    and the weights call's DMA landings still land over the fill."""
    c = _direct_landing_cfg()

    def fill(bufs, compute):
        with torch.cuda.stream(compute):
            bufs["nw"].fill_(0x77)

    run_case(c, kv_first=True, between=fill, name="fill between calls")


def test_pending_calls_sharing_staging_are_einval():
    """The two calls of a plan may be pending together only on buffers of
    their own: a KV call on the pending weights call's staging, or with its
    new arena over the weights' new arena, is refused; the weights call
    still completes."""
    c = configs.get(1)
    table, pool = pagetable.make_for(c)
    pb = model.build(c)
    content = Content(0, c["w_kind"], c["kv_kind"])
    b = problem.build(c, n_live=len(repack.live_blocks(table)), pool=pool)
    plan = b.plan()
    st = plan.stats()
    dev = torch.device("cuda")
    aw = torch.from_numpy(repack.weight_arena(pb, content, "old")).to(dev)
    nw = torch.empty(st.new_arena_bytes, dtype=torch.uint8, device=dev)
    sw = torch.empty(max(st.staging_w, st.staging_kv), dtype=torch.uint8, device=dev)
    ak = torch.from_numpy(repack.kv_arena(pb, content, table, pool, "old")).to(dev)
    nk = torch.empty(st.new_kv_bytes, dtype=torch.uint8, device=dev)
    sk = torch.empty(st.staging_kv, dtype=torch.uint8, device=dev)
    hw = _pinned(repack.packed_weight_inflow(pb, content))
    hk = _pinned(repack.packed_kv_inflow(pb, content, table, pool))
    td = torch.from_numpy(table).to(dev)
    s0, s1 = torch.cuda.current_stream(), torch.cuda.Stream()
    plan.reshard_weights(aw.data_ptr(), aw.numel(), nw.data_ptr(), nw.numel(), hw.data_ptr(), st.inflow_w, None, 0,
                         sw.data_ptr(), sw.numel(), s0.cuda_stream, s1.cuda_stream)

    def kv(new, staging):
        plan.reshard_kv(ak.data_ptr(), ak.numel(), new.data_ptr(), st.new_kv_bytes, td.data_ptr(), table.shape[0],
                        table.shape[1], hk.data_ptr(), st.inflow_kv, None, 0, staging.data_ptr(),
                        st.staging_kv, s0.cuda_stream, s1.cuda_stream)

    for new, staging in ((nk, sw), (nw, sk)):
        with pytest.raises(atp.AtpError) as e:
            kv(new, staging)
        assert e.value.code == atp.EINVAL and "overlaps" in str(e.value)
    plan.sync()
    torch.cuda.synchronize()
    want = repack.weight_arena(pb, content, "new")
    mask = repack.weight_live_mask(pb, "new")
    np.testing.assert_array_equal(nw.cpu().numpy()[mask], want[mask])
