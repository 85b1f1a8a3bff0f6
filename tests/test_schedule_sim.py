"""Replay the library's schedule on the host and compare with the oracle (CPU).

Catches out-of-bounds descriptors, in-place ordering hazards (a level that
reads bytes it or a sibling overwrites, inflow landing on bytes a later
level still reads, outbound reads after an overwrite) and wrong addresses,
before anything runs on a GPU.
"""
import ctypes as C
import random

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

from oracle import model, repack
from paper_2511_11617_amd import atp, problem
from synth import configs, pagetable
from synth.content import KIND_TAG16, Content
from tests.gpu_harness import SQUEEZED_RING_CAP, CachedContent, squeezed_ring_cfg
from tests.schedule_sim import (D2H, H2D, INFLOW, NEW, OLD, OUTBOUND, REPACK, STAGING, Copy, Hazard,
                                 copies, replay)
from tests.test_oracle_repack import med_cfg, tiny_cfg


def sim_case(c, flags=0, staging_cap=0, assign="inorder", mutate=None):
    pb = model.build(c, assign=assign)
    content = CachedContent(Content(c["seed"], c["w_kind"], c["kv_kind"]))
    table, pool = pagetable.make_for(c)
    live = repack.live_blocks(table)
    inplace = bool(flags & atp.INPLACE)
    b = problem.build(c, n_live=len(live), pool=pool, flags=flags, staging_cap=staging_cap)
    plan = b.plan()
    st_ = plan.stats()
    # weights, then KV
    cases = [
        (0, repack.weight_arena(pb, content, "old"), repack.weight_arena(pb, content, "new"),
         repack.weight_live_mask(pb, "new"), repack.packed_weight_inflow(pb, content),
         repack.packed_weight_outbound(pb, content), st_.staging_w),
        (1, repack.kv_arena(pb, content, table, pool, "old", poison=0xDEAD),
         repack.kv_arena(pb, content, table, pool, "new"), repack.kv_live_mask(pb, table, pool, "new"),
         repack.packed_kv_inflow(pb, content, table, pool), repack.packed_kv_outbound(pb, content, table, pool),
         st_.staging_kv),
    ]
    for which, old, want, mask, inflow, outbound, staging in cases:
        cps = copies(plan, which)
        if mutate is not None:
            cps = mutate(which, cps)
        n = max(old.size, want.size)
        bufs = {
            OLD: np.full(n if inplace else old.size, 0xA5, np.uint8),
            NEW: np.full(want.size, 0xA5, np.uint8),
            STAGING: np.full(staging, 0x5A, np.uint8),
            INFLOW: inflow.copy(),
            OUTBOUND: np.full(max(outbound.size, 1), 0x3C, np.uint8),
        }
        bufs[OLD][:old.size] = old
        replay(cps, bufs, live)
        got = (bufs[OLD] if inplace else bufs[NEW])[:want.size]
        bad = np.flatnonzero(got[mask] != want[mask])
        assert bad.size == 0, f"{'kv' if which else 'weights'}: {bad.size} wrong bytes"
        if inplace:
            np.testing.assert_array_equal(bufs[OUTBOUND][:outbound.size], outbound)
        else:
            np.testing.assert_array_equal(bufs[OLD][:old.size], old)  # old arena untouched
    return plan


@pytest.mark.parametrize("inplace", [False, True])
@pytest.mark.parametrize("layout", ["head", "token"])
def test_cfg1(inplace, layout):
    sim_case(configs.get(1, kv_layout=layout, w_kind=KIND_TAG16, kv_kind=KIND_TAG16),
             flags=atp.INPLACE if inplace else 0)


@pytest.mark.parametrize("self_old", [0, 2, 3])
def test_cfg1_survivors_in_place(self_old):
    sim_case(configs.get(1, self_old=self_old, w_kind=KIND_TAG16, kv_kind=KIND_TAG16), flags=atp.INPLACE)


@settings(max_examples=80, deadline=None)
@given(st.integers(0, 2 ** 31), st.booleans(), st.booleans(), st.booleans())
def test_random_small(seed, experts, inplace, no_tail):
    c = tiny_cfg(random.Random(seed), experts)
    sim_case(c, flags=(atp.INPLACE | (atp.NO_TAIL_STAGING if no_tail else 0)) if inplace else 0)


@pytest.mark.parametrize("seed", list(range(10)))
def test_random_medium(seed):
    c = med_cfg(random.Random(9000 + seed), experts=seed % 3 == 0)
    # in place every other time with the level chains resolved by levels alone
    sim_case(c, flags=(atp.INPLACE | (atp.NO_TAIL_STAGING if seed % 4 == 1 else 0)) if seed % 2 else 0)


def test_level_chain_tail_goes_through_staging():
    """The 80-layer TP 8 -> 7 workload's KV geometry (one KV head per old
    rank, two per new one) on a small decoder, in place: the KV shard
    doubles on its own arena, a chain of levels each moving half as much as
    the one before.  With room in staging its tail is staged (read in level
    0, written once its destination is free), leaving few levels; with
    ATP_NO_TAIL_STAGING the chain is resolved by levels alone.  Both replay
    to the oracle's bytes, and the tail costs exactly its bytes of staging."""
    c = configs.get(5, layers=2, hidden=512, n_q=16, n_kv=8, head_dim=64, ffn=1024, n_seq=8, seq_tokens=1024,
                    new_q_widths=None, w_kind=KIND_TAG16, kv_kind=KIND_TAG16)
    tail = sim_case(c, flags=atp.INPLACE, staging_cap=c["staging_cap"]).stats()
    chain = sim_case(c, flags=atp.INPLACE | atp.NO_TAIL_STAGING, staging_cap=c["staging_cap"]).stats()
    assert chain.tail_w == chain.tail_kv == 0
    assert chain.n_levels_kv >= 10  # 512 live blocks: a chain of about log2 of them
    assert tail.tail_kv > 0 and tail.n_levels_kv <= 3
    assert tail.staged_kv - chain.staged_kv == tail.tail_kv
    assert tail.moved_kv == chain.moved_kv and tail.moved_w == chain.moved_w
    # the tail stays within what the cap leaves: a cap at the chain's own
    # need leaves the KV call no room for it
    cap = max(chain.staging_w, chain.staging_kv)
    tight = sim_case(c, flags=atp.INPLACE, staging_cap=cap).stats()
    assert tight.tail_kv == 0 and tight.n_levels_kv == chain.n_levels_kv
    assert max(tight.staging_w, tight.staging_kv) <= cap


@settings(max_examples=40, deadline=None)
@given(st.integers(0, 2 ** 31), st.booleans())
def test_random_small_in_place_under_a_staging_cap(seed, experts):
    """A cap at the unconstrained staging need is accepted; one below it is
    either refused with ATP_ECAPACITY or met by a plan that still replays
    to the oracle's bytes."""
    c = tiny_cfg(random.Random(seed), experts)
    table, pool = pagetable.make_for(c)
    n_live = len(repack.live_blocks(table))
    free = problem.build(c, n_live=n_live, pool=pool, flags=atp.INPLACE).plan().stats()
    need = max(free.staging_w, free.staging_kv)
    plan = sim_case(c, flags=atp.INPLACE, staging_cap=need)
    assert max(plan.stats().staging_w, plan.stats().staging_kv) <= need
    try:
        tight = problem.build(c, n_live=n_live, pool=pool, flags=atp.INPLACE, staging_cap=need - 256).plan()
    except atp.AtpError as e:
        assert e.code == atp.ECAPACITY
        return
    assert max(tight.stats().staging_w, tight.stats().staging_kv) <= need - 256
    sim_case(c, flags=atp.INPLACE, staging_cap=need - 256)


@pytest.mark.slow
@pytest.mark.parametrize("inplace", [False, True])
@pytest.mark.parametrize("n", [2, 3, 4])
def test_large_shapes_one_layer(n, inplace):
    c = configs.scaled(n, layers=1, n_seq=2, seq_tokens=128, w_kind=KIND_TAG16, kv_kind=KIND_TAG16)
    sim_case(c, flags=atp.INPLACE if inplace else 0)


@pytest.mark.slow
def test_cfg5_shape_in_place_two_layers():
    c = configs.scaled(5, layers=2, n_seq=2, seq_tokens=128, w_kind=KIND_TAG16, kv_kind=KIND_TAG16)
    sim_case(c, flags=atp.INPLACE, staging_cap=c["staging_cap"])


def single_target_cfg(self_old):
    """TP 2 -> 1: the survivor ends up holding every tensor whole."""
    return configs.get(1, old_tp=2, new_tp=1, failed=[1 - self_old], self_old=self_old, new_q_widths=None,
                       new_ffn_widths=None, w_kind=KIND_TAG16, kv_kind=KIND_TAG16)


@pytest.mark.parametrize("self_old,inplace", [(0, False), (0, True), (1, False), (1, True)])
def test_single_target_takes_every_tensor_whole(self_old, inplace):
    plan = sim_case(single_target_cfg(self_old), flags=atp.INPLACE if inplace else 0)
    st_ = plan.stats()
    assert st_.self_new_rank == 0 and st_.global_reload == st_.reload_min
    assert st_.retained_w + st_.inflow_w == st_.new_arena_bytes  # shards are 256-aligned, none padded here


def test_no_live_kv_block_plans_no_kv_copy():
    c = configs.get(1)
    table, pool = pagetable.make_for(c)
    n_live = len(repack.live_blocks(table))
    for flags in (0, atp.INPLACE, atp.KV_COMPACT):
        plan = problem.build(c, n_live=0, pool=pool, flags=flags).plan()
        st_ = plan.stats()
        assert copies(plan, 1) == [] and st_.inflow_kv == st_.retained_kv == st_.moved_kv == 0
        # by id the arena keeps every block's place; compact, it holds no block
        full = problem.build(c, n_live=n_live, pool=pool, flags=flags).plan().stats().new_kv_bytes
        assert st_.new_kv_bytes == (0 if flags & atp.KV_COMPACT else full) and full > 0


def test_in_place_ring_under_a_squeezed_staging_cap():
    c = squeezed_ring_cfg()
    plan = sim_case(c, flags=atp.INPLACE, staging_cap=SQUEEZED_RING_CAP)
    st_ = plan.stats()
    # the ring shrank to fit: far less staging than the KV inflow it carries
    assert st_.staging_kv <= SQUEEZED_RING_CAP and st_.staging_kv * 3 < st_.inflow_kv


# ---- the replay catches planted schedule mistakes ---------------------------------------

def _clone(x, **kw):
    y = Copy()
    C.pointer(y)[0] = x
    for k, v in kw.items():
        setattr(y, k, v)
    return y


def _tiny(self_old=0):
    return configs.get(1, self_old=self_old, w_kind=KIND_TAG16, kv_kind=KIND_TAG16)


def test_replay_catches_a_landing_on_repacked_bytes():
    # out of place the landings run beside the repack: a landing that writes
    # bytes a repack copy also writes is a race
    def plant(which, cps):
        if which:
            return cps
        y = min((x for x in cps if x.op == REPACK), key=lambda x: x.run * x.rows)
        return cps + [_clone(y, op=H2D, level=-1)]
    with pytest.raises(Hazard, match="a landing and a level"):
        sim_case(_tiny(), mutate=plant)


def test_replay_catches_two_writers_in_one_level():
    def plant(which, cps):
        ys = [x for x in cps if x.op == REPACK and x.level == 1]
        return cps + [_clone(ys[0])] if ys else cps
    with pytest.raises(Hazard, match="two copies write the same bytes"):
        sim_case(_tiny(), flags=atp.INPLACE, mutate=plant)


def test_replay_catches_an_outbound_read_after_its_overwrite():
    def plant(which, cps):
        return [_clone(x, level=999) if x.op == D2H and x.level >= 1 else x for x in cps]
    with pytest.raises(Hazard, match="outbound read after an overwrite"):
        sim_case(_tiny(self_old=2), flags=atp.INPLACE, mutate=plant)


def test_replay_catches_an_access_past_a_buffer():
    def plant(which, cps):
        if which:
            return cps
        y = next(x for x in cps if x.op == REPACK)
        return [_clone(x, dst_off=x.dst_off + (1 << 40)) if x is y else x for x in cps]
    with pytest.raises(Hazard, match="access outside buffer"):
        sim_case(_tiny(), mutate=plant)
