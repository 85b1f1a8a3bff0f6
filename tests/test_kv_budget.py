"""KV budget under recovery (Sec. III-A): LRU session eviction and the
compact KV layout, on the CPU.

  * the oracle's policy is pinned by hand cases and by a brute-force
    characterisation (the kept sessions are the longest run of most recent
    sessions whose distinct blocks fit);
  * the library's atp_kv_evict_lru matches the oracle on random tables,
    shared blocks and ties included;
  * a reshard of the kept sessions into an ATP_KV_COMPACT arena, replayed
    on the host, equals the oracle's compact arena (the by-id arena gathered
    in live-id order).
"""
import random

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

from oracle import kvbudget, model, repack
from paper_2511_11617_amd import atp, problem
from synth import configs, pagetable
from synth.content import KIND_TAG16, Content
from tests.gpu_harness import CachedContent
from tests.schedule_sim import INFLOW, NEW, OLD, OUTBOUND, STAGING, copies, replay
from tests.test_oracle_repack import tiny_cfg


# ---- the oracle's policy ----------------------------------------------------------

def test_hand_case():
    table = np.array([[0, 1], [2, -1], [3, 4]])
    last = [5, 1, 9]
    # 5 blocks x 100 B = 500 B; evict s1 (400), then s0 (200)
    assert kvbudget.lru_keep(table, last, 100, 500).tolist() == [True, True, True]
    assert kvbudget.lru_keep(table, last, 100, 499).tolist() == [True, False, True]
    assert kvbudget.lru_keep(table, last, 100, 400).tolist() == [True, False, True]
    assert kvbudget.lru_keep(table, last, 100, 399).tolist() == [False, False, True]
    assert kvbudget.lru_keep(table, last, 100, 199).tolist() == [False, False, False]
    np.testing.assert_array_equal(
        kvbudget.evicted_table(table, np.array([False, False, True]), compact=True), [[-1, -1], [-1, -1], [0, 1]])
    np.testing.assert_array_equal(
        kvbudget.evicted_table(table, np.array([True, False, True]), compact=True), [[0, 1], [-1, -1], [2, 3]])


def test_shared_blocks_free_with_their_last_session():
    # block 7 is a shared prefix of all three sessions
    table = np.array([[7, 0], [7, 1], [7, 2]])
    last = [3, 2, 1]
    # 4 distinct blocks; evicting s2 frees only block 2
    assert kvbudget.lru_keep(table, last, 1, 3).tolist() == [True, True, False]
    assert kvbudget.lru_keep(table, last, 1, 2).tolist() == [True, False, False]
    # the shared block goes only with the last session
    assert kvbudget.lru_keep(table, last, 1, 1).tolist() == [False, False, False]


def test_ties_evict_the_lower_session_first():
    table = np.array([[0], [1], [2]])
    assert kvbudget.lru_keep(table, [4, 4, 4], 1, 2).tolist() == [False, True, True]
    assert kvbudget.lru_keep(table, [4, 4, 4], 1, 1).tolist() == [False, False, True]


def _random_table(rng, n_seq, width, pool, shared):
    t = np.full((n_seq, width), -1, np.int32)
    free = list(rng.permutation(pool))
    prefix = [free.pop() for _ in range(shared)]
    for s in range(n_seq):
        n = rng.integers(0, width - shared + 1)
        row = prefix + [free.pop() for _ in range(n)]
        t[s, :len(row)] = row
    return t


@settings(max_examples=200, deadline=None)
@given(st.integers(0, 2 ** 32 - 1))
def test_brute_force_characterisation(seed):
    rng = np.random.default_rng(seed)
    n_seq, width = int(rng.integers(1, 7)), int(rng.integers(1, 5))
    shared = int(rng.integers(0, 2)) if width > 1 else 0
    table = _random_table(rng, n_seq, width, n_seq * width + 4, shared)
    last = rng.integers(0, 4, n_seq)            # many ties
    bb = int(rng.integers(1, 4))
    budget = int(rng.integers(0, bb * (n_seq * width + 1) + 1))
    keep = kvbudget.lru_keep(table, last, bb, budget)
    # hottest first, ties: the higher session index is hotter
    hot = sorted(range(n_seq), key=lambda s: (last[s], s), reverse=True)
    want = np.zeros(n_seq, bool)
    for m in range(n_seq, -1, -1):
        if kvbudget.demand_blocks(table, hot[:m]) * bb <= budget:
            want[hot[:m]] = True
            break
    np.testing.assert_array_equal(keep, want)


# ---- the library against the oracle -----------------------------------------------

@settings(max_examples=200, deadline=None)
@given(st.integers(0, 2 ** 32 - 1), st.booleans())
def test_library_matches_oracle(seed, compact):
    rng = np.random.default_rng(seed)
    n_seq, width = int(rng.integers(0, 9)), int(rng.integers(1, 6))
    shared = int(rng.integers(0, 3)) if width > 2 else 0
    pool = n_seq * width + 5
    table = _random_table(rng, n_seq, width, pool, shared) if n_seq else np.zeros((0, width), np.int32)
    last = rng.integers(0, 5, n_seq)
    bb = int(rng.integers(1, 1 << 20))
    budget = int(rng.integers(0, bb * (n_seq * width + 2)))
    keep, new, st_ = atp.kv_evict_lru(table, last, pool, bb, budget, compact)
    want_keep = kvbudget.lru_keep(table, last, bb, budget)
    np.testing.assert_array_equal(keep, want_keep)
    np.testing.assert_array_equal(new, kvbudget.evicted_table(table, want_keep, compact))
    assert st_.kept_sessions == want_keep.sum() and st_.evicted_sessions == n_seq - want_keep.sum()
    assert st_.live_before == kvbudget.demand_blocks(table, range(n_seq))
    assert st_.live_after == kvbudget.demand_blocks(table, np.flatnonzero(want_keep))
    assert st_.demand_after == st_.live_after * bb


def test_library_rejects_bad_ids():
    for bad in (np.array([[0, 5]]), np.array([[0, -2]])):
        with pytest.raises(atp.AtpError) as e:
            atp.kv_evict_lru(bad, [1], 5, 1, 10)
        assert e.value.code == atp.EINVAL


# ---- compact reshard of the kept sessions (host replay) ---------------------------

def sim_compact(c, last_use, budget_frac, flags=atp.KV_COMPACT):
    pb = model.build(c)
    content = CachedContent(Content(c["seed"], c["w_kind"], c["kv_kind"]))
    full, pool = pagetable.make_for(c)
    bb = pb.kv_arena_bytes("new", pool) // pool
    budget = int(budget_frac * repack.live_blocks(full).size * bb)
    keep = kvbudget.lru_keep(full, last_use, bb, budget)
    table = kvbudget.evicted_table(full, keep, compact=False)
    live = repack.live_blocks(table)
    b = problem.build(c, n_live=len(live), pool=pool, flags=flags)
    plan = b.plan()
    st_ = plan.stats()
    inplace = bool(flags & atp.INPLACE)
    if flags & atp.KV_COMPACT:
        want = repack.kv_arena_compact(pb, content, table, pool)
        mask = np.ones(want.size, bool)
    else:
        want = repack.kv_arena(pb, content, table, pool, "new")
        mask = repack.kv_live_mask(pb, table, pool, "new")
    assert st_.new_kv_bytes == want.size
    old = repack.kv_arena(pb, content, full, pool, "old", poison=0xDEAD)  # every session's blocks
    n = max(old.size, want.size) if inplace else old.size
    bufs = {OLD: np.full(n, 0xA5, np.uint8), NEW: np.full(want.size, 0xA5, np.uint8),
            STAGING: np.full(st_.staging_kv, 0x5A, np.uint8),
            INFLOW: repack.packed_kv_inflow(pb, content, table, pool),
            OUTBOUND: np.full(max(st_.outbound_kv, 1), 0x3C, np.uint8)}
    bufs[OLD][:old.size] = old
    assert bufs[INFLOW].size == st_.inflow_kv
    replay(copies(plan, 1), bufs, live)
    got = (bufs[OLD] if inplace else bufs[NEW])[:want.size]
    bad = np.flatnonzero(got[mask] != want[mask])
    assert bad.size == 0, f"{bad.size} of {mask.sum()} KV bytes wrong"
    return keep


@pytest.mark.parametrize("layout", ["head", "token"])
@pytest.mark.parametrize("frac", [1.0, 0.6, 0.3])
def test_cfg1_compact_after_eviction(layout, frac):
    c = configs.get(1, kv_layout=layout, w_kind=KIND_TAG16, kv_kind=KIND_TAG16)
    last = np.random.default_rng(7).permutation(c["n_seq"])
    keep = sim_compact(c, last, frac)
    assert (keep.sum() < c["n_seq"]) == (frac < 1.0)


@settings(max_examples=40, deadline=None)
@given(st.integers(0, 2 ** 31), st.booleans(), st.floats(0.2, 1.0))
def test_random_small_compact(seed, experts, frac):
    c = tiny_cfg(random.Random(seed), experts)
    last = np.random.default_rng(seed).integers(0, 3, c["n_seq"])
    sim_compact(c, last, frac)


@pytest.mark.parametrize("flags", [0, atp.INPLACE])
def test_cfg1_eviction_ids_kept(flags):
    c = configs.get(1, w_kind=KIND_TAG16, kv_kind=KIND_TAG16)
    sim_compact(c, np.random.default_rng(5).permutation(c["n_seq"]), 0.5, flags)


@settings(max_examples=30, deadline=None)
@given(st.integers(0, 2 ** 31), st.booleans(), st.floats(0.2, 1.0))
def test_random_small_in_place_eviction(seed, experts, frac):
    c = tiny_cfg(random.Random(seed), experts)
    sim_compact(c, np.random.default_rng(seed).integers(0, 3, c["n_seq"]), frac, atp.INPLACE)


def test_compact_in_place_is_rejected():
    c = configs.get(1)
    table, pool = pagetable.make_for(c)
    with pytest.raises(atp.AtpError) as e:
        problem.build(c, n_live=len(repack.live_blocks(table)), pool=pool,
                      flags=atp.KV_COMPACT | atp.INPLACE).plan()
    assert e.value.code == atp.EINVAL
