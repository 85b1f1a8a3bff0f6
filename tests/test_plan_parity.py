"""The library's host planner against the oracle (CPU, no GPU calls).

libatp.so's atp_plan is pure host code; these tests compare every planning
output the C ABI exposes with the oracle on the five workloads and on
random small decoders: survivor-to-target assignment, new ranges, the CMM
task lists, both arena layouts, the packed inflow/outbound order and the
byte statistics (including Eq. 1's minimum reload).
"""
import random

import pytest
from hypothesis import given, settings, strategies as st

from oracle import cmm, model, repack
from paper_2511_11617_amd import atp, problem
from synth import configs, pagetable
from tests.test_oracle_repack import tiny_cfg

SPACES = ["q", "kv"]


def _third(pb):
    return "exp" if "exp" in pb.spaces else "ffn"


def _compare(c, flags=0, staging_cap=0, assign="inorder", variant="cm"):
    table, pool = pagetable.make_for(c)
    n_live = int(len(repack.live_blocks(table)))
    pb = model.build(c, assign=assign, variant=variant)
    b = problem.build(c, n_live=n_live, pool=pool, flags=flags, staging_cap=staging_cap)
    plan = b.plan()
    names = SPACES + [_third(pb)]
    assert plan.owner() == pb.owner
    for s, name in enumerate(names):
        assert plan.ranges(s) == [tuple(r) for r in pb.new[name]], name
        assert plan.tasks(s) == [x.as_tuple() for x in pb.plans[name]], name
    o_offs, o_size = pb.layout("old")
    n_offs, n_size = pb.layout("new")
    for i, t in enumerate(pb.tensors):
        oo, no, nb = plan.layout(i)
        r, cc = t.shard_shape(pb.new_range(t.space))
        assert (oo, no, nb) == (o_offs[i], n_offs[i], r * cc * pb.eb)
    st_ = plan.stats()
    assert st_.self_new_rank == pb.self_new
    assert (st_.old_arena_bytes, st_.new_arena_bytes) == (o_size, n_size)
    assert st_.old_kv_bytes == pb.kv_arena_bytes("old", pool)
    assert st_.new_kv_bytes == pb.kv_arena_bytes("new", pool)
    ret, inf, out = repack.self_bytes(pb, n_live)
    assert st_.retained_w + st_.retained_kv == ret
    assert st_.inflow_w + st_.inflow_kv == inf
    assert st_.outbound_w + st_.outbound_kv == out
    # packed order
    w_in, k_in = repack.inflow_segments(pb, n_live)
    w_out, k_out = repack.outbound_segments(pb, n_live)
    seg = lambda L: [(s.tensor, s.layer, s.which, s.kind, s.unit_begin, s.unit_end,
                      s.host_offset, s.bytes) for s in L]
    assert seg(plan.segments(atp.SEG_INFLOW_W)) == w_in
    assert seg(plan.segments(atp.SEG_INFLOW_KV)) == k_in
    assert seg(plan.segments(atp.SEG_OUTBOUND_W)) == w_out
    assert seg(plan.segments(atp.SEG_OUTBOUND_KV)) == k_out
    # global bytes and Eq. 1
    kv_head = c["layers"] * 2 * n_live * c["block_tokens"] * c["head_dim"] * c["elem_bytes"]
    unit_bytes = {name: 0 for name in names}
    for t in pb.tensors:
        unit_bytes[t.space] += t.unit_bytes(pb.eb)
    unit_bytes["kv"] += kv_head
    rel = sum(cmm.reload_units(pb.plans[n]) * unit_bytes[n] for n in names)
    eq1 = sum(cmm.eq1_min_reload(pb.old[n], pb.failed, pb.new[n]) * unit_bytes[n] for n in names)
    assert st_.global_reload == rel
    assert st_.reload_min == eq1
    if variant == "cm":
        assert eq1 == rel
    return plan, pb


@pytest.mark.parametrize("n", [1, 2, 3, 4, 5])
def test_workloads_match_oracle(n):
    c = configs.get(n)
    if n in (3, 5):   # keep the oracle's page-table walk short; shapes unchanged
        c = configs.scaled(n, n_seq=8)
    flags = atp.INPLACE if c["inplace"] else 0
    _compare(c, flags=flags, staging_cap=c["staging_cap"] or 0)


@pytest.mark.parametrize("n", [2, 3])
def test_failed_rank_sweep(n):
    base = configs.scaled(n, n_seq=4)
    for f in range(base["old_tp"]):
        alive = [i for i in range(base["old_tp"]) if i != f]
        for self_old in (alive[0], alive[-1]):
            _compare(configs.scaled(n, n_seq=4, failed=[f], self_old=self_old))


def test_maxretain_matches_oracle():
    c = configs.scaled(2, n_seq=4, failed=[3], self_old=2)
    _compare(c, flags=atp.ASSIGN_MAXRETAIN, assign="maxretain")


@settings(max_examples=150, deadline=None)
@given(st.integers(0, 2 ** 31), st.booleans())
def test_random_small_match_oracle(seed, experts):
    _compare(tiny_cfg(random.Random(seed), experts))


def test_fig3_tasks_through_library():
    """The worked example of Fig. 3 planned by the library."""
    c = configs.get(1, layers=1, n_q=4, n_kv=4, head_dim=256, hidden=8, ffn=1024, ffn_unit=1,
                    new_q_widths=None, new_ffn_widths=None, new_kv_widths=None,
                    new_rule="floor", failed=[1], self_old=0, kv_rule="ceil")
    b = problem.build(c, n_live=1, pool=1)
    plan = b.plan()
    assert plan.ranges(2) == [(0, 341), (341, 682), (682, 1024)]
    assert plan.tasks(2) == [
        (atp.KEEP, 0, 256, 0, 0, 0), (atp.RELOAD, 256, 341, -1, 0, 0),
        (atp.KEEP, 512, 682, 2, 1, 2), (atp.RELOAD, 341, 512, -1, 1, 2),
        (atp.KEEP, 768, 1024, 3, 2, 3), (atp.P2P, 682, 768, 2, 2, 3)]


@pytest.mark.parametrize("variant,flag", [("greedy", atp.PLAN_GREEDY), ("full", atp.PLAN_FULL)])
@pytest.mark.parametrize("n", [1, 2, 4])
def test_planner_baselines_match_oracle(n, variant, flag):
    c = configs.get(n) if n == 1 else configs.scaled(n, n_seq=4)
    plan, pb = _compare(c, flags=flag, variant=variant)
    cm = _compare(c)[0].stats()
    st_ = plan.stats()
    assert cm.global_reload <= st_.global_reload
    assert st_.global_p2p == 0
    if variant == "full":
        assert st_.retained_w == st_.retained_kv == 0
