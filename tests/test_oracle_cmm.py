"""Pins of the oracle's partitions and CMM plan (CPU).

Pins: the paper's Fig. 3 worked example (exact tasks and totals), the
floor rule of Alg. 1 and the floor/ceil widths of Sec. III-B (hand values),
Eq. 1's closed form, exhaustive searches over per-unit source choices and
over survivor-to-target assignments, and hand-computed byte counts of the
tiny 4 -> 3 workload.
"""
import os
import random

import pytest
from hypothesis import given, settings, strategies as st

from oracle import brute, cmm, model, repack
from synth import configs

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _read_golden(name):
    rows = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                rows.append(line.split())
    return rows


def _ranges(tokens):
    out, cur = [], []
    for t in tokens:
        if t == "|":
            out.append(tuple(cur))
            cur = []
        else:
            cur.append(int(t))
    out.append(tuple(cur))
    return out


# --------------------------------------------------------------------------
# Fig. 3
# --------------------------------------------------------------------------
def test_fig3_worked_example():
    g = _read_golden("fig3_cmm.txt")
    kv = {r[0]: r[1:] for r in g if r[0] != "task"}
    H = int(kv["H"][0])
    old = _ranges(kv["old"])
    failed = [int(kv["failed_gpu"][0]) - 1]
    targets = cmm.floor_targets(H, 3)
    assert targets == _ranges(kv["targets"])
    owner = cmm.assign_inorder(4, failed, 3)
    plan = cmm.cmm(old, failed, targets, owner)
    got = sorted((f"GPU{x.host + 1}", cmm.KIND_NAMES[x.kind], x.begin, x.end,
                  "-" if x.src < 0 else f"GPU{x.src + 1}") for x in plan)
    want = sorted((r[1], r[2], int(r[3]), int(r[4]), r[5]) for r in g if r[0] == "task")
    assert got == want
    tot = {k: sum(x.end - x.begin for x in plan if x.kind == k)
           for k in (cmm.KEEP, cmm.P2P, cmm.RELOAD)}
    assert tot[cmm.RELOAD] == int(kv["total_reload"][0])
    assert tot[cmm.P2P] == int(kv["total_p2p"][0])
    assert tot[cmm.KEEP] == int(kv["total_keep"][0])
    assert cmm.eq1_min_reload(old, failed, targets) == 256
    assert cmm.eq1_closed_form(old, failed, targets) == 256


def test_fig3_task_order():
    """Order reading: targets ascending; within a target the host's own
    range first, then other sources ascending, then reloads."""
    old = [(0, 256), (256, 512), (512, 768), (768, 1024)]
    plan = cmm.cmm(old, [1], cmm.floor_targets(1024, 3), [0, 2, 3])
    assert [x.as_tuple() for x in plan] == [
        (cmm.KEEP, 0, 256, 0, 0, 0), (cmm.RELOAD, 256, 341, -1, 0, 0),
        (cmm.KEEP, 512, 682, 2, 1, 2), (cmm.RELOAD, 341, 512, -1, 1, 2),
        (cmm.KEEP, 768, 1024, 3, 2, 3), (cmm.P2P, 682, 768, 2, 2, 3)]


def test_last_rank_dies_H_includes_dead():
    old = [(0, 4), (4, 8), (8, 12)]
    plan = cmm.cmm(old, [2], cmm.floor_targets(12, 2), [0, 1])
    assert max(x.end for x in plan) == 12
    assert cmm.reload_units(plan) == 4


# --------------------------------------------------------------------------
# partitions
# --------------------------------------------------------------------------
@pytest.mark.parametrize("S,g,want", [
    (688, 3, [229, 229, 230]), (1024, 3, [341, 341, 342]), (10, 4, [2, 3, 2, 3]),
])
def test_floor_rule_widths(S, g, want):
    rs = cmm.floor_targets(S, g)
    assert [b - a for a, b in rs] == want
    assert rs[0][0] == 0 and rs[-1][1] == S


@pytest.mark.parametrize("S,g,want", [
    (688, 3, [230, 229, 229]), (40, 7, [6, 6, 6, 6, 6, 5, 5]),
    (64, 7, [10, 9, 9, 9, 9, 9, 9]), (1088, 3, [363, 363, 362]),
    (128, 3, [43, 43, 42]), (32, 3, [11, 11, 10]), (40, 3, [14, 13, 13]),
    (1088, 7, [156, 156, 156, 155, 155, 155, 155]), (1792, 7, [256] * 7),
])
def test_ceil_first_widths(S, g, want):
    assert cmm.ceil_first_widths(S, g) == want


@given(st.integers(1, 10 ** 6), st.integers(1, 64))
def test_unequal_widths_are_floor_or_ceil(S, g):
    lo, hi = S // g, -(-S // g)
    for w in (cmm.ceil_first_widths(S, g), [b - a for a, b in cmm.floor_targets(S, g)]):
        assert sum(w) == S and all(x in (lo, hi) for x in w)


def test_gqa_ranges_tiny():
    assert cmm.gqa_ranges([(0, 1), (1, 2), (2, 3), (3, 4)], 2) == [(0, 1), (0, 1), (1, 2), (1, 2)]
    assert cmm.gqa_ranges([(0, 2), (2, 3), (3, 4)], 2) == [(0, 1), (1, 2), (1, 2)]
    assert cmm.gqa_ranges([(0, 11), (11, 22), (22, 32)], 8) == [(0, 2), (1, 3), (2, 4)]


# --------------------------------------------------------------------------
# Eq. 1 and exhaustive searches
# --------------------------------------------------------------------------
def _random_layout(rng, H, N):
    cuts = sorted(rng.sample(range(1, H), N - 1)) if N > 1 else []
    b = [0] + cuts + [H]
    return [(b[i], b[i + 1]) for i in range(N)]


@settings(max_examples=300, deadline=None)
@given(st.integers(0, 2 ** 31), st.integers(2, 9), st.integers(9, 4000))
def test_eq1_equals_cmm_reload_disjoint(seed, N, H):
    rng = random.Random(seed)
    old = _random_layout(rng, H, N)
    nf = rng.randint(1, N - 1)
    failed = sorted(rng.sample(range(N), nf))
    M = N - nf
    targets = _random_layout(rng, H, M) if rng.random() < 0.5 else cmm.floor_targets(H, M)
    plan = cmm.cmm(old, failed, targets, cmm.assign_inorder(N, failed, M))
    r = cmm.reload_units(plan)
    assert r == cmm.eq1_min_reload(old, failed, targets)
    assert r == cmm.eq1_closed_form(old, failed, targets)
    dead = sum(old[i][1] - old[i][0] for i in failed)
    assert r == dead   # disjoint sources: exactly the dead ranks' units


def _tiny_cases(n, seed=1234):
    rng = random.Random(seed)
    cases = []
    while len(cases) < n:
        H = rng.randint(1, 9)
        N = rng.randint(2, 4)
        # possibly overlapping (replicated) old ranges covering [0, H)
        old = []
        for i in range(N):
            a = rng.randint(0, H - 1)
            b = rng.randint(a + 1, H)
            old.append((a, b))
        cover = cmm.iv_union(old)
        if cover != [(0, H)]:
            continue
        nf = rng.randint(1, N - 1)
        failed = sorted(rng.sample(range(N), nf))
        M = N - nf
        if M > H:
            continue
        targets = _random_layout(rng, H, M) if M > 1 else [(0, H)]
        cases.append((old, failed, targets))
    return cases


def test_reload_minimal_bruteforce_per_unit():
    for old, failed, targets in _tiny_cases(400):
        M = len(targets)
        plan = cmm.cmm(old, failed, targets, cmm.assign_inorder(len(old), failed, M))
        assert cmm.reload_units(plan) == brute.min_reload_per_unit_choices(old, failed, targets)
        assert cmm.reload_units(plan) == cmm.eq1_min_reload(old, failed, targets)


def test_plan_is_valid_cover():
    """Every unit of every target is delivered exactly once, from a rank
    that holds it (or by reload when no alive rank does)."""
    for old, failed, targets in _tiny_cases(400, seed=99):
        M = len(targets)
        owner = cmm.assign_inorder(len(old), failed, M)
        plan = cmm.cmm(old, failed, targets, owner)
        for j, (u, v) in enumerate(targets):
            seen = []
            for x in plan:
                if x.dst != j:
                    continue
                assert x.host == owner[j]
                for y in range(x.begin, x.end):
                    seen.append(y)
                    if x.kind == cmm.RELOAD:
                        assert brute.holders(old, failed, y) == []
                    else:
                        assert x.src in brute.holders(old, failed, y)
                        assert (x.kind == cmm.KEEP) == (x.src == owner[j])
            assert sorted(seen) == list(range(u, v))


def test_assignment_bruteforce():
    """Reload does not depend on which survivor hosts which target; the
    'maxretain' choice keeps the most units local among all M! choices."""
    for old, failed, targets in _tiny_cases(300, seed=7):
        N, M = len(old), len(targets)
        reloads = set()
        best = -1
        for perm in brute.all_assignments(N, failed, M):
            plan = cmm.cmm(old, failed, targets, perm)
            reloads.add(cmm.reload_units(plan))
            best = max(best, brute.unit_retained(old, perm, targets))
        assert reloads == {brute.unit_reload(old, failed, targets)}
        sp_old, sp_new = {"x": old}, {"x": targets}
        mr = cmm.assign_maxretain(N, failed, M, sp_old, sp_new, {"x": 1})
        assert brute.unit_retained(old, mr, targets) == best


def test_inorder_not_always_optimal():
    """Reading check: in-order hosting can keep fewer bytes than the best
    permutation.  4 -> 3 with old rank 3 failed: on the query heads alone
    (14/13/13) both keep 19 heads, but over every space in bytes (query heads,
    KV heads 3/3/2 with their cache, FFN units) in-order keeps strictly less
    (tests/test_oracle_pins.py counts the bytes from the shapes)."""
    old = cmm.even_ranges(40, 4)
    targets = cmm.ranges_from_widths([14, 13, 13])
    failed = [3]
    inorder = cmm.assign_inorder(4, failed, 3)
    mr = cmm.assign_maxretain(4, failed, 3, {"q": old}, {"q": targets}, {"q": 1})
    assert brute.unit_retained(old, mr, targets) == brute.unit_retained(old, inorder, targets) == 19
    from tests.test_oracle_pins import pin_inorder_strict
    inorder_bytes, best_bytes = pin_inorder_strict()
    assert inorder_bytes < best_bytes


# --------------------------------------------------------------------------
# the tiny workload by hand
# --------------------------------------------------------------------------
def test_cfg1_hand_values():
    g = {r[0]: r[1:] for r in _read_golden("cfg1_hand.txt")}
    pb = model.build(configs.get(1))
    assert pb.new["q"] == _ranges(g["new_q_ranges"])
    assert pb.new["kv"] == _ranges(g["new_kv_ranges"])
    assert pb.old["kv"] == _ranges(g["old_kv_ranges"])
    assert pb.new["ffn"] == _ranges(g["new_ffn_ranges"])
    assert pb.self_new == 0
    n_live = 8 * (128 // 16)
    ret, inf, out = repack.self_bytes(pb, n_live)
    kv_bytes = int(g["kv_arena_bytes"][0])
    assert ret == 2 * int(g["self_retained_per_layer"][0]) + kv_bytes
    assert inf == 2 * int(g["self_inflow_per_layer"][0])
    assert pb.layout("old")[1] == int(g["self_old_arena_bytes"][0])
    assert pb.layout("new")[1] == int(g["self_new_arena_bytes"][0])
    assert pb.kv_arena_bytes("new", n_live) == kv_bytes
    # global reload / P2P bytes per layer over all survivors
    rel = p2p = 0
    for t in pb.tensors:
        if t.layer != 0:
            continue
        ub = t.unit_bytes(pb.eb)
        for x in pb.plans[t.space]:
            if x.kind == cmm.RELOAD:
                rel += (x.end - x.begin) * ub
            elif x.kind == cmm.P2P:
                p2p += (x.end - x.begin) * ub
    assert rel == int(g["global_reload_per_layer"][0])
    assert p2p == int(g["global_p2p_per_layer"][0])


def test_planner_baselines_fig3():
    """Sec. V planner baselines on the Fig. 3 example: Greedy keeps only
    what each host holds and reloads every gap (no cross-device transfer);
    Full Reload reuses nothing.  Table 2's ordering CM < Greedy < Full
    holds in reloaded rows."""
    old = [(0, 256), (256, 512), (512, 768), (768, 1024)]
    targets = cmm.floor_targets(1024, 3)
    owner = [0, 2, 3]
    r = {v: cmm.reload_units(cmm.cmm(old, [1], targets, owner, v)) for v in ("cm", "greedy", "full")}
    assert r == {"cm": 256, "greedy": 85 + 171 + 86, "full": 1024}
    g = cmm.cmm(old, [1], targets, owner, "greedy")
    assert all(x.kind in (cmm.KEEP, cmm.RELOAD) for x in g)


def test_planner_baselines_random():
    for old, failed, targets in _tiny_cases(300, seed=5):
        owner = cmm.assign_inorder(len(old), failed, len(targets))
        cm = cmm.reload_units(cmm.cmm(old, failed, targets, owner))
        gr = cmm.cmm(old, failed, targets, owner, "greedy")
        fu = cmm.cmm(old, failed, targets, owner, "full")
        # Greedy reloads exactly what the host does not hold
        want_gr = sum((v - u) - max(0, min(old[owner[j]][1], v) - max(old[owner[j]][0], u))
                      for j, (u, v) in enumerate(targets))
        assert cmm.reload_units(gr) == want_gr
        assert cmm.reload_units(fu) == sum(v - u for u, v in targets)
        assert cm <= cmm.reload_units(gr) <= cmm.reload_units(fu)
