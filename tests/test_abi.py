"""The C ABI: every function include/atp.h declares is exported by
libatp.so, and planning rejects malformed problems with the documented
codes (CPU; no GPU calls)."""
import ctypes as C
import os
import re
import subprocess

import pytest

from paper_2511_11617_amd import atp, problem
from synth import configs

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "atp.h")


def declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(atp_\w+)\s*\(", src, flags=re.M)))


def test_header_functions_are_exported():
    names = declared()
    assert {"atp_plan", "atp_reshard_weights", "atp_reshard_kv", "atp_sync"} <= set(names)
    out = subprocess.run(["nm", "-D", "--defined-only", atp.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r"\bT (atp_\w+)", out))
    missing = [n for n in names if n not in exported]
    assert not missing, missing
    for n in names:
        assert hasattr(atp.lib, n)


def test_one_hip_runtime_whatever_the_import_order():
    # torch bundles a HIP runtime with the system's soname: loading the
    # library before torch must not leave a second runtime in the process
    code = ("import paper_2511_11617_amd.atp as atp\n"
            "from synth import gpu, pinned\n"
            "gpu.lib(); pinned._lib()\n"
            "import torch\n"
            "rt = atp.hip_runtimes()\n"
            "assert len(rt) == 1 and 'torch' in rt[0], rt\n")
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    r = subprocess.run(["python", "-c", code], cwd=root, capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stderr[-2000:]


def _plan(c, **kw):
    return problem.build(c, **kw).plan()


def test_dead_self_rank_is_einval():
    with pytest.raises(atp.AtpError) as e:
        _plan(configs.get(1, self_old=1))
    assert e.value.code == atp.EINVAL


def test_new_tp_must_match_survivors():
    with pytest.raises(atp.AtpError) as e:
        _plan(configs.get(1, failed=[1, 2]))
    assert e.value.code == atp.EINVAL


def test_non_covering_explicit_ranges_are_einval():
    c = configs.get(1, new_q_widths=None, new_ranges={"q": [(0, 2), (2, 3), (3, 3)]})
    with pytest.raises(atp.AtpError) as e:
        _plan(c)
    assert e.value.code == atp.EINVAL
    assert "cover" in str(e.value)


def test_bad_gqa_reference_is_einval():
    b = problem.build(configs.get(1))
    b.problem.spaces[1].gqa_space = 1   # a space cannot follow itself
    with pytest.raises(atp.AtpError) as e:
        b.plan()
    assert e.value.code == atp.EINVAL


def test_old_and_new_ranges_from_rules():
    """Old ranges from rules (even split, GQA from the query heads) and new
    ranges from widths, all resolved by the library."""
    c = configs.get(2)  # 40 q / 8 KV heads, TP 4 -> 3, q widths 14/13/13, KV widths 3/3/2
    b = problem.build(c)
    sp = b.problem.spaces
    assert (sp[0].old_rule, sp[1].old_rule, sp[2].old_rule) == (atp.RULE_CEIL_FIRST, atp.RULE_GQA,
                                                                 atp.RULE_CEIL_FIRST)
    assert (sp[0].new_rule, sp[1].new_rule, sp[2].new_rule) == (atp.RULE_WIDTHS, atp.RULE_WIDTHS,
                                                                 atp.RULE_CEIL_FIRST)
    p = b.plan()
    assert p.old_ranges(0) == [(0, 10), (10, 20), (20, 30), (30, 40)]
    assert p.old_ranges(1) == [(0, 2), (2, 4), (4, 6), (6, 8)]
    assert p.old_ranges(2) == [(0, 272), (272, 544), (544, 816), (816, 1088)]
    assert p.ranges(0) == [(0, 14), (14, 27), (27, 40)]
    assert p.ranges(1) == [(0, 3), (3, 6), (6, 8)]
    assert p.ranges(2) == [(0, 363), (363, 726), (726, 1088)]
    # the tiny workload: 4 q heads over 2 KV heads, GQA old and new
    p1 = problem.build(configs.get(1)).plan()
    assert p1.old_ranges(1) == [(0, 1), (0, 1), (1, 2), (1, 2)]
    assert p1.ranges(1) == [(0, 1), (1, 2), (1, 2)]


def test_bad_widths_and_old_gqa_reference_are_einval():
    b = problem.build(configs.get(2))
    w = b.problem.spaces[0].new_widths
    w[2] = 12  # 14 + 13 + 12 != 40
    with pytest.raises(atp.AtpError) as e:
        b.plan()
    assert e.value.code == atp.EINVAL and "widths" in str(e.value)
    b = problem.build(configs.get(2))
    b.problem.spaces[0].old_rule = atp.RULE_GQA  # the query-head space cannot follow itself
    b.problem.spaces[0].gqa_space = 0
    with pytest.raises(atp.AtpError) as e:
        b.plan()
    assert e.value.code == atp.EINVAL
    b = problem.build(configs.get(2))
    b.problem.spaces[2].old_rule = 9
    with pytest.raises(atp.AtpError) as e:
        b.plan()
    assert e.value.code == atp.EINVAL and "unknown rule" in str(e.value)


def test_in_place_staging_cap_too_small_is_ecapacity():
    c = configs.scaled(5, layers=2, n_seq=2, seq_tokens=256)
    st = _plan(c, flags=atp.INPLACE, staging_cap=1 << 30).stats()
    need = max(st.staging_w, st.staging_kv)
    _plan(c, flags=atp.INPLACE, staging_cap=need)  # exactly enough
    with pytest.raises(atp.AtpError) as e:  # less than the descriptors alone
        _plan(c, flags=atp.INPLACE, staging_cap=1 << 12)
    assert e.value.code == atp.ECAPACITY


def test_partition_helper():
    assert atp.partition(1024, 3, atp.RULE_FLOOR) == [(0, 341), (341, 682), (682, 1024)]
    assert atp.partition(688, 3, atp.RULE_CEIL_FIRST) == [(0, 230), (230, 459), (459, 688)]
    with pytest.raises(atp.AtpError):
        atp.partition(10, 0, atp.RULE_FLOOR)


def test_planning_is_deterministic():
    c = configs.scaled(5, layers=3, n_seq=2, seq_tokens=256)
    a = _plan(c, flags=atp.INPLACE, staging_cap=2 << 30)
    b = _plan(c, flags=atp.INPLACE, staging_cap=2 << 30)
    sa, sb = a.stats(), b.stats()
    for f, _ in atp.Stats._fields_:
        assert getattr(sa, f) == getattr(sb, f), f


def test_warmup_without_a_gpu_and_with_a_bad_count():
    with pytest.raises(atp.AtpError) as e:
        atp.warmup(0, 0, 5000)
    assert e.value.code == atp.EINVAL
    import torch
    if torch.cuda.is_available():
        pytest.skip("this machine has a GPU: the GPU tests cover atp_warmup")
    with pytest.raises(atp.AtpError) as e:
        atp.warmup(0, 0)
    assert e.value.code == atp.EHIP


def test_staging_overlapping_an_arena_is_einval_before_any_gpu_call():
    """Argument checks run before the first HIP call (fake addresses, no
    GPU): staging may not overlap the arena it repacks."""
    for flags in (0, atp.INPLACE):
        p = _plan(configs.get(1), flags=flags)
        st = p.stats()
        A, N = 1 << 32, 1 << 34  # fake, 256-byte aligned device addresses
        size = max(st.old_arena_bytes, st.new_arena_bytes)
        new = None if flags else N
        inside = A + 4096  # inside the old arena
        with pytest.raises(atp.AtpError) as e:
            p.reshard_weights(A, size, new, st.new_arena_bytes if new else 0, 1 << 36, st.inflow_w,
                              1 << 37, st.outbound_w, inside, st.staging_w, 0, 0)
        assert e.value.code == atp.EINVAL and "staging overlaps" in str(e.value)
        if not flags:  # inside the new arena
            with pytest.raises(atp.AtpError) as e:
                p.reshard_weights(A, size, N, st.new_arena_bytes, 1 << 36, st.inflow_w, 1 << 37, st.outbound_w,
                                  N + 256, st.staging_w, 0, 0)
            assert e.value.code == atp.EINVAL and "staging overlaps" in str(e.value)
        with pytest.raises(atp.AtpError) as e:  # the KV call too
            p.reshard_kv(A, st.old_kv_bytes if flags == 0 else max(st.old_kv_bytes, st.new_kv_bytes),
                         new, st.new_kv_bytes if new else 0, 1 << 38, 8, 8, 1 << 36, st.inflow_kv,
                         1 << 37, st.outbound_kv, A, st.staging_kv, 0, 0)
        assert e.value.code == atp.EINVAL and "staging overlaps" in str(e.value)


def test_old_widths_and_floor_rules_give_the_same_plan_as_explicit_ranges():
    """Old ranges from widths or the floor rule plan exactly like the same
    ranges given explicitly (tasks of every space, statistics)."""
    c = configs.get(1, old_ranges={"q": [(0, 1), (1, 2), (2, 3), (3, 4)]})
    ref = _plan(c)
    for rule in (atp.RULE_WIDTHS, atp.RULE_FLOOR):
        b = problem.build(c)
        sp = b.problem.spaces[0]
        sp.old_rule = rule
        if rule == atp.RULE_WIDTHS:
            w = (C.c_int64 * 4)(1, 1, 1, 1)
            b.keep.append(w)
            sp.old_widths = C.cast(w, C.POINTER(C.c_int64))
        p = b.plan()
        assert p.old_ranges(0) == [(0, 1), (1, 2), (2, 3), (3, 4)]
        for s in range(3):
            assert p.tasks(s) == ref.tasks(s)
        sa, sb = p.stats(), ref.stats()
        for f, _ in atp.Stats._fields_:
            assert getattr(sa, f) == getattr(sb, f), f
    # unequal old widths 2 / 1 / 1 / 0 query heads, the KV heads following them (GQA)
    b = problem.build(configs.get(1))
    sp = b.problem.spaces[0]
    sp.old_rule = atp.RULE_WIDTHS
    w = (C.c_int64 * 4)(2, 1, 1, 0)
    b.keep.append(w)
    sp.old_widths = C.cast(w, C.POINTER(C.c_int64))
    p = b.plan()
    assert p.old_ranges(0) == [(0, 2), (2, 3), (3, 4), (4, 4)]
    assert p.old_ranges(1) == [(0, 1), (1, 2), (1, 2), (2, 2)]
