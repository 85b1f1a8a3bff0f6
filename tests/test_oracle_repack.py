"""Pins of the oracle's repack (CPU).

The new shard has a plain definition (slices of the full tensors); the
oracle also assembles it by executing its own plan.  Pins: the two agree;
concatenating every target's shard reproduces the full tensor; retained plus
inflow bytes equal the new shard; an unchanged partition is a no-op; a
single target receives the whole tensor; the packed buffers hold exactly
the definition's bytes.
"""
import random

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

from oracle import cmm, model, repack
from synth import configs, pagetable
from synth.content import KIND_FP16, KIND_RAW16, KIND_TAG16, Content


def tiny_cfg(rng: random.Random, experts=False):
    """A random small decoder and TP change (odd sizes, unequal widths)."""
    N = rng.randint(2, 5)
    nf = rng.randint(1, N - 1)
    failed = sorted(rng.sample(range(N), nf))
    M = N - nf
    hd = rng.choice([2, 4, 6, 8])
    n_kv = rng.randint(1, 4)
    g = rng.randint(1, 3)
    n_q = n_kv * g
    if n_q < N:
        n_q = n_kv * (-(-N // n_kv))
    kw = dict(
        layers=rng.randint(1, 2), hidden=rng.choice([6, 10, 16]), n_q=n_q, n_kv=n_kv,
        head_dim=hd, old_tp=N, new_tp=M, failed=failed,
        self_old=rng.choice([i for i in range(N) if i not in failed]),
        n_seq=rng.randint(1, 3), seq_tokens=rng.choice([4, 8, 12]), block_tokens=4,
        fragmented=rng.random() < 0.5, pool_factor=1.5, seed=rng.randint(0, 99),
        w_kind=KIND_TAG16, kv_kind=KIND_RAW16,
        new_q_widths=None, new_kv_widths=None, new_ffn_widths=None, new_expert_widths=None,
        kv_layout=rng.choice(["head", "token"]),
    )
    if experts:
        kw.update(experts=rng.randint(N, 3 * N), expert_ffn=rng.choice([2, 4]), ffn=0)
    else:
        unit = rng.choice([1, 2, 3])
        kw.update(ffn=unit * rng.randint(N, 4 * N), ffn_unit=unit, experts=0)
    # old ranges: even split of every space except a random unequal q split
    c = configs.get(1, **kw)
    if rng.random() < 0.5:
        cuts = sorted(rng.sample(range(1, n_q), N - 1))
        b = [0] + cuts + [n_q]
        c["old_ranges"] = {"q": [(b[i], b[i + 1]) for i in range(N)]}
    return c


def med_cfg(rng: random.Random, experts=False):
    """A random medium decoder and TP change: head_dim 64/128 with 16-token
    blocks (2-4 KiB KV head lines), hidden 256-1024, up to TP 8, fragmented
    pools, unequal old q splits, dense or MoE."""
    N = rng.randint(2, 8)
    nf = rng.randint(1, min(3, N - 1))
    failed = sorted(rng.sample(range(N), nf))
    M = N - nf
    hd = rng.choice([64, 128])
    n_kv = rng.choice([1, 2, 4, 8])
    g = rng.choice([1, 2, 4])
    n_q = max(n_kv * g, n_kv * (-(-N // n_kv)))
    kw = dict(layers=rng.randint(1, 3), hidden=rng.choice([256, 512, 1024]), n_q=n_q, n_kv=n_kv,
              head_dim=hd, old_tp=N, new_tp=M, failed=failed,
              self_old=rng.choice([i for i in range(N) if i not in failed]),
              n_seq=rng.randint(1, 12), seq_tokens=rng.choice([64, 128, 256, 512]), block_tokens=16,
              fragmented=rng.random() < 0.5, pool_factor=1.25, seed=rng.randint(0, 999),
              w_kind=KIND_TAG16, kv_kind=rng.choice([KIND_TAG16, KIND_RAW16]),
              new_q_widths=None, new_kv_widths=None, new_ffn_widths=None, new_expert_widths=None,
              kv_layout=rng.choice(["head", "head", "token"]))
    if experts:
        kw.update(experts=rng.randint(N, 3 * N), expert_ffn=rng.choice([64, 128, 256]), ffn=0)
    else:
        unit = rng.choice([1, 8, 16])
        kw.update(ffn=unit * rng.randint(N, 16 * N), ffn_unit=unit, experts=0)
    c = configs.get(1, **kw)
    if rng.random() < 0.5:
        cuts = sorted(rng.sample(range(1, n_q), N - 1))
        b = [0] + cuts + [n_q]
        c["old_ranges"] = {"q": [(b[i], b[i + 1]) for i in range(N)]}
    return c


def _check_cfg(c):
    pb = model.build(c)
    content = Content(c["seed"], c["w_kind"], c["kv_kind"])
    table, pool = pagetable.make_for(c)
    # weights
    old = repack.weight_arena(pb, content, "old")
    want = repack.weight_arena(pb, content, "new")
    inflow = repack.packed_weight_inflow(pb, content)
    got = repack.apply_weights(pb, old, inflow)
    mask = repack.weight_live_mask(pb, "new")
    np.testing.assert_array_equal(got[mask], want[mask])
    # KV
    kold = repack.kv_arena(pb, content, table, pool, "old")
    kwant = repack.kv_arena(pb, content, table, pool, "new")
    kin = repack.packed_kv_inflow(pb, content, table, pool)
    kgot = repack.apply_kv(pb, kold, kin, table, pool)
    km = repack.kv_live_mask(pb, table, pool, "new")
    np.testing.assert_array_equal(kgot[km], kwant[km])
    # byte accounting
    n_live = len(repack.live_blocks(table))
    ret, inf, _ = repack.self_bytes(pb, n_live)
    assert inf == inflow.size + kin.size
    assert ret + inf == mask.sum() + km.sum()
    return pb


def test_cfg1_plan_execution_equals_definition():
    pb = _check_cfg(configs.get(1))
    assert pb.layout("new")[1] == 1099776


@pytest.mark.parametrize("layout", ["head", "token"])
def test_cfg1_kv_layouts(layout):
    _check_cfg(configs.get(1, kv_layout=layout))


@settings(max_examples=60, deadline=None)
@given(st.integers(0, 2 ** 31), st.booleans())
def test_random_tiny_plan_execution_equals_definition(seed, experts):
    _check_cfg(tiny_cfg(random.Random(seed), experts))


@settings(max_examples=40, deadline=None)
@given(st.integers(0, 2 ** 31))
def test_new_shards_concatenate_to_full_tensor(seed):
    rng = random.Random(seed)
    c = tiny_cfg(rng, rng.random() < 0.3)
    pb = model.build(c)
    content = Content(c["seed"], c["w_kind"], c["kv_kind"])
    for t in pb.tensors:
        F = repack.full_tensor(pb, content, t)
        rs = pb.new[t.space]
        axis = 0 if t.kind == model.ROWS else 1
        if all(rs[i][1] == rs[i + 1][0] for i in range(len(rs) - 1)):
            parts = [repack.shard_by_definition(pb, F, t, r) for r in rs]
            np.testing.assert_array_equal(np.concatenate(parts, axis=axis), F)
        else:
            # replicated KV heads (GQA): shards overlap; rebuild unit by unit
            rebuilt = np.zeros_like(F)
            for r in rs:
                sh = repack.shard_by_definition(pb, F, t, r)
                sl = slice(r[0] * t.unit, r[1] * t.unit)
                if axis == 0:
                    rebuilt[sl] = sh
                else:
                    rebuilt[:, sl] = sh
            assert cmm.iv_union(rs) == [(0, pb.spaces[t.space])]
            np.testing.assert_array_equal(rebuilt, F)


def test_identity_partition_is_noop():
    c = configs.get(1, new_tp=4, failed=[], new_q_widths=[1, 1, 1, 1],
                    new_ffn_widths=[172, 172, 172, 172], self_old=2)
    pb = model.build(c)
    content = Content(0, KIND_FP16, KIND_FP16)
    for sp in pb.spaces:
        assert all(x.kind == cmm.KEEP for x in pb.plans[sp])
    assert repack.packed_weight_inflow(pb, content).size == 0
    old = repack.weight_arena(pb, content, "old")
    np.testing.assert_array_equal(repack.apply_weights(pb, old, np.zeros(0, np.uint8)), old)


def test_single_target_gets_full_tensor():
    c = configs.get(1, new_tp=1, failed=[1, 2, 3], new_q_widths=[4],
                    new_ffn_widths=[688], self_old=0)
    pb = model.build(c)
    content = Content(0, KIND_FP16, KIND_FP16)
    offs, _ = pb.layout("new")
    arena = repack.weight_arena(pb, content, "new")
    for t, off in zip(pb.tensors, offs):
        F = repack.full_tensor(pb, content, t)
        got = arena[off:off + F.nbytes].view(np.uint16).reshape(F.shape)
        np.testing.assert_array_equal(got, F)


def test_packed_inflow_holds_definition_bytes():
    """Every inflow byte is a byte of the new shard that is not retained."""
    c = configs.get(1)
    pb = model.build(c)
    content = Content(0, KIND_TAG16, KIND_TAG16)
    inflow = repack.packed_weight_inflow(pb, content)
    assert inflow.size == 2 * 154624
    # Wq of layer 0 is first: rows 64..127 of the full tensor (query head 1)
    F = repack.full_tensor(pb, content, pb.tensors[0])
    np.testing.assert_array_equal(inflow[:32768].view(np.uint16).reshape(64, 256), F[64:128])


def test_outbound_pieces_are_dropped_parts():
    """In cfg 1 this GPU (old 0) sends nothing: FFN [0,172) is all kept."""
    pb = model.build(configs.get(1))
    assert repack.packed_weight_outbound(pb, Content(0, KIND_TAG16, KIND_TAG16)).size == 0
    # old rank 2 sends FFN [459,516) to new rank 2 and keeps [344,459)
    pb2 = model.build(configs.get(1, self_old=2))
    assert repack._outbound_pieces(pb2, "ffn") == [(459, 516)]


@settings(max_examples=30, deadline=None)
@given(st.integers(0, 2 ** 31), st.booleans())
def test_pointwise_definition_matches_materialised(seed, experts):
    """The word-by-word evaluation used for full-size sampling agrees with
    slicing the materialised full tensors, at every byte offset."""
    c = tiny_cfg(random.Random(seed), experts)
    pb = model.build(c)
    content = Content(c["seed"], c["w_kind"], c["kv_kind"])
    arena = repack.weight_arena(pb, content, "new")
    mask = repack.weight_live_mask(pb, "new")
    offs = np.arange(0, arena.size, 2)
    words, valid = repack.expected_weight_words(pb, content, offs)
    np.testing.assert_array_equal(valid, mask[offs])
    np.testing.assert_array_equal(words[valid], arena.view(np.uint16)[valid])
    table, pool = pagetable.make_for(c)
    karena = repack.kv_arena(pb, content, table, pool, "new")
    kmask = repack.kv_live_mask(pb, table, pool, "new")
    koffs = np.arange(0, karena.size, 2)
    kw, kv = repack.expected_kv_words(pb, content, table, pool, koffs)
    np.testing.assert_array_equal(kv, kmask[koffs])
    np.testing.assert_array_equal(kw[kv], karena.view(np.uint16)[kv])
