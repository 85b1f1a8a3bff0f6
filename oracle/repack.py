"""What the reshard must produce, computed two independent ways (oracle).

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py).

The result has a plain definition (Sec. III-B: the new TP layout; Sec. III-C:
a plan moves data without changing it): for target range [a, b) of a space,

  ROWS tensor   new shard = F[a*unit : b*unit, :]
  COLS tensor   new shard = F[:, a*unit : b*unit]
  KV cache      new block p (p = table[s][blk]) holds, for the new KV heads,
                tokens blk*bt .. blk*bt+bt-1 of sequence s

where F is the full, unsharded tensor.  `expected_*` computes exactly this by
slicing the materialised full tensors.  `apply_*` instead executes the
oracle's own CMM plan: KEEP tasks copy from the old local shard, every other
task of this GPU's target takes the next bytes of the packed inflow buffer.
The two must agree (tests), and the HIP library must reproduce the first bit
for bit.

Packed buffers (the contract with the library):
  inflow   for each tensor in arena order, for each non-KEEP task of this
           GPU's target in plan order, the destination rectangle of the new
           shard in row-major order.  KV: for each layer, K then V, for each
           non-KEEP task in plan order, for each live block in ascending id,
           the block's bytes for those heads in destination order.
  outbound (in-place only) for each tensor / KV group in the same order, for
           each P2P task whose source is this GPU, the part of the task this
           GPU does not keep itself, as a rectangle of the old shard.
"""
from __future__ import annotations

import numpy as np

from . import cmm
from .model import COLS, ROWS, Problem


# ----------------------------------------------------------------------------
# full tensors and shards by definition
# ----------------------------------------------------------------------------
def full_tensor(pb: Problem, content, t) -> np.ndarray:
    idx = np.arange(t.rows * t.cols, dtype=np.uint64)
    return content(t.tag, t.layer, idx).reshape(t.rows, t.cols)


def shard_by_definition(pb: Problem, F: np.ndarray, t, rng) -> np.ndarray:
    a, b = rng
    if t.kind == ROWS:
        return F[a * t.unit:b * t.unit, :]
    return F[:, a * t.unit:b * t.unit]


def weight_arena(pb: Problem, content, which: str) -> np.ndarray:
    """This GPU's weight arena (old or new layout) filled by definition."""
    offs, size = pb.layout(which)
    arena = np.zeros(size, dtype=np.uint8)
    for t, off in zip(pb.tensors, offs):
        rng = pb.old_range(t.space) if which == "old" else pb.new_range(t.space)
        sh = shard_by_definition(pb, full_tensor(pb, content, t), t, rng)
        flat = np.ascontiguousarray(sh).view(np.uint8).reshape(-1)
        arena[off:off + flat.size] = flat
    return arena


def weight_live_mask(pb: Problem, which: str) -> np.ndarray:
    """True on arena bytes that belong to a shard (not alignment padding)."""
    offs, size = pb.layout(which)
    m = np.zeros(size, dtype=bool)
    for t, off in zip(pb.tensors, offs):
        rng = pb.old_range(t.space) if which == "old" else pb.new_range(t.space)
        r, c = t.shard_shape(rng)
        m[off:off + r * c * pb.eb] = True
    return m


def _rect(t, rng_local, shard_shape):
    """Row/col slices of a shard for a unit range given in local units."""
    a, b = rng_local
    if t.kind == ROWS:
        return slice(a * t.unit, b * t.unit), slice(0, shard_shape[1])
    return slice(0, shard_shape[0]), slice(a * t.unit, b * t.unit)


def _self_tasks(pb: Problem, space: str):
    return [x for x in pb.plans[space] if x.dst == pb.self_new]


def _outbound_pieces(pb: Problem, space: str):
    """Unit intervals this GPU sends to peers and does not keep itself."""
    mine = pb.new_range(space)
    out = []
    for x in pb.plans[space]:
        if x.kind == cmm.P2P and x.src == pb.self_old:
            for a, b in cmm.iv_subtract([(x.begin, x.end)], mine):
                out.append((a, b))
    return out


def packed_weight_inflow(pb: Problem, content) -> np.ndarray:
    chunks = []
    for t in pb.tensors:
        n0 = pb.new_range(t.space)[0]
        new_sh = shard_by_definition(pb, full_tensor(pb, content, t), t, pb.new_range(t.space))
        for x in _self_tasks(pb, t.space):
            if x.kind == cmm.KEEP:
                continue
            rs, cs = _rect(t, (x.begin - n0, x.end - n0), new_sh.shape)
            chunks.append(np.ascontiguousarray(new_sh[rs, cs]).view(np.uint8).reshape(-1))
    return np.concatenate(chunks) if chunks else np.zeros(0, np.uint8)


def packed_weight_outbound(pb: Problem, content) -> np.ndarray:
    chunks = []
    for t in pb.tensors:
        o0 = pb.old_range(t.space)[0]
        old_sh = shard_by_definition(pb, full_tensor(pb, content, t), t, pb.old_range(t.space))
        for a, b in _outbound_pieces(pb, t.space):
            rs, cs = _rect(t, (a - o0, b - o0), old_sh.shape)
            chunks.append(np.ascontiguousarray(old_sh[rs, cs]).view(np.uint8).reshape(-1))
    return np.concatenate(chunks) if chunks else np.zeros(0, np.uint8)


def apply_weights(pb: Problem, old_arena: np.ndarray, inflow: np.ndarray) -> np.ndarray:
    """Assemble the new arena by executing the oracle's plan."""
    o_offs, _ = pb.layout("old")
    n_offs, n_size = pb.layout("new")
    new = np.zeros(n_size, dtype=np.uint8)
    cur = 0
    dt = np.uint16 if pb.eb == 2 else np.uint8
    for t, oo, no in zip(pb.tensors, o_offs, n_offs):
        o_rng, n_rng = pb.old_range(t.space), pb.new_range(t.space)
        o_shape, n_shape = t.shard_shape(o_rng), t.shard_shape(n_rng)
        o_n = o_shape[0] * o_shape[1]
        n_n = n_shape[0] * n_shape[1]
        old_sh = old_arena[oo:oo + o_n * pb.eb].view(dt).reshape(o_shape)
        new_sh = new[no:no + n_n * pb.eb].view(dt).reshape(n_shape)
        for x in _self_tasks(pb, t.space):
            drs, dcs = _rect(t, (x.begin - n_rng[0], x.end - n_rng[0]), n_shape)
            if x.kind == cmm.KEEP:
                srs, scs = _rect(t, (x.begin - o_rng[0], x.end - o_rng[0]), o_shape)
                new_sh[drs, dcs] = old_sh[srs, scs]
            else:
                h = drs.stop - drs.start
                w = dcs.stop - dcs.start
                nb = h * w * pb.eb
                new_sh[drs, dcs] = inflow[cur:cur + nb].view(dt).reshape(h, w)
                cur += nb
    if cur != inflow.size:
        raise ValueError("inflow buffer size does not match the plan")
    return new


# ----------------------------------------------------------------------------
# paged KV cache
# ----------------------------------------------------------------------------
def kv_full(pb: Problem, content, layer: int, kv: int) -> np.ndarray:
    """Full logical K or V of one layer: [n_seq, seq_tokens, n_kv, head_dim]."""
    c = pb.cfg
    shape = (c["n_seq"], c["seq_tokens"], pb.n_kv, pb.head_dim)
    tag = 10 + kv
    idx = np.arange(np.prod(shape), dtype=np.uint64)
    return content(tag, layer, idx).reshape(shape)


def live_blocks(table: np.ndarray) -> np.ndarray:
    return np.unique(table[table >= 0]).astype(np.int64)


def _block_owner(table: np.ndarray, pool: int):
    seq = np.full(pool, -1, dtype=np.int64)
    blk = np.full(pool, -1, dtype=np.int64)
    for s in range(table.shape[0]):
        for b in range(table.shape[1]):
            p = int(table[s, b])
            if p >= 0 and seq[p] < 0:
                seq[p], blk[p] = s, b
    return seq, blk


def _block_view(arena, pb: Problem, which: str, pool: int, layer: int, kv: int):
    """View of one (layer, K|V) block pool as [pool, heads, bt, hd] (head
    layout) or [pool, bt, heads, hd] (token layout)."""
    a, b = pb.kv_heads(which)
    nh = b - a
    per = pool * nh * pb.block_tokens * pb.head_dim
    g = layer * 2 + kv
    flat = arena.view(np.uint16)[g * per:(g + 1) * per]
    if pb.kv_layout == "head":
        return flat.reshape(pool, nh, pb.block_tokens, pb.head_dim)
    return flat.reshape(pool, pb.block_tokens, nh, pb.head_dim)


def _heads_slice(view, pb, h0, h1, blocks):
    if pb.kv_layout == "head":
        return view[blocks, h0:h1]
    return view[blocks, :, h0:h1]


def kv_arena(pb: Problem, content, table, pool: int, which: str, poison: int = 0):
    """This GPU's KV arena (old or new layout) filled by definition; free
    blocks hold `poison`."""
    size = pb.kv_arena_bytes(which, pool)
    arena = np.full(size // 2, poison, dtype=np.uint16).view(np.uint8)
    seq, blk = _block_owner(table, pool)
    live = live_blocks(table)
    a, b = pb.kv_heads(which)
    bt = pb.block_tokens
    for l in range(pb.n_layers):
        for kv in (0, 1):
            full = kv_full(pb, content, l, kv)
            view = _block_view(arena, pb, which, pool, l, kv)
            for p in live:
                s, lb = seq[p], blk[p]
                tok = full[s, lb * bt:(lb + 1) * bt, a:b, :]          # [bt, nh, hd]
                if pb.kv_layout == "head":
                    view[p] = tok.transpose(1, 0, 2)
                else:
                    view[p] = tok
    return arena


def kv_arena_compact(pb: Problem, content, table, pool: int, which: str = "new") -> np.ndarray:
    """The KV arena indexed by block rank instead of block id: in each
    (layer, K|V) plane, position r holds the live block whose id is the r-th
    smallest (a compact pool of exactly the live blocks)."""
    by_id = kv_arena(pb, content, table, pool, which)
    live = live_blocks(table)
    planes = by_id.reshape(2 * pb.n_layers, pool, -1)
    return np.ascontiguousarray(planes[:, live, :]).reshape(-1)


def packed_kv_inflow(pb: Problem, content, table, pool: int) -> np.ndarray:
    new_arena = kv_arena(pb, content, table, pool, "new")
    live = live_blocks(table)
    n0 = pb.kv_heads("new")[0]
    chunks = []
    for l in range(pb.n_layers):
        for kv in (0, 1):
            view = _block_view(new_arena, pb, "new", pool, l, kv)
            for x in _self_tasks(pb, pb.kv_space):
                if x.kind == cmm.KEEP:
                    continue
                part = _heads_slice(view, pb, x.begin - n0, x.end - n0, live)
                chunks.append(np.ascontiguousarray(part).view(np.uint8).reshape(-1))
    return np.concatenate(chunks) if chunks else np.zeros(0, np.uint8)


def packed_kv_outbound(pb: Problem, content, table, pool: int) -> np.ndarray:
    old_arena = kv_arena(pb, content, table, pool, "old")
    live = live_blocks(table)
    o0 = pb.kv_heads("old")[0]
    chunks = []
    for l in range(pb.n_layers):
        for kv in (0, 1):
            view = _block_view(old_arena, pb, "old", pool, l, kv)
            for a, b in _outbound_pieces(pb, pb.kv_space):
                part = _heads_slice(view, pb, a - o0, b - o0, live)
                chunks.append(np.ascontiguousarray(part).view(np.uint8).reshape(-1))
    return np.concatenate(chunks) if chunks else np.zeros(0, np.uint8)


def apply_kv(pb: Problem, old_arena, inflow, table, pool: int) -> np.ndarray:
    """Assemble the new KV arena by executing the oracle's plan."""
    new = np.zeros(pb.kv_arena_bytes("new", pool), dtype=np.uint8)
    live = live_blocks(table)
    o0 = pb.kv_heads("old")[0]
    n0 = pb.kv_heads("new")[0]
    cur = 0
    for l in range(pb.n_layers):
        for kv in (0, 1):
            ov = _block_view(old_arena, pb, "old", pool, l, kv)
            nv = _block_view(new, pb, "new", pool, l, kv)
            for x in _self_tasks(pb, pb.kv_space):
                dst = _heads_slice(nv, pb, x.begin - n0, x.end - n0, live)
                if x.kind == cmm.KEEP:
                    src = _heads_slice(ov, pb, x.begin - o0, x.end - o0, live)
                else:
                    nb = dst.size * 2
                    src = inflow[cur:cur + nb].view(np.uint16).reshape(dst.shape)
                    cur += nb
                if pb.kv_layout == "head":
                    nv[live, x.begin - n0:x.end - n0] = src
                else:
                    nv[live, :, x.begin - n0:x.end - n0] = src
    if cur != inflow.size:
        raise ValueError("KV inflow buffer size does not match the plan")
    return new


def kv_live_mask(pb: Problem, table, pool: int, which: str) -> np.ndarray:
    """True on KV arena bytes that belong to live blocks."""
    words = np.zeros(pb.kv_arena_bytes(which, pool) // 2, dtype=np.uint16)
    live = live_blocks(table)
    for l in range(pb.n_layers):
        for kv in (0, 1):
            v = _block_view(words.view(np.uint8), pb, which, pool, l, kv)
            v[live] = 1
    return np.repeat(words.astype(bool), 2)


# ----------------------------------------------------------------------------
# the definition evaluated word by word (full-size workloads, sampled)
# ----------------------------------------------------------------------------
def _groups(keys):
    """(key, positions) for every distinct key, via one stable sort."""
    order = np.argsort(keys, kind="stable")
    ks = keys[order]
    cuts = np.flatnonzero(np.diff(ks)) + 1
    for part in np.split(order, cuts):
        if part.size:
            yield int(keys[part[0]]), part


def expected_weight_words(pb: Problem, content, offsets):
    """(words, valid) at even byte offsets of the NEW weight arena: the
    16-bit word the definition puts there, and whether the offset lies in a
    shard (not alignment padding).  Same definition as weight_arena(),
    evaluated one position at a time."""
    offs, _ = pb.layout("new")
    offs = np.asarray(offs, dtype=np.int64)
    q = np.asarray(offsets, dtype=np.int64)
    ti = np.searchsorted(offs, q, side="right") - 1
    words = np.zeros(q.shape, np.uint16)
    valid = np.zeros(q.shape, bool)
    for k, sel in _groups(ti):
        t = pb.tensors[k]
        a, b = pb.new_range(t.space)
        r, c = t.shard_shape((a, b))
        e = (q[sel] - offs[k]) // pb.eb
        ok = e < r * c
        sel, e = sel[ok], e[ok]
        i, j = e // c, e % c
        if t.kind == ROWS:
            gi, gj = i + a * t.unit, j
        else:
            gi, gj = i, j + a * t.unit
        words[sel] = content(t.tag, t.layer, (gi * t.cols + gj).astype(np.uint64))
        valid[sel] = True
    return words, valid


def expected_packed_weight_words(pb: Problem, content, segments, offsets):
    """Words at even byte offsets of a packed weight buffer (inflow or
    outbound): segment (tensor, layer, which, kind, a, b, host_offset,
    bytes) holds units [a, b) of the full tensor as a row-major rectangle."""
    q = np.asarray(offsets, dtype=np.int64)
    starts = np.array([s[6] for s in segments], dtype=np.int64)
    si = np.searchsorted(starts, q, side="right") - 1
    words = np.zeros(q.shape, np.uint16)
    for k, sel in _groups(si):
        ti, _, _, _, a, b, off, _ = segments[k]
        t = pb.tensors[ti]
        e = (q[sel] - off) // pb.eb
        if t.kind == ROWS:
            gi, gj = a * t.unit + e // t.cols, e % t.cols
        else:
            w = (b - a) * t.unit
            gi, gj = e // w, a * t.unit + e % w
        words[sel] = content(t.tag, t.layer, (gi * t.cols + gj).astype(np.uint64))
    return words


def expected_kv_words(pb: Problem, content, table, pool: int, offsets):
    """(words, valid) at even byte offsets of the NEW KV arena; offsets in
    free blocks are not valid.  Same definition as kv_arena()."""
    c = pb.cfg
    a, b = pb.kv_heads("new")
    nh, bt, hd = b - a, pb.block_tokens, pb.head_dim
    block = nh * bt * hd * pb.eb
    q = np.asarray(offsets, dtype=np.int64)
    g, rest = q // (pool * block), q % (pool * block)
    p, inner = rest // block, (rest % block) // pb.eb
    if pb.kv_layout == "head":
        h, t, d = inner // (bt * hd), (inner // hd) % bt, inner % hd
    else:
        t, h, d = inner // (nh * hd), (inner // hd) % nh, inner % hd
    seq, blk = _block_owner(table, pool)
    s, lb = seq[p], blk[p]
    valid = s >= 0
    words = np.zeros(q.shape, np.uint16)
    idx = ((s * c["seq_tokens"] + lb * bt + t) * pb.n_kv + (a + h)) * hd + d
    for grp, sel in _groups(np.where(valid, g, -1)):
        if grp >= 0:
            words[sel] = content(10 + grp % 2, grp // 2, idx[sel].astype(np.uint64))
    return words, valid


# ----------------------------------------------------------------------------
# packed-buffer segment lists (the packing order stated in the docstring)
# ----------------------------------------------------------------------------
def inflow_segments(pb: Problem, n_live: int):
    """[(tensor index or -1, layer, 0=K/1=V, kind, unit_begin, unit_end,
    host_offset, bytes)] of the packed inflow buffers (weights, then KV)."""
    w, at = [], 0
    for ti, t in enumerate(pb.tensors):
        ub = t.unit_bytes(pb.eb)
        for x in _self_tasks(pb, t.space):
            if x.kind != cmm.KEEP:
                n = (x.end - x.begin) * ub
                w.append((ti, t.layer, 0, x.kind, x.begin, x.end, at, n))
                at += n
    k, at = [], 0
    per_head = n_live * pb.block_tokens * pb.head_dim * pb.eb
    for l in range(pb.n_layers):
        for which in (0, 1):
            for x in _self_tasks(pb, pb.kv_space):
                if x.kind != cmm.KEEP:
                    n = (x.end - x.begin) * per_head
                    k.append((-1, l, which, x.kind, x.begin, x.end, at, n))
                    at += n
    return w, k


def outbound_segments(pb: Problem, n_live: int):
    w, at = [], 0
    for ti, t in enumerate(pb.tensors):
        ub = t.unit_bytes(pb.eb)
        for a, b in _outbound_pieces(pb, t.space):
            w.append((ti, t.layer, 0, cmm.P2P, a, b, at, (b - a) * ub))
            at += (b - a) * ub
    k, at = [], 0
    per_head = n_live * pb.block_tokens * pb.head_dim * pb.eb
    for l in range(pb.n_layers):
        for which in (0, 1):
            for a, b in _outbound_pieces(pb, pb.kv_space):
                k.append((-1, l, which, cmm.P2P, a, b, at, (b - a) * per_head))
                at += (b - a) * per_head
    return w, k


# ----------------------------------------------------------------------------
# byte accounting of this GPU's share (definition-level)
# ----------------------------------------------------------------------------
def self_bytes(pb: Problem, n_live: int):
    """Retained / inflow / dropped-outbound bytes of this GPU."""
    ret = inf = out = 0
    for t in pb.tensors:
        ub = t.unit_bytes(pb.eb)
        for x in _self_tasks(pb, t.space):
            if x.kind == cmm.KEEP:
                ret += (x.end - x.begin) * ub
            else:
                inf += (x.end - x.begin) * ub
        out += sum(b - a for a, b in _outbound_pieces(pb, t.space)) * ub
    kv_ub = pb.n_layers * 2 * n_live * pb.block_tokens * pb.head_dim * pb.eb
    for x in _self_tasks(pb, pb.kv_space):
        if x.kind == cmm.KEEP:
            ret += (x.end - x.begin) * kv_ub
        else:
            inf += (x.end - x.begin) * kv_ub
    out += sum(b - a for a, b in _outbound_pieces(pb, pb.kv_space)) * kv_ub
    return ret, inf, out
