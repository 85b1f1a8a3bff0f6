"""Describe a TP-sharded decoder to the library (atp_problem).

A decoder shape is a plain dict (layers, hidden, n_q, n_kv, head_dim, ffn
or experts/expert_ffn, elem_bytes, old_tp, new_tp, failed, self_old, ...).
Spaces: 0 = query heads, 1 = KV heads, 2 = FFN column groups (dense) or
experts (MoE).  Tensors per layer, in arena order: wq, wk, wv (rows), wo
(columns), then w_gate, w_up (rows), w_down (columns), or the expert
tensors e_gate, e_up, e_down (rows of [experts * rows_per_expert, cols]).

Old ranges default to an even split of each space, KV heads following the
query heads (GQA); successive switches pass the previous new ranges as
`old_ranges`.  New ranges are explicit widths when given, else
ceil-first widths, KV heads GQA-derived unless widths are given.
"""
from __future__ import annotations

import ctypes as C

from . import atp

SPACE_Q, SPACE_KV, SPACE_FFN = 0, 1, 2

_TENSORS_DENSE = [("wq", atp.ROWS, SPACE_Q), ("wk", atp.ROWS, SPACE_KV), ("wv", atp.ROWS, SPACE_KV),
                  ("wo", atp.COLS, SPACE_Q), ("w_gate", atp.ROWS, SPACE_FFN),
                  ("w_up", atp.ROWS, SPACE_FFN), ("w_down", atp.COLS, SPACE_FFN)]
_TENSORS_MOE = [("wq", atp.ROWS, SPACE_Q), ("wk", atp.ROWS, SPACE_KV), ("wv", atp.ROWS, SPACE_KV),
                ("wo", atp.COLS, SPACE_Q), ("e_gate", atp.ROWS, SPACE_FFN),
                ("e_up", atp.ROWS, SPACE_FFN), ("e_down", atp.ROWS, SPACE_FFN)]


def _gqa(ranges, g):
    return [(a // g, -(-b // g)) for a, b in ranges]


def tensor_list(shape: dict):
    """[(name, layer, kind, space, rows, cols, unit)] in arena order."""
    L, h, hd = shape["layers"], shape["hidden"], shape["head_dim"]
    nq, nkv = shape["n_q"], shape["n_kv"]
    moe = bool(shape.get("experts"))
    out = []
    for l in range(L):
        for name, kind, sp in (_TENSORS_MOE if moe else _TENSORS_DENSE):
            if name == "wq":
                dims = (nq * hd, h, hd)
            elif name in ("wk", "wv"):
                dims = (nkv * hd, h, hd)
            elif name == "wo":
                dims = (h, nq * hd, hd)
            elif name in ("w_gate", "w_up"):
                dims = (shape["ffn"], h, shape["ffn_unit"])
            elif name == "w_down":
                dims = (h, shape["ffn"], shape["ffn_unit"])
            elif name in ("e_gate", "e_up"):
                E, fe = shape["experts"], shape["expert_ffn"]
                dims = (E * fe, h, fe)
            else:  # e_down
                E, fe = shape["experts"], shape["expert_ffn"]
                dims = (E * h, fe, h)
            out.append((name, l, kind, sp, *dims))
    return out


def space_totals(shape: dict):
    third = shape["experts"] if shape.get("experts") else shape["ffn"] // shape["ffn_unit"]
    return [shape["n_q"], shape["n_kv"], third]


class Built:
    """A Problem plus the arrays it points into."""

    def __init__(self, problem, keep, tensors, n_live, pool, old_ranges):
        self.problem = problem
        self.keep = keep
        self.tensors = tensors
        self.n_live = n_live
        self.pool = pool
        self.old_ranges = old_ranges  # [space][old rank] -> (begin, end)

    def plan(self) -> atp.Plan:
        return atp.Plan(self.problem, keep=self.keep)


def build(shape: dict, n_live: int | None = None, pool: int | None = None, flags: int = 0,
          staging_cap: int = 0, with_kv: bool = True) -> Built:
    N, M = shape["old_tp"], shape["new_tp"]
    totals = space_totals(shape)
    g = shape["n_q"] // shape["n_kv"]
    keep = []
    old_given = shape.get("old_ranges") or {}
    names = ["q", "kv", "exp" if shape.get("experts") else "ffn"]
    old = {}
    old["q"] = old_given.get("q") or atp.partition(totals[0], N, atp.RULE_CEIL_FIRST)
    old["kv"] = old_given.get("kv") or _gqa(old["q"], g)
    old[names[2]] = old_given.get(names[2]) or atp.partition(totals[2], N, atp.RULE_CEIL_FIRST)
    new_widths = {"q": shape.get("new_q_widths"), "kv": shape.get("new_kv_widths"),
                  "ffn": shape.get("new_ffn_widths"), "exp": shape.get("new_expert_widths")}
    new_given = shape.get("new_ranges") or {}
    spaces = (atp.Space * 3)()
    for s, name in enumerate(names):
        sp = spaces[s]
        sp.total_units = totals[s]
        sp.old_tp = N
        sp.new_tp = M
        o = (atp.Range * N)(*[atp.Range(a, b) for a, b in old[name]])
        keep.append(o)
        sp.old_ranges = C.cast(o, C.POINTER(atp.Range))
        rng = new_given.get(name)
        if rng is None and new_widths[name] is not None:
            at, rng = 0, []
            for w in new_widths[name]:
                rng.append((at, at + w))
                at += w
        if rng is not None:
            n = (atp.Range * M)(*[atp.Range(a, b) for a, b in rng])
            keep.append(n)
            sp.new_rule = atp.RULE_EXPLICIT
            sp.new_ranges = C.cast(n, C.POINTER(atp.Range))
        elif name == "kv" and shape.get("kv_rule", "gqa") == "gqa":
            sp.new_rule = atp.RULE_GQA
            sp.gqa_space = SPACE_Q
            sp.gqa_group = g
        else:
            sp.new_rule = atp.RULE_FLOOR if shape.get("new_rule") == "floor" else atp.RULE_CEIL_FIRST
    tl = tensor_list(shape)
    tens = (atp.Tensor * len(tl))()
    eb = shape["elem_bytes"]
    for i, (name, l, kind, sp, rows, cols, unit) in enumerate(tl):
        t = tens[i]
        t.space, t.kind, t.layer, t.elem_bytes = sp, kind, l, eb
        t.rows, t.cols, t.unit = rows, cols, unit
        t.old_offset = atp.OFFSET_AUTO
    keep += [spaces, tens]
    failed = (C.c_int32 * max(1, len(shape["failed"])))(*shape["failed"])
    keep.append(failed)
    pb = atp.Problem()
    pb.n_spaces = 3
    pb.spaces = C.cast(spaces, C.POINTER(atp.Space))
    pb.n_tensors = len(tl)
    pb.tensors = C.cast(tens, C.POINTER(atp.Tensor))
    pb.failed = C.cast(failed, C.POINTER(C.c_int32))
    pb.n_failed = len(shape["failed"])
    pb.self_old_rank = shape["self_old"]
    pb.flags = flags
    pb.staging_cap = staging_cap
    if with_kv:
        bt = shape["block_tokens"]
        if n_live is None:
            n_live = shape["n_seq"] * (-(-shape["seq_tokens"] // bt))
        if pool is None:
            pool = n_live
        kv = atp.KV(SPACE_KV, shape["layers"], bt, shape["head_dim"], eb,
                    atp.KV_TOKEN_MAJOR if shape.get("kv_layout") == "token" else atp.KV_HEAD_MAJOR,
                    pool, n_live)
        keep.append(kv)
        pb.kv = C.pointer(kv)
    return Built(pb, keep, tl, n_live, pool, [old[n] for n in names])
