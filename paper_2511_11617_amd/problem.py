"""Describe a TP-sharded decoder to the library (atp_problem).

A decoder shape is a plain dict (layers, hidden, n_q, n_kv, head_dim, ffn
or experts/expert_ffn, elem_bytes, old_tp, new_tp, failed, self_old, ...).
Spaces: 0 = query heads, 1 = KV heads, 2 = FFN column groups (dense) or
experts (MoE).  Tensors per layer, in arena order: wq, wk, wv (rows), wo
(columns), then w_gate, w_up (rows), w_down (columns), or the expert
tensors e_gate, e_up, e_down (rows of [experts * rows_per_expert, cols]).

Only shapes, widths and rules are passed; the library derives every
range.  Old ranges default to the even split of each space (the
ceil-first rule), KV heads following the query heads (GQA); successive
switches pass the previous new ranges as `old_ranges`.  New ranges are the
stated widths when given, else the ceil-first rule (the floor rule of Alg. 1
on request), KV heads GQA-derived unless widths are given.
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

    def __init__(self, problem, keep, tensors, n_live, pool, n_spaces):
        self.problem = problem
        self.keep = keep
        self.tensors = tensors
        self.n_live = n_live
        self.pool = pool
        self.n_spaces = n_spaces
        self._old = None

    def plan(self) -> atp.Plan:
        return atp.Plan(self.problem, keep=self.keep)

    @property
    def old_ranges(self):
        """[space][old rank] -> (begin, end), as the library resolved them."""
        if self._old is None:
            p = self.plan()
            self._old = [p.old_ranges(s) for s in range(self.n_spaces)]
        return self._old


def build(shape: dict, n_live: int | None = None, pool: int | None = None, flags: int = 0,
          staging_cap: int = 0, with_kv: bool = True) -> Built:
    N, M = shape["old_tp"], shape["new_tp"]
    totals = space_totals(shape)
    g = shape["n_q"] // shape["n_kv"]
    keep = []
    old_given = shape.get("old_ranges") or {}
    names = ["q", "kv", "exp" if shape.get("experts") else "ffn"]
    new_widths = {"q": shape.get("new_q_widths"), "kv": shape.get("new_kv_widths"),
                  "ffn": shape.get("new_ffn_widths"), "exp": shape.get("new_expert_widths")}
    new_given = shape.get("new_ranges") or {}
    spaces = (atp.Space * 3)()

    def ranges(rs):
        arr = (atp.Range * len(rs))(*[atp.Range(a, b) for a, b in rs])
        keep.append(arr)
        return C.cast(arr, C.POINTER(atp.Range))

    for s, name in enumerate(names):
        sp = spaces[s]
        sp.total_units = totals[s]
        sp.old_tp = N
        sp.new_tp = M
        sp.gqa_space = SPACE_Q
        sp.gqa_group = g
        if old_given.get(name) is not None:
            sp.old_rule = atp.RULE_EXPLICIT
            sp.old_ranges = ranges(old_given[name])
        else:
            sp.old_rule = atp.RULE_GQA if name == "kv" else atp.RULE_CEIL_FIRST
        if new_given.get(name) is not None:
            sp.new_rule = atp.RULE_EXPLICIT
            sp.new_ranges = ranges(new_given[name])
        elif new_widths[name] is not None:
            w = (C.c_int64 * M)(*new_widths[name])
            keep.append(w)
            sp.new_rule = atp.RULE_WIDTHS
            sp.new_widths = C.cast(w, C.POINTER(C.c_int64))
        elif name == "kv" and shape.get("kv_rule", "gqa") == "gqa":
            sp.new_rule = atp.RULE_GQA
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
    return Built(pb, keep, tl, n_live, pool, len(names))
