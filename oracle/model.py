"""The TP-sharded decoder, its partitions and arena layouts (oracle).

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py).

Readings of the paper (Sec. III-B layout invariants; Sec. III-C and IV plan
over one linear byte space per rank):
  * planning is done per partition space in units that must not be cut: a
    query head, a KV head, a group of FFN columns, an expert;
  * weights are [out, in] row-major; column-parallel tensors (Wq, Wk, Wv,
    W_gate, W_up, expert tensors) shard rows ("ROWS"), row-parallel tensors
    (Wo, W_down) shard columns ("COLS");
  * a rank's parameters sit in one arena, layer-major, tensor order
    [wq, wk, wv, wo, w_gate, w_up, w_down] (dense) or
    [wq, wk, wv, wo, e_gate, e_up, e_down] (MoE); each shard starts at a
    multiple of 256 bytes;
  * the paged KV cache of a rank is [layer][K, V][physical block][KV head]
    [token][dim] ("head" layout: each block groups its heads) or
    [layer][K, V][block][token][KV head][dim] ("token" layout); block ids
    do not change across the reshard.
"""
from __future__ import annotations

from dataclasses import dataclass, field

from synth.content import TAGS

from . import cmm

ROWS, COLS = 0, 1
ALIGN = 256


def align_up(x: int, a: int = ALIGN) -> int:
    return -(-x // a) * a


@dataclass
class Tensor:
    name: str
    tag: int
    layer: int
    kind: int        # ROWS / COLS
    space: str
    rows: int
    cols: int
    unit: int        # rows (ROWS) or columns (COLS) per unit

    def shard_shape(self, rng):
        a, b = rng
        if self.kind == ROWS:
            return ((b - a) * self.unit, self.cols)
        return (self.rows, (b - a) * self.unit)

    def unit_bytes(self, eb):
        return (self.unit * self.cols if self.kind == ROWS else self.rows * self.unit) * eb


@dataclass
class Problem:
    cfg: dict
    eb: int
    spaces: dict                 # name -> total units
    old: dict                    # name -> list of old ranges (per old rank)
    new: dict                    # name -> list of target ranges (per target j)
    failed: list
    owner: list                  # owner[j] = old rank hosting target j
    self_old: int
    self_new: int
    plans: dict = field(default_factory=dict)   # name -> list[cmm.Task]
    tensors: list = field(default_factory=list)
    n_layers: int = 0
    kv_space: str = "kv"
    block_tokens: int = 16
    head_dim: int = 128
    kv_layout: str = "head"
    n_kv: int = 0

    # -- per-rank geometry -------------------------------------------------
    def old_range(self, space, rank=None):
        return self.old[space][self.self_old if rank is None else rank]

    def new_range(self, space, j=None):
        return self.new[space][self.self_new if j is None else j]

    def layout(self, which: str):
        """(offsets, total bytes) of this GPU's weight arena, old or new."""
        offs, at = [], 0
        for t in self.tensors:
            rng = self.old_range(t.space) if which == "old" else self.new_range(t.space)
            r, c = t.shard_shape(rng)
            offs.append(at)
            at = align_up(at + r * c * self.eb)
        return offs, at

    def kv_heads(self, which: str):
        return self.old_range(self.kv_space) if which == "old" else self.new_range(self.kv_space)

    def kv_block_bytes(self, which: str):
        a, b = self.kv_heads(which)
        return (b - a) * self.block_tokens * self.head_dim * self.eb

    def kv_arena_bytes(self, which: str, pool: int):
        return self.n_layers * 2 * pool * self.kv_block_bytes(which)

    def space_tasks(self, space):
        return self.plans[space]


def _space_defs(cfg):
    sp = {"q": cfg["n_q"], "kv": cfg["n_kv"]}
    if cfg["experts"]:
        sp["exp"] = cfg["experts"]
    else:
        if cfg["ffn"] % cfg["ffn_unit"]:
            raise ValueError("FFN width must be a multiple of its unit")
        sp["ffn"] = cfg["ffn"] // cfg["ffn_unit"]
    return sp


def _tensors(cfg):
    L, h, hd = cfg["layers"], cfg["hidden"], cfg["head_dim"]
    nq, nkv = cfg["n_q"], cfg["n_kv"]
    out = []
    for l in range(L):
        out += [
            Tensor("wq", TAGS["wq"], l, ROWS, "q", nq * hd, h, hd),
            Tensor("wk", TAGS["wk"], l, ROWS, "kv", nkv * hd, h, hd),
            Tensor("wv", TAGS["wv"], l, ROWS, "kv", nkv * hd, h, hd),
            Tensor("wo", TAGS["wo"], l, COLS, "q", h, nq * hd, hd),
        ]
        if cfg["experts"]:
            E, fe = cfg["experts"], cfg["expert_ffn"]
            out += [
                Tensor("e_gate", TAGS["e_gate"], l, ROWS, "exp", E * fe, h, fe),
                Tensor("e_up", TAGS["e_up"], l, ROWS, "exp", E * fe, h, fe),
                Tensor("e_down", TAGS["e_down"], l, ROWS, "exp", E * h, fe, h),
            ]
        else:
            F, u = cfg["ffn"], cfg["ffn_unit"]
            out += [
                Tensor("w_gate", TAGS["w_gate"], l, ROWS, "ffn", F, h, u),
                Tensor("w_up", TAGS["w_up"], l, ROWS, "ffn", F, h, u),
                Tensor("w_down", TAGS["w_down"], l, COLS, "ffn", h, F, u),
            ]
    return out


def _new_ranges(cfg, name, total, M, q_new):
    key = {"q": "new_q_widths", "kv": "new_kv_widths", "ffn": "new_ffn_widths",
           "exp": "new_expert_widths"}[name]
    explicit = (cfg.get("new_ranges") or {}).get(name)
    if explicit is not None:
        return [tuple(r) for r in explicit]
    if name == "kv" and cfg[key] is None and cfg["kv_rule"] == "gqa":
        return cmm.gqa_ranges(q_new, cfg["n_q"] // cfg["n_kv"])
    if cfg[key] is not None:
        w = list(cfg[key])
        if name == "ffn" and cfg["ffn_unit"] != 1 and sum(w) != total:
            raise ValueError("FFN widths are given in units")
        return cmm.ranges_from_widths(w)
    rule = cfg.get("new_rule", "ceil_first")
    if rule == "floor":
        return cmm.floor_targets(total, M)
    return cmm.ranges_from_widths(cmm.ceil_first_widths(total, M))


def _old_ranges(cfg, name, total, N, q_old):
    explicit = (cfg.get("old_ranges") or {}).get(name)
    if explicit is not None:
        return [tuple(r) for r in explicit]
    if name == "kv":
        return cmm.gqa_ranges(q_old, cfg["n_q"] // cfg["n_kv"])
    return cmm.even_ranges(total, N)


def build(cfg: dict, assign: str = "inorder", variant: str = "cm") -> Problem:
    """The oracle's view of workload `cfg` and its per-space CMM plans."""
    N, M = cfg["old_tp"], cfg["new_tp"]
    failed = list(cfg["failed"])
    sp = _space_defs(cfg)
    old, new = {}, {}
    old["q"] = _old_ranges(cfg, "q", sp["q"], N, None)
    new["q"] = _new_ranges(cfg, "q", sp["q"], M, None)
    for name, total in sp.items():
        if name == "q":
            continue
        old[name] = _old_ranges(cfg, name, total, N, old["q"])
        new[name] = _new_ranges(cfg, name, total, M, new["q"])
    tensors = _tensors(cfg)
    eb = cfg["elem_bytes"]
    if assign == "inorder":
        owner = cmm.assign_inorder(N, failed, M)
    else:
        weights = {name: 0 for name in sp}
        for t in tensors:
            weights[t.space] += t.unit_bytes(eb)
        bt, hd = cfg["block_tokens"], cfg["head_dim"]
        live = cfg["n_seq"] * (-(-cfg["seq_tokens"] // bt))
        weights["kv"] += cfg["layers"] * 2 * live * bt * hd * eb
        owner = cmm.assign_maxretain(N, failed, M, old, new, weights)
    self_old = cfg["self_old"]
    if self_old in failed:
        raise ValueError("this GPU must survive")
    pb = Problem(cfg=cfg, eb=eb, spaces=sp, old=old, new=new, failed=failed,
                 owner=owner, self_old=self_old, self_new=owner.index(self_old),
                 tensors=tensors, n_layers=cfg["layers"],
                 block_tokens=cfg["block_tokens"], head_dim=cfg["head_dim"],
                 kv_layout=cfg.get("kv_layout", "head"), n_kv=cfg["n_kv"])
    for name in sp:
        pb.plans[name] = cmm.cmm(old[name], failed, new[name], owner, variant)
    return pb
