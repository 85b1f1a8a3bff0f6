"""Partitions, the CMM planning loop and the minimum reload (oracle).

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py).

Paper passages followed:
  * Alg. 1 (Continuous Minimal Migration), Sec. III-B: H is the largest end
    of any current range, dead ranks included; target j covers
    [floor((j-1) H / M), floor(j H / M)); each target is intersected with
    every alive source range, each non-empty intersection becomes a
    transfer and is removed from the target, and whatever is left becomes a
    reload from host.
  * Sec. III-B, unequal widths: shards may be floor(S/g) or ceil(S/g) wide.
  * Eq. 1, Sec. III-C: the minimum reload is the sum over targets of the
    target size minus the part of it that surviving sources cover.

Readings where the paper is silent:
  * target widths are an input; rules "floor" (Alg. 1) and "ceil_first"
    (larger shards first, as the workloads state) generate them;
  * target j is hosted by the j-th alive old rank in ascending order
    ("inorder"); "maxretain" instead takes the survivor permutation that
    keeps the most bytes local (first such permutation in lexicographic
    order); reload is the same for every permutation;
  * when several alive ranks hold a unit (replicated KV heads), the
    target's own host is asked first, then the others in ascending rank;
  * KV-head ranges follow the query heads (GQA): query heads [a, b) with g
    query heads per KV head need KV heads [floor(a/g), ceil(b/g)).
"""
from __future__ import annotations

import itertools
from dataclasses import dataclass

KEEP, P2P, RELOAD = 0, 1, 2
KIND_NAMES = {KEEP: "KEEP", P2P: "P2P", RELOAD: "RELOAD"}


# ----------------------------------------------------------------------------
# Interval helpers: a "set" is a sorted list of disjoint half-open (a, b).
# ----------------------------------------------------------------------------
def iv_intersect(tar, rng):
    """Pieces of interval set `tar` that lie inside the range `rng`."""
    s, e = rng
    out = []
    for a, b in tar:
        lo, hi = max(a, s), min(b, e)
        if lo < hi:
            out.append((lo, hi))
    return out


def iv_subtract(tar, rng):
    """Interval set `tar` with range `rng` removed."""
    s, e = rng
    out = []
    for a, b in tar:
        if b <= s or a >= e:
            out.append((a, b))
            continue
        if a < s:
            out.append((a, s))
        if b > e:
            out.append((e, b))
    return out


def iv_measure(ivs):
    return sum(b - a for a, b in ivs)


def iv_union(ivs):
    """Union of arbitrary (possibly overlapping) intervals."""
    out = []
    for a, b in sorted(i for i in ivs if i[0] < i[1]):
        if out and a <= out[-1][1]:
            out[-1] = (out[-1][0], max(out[-1][1], b))
        else:
            out.append((a, b))
    return out


# ----------------------------------------------------------------------------
# Partitions
# ----------------------------------------------------------------------------
def floor_targets(H: int, M: int):
    """Alg. 1 target ranges: [floor((j-1)H/M), floor(jH/M)) for j = 1..M."""
    return [((j - 1) * H // M, j * H // M) for j in range(1, M + 1)]


def ranges_from_widths(widths):
    out, at = [], 0
    for w in widths:
        out.append((at, at + w))
        at += w
    return out


def ceil_first_widths(S: int, g: int):
    """Widths ceil(S/g) for the first S mod g shards, floor(S/g) after."""
    q, r = divmod(S, g)
    return [q + 1 if j < r else q for j in range(g)]


def even_ranges(S: int, g: int):
    """The initial equal split (g divides S in every workload)."""
    return ranges_from_widths(ceil_first_widths(S, g))


def gqa_ranges(q_ranges, group: int):
    """KV-head ranges needed by each rank's query-head range."""
    return [(a // group, -(-b // group)) for a, b in q_ranges]


# ----------------------------------------------------------------------------
# Which old rank hosts each target
# ----------------------------------------------------------------------------
def survivors(N: int, failed):
    dead = set(failed)
    return [i for i in range(N) if i not in dead]


def assign_inorder(N: int, failed, M: int):
    alive = survivors(N, failed)
    if len(alive) != M:
        raise ValueError("one target per survivor expected")
    return list(alive)


def retained_weight(space_old, space_new, weights, owner_old, j):
    """Units kept in place if old rank `owner_old` hosts target j, weighted
    by bytes per unit of each space."""
    tot = 0
    for sp, w in weights.items():
        tot += w * iv_measure(iv_intersect([space_new[sp][j]], space_old[sp][owner_old]))
    return tot


def assign_maxretain(N, failed, M, space_old, space_new, weights):
    """Survivor permutation with the most retained bytes (first in
    lexicographic order among equals)."""
    alive = survivors(N, failed)
    if len(alive) != M:
        raise ValueError("one target per survivor expected")
    best, best_val = None, -1
    for perm in itertools.permutations(alive):
        v = sum(retained_weight(space_old, space_new, weights, perm[j], j)
                for j in range(M))
        if v > best_val:
            best, best_val = list(perm), v
    return best


# ----------------------------------------------------------------------------
# Alg. 1
# ----------------------------------------------------------------------------
@dataclass(frozen=True)
class Task:
    kind: int      # KEEP / P2P / RELOAD
    begin: int     # units, half-open
    end: int
    src: int       # old rank holding the data, -1 for a reload
    dst: int       # target index j (0-based)
    host: int      # old rank that hosts target j

    def as_tuple(self):
        return (self.kind, self.begin, self.end, self.src, self.dst, self.host)


def cmm(old_ranges, failed, targets, owner, variant="cm"):
    """The CMM loop of Alg. 1 for one space.

    old_ranges[i] is old rank i's range (dead ranks included); `targets` is
    the list of target ranges; owner[j] is the old rank hosting target j.
    Tasks come out target by target; within a target, transfers in source
    order (host first, then ascending rank), then reloads in range order.

    variant (the planner baselines of Sec. V, Table 2):
      "cm"      Alg. 1
      "greedy"  keep what the host already holds; every gap is reloaded,
                no cross-device transfer
      "full"    no reuse: the whole target is reloaded
    """
    dead = set(failed)
    N = len(old_ranges)
    plan = []
    for j, tgt in enumerate(targets):
        tar = [tgt] if tgt[0] < tgt[1] else []
        order = [owner[j]] + [i for i in range(N) if i != owner[j]]
        for i in order:
            if i in dead or variant == "full" or (variant == "greedy" and i != owner[j]):
                continue
            inter = iv_intersect(tar, old_ranges[i])
            if inter:
                kind = KEEP if i == owner[j] else P2P
                for a, b in inter:
                    plan.append(Task(kind, a, b, i, j, owner[j]))
                tar = iv_subtract(tar, old_ranges[i])
        for a, b in tar:
            plan.append(Task(RELOAD, a, b, -1, j, owner[j]))
    return plan


def eq1_min_reload(old_ranges, failed, targets):
    """Eq. 1: sum over targets of |T_j| minus the measure of T_j covered by
    surviving sources.  Written with a union so that it also holds when
    sources overlap (replicated units)."""
    dead = set(failed)
    tot = 0
    for tgt in targets:
        covered = iv_union([(max(tgt[0], s), min(tgt[1], e))
                            for i, (s, e) in enumerate(old_ranges) if i not in dead])
        tot += (tgt[1] - tgt[0]) - iv_measure(covered)
    return tot


def eq1_closed_form(old_ranges, failed, targets):
    """Eq. 1, second line: H - sum_i sum_j |S_i cap T_j| (disjoint sources
    and a target partition of [0, H))."""
    dead = set(failed)
    H = max(e for _, e in old_ranges)
    kept = 0
    for i, (s, e) in enumerate(old_ranges):
        if i in dead:
            continue
        for u, v in targets:
            kept += max(0, min(e, v) - max(s, u))
    return H - kept


def reload_units(plan):
    return sum(t.end - t.begin for t in plan if t.kind == RELOAD)
