"""Exhaustive searches that pin the CMM plan on tiny inputs (oracle).

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py).

Sec. III-C argues the CMM plan reloads the least possible under the
assumption that a reload byte costs more than any transfer byte (Eq. 1).
These searches check that claim without using the CMM loop: they enumerate
every per-unit source choice, and every survivor-to-target assignment.
"""
from __future__ import annotations

import itertools


def holders(old_ranges, failed, x):
    dead = set(failed)
    return [i for i, (s, e) in enumerate(old_ranges) if i not in dead and s <= x < e]


def min_reload_per_unit_choices(old_ranges, failed, targets, limit=1 << 20):
    """Minimum reload over every plan that, for each unit of each target,
    picks one alive holder or a reload (exhaustive product; tiny inputs)."""
    choices = []
    for u, v in targets:
        for x in range(u, v):
            choices.append(holders(old_ranges, failed, x) + ["R"])
    n = 1
    for c in choices:
        n *= len(c)
    if n > limit:
        raise ValueError("input too large for exhaustive search")
    best = None
    for pick in itertools.product(*choices):
        r = sum(1 for p in pick if p == "R")
        best = r if best is None else min(best, r)
    return best if best is not None else 0


def unit_retained(old_ranges, owner, targets):
    """Units of each target already held by the old rank that hosts it."""
    tot = 0
    for j, (u, v) in enumerate(targets):
        s, e = old_ranges[owner[j]]
        tot += max(0, min(e, v) - max(s, u))
    return tot


def unit_reload(old_ranges, failed, targets):
    """Units of targets that no alive rank holds (counted unit by unit)."""
    return sum(1 for u, v in targets for x in range(u, v)
               if not holders(old_ranges, failed, x))


def all_assignments(N, failed, M):
    dead = set(failed)
    alive = [i for i in range(N) if i not in dead]
    return [list(p) for p in itertools.permutations(alive, M)]
