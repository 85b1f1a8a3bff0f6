"""Host replay of the library's executable schedule (test infrastructure).

Executes the copies that atp_plan_copies exports, with the semantics the
header states, on numpy byte buffers:
  * every access is bounds-checked against its buffer;
  * within one repack level all reads happen before all writes, and a
    level whose copies write bytes that any copy of the same level reads,
    or that two copies write, is reported as a hazard;
  * host inflow landings happen as early as the schedule allows and a later
    level that reads a landed byte is reported; outbound reads happen as
    late as allowed and must not see bytes an earlier level wrote;
  * a landing that waits for nothing runs beside the levels, so the bytes
    it writes must be disjoint from every level's, scatter's and other
    landing's.
The replayed arena is then compared with the oracle by the caller.
"""
from __future__ import annotations

import ctypes as C

import numpy as np

from paper_2511_11617_amd import atp

OLD, NEW, STAGING, INFLOW, OUTBOUND = 0, 1, 2, 3, 4
REPACK, SCATTER, H2D, H2D_RING, D2H = 0, 1, 2, 3, 4


class Copy(C.Structure):
    _fields_ = [("op", C.c_int32), ("level", C.c_int32), ("src_buf", C.c_int32), ("dst_buf", C.c_int32),
                ("flags", C.c_int32), ("after_d2h", C.c_int32), ("src_off", C.c_uint64),
                ("dst_off", C.c_uint64), ("src_pitch", C.c_uint64), ("dst_pitch", C.c_uint64),
                ("src_stride", C.c_uint64), ("dst_stride", C.c_uint64), ("item_begin", C.c_int64),
                ("item_end", C.c_int64), ("run", C.c_uint64), ("rows", C.c_uint64)]


def copies(plan: atp.Plan, which: int):
    fn = atp.lib.atp_plan_copies
    fn.argtypes = [C.c_void_p, C.c_int32, C.POINTER(Copy), C.c_int32, C.POINTER(C.c_int32)]
    fn.restype = C.c_int
    n = C.c_int32()
    atp._check(fn(plan.h, which, None, 0, C.byref(n)))
    arr = (Copy * max(1, n.value))()
    atp._check(fn(plan.h, which, arr, n.value, C.byref(n)))
    return list(arr[:n.value])


class Hazard(AssertionError):
    pass


def _lines(x: Copy, live: np.ndarray):
    """(src_starts, dst_starts) int64 arrays, one entry per line of copy x."""
    if x.flags & 4:  # block range: live blocks with ids in [item_begin, item_end)
        pos = np.arange(np.searchsorted(live, x.item_begin), np.searchsorted(live, x.item_end))
    else:
        pos = np.arange(x.item_begin, x.item_end)
    rel = pos - (pos[0] if len(pos) else 0)
    si = live[pos] if x.flags & 1 else rel
    di = live[pos] if x.flags & 2 else rel
    t = np.arange(x.rows, dtype=np.int64)
    src = (x.src_off + si.astype(np.int64)[:, None] * x.src_stride + t[None, :] * x.src_pitch).reshape(-1)
    dst = (x.dst_off + di.astype(np.int64)[:, None] * x.dst_stride + t[None, :] * x.dst_pitch).reshape(-1)
    return src, dst


def _gather(buf: np.ndarray, starts: np.ndarray, run: int) -> np.ndarray:
    """Bytes of every line, concatenated ([len(starts) * run])."""
    if len(starts) == 0:
        return np.zeros(0, np.uint8)
    if len(starts) <= 64:
        return np.concatenate([buf[s:s + run] for s in starts])
    out = np.empty(len(starts) * run, np.uint8)
    step = max(1, (1 << 24) // max(run, 1))
    ar = np.arange(run, dtype=np.int64)
    for i in range(0, len(starts), step):
        blk = starts[i:i + step]
        out[i * run:(i + len(blk)) * run] = buf[(blk[:, None] + ar[None, :]).reshape(-1)]
    return out


def _scatter(buf: np.ndarray, starts: np.ndarray, run: int, data: np.ndarray):
    if len(starts) == 0:
        return
    if len(starts) <= 64:
        for k, s in enumerate(starts):
            buf[s:s + run] = data[k * run:(k + 1) * run]
        return
    step = max(1, (1 << 24) // max(run, 1))
    ar = np.arange(run, dtype=np.int64)
    for i in range(0, len(starts), step):
        blk = starts[i:i + step]
        buf[(blk[:, None] + ar[None, :]).reshape(-1)] = data[i * run:(i + len(blk)) * run]


def _overlaps(a_lo, a_hi, b_lo, b_hi) -> bool:
    """Does any interval of set A meet any interval of set B?"""
    if len(a_lo) == 0 or len(b_lo) == 0:
        return False
    order = np.argsort(b_lo, kind="stable")
    bl, bh = b_lo[order], np.maximum.accumulate(b_hi[order])
    k = np.searchsorted(bl, a_hi)          # intervals of B starting before a_hi
    has = k > 0
    return bool(np.any(bh[np.maximum(k - 1, 0)][has] > a_lo[has]))


def _self_disjoint(lo, hi) -> bool:
    if len(lo) < 2:
        return True
    o = np.argsort(lo, kind="stable")
    return bool(np.all(lo[o][1:] >= np.maximum.accumulate(hi[o])[:-1]))


def replay(cps, bufs: dict, live: np.ndarray):
    """bufs: {id: np.uint8 array}.  Mutates the buffers."""
    def check(buf, starts, run):
        b = bufs[buf]
        if len(starts) and (starts.min() < 0 or starts.max() + run > b.size):
            raise Hazard(f"access outside buffer {buf} of {b.size} bytes")

    def move(x, src, dst):
        check(x.src_buf, src, x.run)
        check(x.dst_buf, dst, x.run)
        _scatter(bufs[x.dst_buf], dst, x.run, _gather(bufs[x.src_buf], src, x.run))

    levels = sorted({x.level for x in cps if x.op == REPACK})
    landed = {OLD: [], NEW: []}
    written = {OLD: [], NEW: []}
    d2h = [x for x in cps if x.op == D2H]          # issued in list order
    pending = [x for x in cps if x.op == H2D]
    state = {"d2h_done": 0, "levels_done": 0}

    def cat(L):
        if not L:
            return np.zeros(0, np.int64), np.zeros(0, np.int64)
        return np.concatenate([a for a, _ in L]), np.concatenate([b for _, b in L])

    def do_host(x):
        src, dst = _lines(x, live)
        move(x, src, dst)
        if x.op == H2D and x.dst_buf in landed:
            landed[x.dst_buf].append((dst, dst + x.run))

    def do_d2h(x):
        src, _ = _lines(x, live)
        if x.src_buf in written:
            wl, wh = cat(written[x.src_buf])
            if _overlaps(src, src + x.run, wl, wh):
                raise Hazard("outbound read after an overwrite")
        do_host(x)
        state["d2h_done"] += 1

    def d2h_until(pred):
        # outbound copies complete in issue order
        while state["d2h_done"] < len(d2h) and pred(d2h[state["d2h_done"]]):
            do_d2h(d2h[state["d2h_done"]])

    def land_ready():
        # inflow lands as early as its gates allow
        for x in list(pending):
            if (x.level < 0 or x.level < state["levels_done"]) and state["d2h_done"] >= x.after_d2h:
                do_host(x)
                pending.remove(x)

    land_ready()
    for L in levels:
        d2h_until(lambda x: 0 <= x.level <= L)
        land_ready()
        lvl = [x for x in cps if x.op == REPACK and x.level == L]
        moves, rd, wr = [], {}, {}
        for x in lvl:
            src, dst = _lines(x, live)
            check(x.src_buf, src, x.run)
            check(x.dst_buf, dst, x.run)
            moves.append((x, dst, _gather(bufs[x.src_buf], src, x.run)))
            rd.setdefault(x.src_buf, []).append((src, src + x.run))
            wr.setdefault(x.dst_buf, []).append((dst, dst + x.run))
            if x.src_buf in landed:
                ll, lh = cat(landed[x.src_buf])
                if _overlaps(src, src + x.run, ll, lh):
                    raise Hazard(f"level {L} reads bytes that inflow already landed on")
        for buf, W in wr.items():
            wl, wh = cat(W)
            if not _self_disjoint(wl, wh):
                raise Hazard(f"level {L}: two copies write the same bytes")
            if buf in rd:
                rl, rh = cat(rd[buf])
                if _overlaps(wl, wh, rl, rh):
                    raise Hazard(f"level {L} reads and writes the same bytes")
        for x, dst, data in moves:
            _scatter(bufs[x.dst_buf], dst, x.run, data)
            if x.dst_buf in written:
                written[x.dst_buf].append((dst, dst + x.run))
        state["levels_done"] = L + 1
        land_ready()
    # landing ring, after every level: a scatter first waits for the outbound
    # reads it is gated on (outbound reads still happen as late as allowed)
    for x in cps:
        if x.op in (H2D_RING, SCATTER):
            if x.op == SCATTER:
                d2h_until(lambda y: state["d2h_done"] < x.after_d2h)
            src, dst = _lines(x, live)
            move(x, src, dst)
            if x.op == SCATTER and x.dst_buf in written:
                written[x.dst_buf].append((dst, dst + x.run))
    d2h_until(lambda x: True)
    land_ready()
    if pending:
        raise Hazard("inflow landing whose gates never open")
    # a landing that waits for nothing runs beside the levels and scatters:
    # the bytes it writes must be disjoint from theirs and from each other's
    for buf in (OLD, NEW):
        ll = [(d, d + x.run) for x in cps if x.op == H2D and x.level < 0 and x.dst_buf == buf
              for d in [_lines(x, live)[1]]]
        if not ll:
            continue
        lo, hi = np.concatenate([a for a, _ in ll]), np.concatenate([b for _, b in ll])
        if not _self_disjoint(lo, hi):
            raise Hazard("two landings write the same bytes")
        wl, wh = cat(written[buf])
        if _overlaps(lo, hi, wl, wh):
            raise Hazard("a landing and a level or scatter write the same bytes")
