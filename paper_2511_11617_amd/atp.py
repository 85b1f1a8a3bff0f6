"""ctypes binding of libatp.so (include/atp.h), argument marshalling only.

Every step of the reshard runs in the library: planning on the host in
C++, repacking and landing in HIP kernels and HIP copies.  Device and
pinned host buffers are passed as integer addresses (for example
`tensor.data_ptr()`), streams as `torch.cuda.Stream().cuda_stream`.
There is no fallback: if the library is missing, importing this module
raises.
"""
from __future__ import annotations

import ctypes as C
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
# ATP_LIB may name another build of the same library (e.g. a tuning variant)
LIB_PATH = os.environ.get("ATP_LIB") or os.path.join(_HERE, "libatp.so")

# ---- status codes and enums (atp.h) -----------------------------------------
OK, EINVAL, ECAPACITY, EHIP, EALIGN, ESTATE = 0, -1, -2, -3, -4, -5
RULE_EXPLICIT, RULE_FLOOR, RULE_CEIL_FIRST, RULE_GQA, RULE_WIDTHS = 0, 1, 2, 3, 4
ROWS, COLS = 0, 1
OFFSET_AUTO = (1 << 64) - 1
KV_HEAD_MAJOR, KV_TOKEN_MAJOR = 0, 1
ASSIGN_INORDER, ASSIGN_MAXRETAIN = 0, 1
INPLACE = 1 << 4
PLAN_GREEDY = 1 << 8
PLAN_FULL = 1 << 9
KV_COMPACT = 1 << 10
NO_TAIL_STAGING = 1 << 11
KEEP, P2P, RELOAD = 0, 1, 2
SEG_INFLOW_W, SEG_OUTBOUND_W, SEG_INFLOW_KV, SEG_OUTBOUND_KV = 0, 1, 2, 3

EXPORTS = [
    "atp_plan", "atp_plan_free", "atp_reshard_weights", "atp_reshard_kv", "atp_sync",
    "atp_plan_stats", "atp_plan_tasks", "atp_plan_ranges", "atp_plan_old_ranges", "atp_plan_owner",
    "atp_plan_layout", "atp_plan_segments", "atp_plan_launches", "atp_partition",
    "atp_last_error", "atp_st_open", "atp_st_close", "atp_st_find", "atp_load_weights",
    "atp_kv_evict_lru", "atp_daemon_serve", "atp_state_connect", "atp_state_disconnect",
    "atp_state_alloc", "atp_state_open", "atp_state_release", "atp_state_free", "atp_state_put",
    "atp_state_get", "atp_state_list", "atp_state_shutdown", "atp_warmup", "atp_load_reshard_weights",
    "atp_reshard_kv_noalloc", "atp_scratch_bytes", "atp_load_reshard_weights_async", "atp_plan_load_stats",
]


class Range(C.Structure):
    _fields_ = [("begin", C.c_int64), ("end", C.c_int64)]


class Space(C.Structure):
    _fields_ = [("total_units", C.c_int64), ("old_tp", C.c_int32), ("new_tp", C.c_int32),
                ("old_ranges", C.POINTER(Range)), ("new_rule", C.c_int32),
                ("gqa_space", C.c_int32), ("gqa_group", C.c_int32), ("old_rule", C.c_int32),
                ("new_ranges", C.POINTER(Range)), ("old_widths", C.POINTER(C.c_int64)),
                ("new_widths", C.POINTER(C.c_int64))]


class Tensor(C.Structure):
    _fields_ = [("space", C.c_int32), ("kind", C.c_int32), ("layer", C.c_int32),
                ("elem_bytes", C.c_int32), ("rows", C.c_int64), ("cols", C.c_int64),
                ("unit", C.c_int64), ("old_offset", C.c_uint64)]


class KV(C.Structure):
    _fields_ = [("space", C.c_int32), ("num_layers", C.c_int32), ("block_tokens", C.c_int32),
                ("head_dim", C.c_int32), ("elem_bytes", C.c_int32), ("layout", C.c_int32),
                ("num_blocks", C.c_int64), ("live_blocks", C.c_int64)]


class Problem(C.Structure):
    _fields_ = [("n_spaces", C.c_int32), ("spaces", C.POINTER(Space)),
                ("n_tensors", C.c_int32), ("tensors", C.POINTER(Tensor)),
                ("kv", C.POINTER(KV)), ("failed", C.POINTER(C.c_int32)),
                ("n_failed", C.c_int32), ("self_old_rank", C.c_int32),
                ("flags", C.c_int32), ("reserved", C.c_int32), ("staging_cap", C.c_uint64)]


class Timing(C.Structure):
    _fields_ = [("plan_ms", C.c_double), ("wall_ms", C.c_double), ("repack_w_ms", C.c_double),
                ("repack_kv_ms", C.c_double), ("repack_span_ms", C.c_double), ("h2d_ms", C.c_double), ("d2h_ms", C.c_double),
                ("scatter_ms", C.c_double), ("overlap", C.c_double), ("repack_bytes", C.c_uint64),
                ("h2d_bytes", C.c_uint64), ("d2h_bytes", C.c_uint64), ("scatter_bytes", C.c_uint64),
                ("n_launches", C.c_int32), ("reserved", C.c_int32), ("repack_union_ms", C.c_double)]


class Stats(C.Structure):
    _fields_ = [("self_new_rank", C.c_int32), ("n_levels_w", C.c_int32), ("n_levels_kv", C.c_int32),
                ("n_desc_w", C.c_int32), ("n_desc_kv", C.c_int32), ("reserved", C.c_int32)] + [
        (n, C.c_uint64) for n in (
            "old_arena_bytes", "new_arena_bytes", "old_kv_bytes", "new_kv_bytes",
            "retained_w", "inflow_w", "outbound_w", "retained_kv", "inflow_kv", "outbound_kv",
            "moved_w", "moved_kv", "staged_w", "staged_kv", "staging_w", "staging_kv",
            "global_keep", "global_p2p", "global_reload", "reload_min", "tail_w", "tail_kv")]


class Task(C.Structure):
    _fields_ = [("kind", C.c_int32), ("src", C.c_int32), ("dst", C.c_int32), ("host", C.c_int32),
                ("begin", C.c_int64), ("end", C.c_int64)]


class Segment(C.Structure):
    _fields_ = [("tensor", C.c_int32), ("layer", C.c_int32), ("which", C.c_int32),
                ("kind", C.c_int32), ("unit_begin", C.c_int64), ("unit_end", C.c_int64),
                ("host_offset", C.c_uint64), ("bytes", C.c_uint64)]


class Launch(C.Structure):
    _fields_ = [("kind", C.c_int32), ("level", C.c_int32), ("bytes", C.c_uint64), ("ms", C.c_double)]


class StTensor(C.Structure):
    _fields_ = [("file", C.c_int32), ("elem_bytes", C.c_int32), ("ndim", C.c_int32),
                ("shape", C.c_int64 * 8), ("offset", C.c_uint64), ("bytes", C.c_uint64)]


class EvictStats(C.Structure):
    _fields_ = [("kept_sessions", C.c_int32), ("evicted_sessions", C.c_int32),
                ("live_before", C.c_int64), ("live_after", C.c_int64),
                ("demand_before", C.c_uint64), ("demand_after", C.c_uint64)]


class LoadStats(C.Structure):
    _fields_ = [("read_ms", C.c_double), ("bytes", C.c_uint64), ("reads", C.c_uint64),
                ("tensor_bytes", C.c_uint64), ("threads", C.c_int32)]


def hip_runtimes():
    """Distinct libamdhip64 files mapped into this process."""
    try:
        with open("/proc/self/maps") as f:
            return sorted({line.split()[-1] for line in f if "libamdhip64" in line})
    except OSError:
        return []


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with `python -m paper_2511_11617_amd.build`")
    # torch ships its own HIP runtime under the same soname as the system's.
    # Mapping torch's first makes this library bind to it; the other order
    # leaves two runtimes in the process, and this library's calls would then
    # act on streams and memory that the other runtime created.
    try:
        import torch  # noqa: F401
    except ImportError:
        pass
    lib = C.CDLL(LIB_PATH)
    runtimes = hip_runtimes()
    if len(runtimes) > 1:
        raise ImportError("two HIP runtimes are mapped in this process: " + ", ".join(runtimes))
    P = C.c_void_p
    lib.atp_plan.argtypes = [C.POINTER(Problem), C.POINTER(P)]
    lib.atp_plan_free.argtypes = [P]
    lib.atp_plan_free.restype = None
    lib.atp_reshard_weights.argtypes = [P, P, C.c_uint64, P, C.c_uint64, P, C.c_uint64, P, C.c_uint64,
                                        P, C.c_uint64, P, P]
    lib.atp_reshard_kv.argtypes = [P, P, C.c_uint64, P, C.c_uint64, P, C.c_int32, C.c_int32, P,
                                   C.c_uint64, P, C.c_uint64, P, C.c_uint64, P, P]
    lib.atp_reshard_kv_noalloc.argtypes = [P, P, C.c_uint64, P, C.c_uint64, P, C.c_int32, C.c_int32, P,
                                           C.c_uint64, P, C.c_uint64, P, P]
    lib.atp_scratch_bytes.argtypes = []
    lib.atp_scratch_bytes.restype = C.c_uint64
    lib.atp_sync.argtypes = [P, C.POINTER(Timing)]
    lib.atp_warmup.argtypes = [P, P, C.c_int32]
    lib.atp_plan_stats.argtypes = [P, C.POINTER(Stats)]
    lib.atp_plan_tasks.argtypes = [P, C.c_int32, C.POINTER(Task), C.c_int32, C.POINTER(C.c_int32)]
    lib.atp_plan_ranges.argtypes = [P, C.c_int32, C.POINTER(Range), C.c_int32, C.POINTER(C.c_int32)]
    lib.atp_plan_old_ranges.argtypes = [P, C.c_int32, C.POINTER(Range), C.c_int32, C.POINTER(C.c_int32)]
    lib.atp_plan_owner.argtypes = [P, C.POINTER(C.c_int32), C.c_int32, C.POINTER(C.c_int32)]
    lib.atp_plan_layout.argtypes = [P, C.c_int32, C.POINTER(C.c_uint64), C.POINTER(C.c_uint64),
                                    C.POINTER(C.c_uint64)]
    lib.atp_plan_segments.argtypes = [P, C.c_int32, C.POINTER(Segment), C.c_int32, C.POINTER(C.c_int32)]
    lib.atp_plan_launches.argtypes = [P, C.POINTER(Launch), C.c_int32, C.POINTER(C.c_int32)]
    lib.atp_partition.argtypes = [C.c_int64, C.c_int32, C.c_int32, C.POINTER(Range)]
    lib.atp_st_open.argtypes = [C.POINTER(C.c_char_p), C.c_int32, C.POINTER(P)]
    lib.atp_st_close.argtypes = [P]
    lib.atp_st_close.restype = None
    lib.atp_st_find.argtypes = [P, C.c_char_p, C.POINTER(StTensor)]
    lib.atp_load_weights.argtypes = [P, P, C.POINTER(C.c_char_p), C.c_int32, P, C.c_uint64, C.c_int32,
                                     C.POINTER(LoadStats)]
    lib.atp_load_reshard_weights.argtypes = [P, P, C.POINTER(C.c_char_p), C.c_int32, P, C.c_uint64, P,
                                             C.c_uint64, P, C.c_uint64, P, C.c_uint64, P, C.c_uint64, P, P,
                                             C.c_int32, C.POINTER(LoadStats)]
    lib.atp_load_reshard_weights_async.argtypes = [P, P, C.POINTER(C.c_char_p), C.c_int32, P, C.c_uint64, P,
                                                   C.c_uint64, P, C.c_uint64, P, C.c_uint64, P, C.c_uint64, P, P,
                                                   C.c_int32]
    lib.atp_plan_load_stats.argtypes = [P, C.POINTER(LoadStats)]
    lib.atp_kv_evict_lru.argtypes = [P, C.c_int32, C.c_int32, C.c_int64, P, C.c_uint64, C.c_uint64, C.c_int32,
                                     P, P, C.POINTER(EvictStats)]
    lib.atp_daemon_serve.argtypes = [C.c_char_p, C.c_int32]
    lib.atp_state_connect.argtypes = [C.c_char_p, C.POINTER(P)]
    lib.atp_state_disconnect.argtypes = [P]
    lib.atp_state_disconnect.restype = None
    lib.atp_state_alloc.argtypes = [P, C.c_char_p, C.c_uint64, C.POINTER(P)]
    lib.atp_state_open.argtypes = [P, C.c_char_p, C.POINTER(P), C.POINTER(C.c_uint64)]
    lib.atp_state_release.argtypes = [P, P]
    lib.atp_state_free.argtypes = [P, C.c_char_p]
    lib.atp_state_put.argtypes = [P, C.c_char_p, P, C.c_uint64]
    lib.atp_state_get.argtypes = [P, C.c_char_p, P, C.c_uint64, C.POINTER(C.c_uint64)]
    lib.atp_state_list.argtypes = [P, C.c_char_p, C.c_uint64, C.POINTER(C.c_uint64)]
    lib.atp_state_shutdown.argtypes = [P]
    lib.atp_last_error.restype = C.c_char_p
    for f in EXPORTS:
        if f not in ("atp_plan_free", "atp_last_error", "atp_st_close", "atp_state_disconnect"):
            getattr(lib, f).restype = C.c_int
    return lib


lib = _load()


class AtpError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"atp error {code}: {msg}")
        self.code = code


def _check(rc):
    if rc != OK:
        raise AtpError(rc, lib.atp_last_error().decode())
    return rc


def scratch_bytes() -> int:
    """Size of the no-allocation entry point's device scratch array."""
    return int(lib.atp_scratch_bytes())


def partition(total: int, parts: int, rule: int):
    out = (Range * parts)()
    _check(lib.atp_partition(total, parts, rule, out))
    return [(r.begin, r.end) for r in out]


def _list(fn, plan, typ, *args):
    n = C.c_int32()
    _check(fn(plan, *args, None, 0, C.byref(n)))
    arr = (typ * max(n.value, 1))()
    _check(fn(plan, *args, arr, n.value, C.byref(n)))
    return list(arr[:n.value])


def warmup(compute: int, copy: int, events: int = 256) -> None:
    """atp_warmup on the current device: the first reshard's one-time set-up
    (kernels loaded, side stream chosen for these raw stream handles, pooled
    events and pinned buffers) done ahead of time."""
    _check(lib.atp_warmup(compute, copy, events))


class Plan:
    """An atp_plan_t and the ctypes objects its problem points into."""

    def __init__(self, problem: Problem, keep=()):
        self._keep = keep  # arrays referenced by `problem`
        h = C.c_void_p()
        _check(lib.atp_plan(C.byref(problem), C.byref(h)))
        self.h = h

    def close(self):
        if self.h:
            lib.atp_plan_free(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def stats(self) -> Stats:
        s = Stats()
        _check(lib.atp_plan_stats(self.h, C.byref(s)))
        return s

    def tasks(self, space: int):
        return [(t.kind, t.begin, t.end, t.src, t.dst, t.host)
                for t in _list(lib.atp_plan_tasks, self.h, Task, space)]

    def ranges(self, space: int):
        return [(r.begin, r.end) for r in _list(lib.atp_plan_ranges, self.h, Range, space)]

    def old_ranges(self, space: int):
        return [(r.begin, r.end) for r in _list(lib.atp_plan_old_ranges, self.h, Range, space)]

    def owner(self):
        return [int(x) for x in _list(lib.atp_plan_owner, self.h, C.c_int32)]

    def layout(self, t: int):
        o, n, b = C.c_uint64(), C.c_uint64(), C.c_uint64()
        _check(lib.atp_plan_layout(self.h, t, C.byref(o), C.byref(n), C.byref(b)))
        return o.value, n.value, b.value

    def segments(self, which: int):
        return _list(lib.atp_plan_segments, self.h, Segment, which)

    def launches(self):
        return _list(lib.atp_plan_launches, self.h, Launch)

    def reshard_weights(self, arena, arena_bytes, new_arena, new_bytes, inflow, inflow_bytes,
                        outbound, outbound_bytes, staging, staging_bytes, compute, copy):
        _check(lib.atp_reshard_weights(self.h, arena, arena_bytes, new_arena, new_bytes, inflow,
                                       inflow_bytes, outbound, outbound_bytes, staging,
                                       staging_bytes, compute, copy))

    def reshard_kv_noalloc(self, arena, arena_bytes, new_arena, new_bytes, table, n_seq, max_blocks,
                           inflow, inflow_bytes, outbound, outbound_bytes, compute, copy):
        _check(lib.atp_reshard_kv_noalloc(self.h, arena, arena_bytes, new_arena, new_bytes, table, n_seq,
                                          max_blocks, inflow, inflow_bytes, outbound, outbound_bytes,
                                          compute, copy))

    def reshard_kv(self, arena, arena_bytes, new_arena, new_bytes, table, n_seq, max_blocks,
                   inflow, inflow_bytes, outbound, outbound_bytes, staging, staging_bytes,
                   compute, copy):
        _check(lib.atp_reshard_kv(self.h, arena, arena_bytes, new_arena, new_bytes, table, n_seq,
                                  max_blocks, inflow, inflow_bytes, outbound, outbound_bytes,
                                  staging, staging_bytes, compute, copy))

    def sync(self) -> Timing:
        t = Timing()
        _check(lib.atp_sync(self.h, C.byref(t)))
        return t

    def load_weights(self, files: "StFiles", names, inflow, inflow_bytes, threads=0) -> LoadStats:
        """Fill the weight inflow buffer at address `inflow` from `files`."""
        arr = (C.c_char_p * len(names))(*[n.encode() for n in names])
        st = LoadStats()
        _check(lib.atp_load_weights(self.h, files.h, arr, len(names), inflow, inflow_bytes, threads,
                                    C.byref(st)))
        return st

    def load_reshard_weights(self, files: "StFiles", names, arena, arena_bytes, new_arena, new_bytes, inflow,
                             inflow_bytes, outbound, outbound_bytes, staging, staging_bytes, compute, copy,
                             threads=0) -> LoadStats:
        """Range-read the weight inflow from `files` into the pinned buffer at
        `inflow` while the weights reshard is enqueued behind the reads."""
        arr = (C.c_char_p * len(names))(*[n.encode() for n in names])
        st = LoadStats()
        _check(lib.atp_load_reshard_weights(self.h, files.h, arr, len(names), arena, arena_bytes, new_arena,
                                            new_bytes, inflow, inflow_bytes, outbound, outbound_bytes, staging,
                                            staging_bytes, compute, copy, threads, C.byref(st)))
        return st

    def load_reshard_weights_async(self, files: "StFiles", names, arena, arena_bytes, new_arena, new_bytes, inflow,
                                   inflow_bytes, outbound, outbound_bytes, staging, staging_bytes, compute, copy,
                                   threads=0) -> None:
        """The same reload, returning before the reads are done: the inflow
        pieces are issued by sync(); `files`, the names and every buffer stay
        valid until then (the ctypes array of names is kept here)."""
        self._names = (C.c_char_p * len(names))(*[n.encode() for n in names])
        self._files = files
        _check(lib.atp_load_reshard_weights_async(self.h, files.h, self._names, len(names), arena, arena_bytes,
                                                  new_arena, new_bytes, inflow, inflow_bytes, outbound,
                                                  outbound_bytes, staging, staging_bytes, compute, copy, threads))

    def load_stats(self) -> LoadStats:
        st = LoadStats()
        _check(lib.atp_plan_load_stats(self.h, C.byref(st)))
        return st


def kv_evict_lru(table, last_use, num_blocks: int, block_bytes: int, budget_bytes: int, compact=False):
    """LRU session eviction under a KV budget (atp_kv_evict_lru).
    table: int32 [n_seq, max_blocks]; last_use: int64 [n_seq].
    Returns (keep bool array, new table, EvictStats)."""
    import numpy as np
    t = np.ascontiguousarray(table, dtype=np.int32)
    lu = np.ascontiguousarray(last_use, dtype=np.int64)
    if lu.shape != (t.shape[0],):
        raise ValueError("last_use needs one entry per session")
    keep = np.zeros(t.shape[0], np.int32)
    out = np.empty_like(t)
    st = EvictStats()
    _check(lib.atp_kv_evict_lru(t.ctypes.data, t.shape[0], t.shape[1], num_blocks, lu.ctypes.data, block_bytes,
                                budget_bytes, int(bool(compact)), keep.ctypes.data, out.ctypes.data,
                                C.byref(st)))
    return keep.astype(bool), out, st


class StFiles:
    """Opened safetensors files (atp_st_open)."""

    def __init__(self, paths):
        arr = (C.c_char_p * len(paths))(*[os.fsencode(p) for p in paths])
        h = C.c_void_p()
        _check(lib.atp_st_open(arr, len(paths), C.byref(h)))
        self.h = h

    def find(self, name: str):
        t = StTensor()
        _check(lib.atp_st_find(self.h, name.encode(), C.byref(t)))
        return t.file, t.elem_bytes, tuple(t.shape[:t.ndim]), t.offset, t.bytes

    def close(self):
        if self.h:
            lib.atp_st_close(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
