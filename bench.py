"""Benchmark of one surviving GPU's share of a TP reshard on MI355X.

A step is the whole hot path once: plan (partitions, CMM tasks, layouts,
descriptors), repack the retained weight slices and paged-KV head ranges,
land the missing bytes from pinned host memory on a side stream, sync.
Inputs are synthetic (seeded generator), resident in HBM and pinned host
memory before the timed region.

  python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload N]

Prints one JSON line.  `value` is the repack throughput in algorithmic
bytes (one read and one write of every retained byte that moves) per
second of device repack time (the union of the repack kernels' intervals:
the weights and KV repacks may overlap); `ms_per_step` is the wall time
of a whole step, which the PCIe-bound inflow dominates.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

HBM_PEAK_GBPS = 8000.0  # MI355X HBM3E, vendor figure

# HBM bytes per launch of the repack kernel measured with the FETCH_SIZE and
# WRITE_SIZE counters (rocprofv3, one pass each, scaled by what the same
# counters read for a plain 4 GiB copy: x2.0 and x1.0), valid only while the
# kernel sources hash to `src`.
COUNTED_TRAFFIC = {
    "src": "d9999845543f9207",
    "dense-40L-h5120-tp4to3": {"kv": 10738045781, "weights": 9069669589},
}


def kernel_src_hash():
    import hashlib
    d = os.path.join(os.path.dirname(os.path.abspath(__file__)), "paper_2511_11617_amd", "csrc")
    inner = ""
    for f in ("kernels.h", "desc.h"):
        inner += hashlib.sha256(open(os.path.join(d, f), "rb").read()).hexdigest() + "  " + \
            os.path.join("paper_2511_11617_amd", "csrc", f) + "\n"
    return hashlib.sha256(inner.encode()).hexdigest()[:16]


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", type=int, default=2,
                    help="1..5; 2 = dense 40L h5120 TP 4->3 (the headline workload)")
    ap.add_argument("--plan", choices=["cm", "greedy", "full"], default="cm",
                    help="planner: CMM (Alg. 1) or the Greedy / Full Reload baselines of Sec. V")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--kv-budget", type=float, default=None,
                    help="KV budget as a fraction of the new layout's live KV demand: sessions (seeded "
                         "recency) are evicted least recently used first (atp_kv_evict_lru); out of "
                         "place the kept blocks land in a compact arena (ATP_KV_COMPACT)")
    ap.add_argument("--load", action="store_true",
                    help="also time the range-read reload source (atp_load_weights) on a checkpoint "
                         "written for this workload")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="repeat the CPU oracle over the whole workload for at least this long")
    ap.add_argument("--calib-copy-gib", type=float, default=0.0,
                    help="also run a plain device copy of this size (counter calibration)")
    return ap.parse_args()


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "this benchmark measures one GPU's share of the reshard; "
                                   "run it with --gpus 1 (multi-GPU runs are not part of it)"}))
        sys.exit(2)
    import torch

    from paper_2511_11617_amd import atp, problem
    from synth import configs, fill, pagetable
    from synth.content import TAGS, Content
    from synth.pinned import Pinned

    cfg = configs.get(args.workload)
    table, pool = pagetable.make_for(cfg)
    n_live = int(len(np.unique(table[table >= 0])))
    inplace = bool(cfg["inplace"])
    flags = (atp.INPLACE if inplace else 0) | {"cm": 0, "greedy": atp.PLAN_GREEDY,
                                               "full": atp.PLAN_FULL}[args.plan]
    cap = cfg["staging_cap"] or 0
    full_table, evict = table, None
    if args.kv_budget is not None:
        pre = problem.build(cfg, n_live=n_live, pool=pool, flags=flags, staging_cap=cap).plan().stats()
        bb = pre.new_kv_bytes // pool
        last_use = np.random.default_rng(cfg["seed"] + 1).permutation(table.shape[0])
        budget = int(args.kv_budget * n_live * bb)
        keep, table, est = atp.kv_evict_lru(full_table, last_use, pool, bb, budget)
        n_live = int(est.live_after)
        if not inplace:
            flags |= atp.KV_COMPACT
        evict = {"budget_bytes": budget, "block_bytes": int(bb), "kept_sessions": int(est.kept_sessions),
                 "evicted_sessions": int(est.evicted_sessions), "live_before": int(est.live_before),
                 "live_after": int(est.live_after), "demand_before": int(est.demand_before),
                 "demand_after": int(est.demand_after), "compact": bool(flags & atp.KV_COMPACT)}
        log(f"[bench] KV budget {args.kv_budget}: kept {est.kept_sessions} of {table.shape[0]} sessions, "
            f"{est.live_after} of {est.live_before} blocks")
    built = problem.build(cfg, n_live=n_live, pool=pool, flags=flags, staging_cap=cap)
    plan = built.plan()
    st = plan.stats()
    dev = torch.device("cuda")
    u8 = torch.uint8
    content = Content(cfg["seed"], cfg["w_kind"], cfg["kv_kind"])
    self_old = cfg["self_old"]
    layout = atp.KV_TOKEN_MAJOR if cfg.get("kv_layout") == "token" else atp.KV_HEAD_MAJOR
    bt, hd = cfg["block_tokens"], cfg["head_dim"]
    log(f"[bench] workload {args.workload} {cfg['name']}: R_w={st.retained_w / 1e9:.3f} GB "
        f"R_kv={st.retained_kv / 1e9:.3f} GB I={(st.inflow_w + st.inflow_kv) / 1e9:.3f} GB "
        f"levels={st.n_levels_w}/{st.n_levels_kv} inplace={inplace}")

    # ---- buffers ---------------------------------------------------------------
    def arena(old_b, new_b):
        if inplace:
            return torch.empty(max(old_b, new_b, 256), dtype=u8, device=dev), None
        return (torch.empty(max(old_b, 256), dtype=u8, device=dev),
                torch.empty(max(new_b, 256), dtype=u8, device=dev))

    aw, nw = arena(st.old_arena_bytes, st.new_arena_bytes)
    ak, nk = arena(st.old_kv_bytes, st.new_kv_bytes)
    stage_w = torch.empty(max(st.staging_w, 256), dtype=u8, device=dev)
    stage_k = torch.empty(max(st.staging_kv, 256), dtype=u8, device=dev)
    hin_w, hin_k = Pinned(st.inflow_w), Pinned(st.inflow_kv)
    hout_w = Pinned(st.outbound_w if inplace else 1)
    hout_k = Pinned(st.outbound_kv if inplace else 1)
    table_d = torch.from_numpy(table).to(dev)

    # ---- synthetic content -----------------------------------------------------
    t0 = time.time()
    tl = built.tensors
    old_r = built.old_ranges

    def fill_old():
        shards = []
        for i, (name, l, kind, sp, rows, cols, unit) in enumerate(tl):
            a, b = old_r[sp][self_old]
            shards.append((TAGS[name], l, kind == atp.ROWS, rows, cols, unit, a, b, plan.layout(i)[0]))
        fill.weights(aw, content, shards)
        fill.kv_arena(ak, content, full_table, pool, cfg["layers"], old_r[1][self_old], cfg["n_kv"],
                      cfg["seq_tokens"], bt, hd, layout)

    fill_old()
    tmp = torch.empty(max(st.inflow_w, st.inflow_kv, 1), dtype=u8, device=dev)
    shards = []
    for s in plan.segments(atp.SEG_INFLOW_W):
        name, l, kind, sp, rows, cols, unit = tl[s.tensor]
        shards.append((TAGS[name], l, kind == atp.ROWS, rows, cols, unit, s.unit_begin, s.unit_end,
                       s.host_offset))
    fill.weights(tmp, content, shards)
    hin_w.tensor.copy_(tmp[:hin_w.nbytes])
    segs = [(s.layer, s.which, s.unit_begin, s.unit_end, s.host_offset)
            for s in plan.segments(atp.SEG_INFLOW_KV)]
    fill.kv_packed(tmp, content, table, pool, segs, cfg["n_kv"], cfg["seq_tokens"], bt, hd, layout)
    hin_k.tensor.copy_(tmp[:hin_k.nbytes])
    del tmp
    torch.cuda.synchronize()
    log(f"[bench] inputs generated in {time.time() - t0:.1f} s")

    compute = torch.cuda.current_stream()
    copy = torch.cuda.Stream()
    h2d_peak = h2d_probe(torch, [hin_w, hin_k], max(st.inflow_w, st.inflow_kv), copy)
    log(f"[bench] standalone H2D of the inflow buffers: {h2d_peak:.1f} GB/s")
    ptr = lambda t: None if t is None else (t.ptr if isinstance(t, Pinned) else t.data_ptr())

    issue = []  # host time spent enqueuing each call (ms)

    def step():
        p = built.plan()
        i0 = time.perf_counter()
        p.reshard_weights(ptr(aw), aw.numel(), ptr(nw), nw.numel() if nw is not None else 0,
                          ptr(hin_w), st.inflow_w, ptr(hout_w), st.outbound_w if inplace else 0,
                          ptr(stage_w), stage_w.numel(), compute.cuda_stream, copy.cuda_stream)
        i1 = time.perf_counter()
        p.reshard_kv(ptr(ak), ak.numel(), ptr(nk), nk.numel() if nk is not None else 0,
                     ptr(table_d), table.shape[0], table.shape[1], ptr(hin_k), st.inflow_kv,
                     ptr(hout_k), st.outbound_kv if inplace else 0, ptr(stage_k), stage_k.numel(),
                     compute.cuda_stream, copy.cuda_stream)
        i2 = time.perf_counter()
        issue.append(((i1 - i0) * 1e3, (i2 - i1) * 1e3))
        t = p.sync()
        return p, t

    for i in range(args.warmup):
        if inplace and i:
            fill_old()
        step()
        log(f"[bench] warmup {i + 1}/{args.warmup} done")
    recs, launches = [], []
    elapsed = 0.0
    for i in range(args.steps):
        if inplace:
            fill_old()  # restore the old layout (untimed)
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        p, t = step()
        torch.cuda.synchronize()
        elapsed += time.perf_counter() - t1
        recs.append(t)
        launches.append([(x.kind, x.level, x.bytes, x.ms) for x in p.launches()])
        log(f"[bench] step {i + 1}/{args.steps}: wall {t.wall_ms:.1f} ms, repack "
            f"{t.repack_union_ms:.3f} ms, h2d {t.h2d_ms:.1f} ms, d2h {t.d2h_ms:.1f} ms, "
            f"issue {issue[-1][0]:.1f} + {issue[-1][1]:.1f} ms")

    if args.calib_copy_gib > 0:
        n = int(args.calib_copy_gib * (1 << 30))
        src = torch.empty(n, dtype=u8, device=dev)
        dst = torch.empty(n, dtype=u8, device=dev)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    K = args.steps
    alg = 2 * (st.moved_w + st.moved_kv)
    # device repack time: the union of the repack kernels' intervals (the
    # weights and KV repacks may overlap in time)
    rep_ms = sum(t.repack_union_ms for t in recs) / K
    rep_sum_ms = sum(t.repack_w_ms + t.repack_kv_ms for t in recs) / K
    span_ms = sum(t.repack_span_ms for t in recs) / K
    value = alg / (rep_ms * 1e-3) / 1e9 if rep_ms > 0 else 0.0  # Full Reload keeps nothing
    wall_ms = elapsed / K * 1e3
    h2d_ms = sum(t.h2d_ms for t in recs) / K
    # dominant kernel: the repack launch moving the most bytes
    per = {}
    for L in launches:
        for kind, level, b, ms in L:
            if kind in (0, 1):
                per.setdefault((kind, level, b), []).append(ms)
    (dk, dl, db), dms = max(per.items(), key=lambda kv: kv[0][2]) if per else ((0, 0, 0), [0.0])
    traffic = None
    counted = COUNTED_TRAFFIC.get(cfg["name"])
    if counted and args.plan == "cm" and kernel_src_hash() == COUNTED_TRAFFIC["src"]:
        traffic = counted.get("weights" if dk == 0 else "kv")
    dom_ms = sum(dms) / len(dms)
    dom_gbps = 2 * db / (dom_ms * 1e-3) / 1e9 if dom_ms > 0 else 0.0
    kernels = [{"call": "weights" if k == 0 else "kv",
                "level": l, "alg_bytes": 2 * b, "avg_ms": round(sum(v) / len(v), 4),
                "GBps": round(2 * b / (sum(v) / len(v) * 1e-3) / 1e9, 1)}
               for (k, l, b), v in sorted(per.items())][:8]

    out = {
        "metric": "reshard GB/s (fraction of HBM peak) + wall ms per TP k→k-1; reload bytes vs min",
        "value": round(value, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": round(wall_ms, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u8",
        "data": "synthetic",
        "config": {"workload": cfg["name"], "layers": cfg["layers"], "hidden": cfg["hidden"],
                   "tp": f"{cfg['old_tp']}->{cfg['new_tp']}", "failed": cfg["failed"],
                   "self_old_rank": self_old, "self_new_rank": st.self_new_rank,
                   "kv_sequences": cfg["n_seq"], "seq_tokens": cfg["seq_tokens"],
                   "in_place": inplace, "elem": "fp16" if cfg["w_kind"] == 1 else "bf16",
                   "planner": args.plan, "kv_budget": args.kv_budget},
        "hbm_frac": round(value / HBM_PEAK_GBPS, 4),
        "repack_ms": round(rep_ms, 4),
        "repack_sum_ms": round(rep_sum_ms, 4),
        "repack_span_ms": round(span_ms, 4),
        "wall_ms": round(wall_ms, 3),
        "plan_ms": round(sum(t.plan_ms for t in recs) / K, 3),
        "issue_ms": [round(sum(x[0] for x in issue[-K:]) / K, 3), round(sum(x[1] for x in issue[-K:]) / K, 3)],
        "h2d_GBps_pcie_inclusive": round((st.inflow_w + st.inflow_kv) / (h2d_ms * 1e-3) / 1e9, 2)
        if h2d_ms else None,
        "h2d_standalone_GBps": round(h2d_peak, 2),
        "wall_vs_h2d_bound": round((st.inflow_w + st.inflow_kv) / (h2d_peak * 1e9) * 1e3 / wall_ms, 3)
        if h2d_peak else None,
        "overlap": round(sum(t.overlap for t in recs) / K, 3),
        "retained_bytes": int(st.retained_w + st.retained_kv),
        "moved_bytes": int(st.moved_w + st.moved_kv),
        "inflow_bytes": int(st.inflow_w + st.inflow_kv),
        "reload_bytes": int(st.global_reload),
        "reload_min_bytes": int(st.reload_min),
        "kernels": kernels,
        "roofline": {"bound": "hbm", "achieved": round(dom_gbps, 1), "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s", "frac": round(dom_gbps / HBM_PEAK_GBPS, 4), "traffic": traffic,
                     "kernel": "k_copy16", "call": "weights" if dk == 0 else "kv",
                     "alg_bytes_per_launch": int(2 * db), "avg_launch_ms": round(dom_ms, 4)},
    }
    if evict is not None:
        out["kv_evict"] = evict
    if args.load:
        out["load"] = load_leg(args.steps, cfg, plan, st, tl, hin_w, Pinned)
    if not args.no_cpu_baseline and evict is None:  # the oracle's leg runs the by-id layout
        if inplace:
            fill_old()
            torch.cuda.synchronize()
        out["cpu_baseline"] = cpu_baseline(cfg, args.cpu_seconds, aw, ak, hin_w.tensor, hin_k.tensor,
                                           table, pool)
    print(json.dumps(out), flush=True)


def load_leg(steps, cfg, plan, st, tl, hin_w, Pinned):
    """Range-read reload source (atp_load_weights).  The checkpoint has the
    headers of every full weight tensor; as data it holds the intervals this
    plan reads, taken from the synthetic inflow, and holes elsewhere (the full
    model would not fit the scratch disk).  The reads hit a warm page cache."""
    import shutil
    import tempfile

    from paper_2511_11617_amd import atp
    from synth import checkpoint

    if st.inflow_w == 0:
        return {"skipped": "this plan reads no weights"}
    tens = [(n, l, rows, cols) for (n, l, k, sp, rows, cols, u) in tl]
    names = [checkpoint.name(n, l) for (n, l, *_) in tl]
    src = hin_w.tensor.numpy()
    regions = []
    for s in plan.segments(atp.SEG_INFLOW_W):
        n, l, kind, sp, rows, cols, unit = tl[s.tensor]
        a, b = s.unit_begin * unit, s.unit_end * unit
        w = src[s.host_offset:s.host_offset + s.bytes].view(np.uint16)
        if kind == atp.ROWS:
            regions.append((n, l, cols, a, b, 0, cols, w.reshape(b - a, cols)))
        else:
            regions.append((n, l, cols, 0, rows, a, b, w.reshape(rows, b - a)))
    # strided tensors are written whole over the rows they span: allow 3x
    # the read bytes; a memory-backed directory first (no writeback throttle)
    need = 3 * st.inflow_w + (2 << 30)
    where = [x for x in ("/dev/shm", tempfile.gettempdir())
             if os.path.isdir(x) and os.access(x, os.W_OK) and shutil.disk_usage(x).free >= need]
    if not where:
        return {"skipped": f"no scratch directory with {need / 1e9:.1f} GB free"}
    d = tempfile.mkdtemp(prefix="atp_ckpt_", dir=where[0])
    try:
        path = os.path.join(d, "model.safetensors")
        t0 = time.time()
        total = checkpoint.write_stream(path, tens, regions, "fp16" if cfg["w_kind"] == 1 else "bf16")
        write_s = time.time() - t0
        log(f"[bench] checkpoint written in {write_s:.1f} s ({total / 1e9:.1f} GB logical)")
        files = atp.StFiles([path])
        buf = Pinned(st.inflow_w, fill=0xA5)
        ms = []
        for i in range(steps + 1):  # the first pass is a warm-up
            ls = plan.load_weights(files, names, buf.ptr, st.inflow_w)
            if i:
                ms.append(ls.read_ms)
        if not np.array_equal(buf.tensor.numpy(), src):
            raise RuntimeError("range reads returned other bytes than the checkpoint holds")
        files.close()
        buf.close()
    finally:
        shutil.rmtree(d, ignore_errors=True)
    read_ms = sum(ms) / len(ms)
    return {"source": f"safetensors range reads, file in {where[0]} (page cache)", "bytes": int(st.inflow_w),
            "tensor_bytes": int(ls.tensor_bytes), "read_fraction": round(st.inflow_w / ls.tensor_bytes, 4),
            "reads": int(ls.reads), "threads": int(ls.threads), "read_ms": round(read_ms, 3),
            "GBps": round(st.inflow_w / (read_ms * 1e-3) / 1e9, 2), "file_bytes": int(total),
            "write_s": round(write_s, 2)}


def h2d_probe(torch, bufs, max_bytes, stream, chunk=64 << 20):
    """Standalone pinned-host -> device copy rate of the inflow buffers
    (the PCIe ceiling of this run's wall time), GB/s."""
    import ctypes as C
    hip = C.CDLL("libamdhip64.so")
    hip.hipMemcpyAsync.argtypes = [C.c_void_p, C.c_void_p, C.c_size_t, C.c_int, C.c_void_p]
    hip.hipMemcpyAsync.restype = C.c_int
    tot = sum(b.nbytes for b in bufs)
    if tot <= 16:
        return 0.0
    dst = torch.empty(max(max_bytes, 1), dtype=torch.uint8, device="cuda")
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for b in bufs:
        for off in range(0, b.nbytes, chunk):
            n = min(chunk, b.nbytes - off)
            rc = hip.hipMemcpyAsync(C.c_void_p(dst.data_ptr() + off), C.c_void_p(b.ptr + off), n, 1,
                                    C.c_void_p(stream.cuda_stream))
            if rc:
                raise RuntimeError(f"hipMemcpyAsync failed: {rc}")
    e1.record(stream)
    e1.synchronize()
    ms = e0.elapsed_time(e1)
    del dst
    return tot / (ms * 1e-3) / 1e9


def cpu_baseline(cfg, seconds, aw, ak, hin_w, hin_k, table, pool):
    """The oracle's plan execution (old shard + packed inflow -> new shard,
    numpy slicing on one host thread) over the whole workload, repeated
    until `seconds` have passed (at most 8 passes)."""
    from oracle import model, repack

    pb = model.build(cfg)
    _, o_size = pb.layout("old")
    kv_old = pb.kv_arena_bytes("old", pool)
    n_live = len(repack.live_blocks(table))
    old_w = aw[:o_size].cpu().numpy()
    old_k = ak[:kv_old].cpu().numpy()
    ret, inf, _ = repack.self_bytes(pb, n_live)
    in_w = hin_w.numpy()[:sum(s[-1] for s in repack.inflow_segments(pb, n_live)[0])]
    in_k = hin_k.numpy()[:sum(s[-1] for s in repack.inflow_segments(pb, n_live)[1])]
    passes, t0 = 0, time.perf_counter()
    while passes < 8 and (passes == 0 or time.perf_counter() - t0 < seconds):
        repack.apply_weights(pb, old_w, in_w)
        repack.apply_kv(pb, old_k, in_k, table, pool)
        passes += 1
    dt = (time.perf_counter() - t0) / passes
    return {"value": round(2 * ret / dt / 1e9, 3), "unit": "GB/s", "cores": 1, "kind": "oracle",
            "sample": f"whole workload ({cfg['layers']} layers, weights + KV, "
                      f"{2 * ret / 1e9:.2f} GB algorithmic repack + {inf / 1e9:.2f} GB inflow placed), "
                      f"{passes} passes, {dt:.2f} s per pass, numpy on one thread"}


if __name__ == "__main__":
    main()
