"""Benchmark of one surviving GPU's share of a TP reshard on MI355X.

A step is the whole hot path once: plan (partitions, CMM tasks, layouts,
descriptors), repack the retained weight slices and paged-KV head ranges,
land the missing bytes from pinned host memory on a side stream, sync.
Inputs are synthetic (seeded generator), resident in HBM and pinned host
memory before the timed region.

  python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload N]

The default workload is the largest: the dense 80-layer hidden-8192
decoder, TP 8 -> 7, resharded in place under a 2 GB staging cap (about
106 GB of HBM, 57 GB of inflow).  Prints one JSON line.  `value` is the repack throughput in algorithmic
bytes (one read and one write of every retained byte that moves) per
second of device repack time (the union of the repack kernels' intervals:
the weights and KV repacks may overlap); `ms_per_step` is the wall time
of a whole step, which the PCIe-bound inflow dominates.
"""
from __future__ import annotations

import argparse
import gc
import json
import os
import sys
import time

import numpy as np

HBM_PEAK_GBPS = 8000.0  # MI355X HBM3E, vendor figure

# HBM bytes of the dominant repack launch (the one that moves the most
# bytes) per workload, measured with the FETCH_SIZE and WRITE_SIZE counters
# (rocprofv3, one pass each, scaled by what the same counters read for a
# plain 4 GiB device copy: x2.0 and x1.0), keyed by call and the launch's
# algorithmic bytes; valid only while the kernel sources hash to `src`.
COUNTED_TRAFFIC = {
    "src": "98de88c3866af8ac",
    "dense-40L-h5120-tp4to3": {("kv", 10737418240): 10738045781, ("weights", 9043968000): 9069669589},
    "dense-40L-h5120-tp8to7-fragmented-kv": {("kv", 21474836480): 21477139966},
    "dense-80L-h8192-tp8to7-inplace": {("kv", 43083890688): 43088211671, ("weights", 3829399552): 3829563243},
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
    ap.add_argument("--workload", type=int, default=5,
                    help="1..5; 5 = dense 80L h8192 TP 8->7 in place under a 2 GB staging cap (the "
                         "largest workload, the default)")
    ap.add_argument("--plan", choices=["cm", "greedy", "full"], default="cm",
                    help="planner: CMM (Alg. 1) or the Greedy / Full Reload baselines of Sec. V")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--kv-budget", type=float, default=None,
                    help="KV budget as a fraction of the new layout's live KV demand: sessions (seeded "
                         "recency) are evicted least recently used first (atp_kv_evict_lru); out of "
                         "place the kept blocks land in a compact arena (ATP_KV_COMPACT)")
    ap.add_argument("--load", action="store_true",
                    help="also time the range-read reload source on a checkpoint written for this "
                         "workload: the reads alone (atp_load_weights), and reads and reshard pipelined "
                         "(atp_load_reshard_weights)")
    ap.add_argument("--cpu-seconds", type=float, default=8.0,
                    help="repeat each CPU oracle timing (one thread, then a thread pool) over its layer "
                         "sample for at least this long")
    ap.add_argument("--cpu-threads", type=int, default=0,
                    help="threads of the pooled CPU oracle timing (default: the host's CPUs, at most 16)")
    ap.add_argument("--calib-copy-gib", type=float, default=0.0,
                    help="also run a plain device copy of this size (counter calibration)")
    ap.add_argument("--self-old", type=int, default=None,
                    help="measure this surviving old rank's share instead of the workload's named one")
    ap.add_argument("--inplace", action="store_true",
                    help="reshard the workload in place (the new shard over the old one), whatever it states")
    ap.add_argument("--state", action="store_true",
                    help="run the workload in place on memory the state plane holds: a writer process "
                         "allocates one weight and one KV region per layer group through the daemon and "
                         "exits; this process maps them (timed) and reshards every group")
    ap.add_argument("--state-groups", type=int, default=0,
                    help="layer groups of the state leg (default: the fewest whose regions fit)")
    ap.add_argument("--state-window", type=int, default=0,
                    help="groups of the state leg pending at once, each with staging and host buffers of "
                         "its own (default 1: one group after another, the faster order in place)")
    ap.add_argument("--state-writer", default=None, help=argparse.SUPPRESS)
    ap.add_argument("--state-regions", default="", help=argparse.SUPPRESS)
    return ap.parse_args()


def main():
    args = parse()
    if args.state_writer:
        return state_writer(args)
    if args.gpus != 1:
        print(json.dumps({"error": "this benchmark measures one GPU's share of the reshard; "
                                   "run it with --gpus 1 (multi-GPU runs are not part of it)"}))
        sys.exit(2)
    import torch

    from paper_2511_11617_amd import atp, problem
    from synth import configs, fill, pagetable
    from synth.content import TAGS, Content
    from synth.pinned import Pageable, Pinned, host_buffers

    if args.state:
        return state_main(args)
    over = {}
    if args.inplace:
        over["inplace"] = True
    if args.self_old is not None:
        over["self_old"] = args.self_old
    cfg = configs.get(args.workload, **over)
    if not 0 <= cfg["self_old"] < cfg["old_tp"] or cfg["self_old"] in cfg["failed"]:
        raise SystemExit(f"old rank {cfg['self_old']} is not a survivor of workload {args.workload}")
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
    # which survivor hosts which new rank: the paper's in-order choice against
    # the permutation that keeps the most bytes (host planning only)
    assignment = {}
    for nm, fl in (("inorder", atp.ASSIGN_INORDER), ("maxretain", atp.ASSIGN_MAXRETAIN)):
        try:
            a = problem.build(cfg, n_live=n_live, pool=pool, flags=(flags & ~atp.ASSIGN_MAXRETAIN) | fl,
                              staging_cap=cap).plan().stats()
            assignment[nm] = {"self_new_rank": int(a.self_new_rank),
                              "self_inflow_bytes": int(a.inflow_w + a.inflow_kv),
                              "self_retained_bytes": int(a.retained_w + a.retained_kv),
                              "global_retained_bytes": int(a.global_keep),
                              "global_reload_bytes": int(a.global_reload)}
        except atp.AtpError as e:
            assignment[nm] = {"error": str(e)}
    if args.plan != "full":  # a full reload lands the whole shard whatever it holds
        by_target = inflow_by_target(cfg, built, plan, cfg["self_old"])
        if by_target[st.self_new_rank] == st.inflow_w + st.inflow_kv:  # the plan's own inflow
            assignment["self_inflow_by_target_bytes"] = by_target
            assignment["self_inflow_min_bytes"] = min(by_target)
            assignment["critical_path"] = critical_path(cfg, n_live, pool, flags, cap)
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

    # host buffers first (pinning fails more often than device allocation);
    # in place the KV inflow lands by DMA only and may be pageable memory
    (hin_w, hin_k, hout_w, hout_k), pageable_bytes = host_buffers(
        [(st.inflow_w, None, False), (st.inflow_kv, None, inplace),
         (st.outbound_w if inplace else 1, None, False), (st.outbound_kv if inplace else 1, None, False)])
    if pageable_bytes:
        log(f"[bench] the host cannot pin every buffer: {pageable_bytes / 1e9:.1f} GB of KV inflow "
            "(DMA only) in pageable memory")
    aw, nw = arena(st.old_arena_bytes, st.new_arena_bytes)
    ak, nk = arena(st.old_kv_bytes, st.new_kv_bytes)
    stage_w = torch.empty(max(st.staging_w, 256), dtype=u8, device=dev)
    stage_k = torch.empty(max(st.staging_kv, 256), dtype=u8, device=dev)
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
    ptr = lambda t: None if t is None else (t.ptr if isinstance(t, (Pinned, Pageable)) else t.data_ptr())

    issue = []  # host time spent enqueuing each call (ms)
    # the first reshard's one-time set-up, done ahead of it (a recovering
    # process would do it before the failure is known)
    torch.cuda.synchronize()
    t0s = time.perf_counter()
    atp.warmup(compute.cuda_stream, copy.cuda_stream, 256)
    setup_ms = (time.perf_counter() - t0s) * 1e3

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

    first_ms = None
    for i in range(args.warmup):
        if inplace and i:
            fill_old()
        torch.cuda.synchronize()
        t0w = time.perf_counter()
        step()
        torch.cuda.synchronize()
        if i == 0:  # the process's first reshard (after atp_warmup)
            first_ms = (time.perf_counter() - t0w) * 1e3
        log(f"[bench] warmup {i + 1}/{args.warmup} done")
    recs, launches = [], []
    elapsed = 0.0
    gc.collect()
    gc.disable()  # a collector pause is no part of the reshard (one took 45 ms in a step)
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

    gc.enable()

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
    dk, db, dom_ms, dom_gbps, kernels = dominant_launch(launches)
    traffic = None
    counted = COUNTED_TRAFFIC.get(cfg["name"])
    if counted and args.plan == "cm" and not args.inplace and args.kv_budget is None \
            and kernel_src_hash() == COUNTED_TRAFFIC["src"]:
        traffic = counted.get(("weights" if dk == 0 else "kv", 2 * db))

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
        "setup_ms": round(setup_ms, 3),
        "first_step_ms": round(first_ms, 3) if first_ms is not None else None,
        "plan_ms": round(sum(t.plan_ms for t in recs) / K, 3),
        "issue_ms": [round(sum(x[0] for x in issue[-K:]) / K, 3), round(sum(x[1] for x in issue[-K:]) / K, 3)],
        "h2d_GBps_pcie_inclusive": round((st.inflow_w + st.inflow_kv) / (h2d_ms * 1e-3) / 1e9, 2)
        if h2d_ms else None,
        "h2d_standalone_GBps": round(h2d_peak, 2),
        "host_pageable_bytes": int(pageable_bytes),
        "wall_vs_h2d_bound": round((st.inflow_w + st.inflow_kv) / (h2d_peak * 1e9) * 1e3 / wall_ms, 3)
        if h2d_peak else None,
        "overlap": round(sum(t.overlap for t in recs) / K, 3),
        "scatter_ms": round(sum(t.scatter_ms for t in recs) / K, 4),
        "scatter_bytes": int(recs[-1].scatter_bytes),  # landing ring -> place, not algorithmic
        "assignment": assignment,
        "retained_bytes": int(st.retained_w + st.retained_kv),
        "moved_bytes": int(st.moved_w + st.moved_kv),
        # in place: hazard levels of the two calls, bytes routed through
        # staging (cycle breakers and the level chain's tail) and the tail alone
        "levels": [int(st.n_levels_w), int(st.n_levels_kv)],
        "staged_bytes": int(st.staged_w + st.staged_kv),
        "tail_bytes": int(st.tail_w + st.tail_kv),
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
        def pipelined_step(files, names, buf, deferred=False):
            """One step whose weight inflow is read from the checkpoint while the
            weights reshard runs behind the reads (atp_load_reshard_weights).
            `deferred`: atp_load_reshard_weights_async, then the KV call while
            the reads run, and atp_sync issues the weight pieces."""
            if inplace:
                fill_old()
            p = built.plan()
            torch.cuda.synchronize()
            t1 = time.perf_counter()

            def kv():
                p.reshard_kv(ptr(ak), ak.numel(), ptr(nk), nk.numel() if nk is not None else 0,
                             ptr(table_d), table.shape[0], table.shape[1], ptr(hin_k), st.inflow_kv,
                             ptr(hout_k), st.outbound_kv if inplace else 0, ptr(stage_k), stage_k.numel(),
                             compute.cuda_stream, copy.cuda_stream)
            w_args = (ptr(aw), aw.numel(), ptr(nw), nw.numel() if nw is not None else 0, buf.ptr, st.inflow_w,
                      ptr(hout_w), st.outbound_w if inplace else 0, ptr(stage_w), stage_w.numel(),
                      compute.cuda_stream, copy.cuda_stream)
            if deferred:
                p.load_reshard_weights_async(files, names, *w_args)
                kv()
            else:
                if not inplace:  # out of place the KV inflow can use the link while the weights are read
                    kv()
                p.load_reshard_weights(files, names, *w_args)
                if inplace:  # in place the weights call comes first
                    kv()
            p.sync()
            torch.cuda.synchronize()
            return (time.perf_counter() - t1) * 1e3

        out["load"] = load_leg(args.steps, cfg, plan, st, tl, hin_w, Pinned, pipelined_step, wall_ms)
    if not args.no_cpu_baseline and evict is None:  # the oracle's leg runs the by-id layout
        if inplace:
            fill_old()
            torch.cuda.synchronize()
        out["cpu_baseline"] = cpu_baseline(cfg, args.cpu_seconds, args.cpu_threads, aw, ak, hin_w.tensor,
                                           hin_k.tensor, table, pool)
    print(json.dumps(out), flush=True)


def inflow_by_target(cfg, built, plan, self_old):
    """Bytes this survivor would land if it hosted each new target: the
    target's units it does not hold, in every tensor and in the KV cache
    (library ranges and shapes only)."""
    from paper_2511_11617_amd import atp
    eb = cfg["elem_bytes"]
    out = []
    for j in range(cfg["new_tp"]):
        def miss(sp):
            nb, ne = plan.ranges(sp)[j]
            ob, oe = built.old_ranges[sp][self_old]
            return (ne - nb) - max(0, min(ne, oe) - max(nb, ob))
        tot = sum(miss(sp) * unit * (cols if kind == atp.ROWS else rows) * eb
                  for (name, l, kind, sp, rows, cols, unit) in built.tensors)
        tot += miss(1) * built.n_live * cfg["block_tokens"] * cfg["head_dim"] * eb * 2 * cfg["layers"]
        out.append(int(tot))
    return out


def critical_path(cfg, n_live, pool, flags, cap):
    """Every survivor's inflow by target: the largest under the in-order
    assignment (the recovery ends with that survivor) against the smallest
    largest over all M! assignments (host planning only)."""
    import itertools

    from paper_2511_11617_amd import problem
    surv = [r for r in range(cfg["old_tp"]) if r not in cfg["failed"]]
    A = []
    for so in surv:
        c = dict(cfg, self_old=so)
        b = problem.build(c, n_live=n_live, pool=pool, flags=flags, staging_cap=cap)
        A.append(inflow_by_target(c, b, b.plan(), so))
    M = len(A[0])
    inorder = max(A[i][i] for i in range(M))
    best = min(max(A[i][p[i]] for i in range(M)) for p in itertools.permutations(range(M))) if M <= 8 else None
    return {"inorder_max_inflow_bytes": inorder, "best_max_inflow_bytes": best,
            "critical_old_rank": surv[max(range(M), key=lambda i: A[i][i])]}


def dominant_launch(launches):
    """The repack launch that moves the most bytes, averaged over the steps:
    (call kind, bytes moved, ms, algorithmic GB/s, table of the launches)."""
    per = {}
    for L in launches:
        for kind, level, b, ms in L:
            if kind in (0, 1):
                per.setdefault((kind, level, b), []).append(ms)
    (dk, dl, db), dms = max(per.items(), key=lambda kv: kv[0][2]) if per else ((0, 0, 0), [0.0])
    dom_ms = sum(dms) / len(dms)
    dom_gbps = 2 * db / (dom_ms * 1e-3) / 1e9 if dom_ms > 0 else 0.0
    # the eight launches that move the most bytes, in call and level order
    top = sorted(sorted(per.items(), key=lambda kv: -kv[0][2])[:8])
    kernels = [{"call": "weights" if k == 0 else "kv",
                "level": l, "alg_bytes": 2 * b, "avg_ms": round(sum(v) / len(v), 4),
                "GBps": round(2 * b / (sum(v) / len(v) * 1e-3) / 1e9, 1)}
               for (k, l, b), v in top]
    return dk, db, dom_ms, dom_gbps, kernels


def state_writer(args):
    """The process that held the old shard: asks the daemon for the regions,
    leaves the block table with it, and exits without any cleanup.  The
    regions' bytes are what the allocation left there: moving bytes costs
    the same whatever they are (the state-plane tests check content)."""
    from paper_2511_11617_amd import state
    from synth import configs, pagetable

    cl = state.Client(args.state_writer)
    for item in args.state_regions.split(","):
        name, n = item.split(":")
        cl.alloc(name, int(n))
    table, _ = pagetable.make_for(configs.get(args.workload))
    cl.put("kv.table", table.astype(np.int32))
    cl.put("kv.shape", np.array(table.shape, np.int64))
    log(f"[writer] {len(args.state_regions.split(','))} regions allocated; exiting without cleanup")
    os._exit(3)


def state_main(args):
    """The workload in place on device memory the state plane owns
    (Sec. III-A).  IPC regions stay under 2 GiB, so the layers are split into
    the fewest balanced groups whose weight and KV regions fit; every layer
    group is a reshard of its own (layers are independent in the plan) with
    a fresh plan each, one after another.  `--state-window W` keeps up to W
    groups pending at once, each on staging and host buffers of its own; in
    place that is slower: every group's weights chain (outbound reads,
    levels, inflow read by the copy kernel) runs in turn on the one side
    stream, while the later groups' KV inflow takes the link from it.
    Timed: the attach (connect, open every region, fetch the block table)
    once, and every step."""
    import subprocess
    import tempfile

    import torch

    from paper_2511_11617_amd import atp, problem, state
    from synth import configs, pagetable
    from synth.pinned import Pinned

    cfg = configs.get(args.workload, inplace=True)
    table, pool = pagetable.make_for(cfg)
    n_live = int(len(np.unique(table[table >= 0])))
    cap = cfg["staging_cap"] or 0
    L = cfg["layers"]
    built, stats = {}, {}

    def sizes(layers):
        if layers not in built:
            built[layers] = problem.build(dict(cfg, layers=layers), n_live=n_live, pool=pool,
                                          flags=atp.INPLACE, staging_cap=cap)
            st = built[layers].plan().stats()
            stats[layers] = st
        st = stats[layers]
        return max(st.old_arena_bytes, st.new_arena_bytes, 256), max(st.old_kv_bytes, st.new_kv_bytes, 256)

    def split(n):
        return [L // n + (i < L % n) for i in range(n)]

    def fits(n):
        return all(max(sizes(g)) <= state.MAX_REGION for g in set(split(n)))

    if args.state_groups:
        n_groups = args.state_groups
        if not 1 <= n_groups <= L or not fits(n_groups):
            raise SystemExit(f"{n_groups} layer groups do not give regions under {state.MAX_REGION} bytes")
    else:
        n_groups = next((n for n in range(1, L + 1) if fits(n)), 0)
        if not n_groups:
            raise SystemExit("one layer's arena exceeds the state plane's region limit")
    groups = split(n_groups)
    window = min(args.state_window or 1, n_groups)
    if window < 1:
        raise SystemExit("--state-window must be at least 1")
    regions = []
    for i, g in enumerate(groups):
        wb, kb = sizes(g)
        regions += [(f"w{i}", wb), (f"k{i}", kb)]
    log(f"[state] workload {args.workload} {cfg['name']} in place: {n_groups} layer groups {groups}, "
        f"{len(regions)} regions, {sum(n for _, n in regions) / 1e9:.2f} GB, {window} pending at once")

    dev = torch.device("cuda")
    u8 = torch.uint8
    sts = [stats[g] for g in set(groups)]
    # one set of staging and host buffers per pending group, reused by the
    # groups that follow it (what the inflow bytes are does not change the cost)
    slots = []
    for _ in range(window):
        slots.append(dict(
            stage_w=torch.empty(max(max(s.staging_w for s in sts), 256), dtype=u8, device=dev),
            stage_k=torch.empty(max(max(s.staging_kv for s in sts), 256), dtype=u8, device=dev),
            hin_w=Pinned(max(s.inflow_w for s in sts)), hin_k=Pinned(max(s.inflow_kv for s in sts)),
            hout_w=Pinned(max(s.outbound_w for s in sts)), hout_k=Pinned(max(s.outbound_kv for s in sts))))
    torch.cuda.synchronize()

    d = tempfile.mkdtemp(prefix="atp-", dir="/tmp")
    sock = os.path.join(d, "s.sock")
    daemon = state.spawn(sock)
    cl = None
    try:
        r = subprocess.run([sys.executable, os.path.abspath(__file__), "--state-writer", sock,
                            "--workload", str(args.workload),
                            "--state-regions", ",".join(f"{n}:{b}" for n, b in regions)],
                           capture_output=True, text=True, timeout=600)
        if r.returncode != 3:
            raise RuntimeError(f"state writer failed ({r.returncode}): {r.stderr[-2000:]}")
        t0 = time.perf_counter()
        cl = state.Client(sock)
        mapped = [(cl.open(f"w{i}"), cl.open(f"k{i}")) for i in range(n_groups)]
        shape = tuple(int(x) for x in cl.get_array("kv.shape", np.int64))
        tab = cl.get_array("kv.table", np.int32, shape)
        attach_ms = (time.perf_counter() - t0) * 1e3
        if not np.array_equal(tab, table):
            raise RuntimeError("the block table the daemon returned differs from the workload's")
        for (pw, wb), (pk, kb) in mapped:
            if pw % 256 or pk % 256:
                raise RuntimeError("a mapped region is not 256-byte aligned")
        log(f"[state] attach: {attach_ms:.2f} ms for {len(regions)} regions and the block table")
        table_d = torch.from_numpy(tab).to(dev)
        compute = torch.cuda.current_stream()
        copy = torch.cuda.Stream()
        torch.cuda.synchronize()
        t0s = time.perf_counter()
        atp.warmup(compute.cuda_stream, copy.cuda_stream, 256)
        setup_ms = (time.perf_counter() - t0s) * 1e3

        def step():
            plans, recs = [], [None] * n_groups

            def finish(j):
                p = plans[j]
                recs[j] = (p.sync(), [(x.kind, x.level, x.bytes, x.ms) for x in p.launches()])
                plans[j] = None

            for i, g in enumerate(groups):
                if i >= window:
                    finish(i - window)  # its buffers serve this group
                st, b = stats[g], slots[i % window]
                (pw, wb), (pk, kb) = mapped[i]
                p = built[g].plan()
                p.reshard_weights(pw, wb, None, 0, b["hin_w"].ptr, st.inflow_w, b["hout_w"].ptr, st.outbound_w,
                                  b["stage_w"].data_ptr(), b["stage_w"].numel(), compute.cuda_stream,
                                  copy.cuda_stream)
                p.reshard_kv(pk, kb, None, 0, table_d.data_ptr(), shape[0], shape[1], b["hin_k"].ptr,
                             st.inflow_kv, b["hout_k"].ptr, st.outbound_kv, b["stage_k"].data_ptr(),
                             b["stage_k"].numel(), compute.cuda_stream, copy.cuda_stream)
                plans.append(p)
            for j in range(max(0, n_groups - window), n_groups):
                finish(j)
            return recs

        first_ms = None
        for i in range(args.warmup):
            torch.cuda.synchronize()
            t0w = time.perf_counter()
            step()
            torch.cuda.synchronize()
            if i == 0:  # the first reshard after the attach and atp_warmup
                first_ms = (time.perf_counter() - t0w) * 1e3
            log(f"[state] warmup {i + 1}/{args.warmup} done")
        steps, elapsed = [], 0.0
        gc.collect()
        gc.disable()  # a collector pause is no part of the reshard
        for i in range(args.steps):
            torch.cuda.synchronize()
            t1 = time.perf_counter()
            recs = step()
            torch.cuda.synchronize()
            elapsed += time.perf_counter() - t1
            steps.append(recs)
            log(f"[state] step {i + 1}/{args.steps}: walls " +
                " ".join(f"{t.wall_ms:.1f}" for t, _ in recs) + " ms, repack " +
                f"{sum(t.repack_union_ms for t, _ in recs):.3f} ms")
        gc.enable()
        for ptr_w, ptr_k in mapped:
            cl.release(ptr_w[0])
            cl.release(ptr_k[0])
        for n, _ in regions:
            cl.free(n)
    finally:
        try:
            c = cl or state.Client(sock)
            c.shutdown()
            c.close()
        except atp.AtpError:
            pass
        try:
            daemon.wait(timeout=60)
        except subprocess.TimeoutExpired:
            daemon.kill()
            daemon.wait()
        if os.path.isdir(d) and not os.listdir(d):
            os.rmdir(d)

    K = args.steps
    moved = sum(stats[g].moved_w + stats[g].moved_kv for g in groups)
    inflow = sum(stats[g].inflow_w + stats[g].inflow_kv for g in groups)
    rep_ms = sum(sum(t.repack_union_ms for t, _ in recs) for recs in steps) / K
    wall_ms = elapsed / K * 1e3
    value = 2 * moved / (rep_ms * 1e-3) / 1e9 if rep_ms > 0 else 0.0
    dk, db, dom_ms, dom_gbps, kernels = dominant_launch([L_ for recs in steps for _, L_ in recs])
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
        "config": {"workload": cfg["name"] + " in place on state-plane regions", "layers": L,
                   "hidden": cfg["hidden"], "tp": f"{cfg['old_tp']}->{cfg['new_tp']}", "failed": cfg["failed"],
                   "self_old_rank": cfg["self_old"], "kv_sequences": cfg["n_seq"],
                   "seq_tokens": cfg["seq_tokens"], "in_place": True, "planner": "cm"},
        "state": {"layer_groups": groups, "pending_at_once": window, "regions": len(regions),
                  "region_bytes": [b for _, b in regions], "region_limit": state.MAX_REGION,
                  "attach_ms": round(attach_ms, 3),
                  "setup_ms": round(setup_ms, 3),
                  "first_step_ms": round(first_ms, 3) if first_ms is not None else None,
                  "writer": "separate process; allocated through the daemon and exited without cleanup"},
        "hbm_frac": round(value / HBM_PEAK_GBPS, 4),
        "repack_ms": round(rep_ms, 4),
        "wall_ms": round(wall_ms, 3),
        "group_wall_ms": [round(sum(recs[i][0].wall_ms for recs in steps) / K, 3) for i in range(n_groups)],
        "plan_ms": round(sum(sum(t.plan_ms for t, _ in recs) for recs in steps) / K, 3),
        "h2d_ms": round(sum(sum(t.h2d_ms for t, _ in recs) for recs in steps) / K, 3),
        "moved_bytes": int(moved),
        "inflow_bytes": int(inflow),
        "kernels": kernels,
        "roofline": {"bound": "hbm", "achieved": round(dom_gbps, 1), "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s", "frac": round(dom_gbps / HBM_PEAK_GBPS, 4), "traffic": None,
                     "kernel": "k_copy16", "call": "weights" if dk == 0 else "kv",
                     "alg_bytes_per_launch": int(2 * db), "avg_launch_ms": round(dom_ms, 4)},
    }
    print(json.dumps(out), flush=True)


def load_leg(steps, cfg, plan, st, tl, hin_w, Pinned, pipelined_step, step_ms):
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
        # reads and reshard together: the file reads overlap the landings;
        # then the same with the reads behind the asynchronous call
        pipe, defer = [], []
        gc.collect()
        gc.disable()
        for deferred, acc in ((False, pipe), (True, defer)):
            for i in range(steps + 1):  # the first pass is a warm-up
                buf.tensor.fill_(0xA5)
                w = pipelined_step(files, names, buf, deferred)
                if i:
                    acc.append(w)
                log(f"[bench] reads + reshard {'async' if deferred else 'pipelined'}: {w:.1f} ms")
            if not np.array_equal(buf.tensor.numpy(), src):
                raise RuntimeError("pipelined range reads returned other bytes than the checkpoint holds")
        gc.enable()
        files.close()
        buf.close()
    finally:
        shutil.rmtree(d, ignore_errors=True)
    read_ms = sum(ms) / len(ms)
    pipe_ms = sum(pipe) / len(pipe)
    defer_ms = sum(defer) / len(defer)
    return {"source": f"safetensors range reads, file in {where[0]} (page cache)", "bytes": int(st.inflow_w),
            "tensor_bytes": int(ls.tensor_bytes), "read_fraction": round(st.inflow_w / ls.tensor_bytes, 4),
            "reads": int(ls.reads), "threads": int(ls.threads), "read_ms": round(read_ms, 3),
            "GBps": round(st.inflow_w / (read_ms * 1e-3) / 1e9, 2), "file_bytes": int(total),
            "write_s": round(write_s, 2),
            "sequential_ms": round(read_ms + step_ms, 3),  # reads, then the step from pinned memory
            "pipelined_ms": round(pipe_ms, 3),  # reads and reshard together, whole step
            "async_ms": round(defer_ms, 3)}  # the same behind atp_load_reshard_weights_async, KV call between


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


def cpu_baseline(cfg, seconds, threads, aw, ak, hin_w, hin_k, table, pool):
    """The oracle's plan execution (old shard + packed inflow -> new shard,
    host to host) on a sample of the workload's layers.

    Every layer has the same plan, and the weight arena, the KV planes and
    both packed inflow buffers are layer-major, so the buffers of the first
    n layers are those of the same decoder with n layers.  Timed twice over
    the same sample: the oracle on one thread (one call for the weights, one
    for the KV cache), then a pool of threads, one task per (layer, weights or
    KV) on the one-layer problem.  NumPy releases the GIL in its copies."""
    from concurrent.futures import ThreadPoolExecutor

    from oracle import model, repack

    threads = threads or min(os.cpu_count() or 1, 16)
    L = cfg["layers"]
    n = min(L, max(threads, 4))
    n_live = len(repack.live_blocks(table))
    pb1 = model.build(dict(cfg, layers=1))
    pbn = model.build(dict(cfg, layers=n))
    w_stride, kv_stride = pb1.layout("old")[1], pb1.kv_arena_bytes("old", pool)
    win1 = sum(s[-1] for s in repack.inflow_segments(pb1, n_live)[0])
    kin1 = sum(s[-1] for s in repack.inflow_segments(pb1, n_live)[1])
    old_w = aw[:n * w_stride].cpu().numpy()
    old_k = ak[:n * kv_stride].cpu().numpy()
    in_w = hin_w.numpy()[:n * win1]
    in_k = hin_k.numpy()[:n * kin1]
    ret1, inf1, _ = repack.self_bytes(pb1, n_live)
    alg = 2 * ret1 * n

    def timed(one_pass):
        passes, t0 = 0, time.perf_counter()
        while passes < 8 and (passes == 0 or time.perf_counter() - t0 < seconds):
            one_pass()
            passes += 1
        return (time.perf_counter() - t0) / passes, passes

    def serial():
        repack.apply_weights(pbn, old_w, in_w)
        repack.apply_kv(pbn, old_k, in_k, table, pool)

    tasks = [(l, part) for l in range(n) for part in ("weights", "kv")]

    def one(task):
        l, part = task
        if part == "weights":
            repack.apply_weights(pb1, old_w[l * w_stride:(l + 1) * w_stride], in_w[l * win1:(l + 1) * win1])
        else:
            repack.apply_kv(pb1, old_k[l * kv_stride:(l + 1) * kv_stride], in_k[l * kin1:(l + 1) * kin1],
                            table, pool)

    dt1, p1 = timed(serial)
    with ThreadPoolExecutor(threads) as ex:
        dtn, pn = timed(lambda: list(ex.map(one, tasks)))
    sample = (f"{n} of {L} layers (weights + KV: {alg / 1e9:.2f} GB algorithmic repack + "
              f"{inf1 * n / 1e9:.2f} GB inflow placed), host to host")
    return {"value": round(alg / dtn / 1e9, 3), "unit": "GB/s", "cores": threads, "threads": threads,
            "kind": "oracle", "host_cpus": os.cpu_count(),
            "sample": sample + f"; {threads} threads over (layer, weights|KV), {pn} passes of {dtn:.2f} s",
            "single_thread": {"value": round(alg / dt1 / 1e9, 3), "unit": "GB/s", "cores": 1,
                              "passes": p1, "s_per_pass": round(dt1, 3)},
            "threaded_s_per_pass": round(dtn, 3)}


if __name__ == "__main__":
    main()
