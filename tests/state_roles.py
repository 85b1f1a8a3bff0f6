"""Roles of the state-plane GPU tests, run as separate processes (test
infrastructure).

    python tests/state_roles.py writer --socket S --case NAME

`writer` stands in for the inference process that held the old shard: it
asks the daemon for the weight and KV regions (sized for the old and the
new layout, as the state plane provisions them), writes the old arenas the
oracle defines into them, leaves the block table and the per-session last
use with the daemon, and then dies without any cleanup (os._exit).
"""
from __future__ import annotations

import argparse
import ctypes as C
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

from oracle import model, repack  # noqa: E402
from paper_2511_11617_amd import atp, problem, state  # noqa: E402
from synth import configs, pagetable  # noqa: E402
from synth.content import Content  # noqa: E402

H2D, D2H = 1, 2


def case(name: str):
    if name == "tiny":
        return configs.get(1)
    if name == "dense80-2l":
        return configs.scaled(5, layers=2, n_seq=2, seq_tokens=256)
    if name == "dense40-2l":
        return configs.scaled(2, layers=2, n_seq=2, seq_tokens=256, inplace=True)
    raise ValueError(name)


def hip():
    h = C.CDLL("libamdhip64.so")  # torch's runtime, already mapped by the imports above
    h.hipMemcpy.argtypes = [C.c_void_p, C.c_void_p, C.c_size_t, C.c_int]
    h.hipMemcpy.restype = C.c_int
    h.hipDeviceSynchronize.restype = C.c_int
    return h


def copy(h, dst, src, n, kind):
    if n:
        rc = h.hipMemcpy(dst, src, n, kind)
        if rc != 0:
            raise RuntimeError(f"hipMemcpy failed with {rc}")


def region_sizes(c):
    """(weights, kv) region bytes: room for the old and the new layout."""
    table, pool = pagetable.make_for(c)
    n_live = int(len(np.unique(table[table >= 0])))
    st = problem.build(c, n_live=n_live, pool=pool, flags=atp.INPLACE, staging_cap=c["staging_cap"] or 0).plan().stats()
    return (max(st.old_arena_bytes, st.new_arena_bytes, 256), max(st.old_kv_bytes, st.new_kv_bytes, 256))


def writer(sock: str, name: str) -> None:
    c = case(name)
    pb = model.build(c)
    content = Content(c["seed"], c["w_kind"], c["kv_kind"])
    table, pool = pagetable.make_for(c)
    old_w = repack.weight_arena(pb, content, "old")
    old_k = repack.kv_arena(pb, content, table, pool, "old", poison=0xDEAD)
    wb, kb = region_sizes(c)
    assert old_w.size <= wb and old_k.size <= kb
    cl = state.Client(sock)
    pw = cl.alloc("weights", wb)
    pk = cl.alloc("kv", kb)
    h = hip()
    copy(h, pw, old_w.ctypes.data, old_w.size, H2D)
    copy(h, pk, old_k.ctypes.data, old_k.size, H2D)
    if h.hipDeviceSynchronize() != 0:
        raise RuntimeError("hipDeviceSynchronize failed")
    cl.put("kv.table", table.astype(np.int32))
    cl.put("kv.last_use", np.random.default_rng(c["seed"] + 1).permutation(table.shape[0]).astype(np.int64))
    cl.put("case", name.encode())
    print(f"[writer] {name}: weights {old_w.size} B, kv {old_k.size} B written; exiting without cleanup",
          flush=True)
    os._exit(3)


if __name__ == "__main__":
    ap = argparse.ArgumentParser()
    ap.add_argument("role", choices=["writer"])
    ap.add_argument("--socket", required=True)
    ap.add_argument("--case", required=True)
    a = ap.parse_args()
    writer(a.socket, a.case)
