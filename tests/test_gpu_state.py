"""State plane on the GPU (Sec. III-A): the memory of the weights and the KV
cache outlives the inference process that used it, and a fresh process
reshards it in place.

* A writer process allocates a region through the daemon, fills it and dies
  without cleanup; a new process maps the region and reads the same bytes.
* Crash and recover: the writer process (tests/state_roles.py) holds the
  old shards of a TP 4->3 / 8->7 survivor in daemon-owned regions and dies;
  this process maps them, takes the block table from the daemon, runs the
  in-place reshard on the mapped memory and compares every live byte (and
  the outbound buffer) with the oracle.  With a KV budget, the recency the
  writer left with the daemon picks the sessions to keep.
"""
import ctypes as C
import os
import subprocess
import sys
import tempfile
import time

import numpy as np
import pytest
import torch

from oracle import kvbudget, model, repack
from paper_2511_11617_amd import atp, problem, state
from synth import pagetable
from synth.content import Content
from tests import state_roles
from tests.gpu_harness import say

pytestmark = pytest.mark.gpu
ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


@pytest.fixture(scope="module")
def daemon():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    d = tempfile.mkdtemp(prefix="atp-", dir="/tmp")
    path = os.path.join(d, "s.sock")
    say(f"[state] daemon on {path}")
    p = state.spawn(path)
    yield path
    if p.poll() is None:
        try:
            c = state.Client(path)
            c.shutdown()
            c.close()
        except atp.AtpError:
            pass
        try:
            p.wait(timeout=60)
        except subprocess.TimeoutExpired:
            p.kill()
            p.wait()


WRITE_AND_DIE = r"""
import ctypes as C, os, sys
sys.path.insert(0, {root!r})
import numpy as np
from paper_2511_11617_amd import state
from tests import state_roles
c = state.Client({path!r})
p = c.alloc("r", {n})
data = (np.arange({n}, dtype=np.uint64) * 2654435761 % 251).astype(np.uint8)
h = state_roles.hip()
state_roles.copy(h, p, data.ctypes.data, data.size, state_roles.H2D)
assert h.hipDeviceSynchronize() == 0
os._exit(3)
"""


def test_region_outlives_its_writer(daemon):
    n = 64 << 20
    say("[state] writer process")
    r = subprocess.run([sys.executable, "-c", WRITE_AND_DIE.format(root=ROOT, path=daemon, n=n)],
                       capture_output=True, text=True, timeout=300)
    assert r.returncode == 3, r.stderr
    c = state.Client(daemon)
    ptr, size = c.open("r")
    assert size == n and ptr % 256 == 0
    got = np.empty(n, np.uint8)
    h = state_roles.hip()
    state_roles.copy(h, got.ctypes.data, ptr, n, state_roles.D2H)
    want = (np.arange(n, dtype=np.uint64) * 2654435761 % 251).astype(np.uint8)
    np.testing.assert_array_equal(got, want)
    c.release(ptr)
    c.free("r")
    assert "region r " not in c.list()
    c.close()


def _pinned(arr):
    t = torch.empty(max(arr.size, 1), dtype=torch.uint8, pin_memory=True)
    if arr.size:
        t[:arr.size].copy_(torch.from_numpy(arr))
    return t


@pytest.mark.parametrize("name,budget", [("tiny", None), ("dense40-2l", None), ("dense80-2l", None),
                                         ("dense80-2l", 0.5)])
def test_crash_and_recover_in_place(daemon, name, budget):
    say(f"[state] {name}: writer process holds the old shard, then dies")
    r = subprocess.run([sys.executable, os.path.join(ROOT, "tests", "state_roles.py"), "writer", "--socket", daemon,
                        "--case", name], capture_output=True, text=True, timeout=600)
    assert r.returncode == 3, r.stdout + r.stderr

    # ---- the new process: map the surviving state ------------------------------------
    t0 = time.perf_counter()
    cl = state.Client(daemon)
    pw, wb = cl.open("weights")
    pk, kb = cl.open("kv")
    table = cl.get_array("kv.table", np.int32)
    last_use = cl.get_array("kv.last_use", np.int64)
    attach_ms = (time.perf_counter() - t0) * 1e3
    assert cl.get("case") == name.encode()

    c = state_roles.case(name)
    full_table, pool = pagetable.make_for(c)
    table = table.reshape(full_table.shape)
    np.testing.assert_array_equal(table, full_table)
    pb = model.build(c)
    content = Content(c["seed"], c["w_kind"], c["kv_kind"])
    if budget is not None:  # the recency the state plane kept picks the sessions
        bb = pb.kv_arena_bytes("new", pool) // pool
        keep = kvbudget.lru_keep(full_table, last_use, bb, int(budget * len(repack.live_blocks(full_table)) * bb))
        keep_lib, table_lib, _ = atp.kv_evict_lru(full_table, last_use, pool, bb,
                                                  int(budget * len(repack.live_blocks(full_table)) * bb))
        np.testing.assert_array_equal(np.asarray(keep_lib, bool), np.asarray(keep, bool))
        table = kvbudget.evicted_table(full_table, keep, compact=False)
    n_live = int(len(repack.live_blocks(table)))
    plan = problem.build(c, n_live=n_live, pool=pool, flags=atp.INPLACE, staging_cap=c["staging_cap"] or 0).plan()
    st = plan.stats()
    assert max(st.old_arena_bytes, st.new_arena_bytes) <= wb and max(st.old_kv_bytes, st.new_kv_bytes) <= kb

    want_w = repack.weight_arena(pb, content, "new")
    mask_w = repack.weight_live_mask(pb, "new")
    want_k = repack.kv_arena(pb, content, table, pool, "new")
    mask_k = repack.kv_live_mask(pb, table, pool, "new")
    hin_w = _pinned(repack.packed_weight_inflow(pb, content))
    hin_k = _pinned(repack.packed_kv_inflow(pb, content, table, pool))
    hout_w = torch.full((max(st.outbound_w, 1),), 0x3C, dtype=torch.uint8, pin_memory=True)
    hout_k = torch.full((max(st.outbound_kv, 1),), 0x3C, dtype=torch.uint8, pin_memory=True)
    dev = torch.device("cuda")
    stage_w = torch.empty(max(st.staging_w, 256), dtype=torch.uint8, device=dev)
    stage_k = torch.empty(max(st.staging_kv, 256), dtype=torch.uint8, device=dev)
    table_d = torch.from_numpy(table).to(dev)
    compute, copy = torch.cuda.current_stream(), torch.cuda.Stream()
    torch.cuda.synchronize()
    plan.reshard_weights(pw, wb, None, 0, hin_w.data_ptr(), st.inflow_w, hout_w.data_ptr(), st.outbound_w,
                         stage_w.data_ptr(), stage_w.numel(), compute.cuda_stream, copy.cuda_stream)
    plan.reshard_kv(pk, kb, None, 0, table_d.data_ptr(), table.shape[0], table.shape[1], hin_k.data_ptr(),
                    st.inflow_kv, hout_k.data_ptr(), st.outbound_kv, stage_k.data_ptr(), stage_k.numel(),
                    compute.cuda_stream, copy.cuda_stream)
    t = plan.sync()
    torch.cuda.synchronize()
    say(f"[state] {name} budget={budget}: attach {attach_ms:.2f} ms, reshard wall {t.wall_ms:.2f} ms")

    h = state_roles.hip()
    got_w = np.empty(want_w.size, np.uint8)
    got_k = np.empty(want_k.size, np.uint8)
    state_roles.copy(h, got_w.ctypes.data, pw, want_w.size, state_roles.D2H)
    state_roles.copy(h, got_k.ctypes.data, pk, want_k.size, state_roles.D2H)
    assert not np.flatnonzero(got_w[mask_w] != want_w[mask_w]).size
    assert not np.flatnonzero(got_k[mask_k] != want_k[mask_k]).size
    ow = repack.packed_weight_outbound(pb, content)
    ok = repack.packed_kv_outbound(pb, content, table, pool)
    np.testing.assert_array_equal(hout_w.numpy()[:ow.size], ow)
    np.testing.assert_array_equal(hout_k.numpy()[:ok.size], ok)
    plan.close()
    cl.free("weights")  # the daemon is shared by the tests of this module
    cl.free("kv")
    cl.close()
