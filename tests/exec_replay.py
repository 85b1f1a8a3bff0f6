"""Child process of tests/test_exec_replay.py: runs reshards through
libatp.so with the HIP runtime replaced by tests/mockhip (preloaded), and
prints one line per case.  No torch, no GPU.

argv: a JSON list of cases {"w": workload, "inplace": bool, "order":
"weights-first" | "kv-first" | "async-load", "steps": n, "warmup": bool,
"layers": optional layer count}.  "async-load" reads the weight inflow
from a checkpoint of holes (atp_load_reshard_weights_async), issues the KV
call while the reads run and lets atp_sync issue the weight pieces.
"""
import ctypes as C
import json
import os
import sys

sys.modules["torch"] = None  # the binding does without torch; no real HIP runtime is used
sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
mock = C.CDLL(os.environ["ATP_MOCKHIP"])

import numpy as np  # noqa: E402

from paper_2511_11617_amd import atp, problem  # noqa: E402
from synth import checkpoint, configs, pagetable  # noqa: E402


def dmalloc(n):
    p = C.c_void_p()
    assert mock.hipMalloc(C.byref(p), C.c_size_t(max(int(n), 256))) == 0
    return p.value


def hmalloc(n):
    p = C.c_void_p()
    assert mock.hipHostMalloc(C.byref(p), C.c_size_t(max(int(n), 256)), 0) == 0
    return p.value


def stream():
    s = C.c_void_p()
    assert mock.hipStreamCreateWithFlags(C.byref(s), 1) == 0
    return s.value


def run(case):
    c = configs.get(case["w"], inplace=case["inplace"])
    if case.get("layers"):
        c["layers"] = case["layers"]
    table, pool = pagetable.make_for(c)
    n_live = len(np.unique(table[table >= 0]))
    inplace = bool(c["inplace"])
    b = problem.build(c, n_live=n_live, pool=pool, flags=atp.INPLACE if inplace else 0,
                      staging_cap=c["staging_cap"] or (2 << 30 if inplace else 0))
    st = b.plan().stats()
    if inplace:
        aw_n, ak_n = max(st.old_arena_bytes, st.new_arena_bytes), max(st.old_kv_bytes, st.new_kv_bytes)
        aw, nw, ak, nk = dmalloc(aw_n), None, dmalloc(ak_n), None
    else:
        aw_n, ak_n = st.old_arena_bytes, st.old_kv_bytes
        aw, nw, ak, nk = dmalloc(aw_n), dmalloc(st.new_arena_bytes), dmalloc(ak_n), dmalloc(st.new_kv_bytes)
    sw, sk, td = dmalloc(st.staging_w), dmalloc(st.staging_kv), dmalloc(table.nbytes)
    hin_w, hin_k = hmalloc(st.inflow_w), hmalloc(st.inflow_kv)
    hout_w, hout_k = hmalloc(st.outbound_w), hmalloc(st.outbound_kv)
    s0, s1 = stream(), stream()
    if case["warmup"]:
        atp.warmup(s0, s1, 256)
    files = names = None
    if case["order"] == "async-load":
        tl = problem.tensor_list(c)
        path = os.path.join(os.environ["ATP_REPLAY_TMP"], f"w{case['w']}.safetensors")
        checkpoint.write_stream(path, [(n, l, r, cc) for (n, l, k, sp, r, cc, u) in tl], [])
        files = atp.StFiles([path])
        names = [checkpoint.name(n, l) for (n, l, *_) in tl]
    launches = []
    for _ in range(case["steps"]):
        p = b.plan()

        def wcall():
            p.reshard_weights(aw, aw_n, nw, st.new_arena_bytes if nw else 0, hin_w, st.inflow_w, hout_w,
                              st.outbound_w if inplace else 0, sw, max(st.staging_w, 256), s0, s1)

        def kcall():
            p.reshard_kv(ak, ak_n, nk, st.new_kv_bytes if nk else 0, td, table.shape[0], table.shape[1], hin_k,
                         st.inflow_kv, hout_k, st.outbound_kv if inplace else 0, sk, max(st.staging_kv, 256),
                         s0, s1)

        try:
            if case["order"] == "kv-first":
                kcall()
                wcall()
            elif case["order"] == "async-load":
                p.load_reshard_weights_async(files, names, aw, aw_n, nw, st.new_arena_bytes if nw else 0, hin_w,
                                             st.inflow_w, hout_w, st.outbound_w if inplace else 0, sw,
                                             max(st.staging_w, 256), s0, s1)
                kcall()
            else:
                wcall()
                kcall()
        except atp.AtpError as e:
            p.sync()
            return {"refused": e.code, "msg": str(e)}
        t = p.sync()
        if case["order"] == "async-load":
            assert p.load_stats().bytes == st.inflow_w
        launches.append(int(t.n_launches))
    return {"ok": True, "launches": launches, "mock_launches": int(mock.mock_launches()),
            "mock_copies": int(mock.mock_copies()), "streams": int(mock.mock_streams())}


for case in json.loads(sys.argv[1]):
    print(json.dumps({"case": case, **run(case)}), flush=True)
print("replay done", flush=True)
