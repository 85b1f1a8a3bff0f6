"""The executor's host logic on the CPU (no GPU): reshards of the workloads,
in and out of place, in both call orders, with and without atp_warmup, run
through libatp.so in a child process whose HIP runtime is the host-only
stand-in in tests/mockhip.  The stand-in aborts on any copy outside its
allocations or with the wrong host/device sides, and on any use of an
unknown event or stream; the executor must issue every call, sync it and
stay within the bounded side-stream search."""
import json
import os
import subprocess
import sys

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))


@pytest.fixture(scope="module")
def mockhip(tmp_path_factory):
    out = str(tmp_path_factory.mktemp("mockhip") / "libmockhip.so")
    src = os.path.join(HERE, "mockhip")
    r = subprocess.run(["g++", "-O1", "-g", "-fPIC", "-shared", "-std=c++17", "-D__HIP_PLATFORM_AMD__",
                        "-I/opt/rocm/include", f"-Wl,--version-script={src}/mock.map", f"{src}/mock_hip.cpp",
                        "-o", out], capture_output=True, text=True)
    if r.returncode:
        pytest.skip("cannot build the HIP stand-in: " + r.stderr[-500:])
    return out


def _replay(mockhip, cases, tmp=None):
    env = dict(os.environ)
    if tmp is not None:
        env["ATP_REPLAY_TMP"] = str(tmp)
    # appended, so that anything already preloaded stays first
    env["LD_PRELOAD"] = ":".join(x for x in (env.get("LD_PRELOAD", ""), mockhip) if x)
    env["ATP_MOCKHIP"] = mockhip
    r = subprocess.run([sys.executable, os.path.join(HERE, "exec_replay.py"), json.dumps(cases)], env=env,
                       capture_output=True, text=True, timeout=600)
    assert "MOCKHIP FAULT" not in r.stderr, r.stderr[-3000:]
    assert r.returncode == 0 and "replay done" in r.stdout, (r.returncode, r.stdout[-2000:], r.stderr[-3000:])
    return [json.loads(x) for x in r.stdout.splitlines() if x.startswith("{")]


def test_out_of_place_both_orders(mockhip):
    cases = [{"w": w, "inplace": False, "order": o, "steps": 2, "warmup": wu}
             for w in (1, 2, 3, 4) for o in ("weights-first", "kv-first") for wu in (False, True)]
    res = _replay(mockhip, cases)
    assert len(res) == len(cases)
    for i, r in enumerate(res):
        assert r.get("ok"), r
        assert all(n > 0 for n in r["launches"])
        # two caller streams per case so far, plus at most eight side-stream candidates per device
        assert r["streams"] <= 2 * (i + 1) + 8


def test_in_place_weights_first_and_kv_first_refused(mockhip):
    cases = [{"w": 5, "inplace": True, "order": "weights-first", "steps": 2, "warmup": False},
             {"w": 2, "inplace": True, "order": "weights-first", "steps": 2, "warmup": True},
             {"w": 1, "inplace": True, "order": "weights-first", "steps": 3, "warmup": False},
             {"w": 1, "inplace": True, "order": "kv-first", "steps": 1, "warmup": False}]
    res = _replay(mockhip, cases)
    assert [r.get("ok") for r in res[:3]] == [True] * 3
    assert res[0]["launches"][0] > 100  # 22 weight and 25 KV levels, outbound reads, ring scatters
    assert res[3]["refused"] == -5 and "before" in res[3]["msg"]


def test_async_load_with_the_kv_call_between(mockhip, tmp_path):
    """atp_load_reshard_weights_async, the KV call while the reads run, then
    atp_sync issuing the weight pieces: in and out of place, fresh plans in
    a row, with the reads from a checkpoint of holes."""
    cases = [{"w": 1, "inplace": False, "order": "async-load", "steps": 2, "warmup": False},
             {"w": 1, "inplace": True, "order": "async-load", "steps": 2, "warmup": True},
             {"w": 2, "inplace": False, "order": "async-load", "steps": 2, "warmup": False, "layers": 1},
             {"w": 2, "inplace": True, "order": "async-load", "steps": 2, "warmup": False, "layers": 1}]
    res = _replay(mockhip, cases, tmp_path)
    assert [r.get("ok") for r in res] == [True] * 4, res
