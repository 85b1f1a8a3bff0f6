"""State plane on the host (Sec. III-A): the daemon process, its protocol and
its error paths, without touching a GPU.

* named blobs round-trip byte for byte (bytes and numpy arrays), are
  replaced by a second put, and report their size; a too-small buffer is
  ATP_ECAPACITY;
* missing names are ATP_EINVAL, region sizes outside [1, 2 GiB - 1 MiB] are
  refused before the daemon touches a device;
* a client process that dies without disconnecting does not take the daemon
  or its state with it (the state plane's reason to exist);
* a second daemon on a live socket is refused, a stale socket file is
  replaced, shutdown stops the daemon and removes the socket.
"""
import os
import socket
import subprocess
import sys
import tempfile

import numpy as np
import pytest

from paper_2511_11617_amd import atp, state

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture
def daemon():
    d = tempfile.mkdtemp(prefix="atp-", dir="/tmp")
    path = os.path.join(d, "s.sock")
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
            p.wait(timeout=30)
        except subprocess.TimeoutExpired:
            p.kill()
            p.wait()
    os.rmdir(d) if os.path.isdir(d) and not os.listdir(d) else None


def test_blobs_round_trip(daemon):
    c = state.Client(daemon)
    table = np.arange(-1, 4095, dtype=np.int32).reshape(64, 64)
    c.put("kv.table", table)
    np.testing.assert_array_equal(c.get_array("kv.table", np.int32, (64, 64)), table)
    raw = bytes(range(256)) * 5
    c.put("raw", raw)
    assert c.get("raw") == raw
    c.put("raw", b"x")  # replaced
    assert c.get("raw") == b"x"
    c.put("empty", b"")
    assert c.get("empty") == b""
    listing = c.list()
    assert "blob kv.table 16384" in listing and "blob raw 1" in listing
    # a buffer below the size: ECAPACITY, and the size is still reported
    import ctypes as C
    n = C.c_uint64()
    buf = C.create_string_buffer(8)
    rc = atp.lib.atp_state_get(c.h, b"kv.table", buf, 8, C.byref(n))
    assert rc == atp.ECAPACITY and n.value == table.nbytes
    c.close()


def test_missing_names_and_bad_sizes(daemon):
    c = state.Client(daemon)
    for call in (lambda: c.get("nope"), lambda: c.open("nope"), lambda: c.free("nope")):
        with pytest.raises(atp.AtpError) as e:
            call()
        assert e.value.code == atp.EINVAL
    for n in (0, state.MAX_REGION + 1, 4 << 30):
        with pytest.raises(atp.AtpError) as e:
            c.alloc("r", n)
        assert e.value.code == atp.EINVAL and "2 GiB" in str(e.value)
    with pytest.raises(atp.AtpError):
        c.put("", b"x")
    c.close()


def test_allocation_without_a_gpu_is_ehip(daemon):
    import torch
    if torch.cuda.is_available():
        pytest.skip("this machine has a GPU: covered by the GPU state tests")
    c = state.Client(daemon)
    with pytest.raises(atp.AtpError) as e:
        c.alloc("weights", 1 << 20)
    assert e.value.code == atp.EHIP
    assert "region" not in c.list()  # nothing was recorded
    c.close()


CRASHING_CLIENT = r"""
import os, sys
sys.path.insert(0, {root!r})
from paper_2511_11617_amd import state
c = state.Client({path!r})
c.put("session.last_use", bytes(range(200)))
os._exit(3)  # dies without disconnecting
"""


def test_state_survives_a_client_that_dies(daemon):
    r = subprocess.run([sys.executable, "-c", CRASHING_CLIENT.format(root=ROOT, path=daemon)],
                       capture_output=True, text=True, timeout=300)
    assert r.returncode == 3, r.stderr
    c = state.Client(daemon)
    assert c.get("session.last_use") == bytes(range(200))
    c.close()


def test_second_daemon_refused_and_shutdown(daemon):
    r = subprocess.run([sys.executable, "-m", "paper_2511_11617_amd.daemon", "--socket", daemon],
                       cwd=ROOT, capture_output=True, text=True, timeout=300)
    assert r.returncode == 1 and "already serves" in r.stderr
    c = state.Client(daemon)
    c.put("x", b"1")
    c.shutdown()
    c.close()
    for _ in range(200):
        if not os.path.exists(daemon):
            break
        import time
        time.sleep(0.05)
    assert not os.path.exists(daemon)
    with pytest.raises(atp.AtpError) as e:
        state.Client(daemon)
    assert e.value.code == atp.EINVAL


def test_stale_socket_file_is_replaced():
    d = tempfile.mkdtemp(prefix="atp-", dir="/tmp")
    path = os.path.join(d, "s.sock")
    s = socket.socket(socket.AF_UNIX, socket.SOCK_STREAM)
    s.bind(path)
    s.close()  # leaves the file, nobody listens
    assert os.path.exists(path)
    p = state.spawn(path)
    c = state.Client(path)
    c.put("a", b"b")
    assert c.get("a") == b"b"
    c.shutdown()
    c.close()
    assert p.wait(timeout=60) == 0
    os.rmdir(d)


def test_lost_daemon_is_estate(daemon):
    c = state.Client(daemon)
    other = state.Client(daemon)
    other.shutdown()
    other.close()
    import time
    time.sleep(0.2)
    with pytest.raises(atp.AtpError) as e:
        c.put("x", b"1")
    assert e.value.code == atp.ESTATE
    c.close()
