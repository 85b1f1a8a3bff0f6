"""Python binding of the state plane (Sec. III-A): a daemon that owns the
GPU memory of the weights and the KV cache and keeps host metadata, and
the client calls inference processes use to reach it.  Marshalling only:
the daemon and the client are the library's C ABI (atp_daemon_serve,
atp_state_*).

    p = spawn("/tmp/atp.sock")          # daemon process, ready on return
    c = Client("/tmp/atp.sock")
    ptr = c.alloc("weights", nbytes)     # device pointer in this process
    c.put("kv.table", table)             # numpy array or bytes
    ...                                  # the process may die here
    c = Client("/tmp/atp.sock")          # a new process
    ptr, nbytes = c.open("weights")
    table = c.get_array("kv.table", np.int32)
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess
import sys
import time

import numpy as np

from . import atp

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
MAX_REGION = (2 << 30) - (1 << 20)


def serve(path: str, device: int = 0) -> None:
    """Run the daemon in this thread until a client asks it to shut down."""
    atp._check(atp.lib.atp_daemon_serve(path.encode(), device))


def spawn(path: str, device: int = 0, timeout: float = 120.0) -> subprocess.Popen:
    """Start a daemon process on `path` and return once it answers."""
    p = subprocess.Popen([sys.executable, "-m", "paper_2511_11617_amd.daemon", "--socket", path,
                          "--device", str(device)], cwd=ROOT, stdout=subprocess.PIPE,
                         stderr=subprocess.PIPE, text=True)
    t0 = time.time()
    while True:
        if p.poll() is not None:
            out, err = p.communicate()
            raise RuntimeError(f"state daemon exited with {p.returncode}: {err.strip() or out.strip()}")
        try:
            Client(path).close()
            return p
        except atp.AtpError:
            pass
        if time.time() - t0 > timeout:
            p.kill()
            p.wait()
            raise TimeoutError(f"state daemon on {path} did not answer within {timeout} s")
        time.sleep(0.05)


class Client:
    def __init__(self, path: str):
        h = C.c_void_p()
        atp._check(atp.lib.atp_state_connect(path.encode(), C.byref(h)))
        self.h = h

    def close(self):
        if self.h:
            atp.lib.atp_state_disconnect(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def alloc(self, name: str, nbytes: int) -> int:
        p = C.c_void_p()
        atp._check(atp.lib.atp_state_alloc(self.h, name.encode(), int(nbytes), C.byref(p)))
        return p.value

    def open(self, name: str):
        p, n = C.c_void_p(), C.c_uint64()
        atp._check(atp.lib.atp_state_open(self.h, name.encode(), C.byref(p), C.byref(n)))
        return p.value, n.value

    def release(self, ptr: int) -> None:
        atp._check(atp.lib.atp_state_release(self.h, C.c_void_p(ptr)))

    def free(self, name: str) -> None:
        atp._check(atp.lib.atp_state_free(self.h, name.encode()))

    def put(self, name: str, data) -> None:
        b = np.ascontiguousarray(data).view(np.uint8).reshape(-1) if isinstance(data, np.ndarray) \
            else np.frombuffer(bytes(data), dtype=np.uint8)
        atp._check(atp.lib.atp_state_put(self.h, name.encode(), b.ctypes.data if b.size else None, b.size))

    def get(self, name: str) -> bytes:
        n = C.c_uint64()
        atp._check(atp.lib.atp_state_get(self.h, name.encode(), None, 0, C.byref(n)))
        buf = C.create_string_buffer(max(n.value, 1))
        atp._check(atp.lib.atp_state_get(self.h, name.encode(), buf, n.value, C.byref(n)))
        return buf.raw[:n.value]

    def get_array(self, name: str, dtype, shape=None) -> np.ndarray:
        a = np.frombuffer(self.get(name), dtype=dtype).copy()
        return a.reshape(shape) if shape is not None else a

    def list(self) -> str:
        n = C.c_uint64()
        atp._check(atp.lib.atp_state_list(self.h, None, 0, C.byref(n)))
        buf = C.create_string_buffer(n.value)
        atp._check(atp.lib.atp_state_list(self.h, buf, n.value, C.byref(n)))
        return buf.value.decode()

    def shutdown(self) -> None:
        atp._check(atp.lib.atp_state_shutdown(self.h))
