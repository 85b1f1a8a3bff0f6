"""Build the reshard library (libatp.so) and the synthetic-input helper
library (synth/libatp_synth.so) for gfx950 with hipcc.

Run as `python -m paper_2511_11617_amd.build` or through
`__graft_entry__.build()`.  Always recompiles.
"""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libatp.so")
SYNTH_SRC = os.path.join(ROOT, "synth", "csrc", "synth.hip")
SYNTH_LIB = os.path.join(ROOT, "synth", "libatp_synth.so")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
# Packed fp32 instructions stay off in device code (no float math here, but
# the flag keeps every HIP translation unit built the same way).
DEVICE_FLAGS = ["--offload-arch=" + ARCH, "-O3", "-fPIC", "-std=c++17",
                "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
                "-Wall", "-Wno-unused-function"]
HOST_FLAGS = ["-O2", "-fPIC", "-pthread", "-std=c++17", "-Wall", "-Wextra", "-Wno-unused-parameter",
              "-I/opt/rocm/include", "-D__HIP_PLATFORM_AMD__"]


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(" ".join(cmd) + "\n" + r.stdout + r.stderr)
        raise RuntimeError(f"build failed: {cmd[0]} exited {r.returncode}")
    return r


def build_atp(out_dir: str | None = None, lib_path: str = LIB, defines=()) -> str:
    """Compile libatp.so; `defines` (e.g. ["ATP_UNROLL=4"]) select a launch
    shape other than the default (see csrc/desc.h)."""
    out_dir = out_dir or os.path.join(HERE, "_build")
    os.makedirs(out_dir, exist_ok=True)
    dflags = ["-D" + d for d in defines]
    objs = []
    for src in ("plan.cpp", "loader.cpp", "kvbudget.cpp", "state.cpp", "capi.cpp"):
        obj = os.path.join(out_dir, src + ".o")
        _run(["g++", *HOST_FLAGS, *dflags, "-c", os.path.join(CSRC, src), "-o", obj])
        objs.append(obj)
    obj = os.path.join(out_dir, "exec.hip.o")
    _run([HIPCC, *DEVICE_FLAGS, *dflags, "-c", os.path.join(CSRC, "exec.hip"), "-o", obj])
    objs.append(obj)
    tmp = lib_path + ".tmp"
    _run([HIPCC, "--offload-arch=" + ARCH, "-shared", "-fPIC", "-pthread", *objs, "-o", tmp])
    os.replace(tmp, lib_path)
    return lib_path


def build_synth() -> str:
    tmp = SYNTH_LIB + ".tmp"
    _run([HIPCC, *DEVICE_FLAGS, "-shared", SYNTH_SRC, "-o", tmp])
    os.replace(tmp, SYNTH_LIB)
    return SYNTH_LIB


def build_all() -> None:
    build_atp()
    if os.path.exists(SYNTH_SRC):
        build_synth()


if __name__ == "__main__":
    build_all()
    print("built", LIB)
