"""State daemon process (Sec. III-A): `python -m paper_2511_11617_amd.daemon
--socket PATH [--device N]`.  Owns the regions it allocates until a client
asks it to shut down; see state.py."""
from __future__ import annotations

import argparse
import sys


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--socket", required=True)
    ap.add_argument("--device", type=int, default=0)
    a = ap.parse_args()
    from . import atp, state  # loads torch's HIP runtime first (one runtime per process)
    try:
        state.serve(a.socket, a.device)
    except atp.AtpError as e:
        print(f"state daemon: {e}", file=sys.stderr, flush=True)
        return 1
    return 0


if __name__ == "__main__":
    sys.exit(main())
