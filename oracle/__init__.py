"""CPU oracle for the state-preserving TP reshard (AnchorTP, arXiv 2511.11617).

TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke entry point and the
CPU-baseline leg of the benchmark may import this package.  It shares no
code with the HIP library and never imports it; the two meet only through
the seeded input generators in `synth`.

Modules
  cmm      target partitions (Alg. 1 floor rule, ceil-first, GQA-consistent),
           the Continuous Minimal Migration loop (Alg. 1) and the minimum
           reload of Eq. 1.
  model    the decoder's TP-sharded tensors and paged KV cache, shard
           geometry and arena layouts.
  repack   the new shard by definition (slicing the full tensors) and by
           executing the oracle's own plan (old shard + packed inflow).
  brute    exhaustive searches used to pin the plan on tiny inputs.
  hazard   replays an in-place copy schedule on a shadow copy of the arena.

Every function is pinned by CPU tests (tests/test_oracle_*.py) to the
paper's worked example (Fig. 3), hand-computed shard splits, Eq. 1's closed
form, brute force and invariants; nothing is "parity unpinned".
"""
