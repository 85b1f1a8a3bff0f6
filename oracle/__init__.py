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
  kvbudget the least-recently-used session eviction of the KV budget.

Every function is pinned by CPU tests (tests/test_oracle_*.py,
tests/test_kv_budget.py) to something other than itself: the paper's worked
example (Fig. 3), hand-computed shard splits and hand-located words of the
tiny workload (tests/golden/), Eq. 1's closed form, brute force, and
invariants (every target's new shards and KV blocks together rebuild the
full tensors; outbound bytes are what the receiving peers' new shards hold).
tests/test_oracle_mutants.py plants one-line index mistakes in the oracle
and requires a pin to fail on each.
"""
