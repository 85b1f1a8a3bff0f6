"""Bit-exact parity of the HIP reshard with the oracle (GPU, through the C ABI).

Small cases the oracle materialises in seconds: the tiny 4 -> 3 workload,
random small decoders (odd sizes, unaligned runs, replicated KV heads,
fragmented block tables, both KV layouts, 16-bit payloads with NaN / Inf
/ -0 patterns), the per-layer shapes of the four large workloads with few
layers and sequences, out of place (destination poisoned first) and in
place.
"""
import random

import pytest
import torch

from paper_2511_11617_amd import atp
from synth import configs
from synth.content import KIND_RAW16, KIND_TAG16
from tests.gpu_harness import SQUEEZED_RING_CAP, run_case, squeezed_ring_cfg
from tests.test_oracle_repack import med_cfg, tiny_cfg
from tests.test_schedule_sim import single_target_cfg

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


@pytest.mark.parametrize("layout", ["head", "token"])
@pytest.mark.parametrize("payload", ["normal", "raw"])
def test_cfg1_out_of_place(layout, payload):
    kw = {"kv_layout": layout}
    if payload == "raw":
        kw.update(w_kind=KIND_RAW16, kv_kind=KIND_RAW16)
    run_case(configs.get(1, **kw), name="cfg1")


@pytest.mark.parametrize("self_old", [0, 2, 3])
def test_cfg1_every_survivor(self_old):
    run_case(configs.get(1, self_old=self_old), name="cfg1-survivor")


@pytest.mark.parametrize("no_tail", [False, True])
@pytest.mark.parametrize("layout", ["head", "token"])
def test_cfg1_in_place(layout, no_tail):
    flags = atp.INPLACE | (atp.NO_TAIL_STAGING if no_tail else 0)
    run_case(configs.get(1, kv_layout=layout), flags=flags, name="cfg1-inplace" + ("-levels" if no_tail else ""))


@pytest.mark.parametrize("seed", list(range(24)))
def test_random_small(seed):
    rng = random.Random(seed)
    c = tiny_cfg(rng, experts=seed % 3 == 0)
    run_case(c, name=f"random-{seed}")


@pytest.mark.parametrize("seed", list(range(6)))
def test_random_small_kv_call_first(seed):
    """Out of place the two calls may come in either order."""
    rng = random.Random(500 + seed)
    run_case(tiny_cfg(rng, experts=seed % 2 == 1), kv_first=True, name=f"random-kv-first-{seed}")


@pytest.mark.parametrize("mode", ["out-of-place", "in-place", "kv-first"])
@pytest.mark.parametrize("seed", list(range(20)))
def test_random_medium(seed, mode):
    """Random medium decoders: real 2-4 KiB KV head lines (wide tiles),
    multi-tile weight lines, up to TP 8, fragmented pools."""
    c = med_cfg(random.Random(9000 + seed), experts=seed % 3 == 0)
    # in place, odd seeds resolve their level chains by levels alone
    flags = (atp.INPLACE | (atp.NO_TAIL_STAGING if seed % 2 else 0)) if mode == "in-place" else 0
    run_case(c, flags=flags, kv_first=mode == "kv-first", name=f"random-medium-{seed}-{mode}")


@pytest.mark.parametrize("seed", list(range(24)))
def test_random_small_in_place(seed):
    rng = random.Random(1000 + seed)
    c = tiny_cfg(rng, experts=seed % 3 == 0)
    # odd seeds resolve their level chains by levels alone
    flags = atp.INPLACE | (atp.NO_TAIL_STAGING if seed % 2 else 0)
    run_case(c, flags=flags, name=f"random-inplace-{seed}" + ("-levels" if seed % 2 else ""))


@pytest.mark.parametrize("inplace", [False, True])
@pytest.mark.parametrize("n", [2, 3, 4])
def test_large_shapes_one_layer(n, inplace):
    c = configs.scaled(n, layers=1, n_seq=2, seq_tokens=256, w_kind=KIND_TAG16, kv_kind=KIND_TAG16)
    run_case(c, flags=atp.INPLACE if inplace else 0, name=f"cfg{n}-1layer" + ("-inplace" if inplace else ""))


@pytest.mark.parametrize("self_old,inplace", [(0, False), (0, True), (1, False), (1, True)])
def test_single_target_takes_every_tensor_whole(self_old, inplace):
    run_case(single_target_cfg(self_old), flags=atp.INPLACE if inplace else 0,
             name=f"tp2to1-self{self_old}" + ("-inplace" if inplace else ""))


def test_in_place_ring_under_a_squeezed_staging_cap():
    c = squeezed_ring_cfg()
    run_case(c, flags=atp.INPLACE, staging_cap=SQUEEZED_RING_CAP, name="ring-squeezed-inplace")


def test_cfg5_shape_in_place_two_layers():
    c = configs.scaled(5, layers=2, n_seq=2, seq_tokens=256, w_kind=KIND_TAG16, kv_kind=KIND_TAG16)
    run_case(c, flags=atp.INPLACE, staging_cap=c["staging_cap"], name="cfg5-2layers-inplace")


@pytest.mark.parametrize("no_tail", [False, True])
def test_kv_level_chain_in_place(no_tail):
    """The 80-layer TP 8 -> 7 workload's KV geometry on a small decoder: the
    KV shard doubles on its own arena (a chain of about 12 levels), its tail
    through staging or every level launched."""
    c = configs.get(5, layers=2, hidden=512, n_q=16, n_kv=8, head_dim=64, ffn=1024, n_seq=8, seq_tokens=1024,
                    new_q_widths=None, w_kind=KIND_TAG16, kv_kind=KIND_TAG16)
    flags = atp.INPLACE | (atp.NO_TAIL_STAGING if no_tail else 0)
    run_case(c, flags=flags, staging_cap=c["staging_cap"], name="kv-chain-inplace" + ("-levels" if no_tail else ""))


@pytest.mark.parametrize("variant,flag", [("greedy", atp.PLAN_GREEDY), ("full", atp.PLAN_FULL)])
@pytest.mark.parametrize("inplace", [False, True])
def test_planner_baselines(variant, flag, inplace):
    flags = flag | (atp.INPLACE if inplace else 0)
    run_case(configs.get(1), flags=flags, variant=variant, name=f"cfg1-{variant}")
