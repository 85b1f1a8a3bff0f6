"""KV budget under recovery on the GPU (through the C ABI): the sessions the
oracle's LRU policy keeps are resharded, into the by-id arena or an
ATP_KV_COMPACT arena, and the result equals the oracle's byte for byte."""
import random

import numpy as np
import pytest
import torch

from paper_2511_11617_amd import atp
from synth import configs
from synth.content import KIND_TAG16
from tests.gpu_harness import run_case
from tests.test_oracle_repack import tiny_cfg

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    yield
    torch.cuda.synchronize()


@pytest.mark.parametrize("layout", ["head", "token"])
@pytest.mark.parametrize("frac", [0.5, 0.25])
def test_cfg1_compact_after_eviction(layout, frac):
    c = configs.get(1, kv_layout=layout, w_kind=KIND_TAG16, kv_kind=KIND_TAG16)
    last = np.random.default_rng(3).permutation(c["n_seq"])
    run_case(c, flags=atp.KV_COMPACT, evict=(last, frac), name=f"cfg1-compact-{layout}-{frac}")


@pytest.mark.parametrize("flags", [0, atp.INPLACE])
def test_cfg1_eviction_ids_kept(flags):
    c = configs.get(1, w_kind=KIND_TAG16, kv_kind=KIND_TAG16)
    last = np.random.default_rng(5).permutation(c["n_seq"])
    run_case(c, flags=flags, evict=(last, 0.5), name=f"cfg1-evict-flags{flags}")


@pytest.mark.parametrize("flags", [atp.KV_COMPACT, 0, atp.INPLACE])
def test_cfg1_zero_budget_evicts_every_session(flags):
    """No live block is left: the KV call moves and lands nothing, and the
    weights are resharded as usual."""
    c = configs.get(1, w_kind=KIND_TAG16, kv_kind=KIND_TAG16)
    last = np.random.default_rng(7).permutation(c["n_seq"])
    run_case(c, flags=flags, evict=(last, 0.0), name=f"cfg1-evict-all-flags{flags}")


@pytest.mark.parametrize("seed", [2, 11, 40])
def test_tiny_compact_after_eviction(seed):
    c = tiny_cfg(random.Random(seed), experts=seed % 2 == 1)
    last = np.random.default_rng(seed).integers(0, 3, c["n_seq"])
    run_case(c, flags=atp.KV_COMPACT, evict=(last, 0.6), name=f"tiny{seed}-compact")
