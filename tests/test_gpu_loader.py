"""Reload from a checkpoint, end to end on the GPU: the library's range-read
loader fills the pinned weight inflow buffer from a safetensors file, the
reshard lands it, and the new arena equals the oracle's new shard byte for
byte (through the C ABI)."""
import random

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


@pytest.mark.parametrize("flags", [0, atp.INPLACE])
def test_cfg1_from_checkpoint(tmp_path, flags):
    run_case(configs.get(1, w_kind=KIND_TAG16), flags=flags, ckpt_dir=tmp_path, name="cfg1-ckpt")


@pytest.mark.parametrize("seed,experts", [(3, True), (8, False), (21, True)])
def test_tiny_from_checkpoint(tmp_path, seed, experts):
    run_case(tiny_cfg(random.Random(seed), experts), ckpt_dir=tmp_path, name=f"tiny{seed}-ckpt")


def test_full_reload_from_checkpoint(tmp_path):
    run_case(configs.get(1, w_kind=KIND_TAG16), flags=atp.PLAN_FULL, variant="full", ckpt_dir=tmp_path,
             name="cfg1-full-ckpt")
