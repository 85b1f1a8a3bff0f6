"""Several plans pending together on one GPU (through the C ABI).

Each plan owns its events, descriptor buffers and staging; plans issued on
the same (compute, copy) stream pair share the side stream that the
executor picks for that pair.  Here two or three plans, each on arenas of
its own, are issued back to back before any of them is synced, then synced
in issue order or in reverse, and every byte of every plan (and in place,
its outbound buffer) is compared with the oracle: in place, out of place,
mixed, and two layer groups of one decoder as a state-plane process
reshards them.
"""
import random

import pytest
import torch

from paper_2511_11617_amd import atp
from synth import configs
from synth.content import KIND_TAG16
from tests.gpu_harness import prepare_case, say
from tests.test_oracle_repack import med_cfg, tiny_cfg

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def run_together(cases, reverse_sync=False):
    """Prepare every case, issue them all on one stream pair, then sync and
    check each; `cases` holds (config, flags, name)."""
    compute = torch.cuda.current_stream()
    copy = torch.cuda.Stream()
    issues = [prepare_case(c, flags=f, name=n, streams=(compute, copy)) for c, f, n in cases]
    torch.cuda.synchronize()
    finishes = [issue() for issue in issues]
    say(f"[gpu case] {len(finishes)} plans pending")
    order = list(range(len(finishes)))
    if reverse_sync:
        order.reverse()
    for i in order:
        finishes[i]()


@pytest.mark.parametrize("reverse_sync", [False, True])
@pytest.mark.parametrize("mode", ["out-of-place", "in-place", "mixed"])
def test_two_plans_pending(mode, reverse_sync):
    a = configs.get(1)
    b = med_cfg(random.Random(17))
    fa = atp.INPLACE if mode in ("in-place", "mixed") else 0
    fb = atp.INPLACE if mode == "in-place" else 0
    run_together([(a, fa, f"cfg1-{mode}"), (b, fb, f"medium17-{mode}")], reverse_sync)


@pytest.mark.parametrize("seed", range(6))
def test_three_random_plans_pending(seed):
    rng = random.Random(500 + seed)
    cases = []
    for i in range(3):
        c = tiny_cfg(rng, experts=rng.random() < 0.5) if i < 2 else med_cfg(rng)
        cases.append((c, atp.INPLACE if rng.random() < 0.5 else 0, f"random{seed}-{i}"))
    run_together(cases, reverse_sync=seed % 2 == 1)


@pytest.mark.parametrize("inplace", [False, True])
def test_two_layer_groups_of_one_decoder(inplace):
    # the shape a state-plane process reshards group by group: two groups of
    # layers of the headline decoder, pending together
    c = configs.scaled(2, layers=2, n_seq=2, seq_tokens=256, w_kind=KIND_TAG16, kv_kind=KIND_TAG16)
    f = atp.INPLACE if inplace else 0
    run_together([(c, f, "dense40-group0"), (dict(c, seed=c["seed"] + 1), f, "dense40-group1")])
