"""Pins of the seeded input generator (CPU)."""
import numpy as np
import torch

from synth import configs, pagetable
from synth.content import (KIND_BF16, KIND_FP16, KIND_RAW16, f32_to_bf16_bits,
                           f32_to_fp16_bits, values16, words)


def test_splitmix64_published_sequence():
    # SplitMix64 seeded with 0: its first three outputs (Steele et al. 2014;
    # the reference C implementation prints these for x = 0).
    w = words(0, np.array([0, 1, 2]))
    assert [int(x) for x in w] == [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F]


def _probe_floats():
    rng = np.random.default_rng(5)
    parts = [
        rng.normal(0, 0.02, 200000), rng.normal(0, 1, 200000),
        rng.uniform(-1e-7, 1e-7, 200000), rng.uniform(-7e-5, 7e-5, 200000),
        np.array([0.0, -0.0, 2 ** -24, 2 ** -25, 3 * 2 ** -26, 2 ** -14, 65504.0]),
    ]
    return np.concatenate(parts).astype(np.float32)


def test_fp16_rounding_matches_numpy():
    f = _probe_floats()
    np.testing.assert_array_equal(f32_to_fp16_bits(f), f.astype(np.float16).view(np.uint16))


def test_bf16_rounding_matches_torch():
    f = _probe_floats()
    want = torch.from_numpy(f).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(f32_to_bf16_bits(f), want)


def test_near_normal_moments():
    idx = np.arange(1 << 20, dtype=np.uint64)
    w = values16(12345, idx, KIND_BF16, 0.02)
    x = torch.from_numpy(w.view(np.int16)).view(torch.bfloat16).float().numpy()
    assert abs(x.mean()) < 1e-3 and abs(x.std() - 0.02) < 5e-4
    h = values16(12345, idx, KIND_FP16, 1.0).view(np.float16).astype(np.float32)
    assert abs(h.mean()) < 5e-3 and abs(h.std() - 1.0) < 5e-3


def test_raw_payload_covers_nan_and_negzero():
    w = values16(7, np.arange(1 << 20, dtype=np.uint64), KIND_RAW16, 0.0)
    f = w.view(np.float16)
    assert np.isnan(f).any() and np.isinf(f).any() and (w == 0x8000).any()


def test_fragmented_table_is_seeded_permutation():
    c = configs.get(3)
    t, pool = pagetable.make_for(configs.scaled(3, n_seq=4, seq_tokens=256))
    live = t[t >= 0]
    assert len(np.unique(live)) == live.size and live.max() < pool
    assert pool == int(np.ceil(1.125 * live.size))
    t2, _ = pagetable.make_for(configs.scaled(3, n_seq=4, seq_tokens=256))
    np.testing.assert_array_equal(t, t2)
    assert c["fragmented"]
