"""Seeded synthetic content for the reshard workloads (CPU side).

This module is an input generator only.  It holds none of the reshard
method's arithmetic: it answers "what 16-bit word does element `idx` of the
full, unsharded logical tensor (`tag`, `layer`) hold?", so that any slice of
any tensor can be produced without materialising the model.

Generator (published definitions, restated):

* SplitMix64 (Steele, Lea, Flood, "Fast splittable pseudorandom number
  generators", OOPSLA 2014).  The generator's state advances by the odd
  constant GAMMA = 0x9E3779B97F4A7C15 and each output is the state passed
  through the "mix64" finaliser
      z ^= z >> 30; z *= 0xBF58476D1CE4E5B9;
      z ^= z >> 27; z *= 0x94D049BB133111EB;
      z ^= z >> 31.
  Used counter-style: word(key, idx) = mix64(key + (idx + 1) * GAMMA), i.e.
  the (idx+1)-th output of a SplitMix64 stream seeded with `key`.
* Near-normal values without transcendental functions (Irwin-Hall, n = 4):
  the four 16-bit fields of the word are summed and centred; the integer
  s in [-131070, 131070] has variance 4 * (65536^2 - 1) / 12.  The value is
  float32(s) * float32(sigma / std), a single IEEE binary32 multiply, then
  rounded to bf16 or fp16 with round-to-nearest-even done on the integer
  bits.  Every step is exact integer arithmetic or one correctly rounded
  multiply, so the HIP twin of this generator (synth/csrc/synth.hip) yields
  identical bits.

Payload kinds:
  KIND_BF16 / KIND_FP16 : near-normal values (weights sigma 0.02, KV sigma 1)
  KIND_TAG16            : low 16 bits of the word (distinct-ish tags)
  KIND_RAW16            : top 16 bits of the word (any bit pattern,
                          including NaN / Inf / -0 encodings)
"""
from __future__ import annotations

import numpy as np

GAMMA = 0x9E3779B97F4A7C15
MIX1 = 0xBF58476D1CE4E5B9
MIX2 = 0x94D049BB133111EB
MASK64 = (1 << 64) - 1

KIND_BF16 = 0
KIND_FP16 = 1
KIND_TAG16 = 2
KIND_RAW16 = 3

# Standard deviation of the centred sum of four uniform 16-bit integers.
IH_STD = float(np.sqrt((65536.0 ** 2 - 1.0) / 3.0))

# Tensor tags (content streams).  Names follow the usual decoder notation.
TAGS = {
    "wq": 0, "wk": 1, "wv": 2, "wo": 3,
    "w_gate": 4, "w_up": 5, "w_down": 6,
    "e_gate": 7, "e_up": 8, "e_down": 9,
    "k_cache": 10, "v_cache": 11,
}


def mix64_int(z: int) -> int:
    """SplitMix64 finaliser on a Python int (scalar reference)."""
    z &= MASK64
    z = ((z ^ (z >> 30)) * MIX1) & MASK64
    z = ((z ^ (z >> 27)) * MIX2) & MASK64
    return z ^ (z >> 31)


def stream_key(seed: int, tag: int, layer: int) -> int:
    """Key of the content stream of tensor `tag` in `layer`."""
    return mix64_int(mix64_int(seed) + (tag << 20) + layer)


def _mix64(z: np.ndarray) -> np.ndarray:
    with np.errstate(over="ignore"):
        z = (z ^ (z >> np.uint64(30))) * np.uint64(MIX1)
        z = (z ^ (z >> np.uint64(27))) * np.uint64(MIX2)
    return z ^ (z >> np.uint64(31))


def words(key: int, idx: np.ndarray) -> np.ndarray:
    """64-bit SplitMix64 words for flat indices `idx` (any int array)."""
    idx = np.asarray(idx, dtype=np.uint64)
    with np.errstate(over="ignore"):
        z = np.uint64(key) + (idx + np.uint64(1)) * np.uint64(GAMMA)
    return _mix64(z)


def f32_to_bf16_bits(f: np.ndarray) -> np.ndarray:
    """Round-to-nearest-even float32 -> bf16 (finite inputs)."""
    b = np.ascontiguousarray(f, dtype=np.float32).view(np.uint32)
    lsb = (b >> np.uint32(16)) & np.uint32(1)
    return ((b + np.uint32(0x7FFF) + lsb) >> np.uint32(16)).astype(np.uint16)


def f32_to_fp16_bits(f: np.ndarray) -> np.ndarray:
    """Round-to-nearest-even float32 -> IEEE binary16 on the integer bits.

    Finite inputs with |x| < 65520 (the values produced here are far
    smaller); subnormal results are rounded like normal ones."""
    b = np.ascontiguousarray(f, dtype=np.float32).view(np.uint32).astype(np.int64)
    sign = (b >> 16) & 0x8000
    e = (b >> 23) & 0xFF
    m = b & 0x7FFFFF
    out = np.zeros(b.shape, dtype=np.int64)
    # normal binary16 results: biased exponent e - 112 in [1, 30]
    nrm = e >= 113
    mant = m >> 13
    rem = m & 0x1FFF
    up = (rem > 0x1000) | ((rem == 0x1000) & ((mant & 1) == 1))
    out = np.where(nrm, ((e - 112) << 10) + mant + up.astype(np.int64), out)
    # subnormal results: value = full * 2^(e-150) = k * 2^-24, k = full >> (126-e)
    sub = (~nrm) & (e >= 102)
    full = m | 0x800000
    sh = np.clip(126 - e, 1, 62)
    k = full >> sh
    rem2 = full & ((np.int64(1) << sh) - 1)
    half = np.int64(1) << (sh - 1)
    up2 = (rem2 > half) | ((rem2 == half) & ((k & 1) == 1))
    out = np.where(sub, k + up2.astype(np.int64), out)
    return (sign | out).astype(np.uint16)


def values16(key: int, idx: np.ndarray, kind: int, sigma: float) -> np.ndarray:
    """The 16-bit payload words of stream `key` at flat indices `idx`."""
    w = words(key, idx)
    if kind == KIND_TAG16:
        return (w & np.uint64(0xFFFF)).astype(np.uint16)
    if kind == KIND_RAW16:
        return (w >> np.uint64(48)).astype(np.uint16)
    s = ((w & np.uint64(0xFFFF)) + ((w >> np.uint64(16)) & np.uint64(0xFFFF))
         + ((w >> np.uint64(32)) & np.uint64(0xFFFF)) + (w >> np.uint64(48)))
    s = s.astype(np.int64) - 131070
    scale = np.float32(sigma / IH_STD)
    f = s.astype(np.float32) * scale
    if kind == KIND_BF16:
        return f32_to_bf16_bits(f)
    if kind == KIND_FP16:
        return f32_to_fp16_bits(f)
    raise ValueError(f"unknown payload kind {kind}")


def scale_f32(sigma: float) -> np.float32:
    """The binary32 multiplier applied to the centred integer sum."""
    return np.float32(sigma / IH_STD)


class Content:
    """Content provider for one workload: (tag, layer, flat idx) -> uint16."""

    def __init__(self, seed: int, w_kind: int, kv_kind: int,
                 w_sigma: float = 0.02, kv_sigma: float = 1.0):
        self.seed = seed
        self.w_kind = w_kind
        self.kv_kind = kv_kind
        self.w_sigma = w_sigma
        self.kv_sigma = kv_sigma

    def key(self, tag: int, layer: int) -> int:
        return stream_key(self.seed, tag, layer)

    def kind_sigma(self, tag: int):
        if tag in (TAGS["k_cache"], TAGS["v_cache"]):
            return self.kv_kind, self.kv_sigma
        return self.w_kind, self.w_sigma

    def __call__(self, tag: int, layer: int, idx: np.ndarray) -> np.ndarray:
        kind, sigma = self.kind_sigma(tag)
        return values16(self.key(tag, layer), idx, kind, sigma)
