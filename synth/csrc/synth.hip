// synth.hip — GPU twin of synth/content.py (seeded input generator).
//
// Test and benchmark infrastructure only: fills device buffers with the
// same 16-bit words the CPU generator defines, so that full-size inputs
// need not be generated on the host.  Holds none of the reshard's logic.
//
// word(key, idx) = mix64(key + (idx + 1) * GAMMA)  (SplitMix64, Steele,
// Lea, Flood 2014); near-normal payload = float32(sum of the four 16-bit
// fields - 131070) * scale, rounded to bf16 / fp16 on the integer bits.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

constexpr uint64_t GAMMA = 0x9E3779B97F4A7C15ull;
constexpr uint64_t MIX1 = 0xBF58476D1CE4E5B9ull;
constexpr uint64_t MIX2 = 0x94D049BB133111EBull;

__device__ __forceinline__ uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * MIX1;
  z = (z ^ (z >> 27)) * MIX2;
  return z ^ (z >> 31);
}

__device__ __forceinline__ uint16_t f32_to_bf16(uint32_t b) {
  return uint16_t((b + 0x7FFFu + ((b >> 16) & 1u)) >> 16);
}

__device__ __forceinline__ uint16_t f32_to_fp16(uint32_t b) {
  uint32_t sign = (b >> 16) & 0x8000u;
  int32_t e = int32_t((b >> 23) & 0xFF);
  uint32_t m = b & 0x7FFFFFu;
  uint32_t out = 0;
  if (e >= 113) {
    uint32_t mant = m >> 13, rem = m & 0x1FFFu;
    uint32_t up = (rem > 0x1000u) || (rem == 0x1000u && (mant & 1u));
    out = (uint32_t(e - 112) << 10) + mant + up;
  } else if (e >= 102) {
    uint32_t full = m | 0x800000u;
    uint32_t sh = uint32_t(126 - e);
    uint32_t k = full >> sh;
    uint32_t rem = full & ((1u << sh) - 1u), half = 1u << (sh - 1);
    uint32_t up = (rem > half) || (rem == half && (k & 1u));
    out = k + up;
  }
  return uint16_t(sign | out);
}

enum { KIND_BF16 = 0, KIND_FP16 = 1, KIND_TAG16 = 2, KIND_RAW16 = 3 };

__device__ __forceinline__ uint16_t value16(uint64_t key, uint64_t idx, int kind, float scale) {
  uint64_t w = mix64(key + (idx + 1) * GAMMA);
  if (kind == KIND_TAG16) return uint16_t(w & 0xFFFF);
  if (kind == KIND_RAW16) return uint16_t(w >> 48);
  int32_t s = int32_t((w & 0xFFFF) + ((w >> 16) & 0xFFFF) + ((w >> 32) & 0xFFFF) + (w >> 48)) - 131070;
  float f = __fmul_rn(float(s), scale);
  uint32_t b = __float_as_uint(f);
  return kind == KIND_BF16 ? f32_to_bf16(b) : f32_to_fp16(b);
}

}  // namespace

extern "C" {

// One 3-level region: element (i0, i1, i2) of a full logical tensor with
// flat index idx0 + i0*is0 + i1*is1 + i2*is2 goes to byte
// dst_off + i0*ds0 + i1*ds1 + i2*2 of the buffer.
struct SynthRegion {
  uint64_t key;
  int32_t kind;
  float scale;
  uint64_t dst_off;
  int64_t n0, n1, n2;
  int64_t ds0, ds1;
  int64_t idx0, is0, is1, is2;
};

}

__global__ void k_fill(char *dst, SynthRegion r) {
  const int64_t total = r.n0 * r.n1 * r.n2;
  for (int64_t e = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; e < total; e += int64_t(gridDim.x) * blockDim.x) {
    int64_t i2 = e % r.n2, t = e / r.n2;
    int64_t i1 = t % r.n1, i0 = t / r.n1;
    uint64_t idx = uint64_t(r.idx0 + i0 * r.is0 + i1 * r.is1 + i2 * r.is2);
    uint16_t v = value16(r.key, idx, r.kind, r.scale);
    *reinterpret_cast<uint16_t *>(dst + r.dst_off + i0 * r.ds0 + i1 * r.ds1 + i2 * 2) = v;
  }
}

// KV blocks: item k is (seq[k], blk[k]) written at block position pos[k]
// of a pool with `block_stride` bytes per block; heads [h0, h1) of
// n_kv; layout 0 = [heads][bt][hd], 1 = [bt][heads][hd].
__global__ void k_fill_kv(char *dst, uint64_t base, const int32_t *seq, const int32_t *blk, const int64_t *pos,
                          int64_t n_items, int64_t block_stride, int32_t layout, int32_t h0, int32_t h1,
                          int32_t n_kv, int64_t seq_tokens, int32_t bt, int32_t hd, uint64_t key, int32_t kind,
                          float scale) {
  const int64_t nh = h1 - h0, per = nh * bt * hd, total = n_items * per;
  for (int64_t e = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; e < total; e += int64_t(gridDim.x) * blockDim.x) {
    int64_t k = e / per, r = e % per;
    int64_t h, t, d;
    if (layout == 0) {
      h = r / (int64_t(bt) * hd);
      t = (r / hd) % bt;
    } else {
      t = r / (nh * hd);
      h = (r / hd) % nh;
    }
    d = r % hd;
    int64_t s = seq[k], b = blk[k];
    uint64_t idx = uint64_t(((s * seq_tokens + b * bt + t) * n_kv + (h0 + h)) * hd + d);
    uint16_t v = value16(key, idx, kind, scale);
    *reinterpret_cast<uint16_t *>(dst + base + pos[k] * block_stride + r * 2) = v;
  }
}

extern "C" {

int synth_fill(void *dst, const SynthRegion *regions, int n, void *stream) {
  hipStream_t s = static_cast<hipStream_t>(stream);
  for (int i = 0; i < n; ++i) {
    int64_t total = regions[i].n0 * regions[i].n1 * regions[i].n2;
    if (total <= 0) continue;
    int64_t blocks = (total + 255) / 256;
    if (blocks > 65536) blocks = 65536;
    hipLaunchKernelGGL(k_fill, dim3(unsigned(blocks)), dim3(256), 0, s, static_cast<char *>(dst), regions[i]);
  }
  return int(hipGetLastError());
}

int synth_fill_kv(void *dst, uint64_t base, const int32_t *seq, const int32_t *blk, const int64_t *pos,
                  int64_t n_items, int64_t block_stride, int32_t layout, int32_t h0, int32_t h1, int32_t n_kv,
                  int64_t seq_tokens, int32_t bt, int32_t hd, uint64_t key, int32_t kind, float scale,
                  void *stream) {
  int64_t total = n_items * (h1 - h0) * int64_t(bt) * hd;
  if (total <= 0) return 0;
  int64_t blocks = (total + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  hipLaunchKernelGGL(k_fill_kv, dim3(unsigned(blocks)), dim3(256), 0, static_cast<hipStream_t>(stream),
                     static_cast<char *>(dst), base, seq, blk, pos, n_items, block_stride, layout, h0, h1, n_kv,
                     seq_tokens, bt, hd, key, kind, scale);
  return int(hipGetLastError());
}

}
