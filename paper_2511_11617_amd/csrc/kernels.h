// kernels.h — gfx950 (CDNA4) kernels of the reshard library.
//
// The reshard moves bytes without arithmetic, so every kernel here is bound
// by HBM bandwidth; there is no matrix work and no MFMA.
//   k_prepare     one workgroup turns the plan into per-tile work: it
//                 compacts the block table into the sorted list of live
//                 blocks (wavefront prefix sums over block flags), resolves
//                 block-id ranges into list positions and scans the tile
//                 counts of every descriptor (wavefront prefix sums).
//   k_copy16      descriptor-driven copy in 16-byte chunks, 2 independent
//                 loads in flight per thread, non-temporal hints; a tile is
//                 512 consecutive chunks (8 KiB) of one descriptor.
//   k_copy_bytes  the same for runs that are not 16-byte aligned (odd
//                 column counts): a tile stages one 8 KiB line segment in
//                 LDS with aligned 16-byte loads and writes it out with
//                 aligned 16-byte stores, funnel-shifting bytes between
//                 neighbouring LDS words; ragged ends use byte stores.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "desc.h"

namespace atp {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

enum : int32_t { ERR_BAD_BLOCK = 1, ERR_LIVE_COUNT = 2 };

__device__ __forceinline__ uint32_t divq(uint32_t n, uint64_t magic) {
  return magic ? uint32_t(__umul64hi(uint64_t(n), magic)) : n;
}

__device__ __forceinline__ char *slot_base(uint32_t slot, char *b0, char *b1, char *b2) {
  return slot == BUF_IN ? b0 : (slot == BUF_OUT ? b1 : b2);
}

// Exclusive prefix sum over the 1024 threads of a workgroup (wave64 scans
// with lane shuffles, then one scan of the 16 wave totals).
template <typename T>
__device__ T block_exclusive_scan(T v, T *lds16, T *total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
  T x = v;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    T y = __shfl_up(x, d, 64);
    if (lane >= d) x += y;
  }
  if (lane == 63) lds16[wave] = x;
  __syncthreads();
  if (wave == 0) {
    T w = lane < nw ? lds16[lane] : T(0);
#pragma unroll
    for (int d = 1; d < 16; d <<= 1) {
      T y = __shfl_up(w, d, 64);
      if (lane >= d) w += y;
    }
    if (lane < nw) lds16[lane] = w;
  }
  __syncthreads();
  T base = wave ? lds16[wave - 1] : T(0);
  *total = lds16[nw - 1];
  __syncthreads();
  return base + x - v;
}

struct PrepArgs {
  Desc *descs;
  int32_t n_desc;
  int32_t kv;            // 1: compact the block table first
  int64_t *prefix;       // [n_desc + 1] tile prefix
  int32_t *err;          // error word (meta area)
  const int32_t *table;  // block table, n_entries int32
  int64_t n_entries;
  int32_t *flags;        // [n_blocks]
  int32_t *pref;         // [n_blocks + 1]
  int32_t *live;         // [n_blocks] sorted live block ids
  int64_t n_blocks;
  int64_t expect_live;
};

__global__ void __launch_bounds__(1024) k_prepare(PrepArgs a) {
  __shared__ int64_t s64[16];
  __shared__ int32_t s32[16];
  __shared__ int32_t s_err;
  const int tid = threadIdx.x, nt = blockDim.x;
  if (tid == 0) s_err = 0;
  __syncthreads();
  if (a.kv) {
    for (int64_t p = tid; p < a.n_blocks; p += nt) a.flags[p] = 0;
    __syncthreads();
    for (int64_t e = tid; e < a.n_entries; e += nt) {
      int32_t v = a.table[e];
      if (v >= 0) {
        if (v < a.n_blocks)
          a.flags[v] = 1;
        else
          atomicOr(&s_err, ERR_BAD_BLOCK);
      }
    }
    __syncthreads();
    // compact: pref = exclusive scan of flags, live[pref[p]] = p
    int64_t per = (a.n_blocks + nt - 1) / nt;
    int64_t p0 = tid * per, p1 = p0 + per < a.n_blocks ? p0 + per : a.n_blocks;
    int32_t sum = 0;
    for (int64_t p = p0; p < p1; ++p) sum += a.flags[p];
    int32_t tot;
    int32_t run = block_exclusive_scan<int32_t>(sum, s32, &tot);
    for (int64_t p = p0; p < p1; ++p) {
      a.pref[p] = run;
      if (a.flags[p]) a.live[run++] = int32_t(p);
    }
    if (tid == 0) {
      a.pref[a.n_blocks] = tot;
      if (tot != a.expect_live) atomicOr(&s_err, ERR_LIVE_COUNT);
    }
    __syncthreads();
  }
  const bool bad = s_err != 0;
  // resolve block ranges, count tiles, scan
  int64_t per = (a.n_desc + nt - 1) / nt;
  int64_t d0 = tid * per, d1 = d0 + per < a.n_desc ? d0 + per : a.n_desc;
  int64_t sum = 0;
  for (int64_t d = d0; d < d1; ++d) {
    Desc &x = a.descs[d];
    if (x.flags & DF_BLOCKRANGE) {
      int64_t b0 = x.o_begin < 0 ? 0 : (x.o_begin > a.n_blocks ? a.n_blocks : x.o_begin);
      int64_t b1 = x.o_end < 0 ? 0 : (x.o_end > a.n_blocks ? a.n_blocks : x.o_end);
      x.o_begin = a.pref[b0];
      x.o_end = b1 > b0 ? a.pref[b1] : x.o_begin;
      x.flags &= ~DF_BLOCKRANGE;
    }
    if (bad) x.o_end = x.o_begin;  // an invalid table moves nothing
    uint64_t lines = uint64_t(x.o_end - x.o_begin) * x.rows;
    uint64_t tiles;
    if (x.flags & DF_ALIGNED)
      tiles = (lines * (x.run >> 4) + tile_chunks(x.flags) - 1) / tile_chunks(x.flags);
    else
      tiles = lines * ((x.run + kSegBytes - 1) / kSegBytes);
    a.prefix[d] = int64_t(tiles);  // temporarily the count
    sum += int64_t(tiles);
  }
  int64_t tot;
  int64_t run = block_exclusive_scan<int64_t>(sum, s64, &tot);
  for (int64_t d = d0; d < d1; ++d) {
    int64_t c = a.prefix[d];
    a.prefix[d] = run;
    run += c;
  }
  if (tid == 0) {
    a.prefix[a.n_desc] = tot;
    *a.err = s_err;
  }
}

// Descriptor of tile t: the last d in [d0, d1) with prefix[d] <= t.
__device__ __forceinline__ int find_desc(const int64_t *__restrict__ prefix, int d0, int d1, int64_t t) {
  int lo = d0, hi = d1 - 1;
  while (lo < hi) {
    int mid = (lo + hi + 1) >> 1;
    if (prefix[mid] <= t)
      lo = mid;
    else
      hi = mid - 1;
  }
  return lo;
}

struct LineAddr {
  char *src, *dst;
};

// The live-block list and the descriptors are never written while a copy
// kernel runs, so a wave-uniform index may read them through the scalar
// cache (constant address space) instead of a per-lane vector load.
typedef const int32_t __attribute__((address_space(4))) *const_i32_p;

// Addresses of line `line` of descriptor x.  UNIFORM: `line` is the same on
// every lane of the wave, and the block id comes in through a scalar load.
template <bool UNIFORM>
__device__ __forceinline__ LineAddr line_addr(const Desc &x, uint32_t line, char *b0, char *b1, char *b2,
                                              const int32_t *__restrict__ live) {
  uint32_t orel = divq(line, x.magic_rows);
  uint32_t r = line - orel * x.rows;
  int64_t o = x.o_begin + orel;
  uint64_t id = 0;
  if (x.flags & (DF_SRC_IND | DF_DST_IND))
    id = UNIFORM ? uint64_t(((const_i32_p)(live))[o]) : uint64_t(live[o]);
  uint64_t si = (x.flags & DF_SRC_IND) ? id : uint64_t(orel);
  uint64_t di = (x.flags & DF_DST_IND) ? id : uint64_t(orel);
  char *sb = slot_base((x.flags >> DF_SRC_SHIFT) & 3, b0, b1, b2);
  char *db = slot_base((x.flags >> DF_DST_SHIFT) & 3, b0, b1, b2);
  LineAddr la;
  la.src = sb + x.src_off + si * x.src_ostride + uint64_t(r) * x.src_pitch;
  la.dst = db + x.dst_off + di * x.dst_ostride + uint64_t(r) * x.dst_pitch;
  return la;
}

// Streaming 16-byte accesses: nothing is read twice, so both sides carry
// the non-temporal hint by default.  The pointers are cast to the global
// address space, which keeps the accesses global_* rather than flat_*
// where the compiler cannot infer it.
typedef u32x4 __attribute__((address_space(1))) global_u32x4;

__device__ __forceinline__ u32x4 load16(const u32x4 *p) {
#if ATP_NT_LOAD
  return __builtin_nontemporal_load((const global_u32x4 *)(p));
#else
  return *(const global_u32x4 *)(p);
#endif
}

__device__ __forceinline__ void store16(u32x4 *p, u32x4 v) {
#if ATP_NT_STORE
  __builtin_nontemporal_store(v, (global_u32x4 *)(p));
#else
  *(global_u32x4 *)(p) = v;
#endif
}

// First tile of this workgroup.  Workgroups are dealt round-robin to the
// 8 XCDs; with ATP_XCD_MAP each XCD gets a contiguous run of tiles instead
// of every 8th one.
__device__ __forceinline__ int64_t tile_of_block() {
#if ATP_XCD_MAP
  const uint32_t G = gridDim.x, b = blockIdx.x, q = G >> 3, r = G & 7, xcd = b & 7, i = b >> 3;
  return xcd < r ? int64_t(xcd) * (q + 1) + i : int64_t(r) * (q + 1) + int64_t(xcd - r) * q + i;
#else
  return blockIdx.x;
#endif
}

// Each tile resolves every address first (descriptor by value, block ids
// through scalar loads), then issues all of its loads, then all stores, so
// that no load waits behind another's address computation.  Lanes past the
// end of the tile load its last chunk again (a valid address) and store
// nothing: unconditional loads keep the compiler from waiting on each one.
// U chunks per thread: every descriptor of a launch has DF_WIDE exactly when
// U == kWideUnroll (the prepare kernel counted its tiles that way).
template <int U>
__global__ void __launch_bounds__(kThreads) k_copy16(const Desc *__restrict__ descs, const int64_t *__restrict__ prefix,
                                                     int d0, int d1, char *b0, char *b1, char *b2,
                                                     const int32_t *__restrict__ live) {
  constexpr int64_t kTile = int64_t(kThreads) * U;
  const int64_t T0 = prefix[d0], T1 = prefix[d1];
  for (int64_t t = T0 + tile_of_block(); t < T1; t += gridDim.x) {
    const int d = find_desc(prefix, d0, d1, t);
    const Desc x = descs[d];
    const uint32_t cpl = x.run >> 4;
    const uint64_t total = uint64_t(x.o_end - x.o_begin) * x.rows * cpl;
    const uint64_t cbase = uint64_t(t - prefix[d]) * kTile;
    const uint64_t clast = (cbase + kTile < total ? cbase + kTile : total) - 1;
    const uint32_t l0 = divq(uint32_t(cbase), x.magic_line);
    u32x4 v[U];
    if (l0 == divq(uint32_t(clast), x.magic_line)) {
      // the whole tile lies in one line: one address computation per tile
      const LineAddr la = line_addr<true>(x, l0, b0, b1, b2, live);
      const uint32_t col0 = uint32_t(cbase) - l0 * cpl;
      const uint32_t n = uint32_t(clast - cbase) + 1;
      const u32x4 *s = reinterpret_cast<const u32x4 *>(la.src) + col0;
      u32x4 *dd = reinterpret_cast<u32x4 *>(la.dst) + col0;
#pragma unroll
      for (int k = 0; k < U; ++k) {
        const uint32_t i = threadIdx.x + k * kThreads;
        v[k] = load16(s + (i < n ? i : n - 1));
      }
#pragma unroll
      for (int k = 0; k < U; ++k) {
        const uint32_t i = threadIdx.x + k * kThreads;
        if (i < n) store16(dd + i, v[k]);
      }
      continue;
    }
    // several lines per tile: resolve the line once per wavefront when its
    // 64 chunks share one (short KV head runs), else per lane
    const u32x4 *sp[U];
    u32x4 *dp[U];
    const uint32_t wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
#pragma unroll
    for (int k = 0; k < U; ++k) {
      const uint64_t g0r = cbase + uint64_t(k) * kThreads + wv * 64;
      const uint64_t g0 = g0r < clast ? g0r : clast;
      const uint64_t gl = g0r + 63 < clast ? g0r + 63 : clast;
      const uint64_t cr = cbase + threadIdx.x + uint64_t(k) * kThreads;
      const uint64_t c = cr < clast ? cr : clast;
      const uint32_t lf = divq(uint32_t(g0), x.magic_line);
      if (lf == divq(uint32_t(gl), x.magic_line)) {
        const LineAddr la = line_addr<true>(x, lf, b0, b1, b2, live);
        const uint32_t col = uint32_t(c) - lf * cpl;
        sp[k] = reinterpret_cast<const u32x4 *>(la.src) + col;
        dp[k] = reinterpret_cast<u32x4 *>(la.dst) + col;
      } else {
        const uint32_t line = divq(uint32_t(c), x.magic_line);
        const uint32_t col = uint32_t(c) - line * cpl;
        const LineAddr la = line_addr<false>(x, line, b0, b1, b2, live);
        sp[k] = reinterpret_cast<const u32x4 *>(la.src) + col;
        dp[k] = reinterpret_cast<u32x4 *>(la.dst) + col;
      }
    }
#pragma unroll
    for (int k = 0; k < U; ++k) v[k] = load16(sp[k]);
#pragma unroll
    for (int k = 0; k < U; ++k)
      if (cbase + threadIdx.x + uint64_t(k) * kThreads <= clast) store16(dp[k], v[k]);
  }
}

__global__ void __launch_bounds__(kThreads) k_copy_bytes(const Desc *__restrict__ descs,
                                                         const int64_t *__restrict__ prefix, int d0, int d1, char *b0,
                                                         char *b1, char *b2, const int32_t *__restrict__ live) {
  __shared__ uint32_t lds[kSegBytes / 4 + 16];
  const int64_t T0 = prefix[d0], T1 = prefix[d1];
  const int tid = threadIdx.x;
  for (int64_t t = T0 + blockIdx.x; t < T1; t += gridDim.x) {
    const int d = find_desc(prefix, d0, d1, t);
    const Desc x = descs[d];
    const uint32_t spl = uint32_t((x.run + kSegBytes - 1) / kSegBytes);
    const uint32_t tin = uint32_t(t - prefix[d]);
    const uint32_t line = divq(tin, x.magic_line);
    const uint32_t seg = tin - line * spl;
    LineAddr la = line_addr<true>(x, line, b0, b1, b2, live);
    const uint64_t skip = uint64_t(seg) * kSegBytes;
    const char *src = la.src + skip;
    char *dst = la.dst + skip;
    const uint32_t n = uint32_t((x.run - skip) < uint64_t(kSegBytes) ? (x.run - skip) : kSegBytes);
    // stage [src, src + n) through LDS in aligned 16-byte groups
    const uintptr_t s_al = uintptr_t(src) & ~uintptr_t(15);
    const uint32_t head = uint32_t(uintptr_t(src) - s_al);
    const uint32_t ngroups = (head + n + 15) >> 4;
    for (uint32_t g = tid; g < ngroups; g += kThreads) {
      u32x4 w = *reinterpret_cast<const u32x4 *>(s_al + 16 * uintptr_t(g));
      lds[4 * g + 0] = w.x;
      lds[4 * g + 1] = w.y;
      lds[4 * g + 2] = w.z;
      lds[4 * g + 3] = w.w;
    }
    __syncthreads();
    const uintptr_t d_lo = uintptr_t(dst), d_hi = d_lo + n;
    uintptr_t a_lo = (d_lo + 15) & ~uintptr_t(15), a_hi = d_hi & ~uintptr_t(15);
    if (a_lo > a_hi) a_lo = a_hi = d_hi;  // no whole aligned chunk inside
    const uint32_t nfull = uint32_t((a_hi - a_lo) >> 4);
    for (uint32_t ch = tid; ch < nfull; ch += kThreads) {
      const uint32_t off = head + uint32_t(a_lo - d_lo) + 16 * ch;  // byte offset in the staged window
      const uint32_t w0 = off >> 2, sh = off & 3;
      u32x4 o;
      if (sh == 0) {
        o.x = lds[w0];
        o.y = lds[w0 + 1];
        o.z = lds[w0 + 2];
        o.w = lds[w0 + 3];
      } else {
        const uint32_t l0 = lds[w0], l1 = lds[w0 + 1], l2 = lds[w0 + 2], l3 = lds[w0 + 3], l4 = lds[w0 + 4];
        o.x = __builtin_amdgcn_alignbyte(l1, l0, sh);
        o.y = __builtin_amdgcn_alignbyte(l2, l1, sh);
        o.z = __builtin_amdgcn_alignbyte(l3, l2, sh);
        o.w = __builtin_amdgcn_alignbyte(l4, l3, sh);
      }
      __builtin_nontemporal_store(o, reinterpret_cast<u32x4 *>(a_lo) + ch);
    }
    // ragged ends, one byte per thread
    const uint32_t nhead = uint32_t(a_lo - d_lo), ntail = uint32_t(d_hi - a_hi);
    const unsigned char *lb = reinterpret_cast<const unsigned char *>(lds);
    for (uint32_t i = tid; i < nhead + ntail; i += kThreads) {
      const uint32_t pos = i < nhead ? i : uint32_t(a_hi - d_lo) + (i - nhead);
      reinterpret_cast<unsigned char *>(d_lo)[pos] = lb[head + pos];
    }
    __syncthreads();
  }
}

}  // namespace atp
