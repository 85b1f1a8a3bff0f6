// desc.h — copy descriptors shared by the host planner and the gfx950
// kernels of the reshard library.
//
// A descriptor is one copy family (Sec. III-C: tasks on interval boundaries,
// lowered to bytes):
//   for every outer item o in [o_begin, o_end)
//     for every line t in [0, rows)
//       copy `run` bytes
//         from src_base + src_off + idx_src(o) * src_ostride + t * src_pitch
//         to   dst_base + dst_off + idx_dst(o) * dst_ostride + t * dst_pitch
// where idx(o) = o - o_begin on a direct side and live[o] (a physical KV
// block id from the compacted block table) on an indirect side.  Weight
// tensors use outer items = rows of the matrix; KV uses outer items = live
// blocks and lines = tokens (token-major) or one line per block.
#pragma once
#include <stdint.h>

namespace atp {

// base-pointer slots a descriptor reads from / writes to
enum : uint32_t { BUF_IN = 0, BUF_OUT = 1, BUF_STAGE = 2 };

enum : uint32_t {
  DF_SRC_SHIFT = 0,       // 2 bits: source buffer slot
  DF_DST_SHIFT = 2,       // 2 bits: destination buffer slot
  DF_SRC_IND = 1u << 4,   // source index through the live-block list
  DF_DST_IND = 1u << 5,   // destination index through the live-block list
  DF_BLOCKRANGE = 1u << 6,// [o_begin, o_end) are block ids; the prepare
                          // kernel rewrites them as live-list positions
  DF_ALIGNED = 1u << 7,   // every offset, pitch, stride and run is a
                          // multiple of 16: the 16-byte vector kernel
  DF_WIDE = 1u << 8,      // aligned, tiled kWideUnroll chunks per thread
};

// Launch shape of the vector kernel: 256 threads, ATP_UNROLL independent
// 16-byte chunks per thread per tile; one workgroup per tile unless
// ATP_PERSIST (grid-stride over tiles with a fixed grid).
#ifndef ATP_UNROLL
#define ATP_UNROLL 2
#endif
#ifndef ATP_PERSIST
#define ATP_PERSIST 0
#endif
#ifndef ATP_NT_LOAD
#define ATP_NT_LOAD 1
#endif
#ifndef ATP_NT_STORE
#define ATP_NT_STORE 1
#endif
#ifndef ATP_XCD_MAP
#define ATP_XCD_MAP 1
#endif
constexpr int kThreads = 256;
constexpr int kUnroll = ATP_UNROLL;
constexpr int64_t kTileChunks = kThreads * kUnroll;
// Short aligned KV lines (a head of one block, 4 KiB or less) take tiles
// twice as wide, which keeps more bytes in flight per thread: the largest KV
// level of the 80-layer TP 8->7 reshard ran 5 % faster so, while the
// weights' long lines ran slower.
constexpr int kWideUnroll = 2 * ATP_UNROLL;
constexpr int64_t kWideTileChunks = kThreads * kWideUnroll;
constexpr uint64_t kWideMaxRun = 4096;
// 16-byte chunks per tile of a vector-kernel descriptor
constexpr int64_t tile_chunks(uint32_t flags) { return (flags & DF_WIDE) ? kWideTileChunks : kTileChunks; }
// bytes per tile of the 2-byte-granular (LDS funnel-shift) kernel
constexpr int64_t kSegBytes = 8192;

struct alignas(16) Desc {
  uint64_t src_off, dst_off;
  uint64_t src_pitch, dst_pitch;
  uint64_t src_ostride, dst_ostride;
  int64_t o_begin, o_end;
  uint32_t run, rows;
  uint32_t flags, pad;
  // exact 32-bit division by a host-known divisor d >= 2:
  // q = umulhi64(n, m) with m = ceil(2^64 / d); m = 0 means d == 1
  uint64_t magic_line;  // divisor: 16-byte chunks per line (vector kernel)
                        //          or segments per line (2-byte kernel)
  uint64_t magic_rows;  // divisor: rows
};

static_assert(sizeof(Desc) == 96, "descriptor layout");

}  // namespace atp
