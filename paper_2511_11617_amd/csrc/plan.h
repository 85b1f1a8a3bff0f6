// plan.h — host-side planner of the reshard library (no HIP dependency).
//
// Stage 1 of Sec. III-C (logical, topology-agnostic): partitions, the CMM
// loop of Alg. 1 per space and the Eq. 1 statistics.  Then this GPU's share
// is lowered to byte-level copy families and, for an in-place reshard,
// ordered into hazard-free levels with a bounded staging buffer; this is
// the single pre-allocation pass of Sec. III-C (every size is known before
// any byte moves).
#pragma once

#include <stdint.h>

#include <stdexcept>
#include <string>
#include <vector>

#include "../../include/atp.h"
#include "desc.h"

namespace atp {

struct Error : std::runtime_error {
  int code;
  Error(int c, const std::string &m) : std::runtime_error(m), code(c) {}
};

struct Rng {
  int64_t b, e;
};

// A copy family before it becomes a device descriptor.  Offsets are bytes
// relative to the base of the buffer slot named in `flags`.
struct Fam {
  uint64_t src_off = 0, dst_off = 0;
  uint64_t src_pitch = 0, dst_pitch = 0;
  uint64_t src_ostride = 0, dst_ostride = 0;
  int64_t o_begin = 0, o_end = 1;
  uint64_t run = 0, rows = 1;
  uint32_t flags = 0;
  uint64_t bytes() const { return uint64_t(o_end - o_begin) * rows * run; }
};

struct SpacePlan {
  int64_t H = 0;
  int N = 0, M = 0;
  std::vector<Rng> old_r, new_r;
  std::vector<atp_task> tasks;
  uint64_t unit_bytes = 0;  // bytes per unit summed over tensors (+ KV)
};

struct TensorPlan {
  atp_tensor t;
  Rng old_r, new_r;
  uint64_t old_off = 0, new_off = 0, old_bytes = 0, new_bytes = 0;
};

// One kernel launch over a contiguous descriptor range.
struct Launch {
  int level = 0;
  int kind = 0;        // 0 repack, 2 scatter, 3 outbound read, 4 host read
  bool aligned = true;
  bool wide = false;   // aligned, with tiles of kWideTileChunks (DF_WIDE)
  int d0 = 0, d1 = 0;
  uint64_t bytes = 0;  // bytes copied (upper bound for block ranges)
  uint64_t tiles_max = 0;
  std::vector<int> wait_outbound;  // outbound copies that must finish first
};

// Host <-> device copy of packed bytes.
struct HostCopy {
  uint64_t host_off = 0;
  uint64_t dev_off = 0;       // device offset (arena or staging slot)
  uint64_t bytes = 0;
  int dev_buf = BUF_OUT;      // BUF_OUT for direct landing, BUF_STAGE ring
  // while planning a landing in place: the last level that reads its
  // destination and the number of outbound copies (in issue order) that must
  // finish first; a planned direct landing always has neither
  int gate_level = -1;
  int gate_pos = 0;
  // strided device side (outbound): rows x run at dev pitch
  uint64_t rows = 1, run = 0, dev_pitch = 0;
};

// Landing-ring chunk: H2D into a slot, then scatter launch(es) from it.
struct Chunk {
  int slot = 0;
  std::vector<HostCopy> copies;   // into the slot
  std::vector<Launch> scatters;   // aligned and/or 2-byte-granular
};

// Everything one reshard call (weights or KV) executes.
struct CallPlan {
  std::vector<Fam> fams;        // final families, index = descriptor index
  std::vector<Launch> levels;   // repack launches in order
  std::vector<HostCopy> directs;
  std::vector<Chunk> chunks;
  std::vector<HostCopy> outbound;
  std::vector<int> out_order;   // outbound issue order (by the level needing it)
  // Inflow other than large contiguous gaps is read by the copy kernel
  // straight from the pinned inflow buffer (host_reads): out of place from
  // the call's start, in place after the call's last level.  In place, no
  // host-to-device copy command waits long for an event: such a command
  // holds up every later host-to-device copy of the process on the DMA
  // engine (the in-place KV inflow takes the landing ring, which waits only
  // for its own scatters).  The weights' outbound
  // reads are copy-kernel descriptors too (out_d0 + k for position k of
  // out_order), writing straight into the pinned outbound buffer: the
  // runtime's own device-to-host copies are wide blit kernels that starve
  // the HBM-bound repack beside them.
  std::vector<Launch> host_reads;
  int out_d0 = -1;
  std::vector<uint64_t> out_tiles;
  std::vector<uint8_t> out_aligned;
  std::vector<atp_segment> seg_in, seg_out;
  int n_levels = 0;
  uint64_t retained = 0, moved = 0, staged = 0, tail = 0;
  uint64_t inflow = 0, outbound_bytes = 0;
  // staging layout
  uint64_t off_meta = 0, off_desc = 0, off_prefix = 0, off_kvflags = 0,
           off_kvpref = 0, off_kvlive = 0, off_ring = 0, off_stage = 0,
           ring_slot = 0, staging_need = 0;
  int n_slots = 0;
  uint64_t old_bytes = 0, new_bytes = 0;
};

struct Plan {
  atp_problem prob{};
  std::vector<atp_space> spaces_in;
  std::vector<atp_tensor> tensors_in;
  atp_kv kv{};
  bool has_kv = false;
  std::vector<int> failed;
  int flags = 0;
  bool inplace = false;

  std::vector<SpacePlan> sp;
  std::vector<TensorPlan> tp;
  std::vector<int> owner;  // owner[j] = old rank hosting target j
  int self_old = 0, self_new = 0;

  CallPlan w, k;
  atp_stats stats{};
  double plan_ms = 0;

  void *exec = nullptr;  // executor state (exec.hip)
  // read statistics of the last atp_load_reshard_weights_async, once synced
  atp_load_stats load_stats{};
  bool load_stats_valid = false;
};

// Build a plan; throws Error.
Plan *make_plan(const atp_problem *p);
void partition(int64_t total, int parts, int rule, std::vector<Rng> &out);

}  // namespace atp
