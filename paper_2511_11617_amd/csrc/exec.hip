// exec.hip — executor of the reshard library (Sec. III-C physical stage on
// one GPU): uploads the plan's descriptors into the caller's staging
// buffer, launches the prepare and repack kernels level by level, lands the
// missing bytes from the pinned host buffer (DMA copies of large contiguous
// gaps straight into place; every other piece read by the copy kernel from
// the host buffer, out of place beside the repack on a side stream that
// feeds a hardware queue of its own, in place after the last level; the
// in-place KV inflow through the landing ring plus a scatter kernel), reads
// dropped outbound bytes out before an in-place overwrite (the copy kernel
// writing the host buffer, on the side stream), and orders all of it with
// HIP events.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <chrono>
#include <map>
#include <memory>
#include <mutex>
#include <cstdio>
#include <cstring>
#include <string>
#include <tuple>
#include <vector>

#include "exec.h"
#include "kernels.h"
#include "plan.h"

namespace atp {
namespace {

// A failed call also stays the thread's last HIP error, which the caller's
// next launch check (torch's, say) would report as its own: the error is
// reported here, so it is cleared.
void hip_check(hipError_t e, const char *what) {
  if (e == hipSuccess) return;
  (void)hipGetLastError();
  throw Error(ATP_EHIP, std::string(what) + ": " + hipGetErrorString(e));
}
#define HIPCHK(x) hip_check((x), #x)

uint64_t magic_of(uint64_t d) {
  if (d <= 1) return 0;
  unsigned __int128 m = ((((unsigned __int128)1) << 64) + d - 1) / d;  // ceil(2^64 / d)
  return uint64_t(m);
}

// A half-open byte range of device memory a call touches.
struct Span {
  uintptr_t b = 0, e = 0;
  bool meets(const Span &o) const { return b < e && o.b < o.e && b < o.e && o.b < e; }
};

struct CallState {
  bool pending = false;
  bool on_scratch = false;  // the pending call runs on the device's scratch array
  Span old_arena, new_arena, staging;  // what the pending call reads and writes
  Desc *desc_host = nullptr;  // pinned copy of the descriptors
  size_t desc_cap = 0;
  int32_t *err_host = nullptr;  // pinned error word
  hipEvent_t start = nullptr;  // marks the caller's work queued before the call
  hipEvent_t tail_compute = nullptr, tail_copy = nullptr, tail_side = nullptr;
  hipEvent_t rep0 = nullptr, rep1 = nullptr, h2d0 = nullptr, h2d1 = nullptr, d2h0 = nullptr, d2h1 = nullptr;
  hipEvent_t hr1 = nullptr;  // end of the copy kernel's host reads (inflow ends with the later of h2d1, hr1)
  struct LaunchRec {
    int kind, level;
    uint64_t bytes;
    hipEvent_t e0, e1;
  };
  std::vector<LaunchRec> launches;
  uint64_t h2d_bytes = 0, d2h_bytes = 0, scatter_bytes = 0, repack_bytes = 0;
  hipStream_t compute = nullptr, copy = nullptr;  // the caller's streams of the pending call
  // A weights call whose inflow buffer is still being read: its awaited
  // pieces are issued by atp_sync (then the tails are recorded again).
  std::function<void()> finish_issue;
};

// Process-wide recycling of HIP objects per device.  Each plan owns what it
// takes until it is freed; creating events, streams and pinned buffers for
// every plan would otherwise cost tens of milliseconds per reshard.
struct DevicePool {
  std::vector<hipEvent_t> sync_ev, time_ev;
  std::vector<hipStream_t> streams;  // side streams (choose_side); never destroyed, so that no new
                                     // stream reuses a handle the probe cache knows
  std::vector<std::pair<void *, size_t>> pinned;
};
std::mutex g_pool_mu;
std::map<int, DevicePool> g_pools;

struct Exec {
  int device = -1;
  int grid_max = 2048;
  // Set while a call of the no-allocation entry point is being issued:
  // events, pinned buffers and the side stream then come from the pools
  // atp_warmup filled, and running short is an error, not an allocation.
  bool no_alloc = false;
  // In place: `side` runs the outbound gathers and their device-to-host
  // copies, the weight levels that wait for them and the weight inflow the
  // copy kernel reads after them.  Out of place it runs the copy kernel's
  // host reads.  It feeds another hardware queue than the caller's streams
  // and is shared process-wide (choose_side).
  hipStream_t side = nullptr;
  hipStream_t side_for_compute = nullptr, side_for_copy = nullptr;
  std::vector<hipEvent_t> sync_pool, time_pool;
  size_t sync_used = 0, time_used = 0;
  CallState w, k;
  bool wall_started = false;
  std::chrono::steady_clock::time_point wall0;
  atp_timing last{};
  std::vector<atp_launch> last_launches;

  hipEvent_t ev_sync() {
    if (sync_used == sync_pool.size()) {
      hipEvent_t e = nullptr;
      {
        std::lock_guard<std::mutex> g(g_pool_mu);
        auto &v = g_pools[device].sync_ev;
        if (!v.empty()) {
          e = v.back();
          v.pop_back();
        }
      }
      if (!e && no_alloc) throw Error(ATP_ESTATE, "no pooled event left: call atp_warmup with more events first");
      if (!e) HIPCHK(hipEventCreateWithFlags(&e, hipEventDisableTiming));
      sync_pool.push_back(e);
    }
    return sync_pool[sync_used++];
  }
  hipEvent_t ev_time() {
    if (time_used == time_pool.size()) {
      hipEvent_t e = nullptr;
      {
        std::lock_guard<std::mutex> g(g_pool_mu);
        auto &v = g_pools[device].time_ev;
        if (!v.empty()) {
          e = v.back();
          v.pop_back();
        }
      }
      if (!e && no_alloc) throw Error(ATP_ESTATE, "no pooled event left: call atp_warmup with more events first");
      if (!e) HIPCHK(hipEventCreate(&e));
      time_pool.push_back(e);
    }
    return time_pool[time_used++];
  }
  void *pinned(size_t bytes, size_t *cap) {
    {
      std::lock_guard<std::mutex> g(g_pool_mu);
      auto &v = g_pools[device].pinned;
      size_t best = v.size();  // the smallest pooled buffer that fits
      for (size_t i = 0; i < v.size(); ++i)
        if (v[i].second >= bytes && (best == v.size() || v[i].second < v[best].second)) best = i;
      if (best < v.size()) {
        void *p = v[best].first;
        *cap = v[best].second;
        v.erase(v.begin() + long(best));
        return p;
      }
    }
    if (no_alloc)
      throw Error(ATP_ESTATE, "no pooled pinned buffer of " + std::to_string(bytes) +
                                  " bytes: call atp_warmup on this device first");
    void *p = nullptr;
    HIPCHK(hipHostMalloc(&p, bytes, hipHostMallocDefault));
    *cap = bytes;
    return p;
  }
  ~Exec() {
    // hand everything back for the next plan on this device
    std::lock_guard<std::mutex> g(g_pool_mu);
    DevicePool &pl = g_pools[device];
    pl.sync_ev.insert(pl.sync_ev.end(), sync_pool.begin(), sync_pool.end());
    pl.time_ev.insert(pl.time_ev.end(), time_pool.begin(), time_pool.end());
    for (CallState *c : {&w, &k}) {
      if (c->desc_host) pl.pinned.push_back({c->desc_host, c->desc_cap * sizeof(Desc)});
      if (c->err_host) pl.pinned.push_back({c->err_host, 256});
    }
  }
};

Exec &exec_of(Plan &P) {
  if (!P.exec) {
    Exec *e = new Exec();
    HIPCHK(hipGetDevice(&e->device));
    int cus = 0;
    HIPCHK(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, e->device));
    e->grid_max = std::max(1, cus) * 8;
    P.exec = e;
  }
  return *static_cast<Exec *>(P.exec);
}

// ---- hardware queues -------------------------------------------------------------
// HIP feeds every stream of a process into one of a few hardware queues (four
// by default), and a queue runs its commands in order whichever stream they
// came from.  A stream that waits for 200 ms of outbound reads therefore
// stalls every other stream on its queue.  Whether two streams share a queue
// is observed directly: an empty kernel on `b` finishes before a bounded
// spin kernel queued on `a` ends only if the two queues differ.

__global__ void k_spin(uint32_t iters) {
  for (uint32_t i = 0; i < iters; ++i) __builtin_amdgcn_s_sleep(127);  // about 8 K clocks each
}
__global__ void k_nop() {}

// The probe sits on the first reshard of a process (per caller stream pair),
// so it is kept short: on another queue the empty kernel ends within
// microseconds of its launch, on the same queue only after the spin.
constexpr uint32_t kSpinIters = 100;     // about 0.34 ms at 2.4 GHz
constexpr float kSpinMarginMs = 0.15f;   // the empty kernel must finish this much earlier

// Workgroups of the launches that move bytes over PCIe with the copy kernel
// (persistent grids over their tiles).  Host reads: 32 workgroups carry a
// full x16 Gen5 link from pinned host memory (57 GB/s; 16 reach 50).  The
// long-latency host reads they keep in flight slow an HBM-bound repack
// running beside them, the more the wider the grid: the 40-layer TP 4->3
// repack ran at 6.14 / 5.97 / 5.55 / 2.63 / 1.12 TB/s beside 32 / 48 / 64 /
// 80 / 128 host-read workgroups (6.2 alone).  The outbound reads get a narrow
// grid: wide device-to-host writers (the runtime's 512-workgroup blits)
// slowed a concurrent HBM-bound repack several-fold; 8 workgroups leave a
// concurrent HBM copy at full speed while writing 17 GB/s beside it (41 GB/s
// alone).
#ifndef ATP_HOST_READ_GRID
#define ATP_HOST_READ_GRID 32
#endif
constexpr uint64_t kHostReadGrid = ATP_HOST_READ_GRID;
constexpr uint64_t kOutboundGrid = 8;
// host-read launch pieces while the inflow buffer is still being filled
constexpr uint64_t kPipeBytes = 64ull << 20;
std::map<std::pair<hipStream_t, hipStream_t>, bool> g_same_queue;  // under g_pool_mu

bool same_queue(Exec &E, hipStream_t a, hipStream_t b) {
  if (a == b) return true;
  {
    std::lock_guard<std::mutex> g(g_pool_mu);
    auto it = g_same_queue.find({a, b});
    if (it != g_same_queue.end()) return it->second;
  }
  hipEvent_t ea = E.ev_time(), eb = E.ev_time();
  hipLaunchKernelGGL(k_spin, dim3(1), dim3(64), 0, a, kSpinIters);
  HIPCHK(hipGetLastError());
  HIPCHK(hipEventRecord(ea, a));
  hipLaunchKernelGGL(k_nop, dim3(1), dim3(64), 0, b);
  HIPCHK(hipGetLastError());
  HIPCHK(hipEventRecord(eb, b));
  HIPCHK(hipEventSynchronize(ea));
  HIPCHK(hipEventSynchronize(eb));
  float ms = 0;
  HIPCHK(hipEventElapsedTime(&ms, eb, ea));  // spin end minus empty-kernel end
  const bool same = ms < kSpinMarginMs;
  std::lock_guard<std::mutex> g(g_pool_mu);
  g_same_queue[{a, b}] = g_same_queue[{b, a}] = same;
  return same;
}

// The side stream for a pair of caller streams: one on a hardware queue that
// neither caller stream uses, chosen once per (device, compute, copy) and
// shared by every plan (work from several plans on it is merely serialised).
// Candidates are the device's earlier side streams first, then new ones, at
// most kSideStreams per device in all.  When none qualifies, the first is
// used and the outbound work then holds up the caller's stream on that queue
// (the reshard stays correct).
constexpr size_t kSideStreams = 8;
std::map<std::tuple<int, hipStream_t, hipStream_t>, hipStream_t> g_side;  // under g_pool_mu

void choose_side(Exec &E, hipStream_t compute, hipStream_t copy) {
  if (E.side && E.side_for_compute == compute && E.side_for_copy == copy) return;
  const auto key = std::make_tuple(E.device, compute, copy);
  std::vector<hipStream_t> known;
  {
    std::lock_guard<std::mutex> g(g_pool_mu);
    auto it = g_side.find(key);
    if (it != g_side.end()) {
      E.side = it->second;
      E.side_for_compute = compute;
      E.side_for_copy = copy;
      return;
    }
    known = g_pools[E.device].streams;
  }
  hipStream_t pick = nullptr;
  for (size_t i = 0; !pick; ++i) {
    hipStream_t s = nullptr;
    if (i < known.size()) {
      s = known[i];
    } else if (i < kSideStreams) {
      if (E.no_alloc)
        throw Error(ATP_ESTATE, "no side stream chosen for these streams: call atp_warmup(compute, copy) first");
      HIPCHK(hipStreamCreateWithFlags(&s, hipStreamNonBlocking));  // default priority
      std::lock_guard<std::mutex> g(g_pool_mu);
      g_pools[E.device].streams.push_back(s);
      known.push_back(s);
    } else {
      break;
    }
    if (!same_queue(E, compute, s) && !same_queue(E, copy, s)) pick = s;
  }
  if (!pick) {
    if (known.empty()) throw Error(ATP_EHIP, "no stream for the in-place outbound work");
    pick = known.front();
    fprintf(stderr, "atp: no hardware queue free of the caller's streams among %zu streams; the in-place "
                    "outbound work shares one\n", known.size());
  }
  {
    std::lock_guard<std::mutex> g(g_pool_mu);
    E.side = g_side.insert({key, pick}).first->second;  // another thread may have chosen first
  }
  E.side_for_compute = compute;
  E.side_for_copy = copy;
}

// The copy kernel reads or writes a host buffer only through its device
// address; memory not pinned by HIP would fault the GPU, so it is refused.
void check_kernel_host_buffer(const void *p, uint64_t bytes, const char *what) {
  if (!bytes) return;
  if (!p) throw Error(ATP_EINVAL, std::string(what) + " is NULL");
  if (reinterpret_cast<uintptr_t>(p) % 256)
    throw Error(ATP_EALIGN, std::string(what) + " must be 256-byte aligned (the copy kernel accesses it directly)");
  for (const char *q : {static_cast<const char *>(p), static_cast<const char *>(p) + bytes - 1}) {
    hipPointerAttribute_t a{};
    if (hipPointerGetAttributes(&a, q) != hipSuccess || a.type != hipMemoryTypeHost || a.hostPointer == nullptr ||
        a.devicePointer != a.hostPointer) {
      (void)hipGetLastError();
      throw Error(ATP_EINVAL, std::string(what) +
                                  " must be pinned host memory from hipHostMalloc "
                                  "(the copy kernel accesses it directly)");
    }
  }
}

void build_descs(Exec &E, const CallPlan &c, CallState &cs) {
  size_t n = c.fams.size();
  if (cs.desc_host) return;  // the descriptors of a plan never change
  size_t cap = 0;
  cs.desc_host = static_cast<Desc *>(E.pinned(std::max<size_t>(n, 1) * sizeof(Desc), &cap));
  cs.desc_cap = cap / sizeof(Desc);
  for (size_t i = 0; i < n; ++i) {
    const Fam &f = c.fams[i];
    Desc d{};
    d.src_off = f.src_off;
    d.dst_off = f.dst_off;
    d.src_pitch = f.src_pitch;
    d.dst_pitch = f.dst_pitch;
    d.src_ostride = f.src_ostride;
    d.dst_ostride = f.dst_ostride;
    d.o_begin = f.o_begin;
    d.o_end = f.o_end;
    d.run = uint32_t(f.run);
    d.rows = uint32_t(f.rows);
    d.flags = f.flags;
    if (f.flags & DF_ALIGNED)
      d.magic_line = magic_of(f.run / 16);
    else
      d.magic_line = magic_of((f.run + kSegBytes - 1) / kSegBytes);
    d.magic_rows = magic_of(f.rows);
    cs.desc_host[i] = d;
  }
}

// Largest byte offset + 1 a family touches on one side.
uint64_t extent(const Fam &f, bool src, int64_t n_blocks, int64_t live) {
  uint64_t off = src ? f.src_off : f.dst_off, os = src ? f.src_ostride : f.dst_ostride,
           pitch = src ? f.src_pitch : f.dst_pitch;
  bool ind = f.flags & (src ? DF_SRC_IND : DF_DST_IND);
  int64_t items;
  if (ind)
    items = n_blocks;  // any block id
  else if (f.flags & DF_BLOCKRANGE)
    items = std::min<int64_t>(f.o_end - f.o_begin, live);
  else
    items = f.o_end - f.o_begin;
  if (items <= 0 || f.run == 0) return 0;
  return off + uint64_t(items - 1) * os + (f.rows - 1) * pitch + f.run;
}

void check_extents(const CallPlan &c, bool kvcall, const Plan &P, uint64_t in_bytes, uint64_t out_bytes,
                   uint64_t stage_bytes, uint64_t inflow_bytes, uint64_t outbound_bytes) {
  int64_t nb = kvcall ? P.kv.num_blocks : 0, live = kvcall ? P.kv.live_blocks : 0;
  // the host-read launches bind slot IN to the pinned inflow buffer, the
  // outbound launches slot OUT to the pinned outbound buffer
  const int h0 = c.host_reads.empty() ? -1 : c.host_reads.front().d0;
  const int h1 = c.host_reads.empty() ? -1 : c.host_reads.back().d1;
  auto fits = [](uint64_t off, uint64_t bytes, uint64_t lim) { return bytes <= lim && off <= lim - bytes; };
  for (const HostCopy &h : c.directs)
    if (!fits(h.host_off, h.bytes, inflow_bytes) || !fits(h.dev_off, h.bytes, out_bytes))
      throw Error(ATP_ECAPACITY, "an inflow landing would run past the end of a buffer");
  for (const Chunk &ch : c.chunks)
    for (const HostCopy &h : ch.copies)
      if (!fits(h.host_off, h.bytes, inflow_bytes) || !fits(h.dev_off, h.bytes, stage_bytes))
        throw Error(ATP_ECAPACITY, "an inflow landing would run past the end of a buffer");
  const int o0 = c.out_d0, o1 = c.out_d0 < 0 ? -1 : c.out_d0 + int(c.out_order.size());
  for (int d = 0; d < int(c.fams.size()); ++d) {
    const Fam &f = c.fams[size_t(d)];
    const bool host_read = d >= h0 && d < h1, outbound = d >= o0 && d < o1;
    for (int side = 0; side < 2; ++side) {
      uint32_t slot = (f.flags >> (side == 0 ? DF_SRC_SHIFT : DF_DST_SHIFT)) & 3;
      uint64_t e = extent(f, side == 0, nb, live);
      uint64_t lim = slot == BUF_IN ? in_bytes : slot == BUF_OUT ? out_bytes : stage_bytes;
      if (host_read && slot == BUF_IN) lim = inflow_bytes;
      if (outbound && slot == BUF_OUT) lim = outbound_bytes;
      if (e > lim) throw Error(ATP_ECAPACITY, "a copy would run past the end of a buffer");
    }
    uint64_t lines = uint64_t(kvcall ? std::max<int64_t>(nb, f.o_end - f.o_begin) : f.o_end - f.o_begin) * f.rows;
    if (lines * (f.run / 16 + 1) >= (uint64_t(1) << 32)) throw Error(ATP_EINVAL, "copy family too large");
  }
  // a launch's kernel tiles its descriptors the way the prepare kernel
  // counted them: the flags of every descriptor must match the launch
  auto same_shape = [&](const Launch &L) {
    for (int d = L.d0; d < L.d1; ++d) {
      const uint32_t fl = c.fams[size_t(d)].flags;
      if (((fl & DF_ALIGNED) != 0) != L.aligned || ((fl & DF_WIDE) != 0) != (L.aligned && L.wide))
        throw Error(ATP_EINVAL, "internal: a launch mixes descriptor shapes");
    }
  };
  for (const Launch &L : c.levels) same_shape(L);
  for (const Launch &L : c.host_reads) same_shape(L);
  for (const Chunk &ch : c.chunks)
    for (const Launch &L : ch.scatters) same_shape(L);
  for (size_t k = 0; k < c.out_aligned.size(); ++k)
    if (((c.fams[size_t(c.out_d0) + k].flags & DF_ALIGNED) != 0) != (c.out_aligned[k] != 0) ||
        (c.fams[size_t(c.out_d0) + k].flags & DF_WIDE))
      throw Error(ATP_EINVAL, "internal: an outbound read has the wrong shape");
}

void launch_copy(Exec &E, const Launch &L, const Desc *dev_desc, const int64_t *dev_prefix, char *b0, char *b1,
                 char *b2, const int32_t *live, hipStream_t s, uint64_t grid_cap = 0) {
  // one workgroup per tile, or a fixed persistent grid (the kernels loop
  // over the tiles of the launch)
  uint64_t cap = grid_cap ? grid_cap : ATP_PERSIST ? uint64_t(E.grid_max) : (uint64_t(1) << 30);
  uint64_t g = std::min<uint64_t>(std::max<uint64_t>(L.tiles_max, 1), cap);
  if (L.aligned && L.wide)
    hipLaunchKernelGGL((k_copy16<kWideUnroll>), dim3(unsigned(g)), dim3(kThreads), 0, s, dev_desc, dev_prefix, L.d0,
                       L.d1, b0, b1, b2, live);
  else if (L.aligned)
    hipLaunchKernelGGL((k_copy16<kUnroll>), dim3(unsigned(g)), dim3(kThreads), 0, s, dev_desc, dev_prefix, L.d0,
                       L.d1, b0, b1, b2, live);
  else
    hipLaunchKernelGGL(k_copy_bytes, dim3(unsigned(g)), dim3(kThreads), 0, s, dev_desc, dev_prefix, L.d0, L.d1, b0,
                       b1, b2, live);
  HIPCHK(hipGetLastError());
}

// ---- issuing one call ----------------------------------------------------------------
// Every event recorded on a stream costs it a few microseconds (about 4.5 us
// each on the MI355X, against 2 us between two bare launches), so the
// launches of a stream share their timing marks: a launch that comes right
// after a timed one starts at that launch's end mark, and the events other
// streams wait on are those same marks.  mark[s] is the end mark of the last
// command queued on s when that command was a timed launch; other(s) forgets
// it when anything else is queued there.  The Issuer also lands the inflow
// pieces that are not repack: DMA copies of large gaps and the copy kernel's
// reads of the pinned host buffer.  A deferred issue (the weights call of
// atp_load_reshard_weights_async) keeps a copy of it, with marks of its own.
struct Issuer {
  Exec &E;
  CallState &cs;
  const CallPlan &c;
  int64_t nb, live;  // KV pool size and live blocks (0 for the weights call)
  char *b_out, *b_st;
  const char *host_in;
  Desc *dev_desc;
  int64_t *dev_prefix;
  int32_t *dev_live;
  hipStream_t copy;
  std::map<hipStream_t, hipEvent_t> mark;

  void other(hipStream_t st) { mark.erase(st); }
  void record(hipEvent_t e, hipStream_t st) {
    HIPCHK(hipEventRecord(e, st));
    other(st);
  }
  template <class F>
  CallState::LaunchRec timed(int kind, int level, uint64_t bytes, hipStream_t st, const F &launch) {
    CallState::LaunchRec r{kind, level, bytes, nullptr, E.ev_time()};
    auto it = mark.find(st);
    if (it != mark.end()) {
      r.e0 = it->second;
    } else {
      r.e0 = E.ev_time();
      HIPCHK(hipEventRecord(r.e0, st));
    }
    launch();
    HIPCHK(hipEventRecord(r.e1, st));
    mark[st] = r.e1;
    cs.launches.push_back(r);
    return r;
  }
  // an event that fires once everything queued on st so far is done: the
  // last end mark there, or a fresh event (a fresh timing event is then the
  // mark a following launch starts at)
  hipEvent_t mark_or_record(hipStream_t st, bool timing) {
    auto it = mark.find(st);
    if (it != mark.end()) return it->second;
    hipEvent_t e = timing ? E.ev_time() : E.ev_sync();
    HIPCHK(hipEventRecord(e, st));
    if (timing) mark[st] = e;
    return e;
  }
  // a large contiguous gap straight into place by DMA
  void direct(const HostCopy &h) {
    HIPCHK(hipMemcpyAsync(b_out + h.dev_off, host_in + h.host_off, h.bytes, hipMemcpyHostToDevice, copy));
    cs.h2d_bytes += h.bytes;
  }
  // the copy kernel reads inflow pieces from the pinned host buffer into
  // their final place (kind 4 launches)
  void host_read(const Launch &L, hipStream_t s) {
    timed(4, -1, L.bytes, s, [&] {
      launch_copy(E, L, dev_desc, dev_prefix, const_cast<char *>(host_in), b_out, b_st, dev_live, s, kHostReadGrid);
    });
    cs.h2d_bytes += L.bytes;
  }
  void end_host_reads(hipStream_t s) { cs.hr1 = mark_or_record(s, true); }
  // While the inflow buffer is still being filled, the direct landings and
  // the host reads (each launch cut at descriptor boundaries into pieces of
  // at least kPipeBytes) are issued in the order of the end of the bytes
  // they read, each once `await` says those bytes are in.
  void awaited(hipStream_t s, const std::function<void(uint64_t)> &await) {
    struct Piece {
      uint64_t end;
      const HostCopy *direct;
      Launch L;
    };
    std::vector<Piece> pieces;
    for (const HostCopy &h : c.directs) pieces.push_back({h.host_off + h.bytes, &h, Launch{}});
    for (const Launch &L : c.host_reads) {
      Launch piece = L;
      piece.bytes = 0;
      uint64_t end = 0;
      for (int d = L.d0; d < L.d1; ++d) {
        const Fam &f = c.fams[size_t(d)];
        piece.bytes += (f.o_end - f.o_begin) * f.rows * f.run;
        end = std::max(end, extent(f, true, nb, live));  // source side: the inflow buffer
        if (piece.bytes >= kPipeBytes || d + 1 == L.d1) {
          piece.d1 = d + 1;
          pieces.push_back({end, nullptr, piece});
          piece.d0 = d + 1;
          piece.bytes = 0;
          end = 0;
        }
      }
    }
    std::stable_sort(pieces.begin(), pieces.end(), [](const Piece &x, const Piece &y) { return x.end < y.end; });
    for (const Piece &x : pieces) {
      await(x.end);
      if (x.direct) {
        direct(*x.direct);
      } else {
        other(s);  // the launch starts once the host has waited: it gets a start mark of its own
        host_read(x.L, s);
      }
    }
    if (!c.host_reads.empty()) end_host_reads(s);
  }
};

// ---- the scratch array of the no-allocation entry point --------------------------
// Callers that cannot allocate (code under HIP graph capture, tight serving
// loops) reshard on this file-scope device array instead of a staging
// buffer of their own.  Each device holds its own copy at its own address,
// looked up once per device with that device current; host code uses that
// address, never the array's name.
constexpr uint64_t kScratchBytes = 64ull << 20;
__device__ __align__(256) char scratch[kScratchBytes];
std::map<int, void *> g_scratch;     // device -> address of its copy (under g_pool_mu)
std::map<int, bool> g_scratch_busy;  // a call on it is pending (under g_pool_mu)

void *scratch_of(int dev) {
  std::lock_guard<std::mutex> g(g_pool_mu);
  auto it = g_scratch.find(dev);
  if (it != g_scratch.end()) return it->second;
  void *p = nullptr;
  HIPCHK(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
  if (!p || reinterpret_cast<uintptr_t>(p) % 256) throw Error(ATP_EHIP, "scratch array has no usable device address");
  g_scratch[dev] = p;
  return p;
}

void release_scratch(Exec &E, CallState &cs) {
  if (!cs.on_scratch) return;
  cs.on_scratch = false;
  std::lock_guard<std::mutex> g(g_pool_mu);
  g_scratch_busy[E.device] = false;
}

}  // namespace

uint64_t scratch_bytes() { return kScratchBytes; }

void exec_call(Plan &P, bool kvcall, void *arena, uint64_t arena_bytes, void *new_arena, uint64_t new_bytes,
               const void *inflow_host, uint64_t inflow_bytes, void *outbound_host, uint64_t outbound_bytes,
               const int32_t *table, int64_t n_entries, void *staging, uint64_t staging_bytes, hipStream_t compute,
               hipStream_t copy, const std::function<void(uint64_t)> *await, bool on_scratch, bool defer,
               std::function<void()> after_issue) {
  CallPlan &c = kvcall ? P.k : P.w;
  if (defer && (!await || kvcall)) throw Error(ATP_EINVAL, "internal: only a weights call that awaits its inflow is deferred");
  if (on_scratch) {
    // the device's scratch array in place of a staging buffer
    if (c.staging_need > kScratchBytes)
      throw Error(ATP_ECAPACITY, std::string(kvcall ? "kv" : "weights") + ": the plan needs " +
                                     std::to_string(c.staging_need) + " bytes of scratch; the no-allocation entry "
                                     "point has " + std::to_string(kScratchBytes) +
                                     " (plan with a staging cap no larger)");
    int dev = -1;
    HIPCHK(hipGetDevice(&dev));
    staging = scratch_of(dev);
    staging_bytes = kScratchBytes;
  }
  // Every argument is checked before the first HIP call.  The executor's
  // state exists from the plan's first call on; before it nothing is pending.
  Exec *Ep = static_cast<Exec *>(P.exec);
  if (Ep && (kvcall ? Ep->k : Ep->w).pending) throw Error(ATP_ESTATE, "reshard called again before atp_sync");
  // In place, a weights call issued while the KV call is pending ended one
  // process with a host fault whose cause is not known; that order is
  // refused until it is.
  if (P.inplace && !kvcall && Ep && Ep->k.pending)
    throw Error(ATP_ESTATE, "in place, call atp_reshard_weights before atp_reshard_kv (or after atp_sync)");
  const char *what = kvcall ? "kv" : "weights";
  // ---- argument checks ------------------------------------------------------
  if (!arena) throw Error(ATP_EINVAL, std::string(what) + ": arena is NULL");
  if (reinterpret_cast<uintptr_t>(arena) % 256 || (new_arena && reinterpret_cast<uintptr_t>(new_arena) % 256) ||
      reinterpret_cast<uintptr_t>(staging) % 256)
    throw Error(ATP_EALIGN, std::string(what) + ": device buffers must be 256-byte aligned");
  if (P.inplace) {
    if (new_arena && new_arena != arena) throw Error(ATP_EINVAL, std::string(what) + ": in place takes no new arena");
    new_arena = arena;
    if (arena_bytes < std::max(c.old_bytes, c.new_bytes))
      throw Error(ATP_ECAPACITY, std::string(what) + ": arena smaller than the old or the new layout");
    new_bytes = arena_bytes;
  } else {
    if (!new_arena) throw Error(ATP_EINVAL, std::string(what) + ": out of place needs a new arena");
    if (arena_bytes < c.old_bytes) throw Error(ATP_ECAPACITY, std::string(what) + ": arena smaller than the old layout");
    if (new_bytes < c.new_bytes) throw Error(ATP_ECAPACITY, std::string(what) + ": new arena smaller than the new layout");
    uintptr_t a0 = uintptr_t(arena), a1 = a0 + c.old_bytes, n0 = uintptr_t(new_arena), n1 = n0 + c.new_bytes;
    if (a0 < n1 && n0 < a1) throw Error(ATP_EINVAL, std::string(what) + ": old and new arenas overlap");
  }
  if (!staging || staging_bytes < c.staging_need)
    throw Error(ATP_ECAPACITY, std::string(what) + ": staging needs " + std::to_string(c.staging_need) + " bytes");
  if (inflow_bytes != c.inflow || (c.inflow && !inflow_host))
    throw Error(ATP_EINVAL, std::string(what) + ": inflow buffer must hold exactly " + std::to_string(c.inflow) +
                                " bytes");
  bool do_out = P.inplace && c.outbound_bytes > 0;
  if (do_out && (outbound_bytes < c.outbound_bytes || !outbound_host))
    throw Error(ATP_EINVAL, std::string(what) + ": outbound buffer must hold " + std::to_string(c.outbound_bytes) +
                                " bytes");
  if (kvcall && (!table || n_entries <= 0)) throw Error(ATP_EINVAL, "kv: block table missing");
  check_extents(c, kvcall, P, P.inplace ? arena_bytes : c.old_bytes, P.inplace ? arena_bytes : new_bytes,
                staging_bytes, inflow_bytes, do_out ? outbound_bytes : 0);
  // Device memory this call touches: the arenas (in place one span of the
  // larger layout) and the part of staging it uses for descriptors, prefix
  // sums, block lists, the landing ring and staged pieces.  Staging may not
  // meet an arena, and neither may meet what a pending call of the other
  // kind touches (both would write there while the other still reads).
  const uintptr_t a0 = reinterpret_cast<uintptr_t>(arena), n0 = reinterpret_cast<uintptr_t>(new_arena),
                  s0 = reinterpret_cast<uintptr_t>(staging);
  Span my_old{a0, a0 + (P.inplace ? std::max(c.old_bytes, c.new_bytes) : c.old_bytes)};
  Span my_new = P.inplace ? Span{} : Span{n0, n0 + c.new_bytes};
  Span my_st{s0, s0 + c.staging_need};
  if (my_st.meets(my_old) || my_st.meets(my_new))
    throw Error(ATP_EINVAL, std::string(what) + ": staging overlaps an arena");
  if (Ep) {
    const CallState &o = kvcall ? Ep->w : Ep->k;
    if (o.pending)
      for (const Span &mine : {my_old, my_new, my_st})
        for (const Span &theirs : {o.old_arena, o.new_arena, o.staging})
          if (mine.meets(theirs))
            throw Error(ATP_EINVAL, std::string(what) + ": an arena or staging buffer overlaps one of the pending " +
                                        (kvcall ? "weights" : "kv") + " call");
  }
  if (!c.host_reads.empty()) check_kernel_host_buffer(inflow_host, inflow_bytes, "inflow buffer");
  if (do_out && c.out_d0 >= 0) check_kernel_host_buffer(outbound_host, c.outbound_bytes, "outbound buffer");

  Exec &E = exec_of(P);
  CallState &cs = kvcall ? E.k : E.w;
  if (on_scratch) {
    std::lock_guard<std::mutex> g(g_pool_mu);
    if (g_scratch_busy[E.device])
      throw Error(ATP_ESTATE, "the device's scratch array is in use by a pending call: atp_sync it first");
    g_scratch_busy[E.device] = true;
  }
  // from here on the call either is issued (pending) or, if it fails after
  // queuing work, waits until nothing it queued can still be running (the
  // caller may then free its buffers) and gives back the scratch array
  struct Undo {
    Exec &E;
    CallState &cs;
    hipStream_t s0, s1;
    bool armed = true, enqueued = false;
    ~Undo() {
      E.no_alloc = false;
      if (!armed) return;
      if (enqueued)
        for (hipStream_t s : {s0, s1, E.side})
          if (s && hipStreamSynchronize(s) != hipSuccess) (void)hipGetLastError();
      release_scratch(E, cs);
    }
  } undo{E, cs, compute, copy};
  cs.on_scratch = on_scratch;
  E.no_alloc = on_scratch;

  int dev = -1;
  HIPCHK(hipGetDevice(&dev));
  if (dev != E.device) throw Error(ATP_EINVAL, "plan used on another device than its first call");
  if (!E.w.pending && !E.k.pending) {
    E.sync_used = E.time_used = 0;
    E.wall_started = true;
    E.wall0 = std::chrono::steady_clock::now();
  }
  if (!cs.err_host) {
    size_t cap = 0;
    cs.err_host = static_cast<int32_t *>(E.pinned(256, &cap));
  }
  *cs.err_host = 0;
  cs.old_arena = my_old;
  cs.new_arena = my_new;
  cs.staging = my_st;
  cs.launches.clear();
  cs.h2d_bytes = cs.d2h_bytes = cs.scatter_bytes = cs.repack_bytes = 0;
  build_descs(E, c, cs);

  char *b_in = static_cast<char *>(arena), *b_out = static_cast<char *>(new_arena),
       *b_st = static_cast<char *>(staging);
  const char *host_in = static_cast<const char *>(inflow_host);
  char *host_out = static_cast<char *>(outbound_host);
  Desc *dev_desc = reinterpret_cast<Desc *>(b_st + c.off_desc);
  int64_t *dev_prefix = reinterpret_cast<int64_t *>(b_st + c.off_prefix);
  int32_t *dev_err = reinterpret_cast<int32_t *>(b_st + c.off_meta);
  int32_t *dev_live = kvcall ? reinterpret_cast<int32_t *>(b_st + c.off_kvlive) : nullptr;

  Issuer is{E, cs, c, kvcall ? P.kv.num_blocks : 0, kvcall ? P.kv.live_blocks : 0, b_out, b_st, host_in,
            dev_desc, dev_prefix, dev_live, copy, {}};
  cs.compute = compute;
  cs.copy = copy;
  cs.finish_issue = nullptr;

  // The side stream runs, in place, the weights call's outbound reads,
  // levels and host reads and the KV call's outbound copies; out of place,
  // the host reads of both calls, beside the repack on `compute`.  It is
  // chosen before this call queues anything: the probe waits for what the
  // caller's streams already hold.
  const bool early_reads = !P.inplace && !c.host_reads.empty();
  const bool use_side = do_out || early_reads;
  if (use_side) choose_side(E, compute, copy);

  // every stream of this call starts after what the caller has queued on
  // `compute` when the call is made (with the other call of the plan
  // pending, that includes the other call's work on `compute`)
  cs.start = E.ev_sync();
  undo.enqueued = true;
  HIPCHK(hipEventRecord(cs.start, compute));
  HIPCHK(hipStreamWaitEvent(copy, cs.start, 0));

  // direct landings wait for nothing (the planner routes every landing that
  // would wait for a level or an outbound read elsewhere): they go first, so
  // that the link is busy at once.  While the inflow buffer is still being
  // filled (`await`) they go after the levels instead, with the host reads,
  // so that the host does not wait for the reads before the repack is queued.
  cs.h2d0 = E.ev_time();
  HIPCHK(hipEventRecord(cs.h2d0, copy));
  if (!await)
    for (const HostCopy &h : c.directs) is.direct(h);

  // ---- upload descriptors, prepare ----------------------------------------------
  if (!c.fams.empty())
    HIPCHK(hipMemcpyAsync(dev_desc, cs.desc_host, c.fams.size() * sizeof(Desc), hipMemcpyHostToDevice, compute));
  PrepArgs pa{};
  pa.descs = dev_desc;
  pa.n_desc = int32_t(c.fams.size());
  pa.kv = kvcall;
  pa.prefix = dev_prefix;
  pa.err = dev_err;
  if (kvcall) {
    pa.table = table;
    pa.n_entries = n_entries;
    pa.flags = reinterpret_cast<int32_t *>(b_st + c.off_kvflags);
    pa.pref = reinterpret_cast<int32_t *>(b_st + c.off_kvpref);
    pa.live = dev_live;
    pa.n_blocks = P.kv.num_blocks;
    pa.expect_live = P.kv.live_blocks;
  }
  // k_prepare is the only writer of the error word: it stores it once
  hipLaunchKernelGGL(k_prepare, dim3(1), dim3(1024), 0, compute, pa);
  HIPCHK(hipGetLastError());
  is.other(compute);
  hipEvent_t prepared = nullptr;  // descriptors, prefix sums and live blocks in place
  if (use_side) {
    prepared = E.ev_sync();
    is.record(prepared, compute);
  }

  cs.hr1 = nullptr;
  // out of place: at once, on the side stream, beside the repack (the two
  // write disjoint bytes of the new arena)
  if (early_reads) {
    HIPCHK(hipStreamWaitEvent(E.side, prepared, 0));
    is.other(E.side);
    if (!await) {
      for (const Launch &L : c.host_reads) is.host_read(L, E.side);
      is.end_host_reads(E.side);
    }
  }

  // ---- outbound (in place): read before overwrite ---------------------------------
  // The weights call's outbound reads are copy-kernel launches on the side
  // stream that write straight into the pinned outbound buffer, in the
  // plan's order (by the first level that overwrites them), each level right
  // after the reads it needs (stream order on that one stream is the gate).
  // That work and the weight inflow read after it stay off the caller's
  // streams, so that they do not hold up the other call's work queued
  // behind them.
  size_t issued = 0;  // outbound pieces read out so far, in plan order
  const bool split = do_out && !kvcall;
  hipStream_t late_comp = compute;
  if (split) {
    late_comp = E.side;  // the outbound launches read the descriptors
    HIPCHK(hipStreamWaitEvent(late_comp, prepared, 0));
    is.other(late_comp);
  }
  std::vector<size_t> pos_of(c.outbound.size(), 0);
  for (size_t p = 0; p < c.out_order.size(); ++p) pos_of[size_t(c.out_order[p])] = p;
  auto issue_outbound = [&](size_t upto) {  // read out the first `upto` pieces
    while (issued < upto) {
      // one launch per run of positions with the same alignment
      Launch L;
      L.kind = 3;
      L.aligned = c.out_aligned[issued] != 0;
      L.d0 = c.out_d0 + int(issued);
      for (; issued < upto && (c.out_aligned[issued] != 0) == L.aligned; ++issued) {
        L.tiles_max += c.out_tiles[issued];
        L.bytes += c.outbound[size_t(c.out_order[issued])].bytes;
      }
      L.d1 = c.out_d0 + int(issued);
      const CallState::LaunchRec r = is.timed(3, -1, L.bytes, late_comp, [&] {
        launch_copy(E, L, dev_desc, dev_prefix, b_in, host_out, b_st, dev_live, late_comp, kOutboundGrid);
      });
      if (!cs.d2h0) cs.d2h0 = r.e0;
      cs.d2h1 = r.e1;
      cs.d2h_bytes += L.bytes;
    }
  };
  cs.d2h0 = cs.d2h1 = nullptr;

  // ---- repack levels ---------------------------------------------------------------
  hipEvent_t level0_end = nullptr;  // the KV outbound gathered at level 0 is copied out after it
  cs.rep0 = nullptr;
  for (size_t i = 0; i < c.levels.size(); ++i) {
    const Launch &L = c.levels[i];
    if (split) {
      size_t need = 0;
      for (int o : L.wait_outbound) need = std::max(need, pos_of[size_t(o)] + 1);
      issue_outbound(need);
    }
    const CallState::LaunchRec r = is.timed(kvcall ? 1 : 0, L.level, L.bytes, late_comp, [&] {
      launch_copy(E, L, dev_desc, dev_prefix, b_in, b_out, b_st, dev_live, late_comp);
    });
    if (!cs.rep0) cs.rep0 = r.e0;
    cs.repack_bytes += 2 * L.bytes;
    if (L.level == 0) level0_end = r.e1;
  }
  if (split) issue_outbound(c.out_order.size());  // pieces no level waits for
  if (!cs.rep0) cs.rep0 = is.mark_or_record(late_comp, true);
  cs.rep1 = is.mark_or_record(late_comp, true);  // also: prepare and every level are done

  // in place: the copy kernel reads every gated or strided inflow piece from
  // the pinned host buffer into its final place, after the last level (and,
  // for the weights, after every outbound read)
  const hipStream_t await_stream = P.inplace ? late_comp : E.side;
  if (await && !defer) {
    is.awaited(await_stream, *await);
  } else if (!await && P.inplace && !c.host_reads.empty()) {
    for (const Launch &L : c.host_reads) is.host_read(L, late_comp);
    is.end_host_reads(late_comp);
  }

  // KV outbound gathered into staging at level 0: copy it out after that level
  if (do_out && kvcall) {
    if (level0_end) HIPCHK(hipStreamWaitEvent(E.side, level0_end, 0));
    cs.d2h0 = E.ev_time();
    is.record(cs.d2h0, E.side);
    for (size_t o = 0; o < c.outbound.size(); ++o) {
      const HostCopy &h = c.outbound[o];
      HIPCHK(hipMemcpyAsync(host_out + h.host_off, b_st + h.dev_off, h.bytes, hipMemcpyDeviceToHost, E.side));
      cs.d2h_bytes += h.bytes;
    }
    cs.d2h1 = E.ev_time();
    is.record(cs.d2h1, E.side);
  }

  // ---- inflow ------------------------------------------------------------------------
  // (direct landings went first, none of them waits for anything; the copy
  // kernel's host reads are issued above)
  // ring (the in-place KV call only): H2D into a slot, then a scatter from it
  // after every level; a chunk reuses its slot once the slot's previous
  // scatter is done
  std::vector<hipEvent_t> slot_free(c.chunks.size(), nullptr);
  for (size_t i = 0; i < c.chunks.size(); ++i) {
    const Chunk &ch = c.chunks[i];
    if (i >= size_t(c.n_slots) && slot_free[i - c.n_slots])
      HIPCHK(hipStreamWaitEvent(copy, slot_free[i - c.n_slots], 0));
    for (const HostCopy &h : ch.copies) {
      HIPCHK(hipMemcpyAsync(b_st + h.dev_off, host_in + h.host_off, h.bytes, hipMemcpyHostToDevice, copy));
      cs.h2d_bytes += h.bytes;
    }
    hipEvent_t landed = E.ev_sync();
    HIPCHK(hipEventRecord(landed, copy));
    HIPCHK(hipStreamWaitEvent(late_comp, landed, 0));
    is.other(late_comp);
    for (const Launch &L : ch.scatters) {
      is.timed(2, -1, L.bytes, late_comp,
               [&] { launch_copy(E, L, dev_desc, dev_prefix, b_in, b_out, b_st, dev_live, late_comp); });
      cs.scatter_bytes += L.bytes;
    }
    slot_free[i] = is.mark_or_record(late_comp, false);  // the chunk's last scatter is done
  }
  cs.h2d1 = E.ev_time();  // the inflow ends with the later of this and hr1
  HIPCHK(hipEventRecord(cs.h2d1, copy));

  // ---- tails ----------------------------------------------------------------------
  HIPCHK(hipMemcpyAsync(cs.err_host, dev_err, sizeof(int32_t), hipMemcpyDeviceToHost, compute));
  cs.tail_compute = E.ev_sync();
  HIPCHK(hipEventRecord(cs.tail_compute, compute));
  cs.tail_copy = E.ev_sync();
  HIPCHK(hipEventRecord(cs.tail_copy, copy));
  cs.tail_side = nullptr;
  if (use_side) {
    // the side stream is not joined back into the caller's streams (that
    // would hold up the other call's work); atp_sync waits for it
    cs.tail_side = E.ev_sync();
    HIPCHK(hipEventRecord(cs.tail_side, E.side));
  }
  if (defer) {
    // the awaited pieces wait for the reads: atp_sync issues them (the
    // caller may queue the KV call meanwhile), then records the tails again
    auto d = std::make_shared<Issuer>(is);
    d->mark.clear();
    const std::function<void(uint64_t)> aw = *await;
    const hipStream_t side = use_side ? E.side : nullptr;
    cs.finish_issue = [d, aw, after_issue, await_stream, compute, copy, side]() {
      Exec &E = d->E;
      CallState &cs = d->cs;
      d->awaited(await_stream, aw);
      cs.h2d1 = E.ev_time();
      HIPCHK(hipEventRecord(cs.h2d1, copy));
      cs.tail_compute = E.ev_sync();
      HIPCHK(hipEventRecord(cs.tail_compute, compute));
      cs.tail_copy = E.ev_sync();
      HIPCHK(hipEventRecord(cs.tail_copy, copy));
      if (side) {
        cs.tail_side = E.ev_sync();
        HIPCHK(hipEventRecord(cs.tail_side, side));
      }
      if (after_issue) after_issue();
    };
  }
  cs.pending = true;
  undo.armed = false;
}

int exec_sync(Plan &P, atp_timing *out) {
  if (!P.exec) throw Error(ATP_ESTATE, "nothing to synchronise");
  Exec &E = *static_cast<Exec *>(P.exec);
  int rc = ATP_OK;
  std::string msg;
  atp_timing t{};
  t.plan_ms = P.plan_ms;
  E.last_launches.clear();
  auto ms = [](hipEvent_t a, hipEvent_t b) {
    float f = 0;
    if (a && b && hipEventElapsedTime(&f, a, b) == hipSuccess) return double(f);
    return 0.0;
  };
  // a deferred issue first: its pieces wait for the reads, then its tails
  // are recorded again; if it fails (a read, a HIP call), everything the
  // plan queued drains before the error is returned
  for (CallState *c : {&E.w, &E.k}) {
    if (!c->pending || !c->finish_issue) continue;
    std::function<void()> f = std::move(c->finish_issue);
    c->finish_issue = nullptr;
    try {
      f();
    } catch (const std::exception &e) {
      if (rc == ATP_OK) {
        const Error *ae = dynamic_cast<const Error *>(&e);
        rc = ae ? ae->code : ATP_EINVAL;
        msg = e.what();
      }
      for (hipStream_t s : {c->compute, c->copy, E.side})
        if (s && hipStreamSynchronize(s) != hipSuccess) (void)hipGetLastError();
    }
  }
  double h2d_ms = 0, rep_ms = 0;
  hipEvent_t h2d_first = nullptr, h2d_last = nullptr;  // union span of both calls
  const bool was_pending[2] = {E.w.pending, E.k.pending};
  for (int which = 0; which < 2; ++which) {
    CallState &cs = which == 0 ? E.w : E.k;
    if (!cs.pending) continue;
    for (hipEvent_t e : {cs.tail_compute, cs.tail_copy, cs.tail_side}) {
      if (!e) continue;
      hipError_t err = hipEventSynchronize(e);
      if (err != hipSuccess) (void)hipGetLastError();  // reported below, as for hip_check
      if (err != hipSuccess && rc == ATP_OK) {
        rc = ATP_EHIP;
        msg = std::string("reshard failed on the GPU: ") + hipGetErrorString(err);
      }
    }
    cs.pending = false;
    release_scratch(E, cs);
    if (*cs.err_host && rc == ATP_OK) {
      rc = ATP_EINVAL;
      msg = "block table invalid:";
      if (*cs.err_host & ERR_BAD_BLOCK) msg += " a block id is >= num_blocks;";
      if (*cs.err_host & ERR_LIVE_COUNT) msg += " the number of distinct live blocks differs from kv.live_blocks;";
    }
    // busy time of the repack kernels (levels), and the span they cover
    double busy = 0;
    for (const auto &L : cs.launches)
      if (L.kind < 2) busy += ms(L.e0, L.e1);
    (which == 0 ? t.repack_w_ms : t.repack_kv_ms) = busy;
    t.repack_span_ms += ms(cs.rep0, cs.rep1);
    rep_ms += busy;
    // union span of both calls: the earlier start, the later end
    if (cs.h2d0 && (!h2d_first || ms(cs.h2d0, h2d_first) > 0)) h2d_first = cs.h2d0;
    for (hipEvent_t e : {cs.h2d1, cs.hr1})
      if (e && (!h2d_last || ms(h2d_last, e) > 0)) h2d_last = e;
    t.d2h_ms = std::max(t.d2h_ms, ms(cs.d2h0, cs.d2h1));
    for (const auto &L : cs.launches) {
      double m = ms(L.e0, L.e1);
      if (L.kind == 2) t.scatter_ms += m;
      E.last_launches.push_back({L.kind, L.level, L.bytes, m});
    }
    t.repack_bytes += cs.repack_bytes;
    t.h2d_bytes += cs.h2d_bytes;
    t.d2h_bytes += cs.d2h_bytes;
    t.scatter_bytes += cs.scatter_bytes;
  }
  h2d_ms = ms(h2d_first, h2d_last);
  t.h2d_ms = h2d_ms;
  // union of the repack kernels' intervals over both calls, on a common
  // time origin (the start of the inflow)
  if (h2d_first) {
    std::vector<std::pair<double, double>> iv;
    for (int which = 0; which < 2; ++which)
      if (was_pending[which])
        for (const auto &L : (which == 0 ? E.w : E.k).launches)
          if (L.kind < 2 && L.e0 && L.e1) iv.push_back({ms(h2d_first, L.e0), ms(h2d_first, L.e1)});
    std::sort(iv.begin(), iv.end());
    double cur_lo = 0, cur_hi = 0;
    bool open = false;
    for (const auto &x : iv) {
      if (open && x.first <= cur_hi) {
        cur_hi = std::max(cur_hi, x.second);
        continue;
      }
      if (open) t.repack_union_ms += cur_hi - cur_lo;
      cur_lo = x.first;
      cur_hi = x.second;
      open = true;
    }
    if (open) t.repack_union_ms += cur_hi - cur_lo;
  }
  t.wall_ms = E.wall_started
                  ? std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - E.wall0).count()
                  : 0;
  E.wall_started = false;
  double lo = std::min(rep_ms, h2d_ms);
  if (lo > 0) t.overlap = std::min(1.0, std::max(0.0, (rep_ms + h2d_ms - t.wall_ms) / lo));
  t.n_launches = int32_t(E.last_launches.size());
  E.last = t;
  if (out) *out = t;
  if (rc != ATP_OK) throw Error(rc, msg);
  return ATP_OK;
}

void exec_free(Plan &P) {
  if (P.exec) {
    Exec *E = static_cast<Exec *>(P.exec);
    // drain anything still queued before the pinned buffers go away
    for (CallState *c : {&E->w, &E->k}) {
      if (c->pending)
        for (hipEvent_t e : {c->tail_compute, c->tail_copy, c->tail_side})
          if (e) (void)hipEventSynchronize(e);
      c->finish_issue = nullptr;  // a deferred issue never run: its readers stop and join
      release_scratch(*E, *c);
    }
    delete E;
    P.exec = nullptr;
  }
}

// The per-process set-up a first reshard on this device would otherwise
// pay (about 5 ms on the 40-layer TP 4->3 workload): the kernels' code is
// loaded, the side stream for (compute, copy) is chosen, and pooled events
// and pinned descriptor buffers are created, all on the current device.
void exec_warmup(void *compute_, void *copy_, int events) {
  if (events < 0 || events > 4096) throw Error(ATP_EINVAL, "warmup: events must be in [0, 4096]");
  hipStream_t compute = static_cast<hipStream_t>(compute_), copy = static_cast<hipStream_t>(copy_);
  Exec E;  // hands its events back to the device pool when it goes
  HIPCHK(hipGetDevice(&E.device));
  hipFuncAttributes fa;
  HIPCHK(hipFuncGetAttributes(&fa, reinterpret_cast<const void *>(&k_copy16<kUnroll>)));
  HIPCHK(hipFuncGetAttributes(&fa, reinterpret_cast<const void *>(&k_copy16<kWideUnroll>)));
  HIPCHK(hipFuncGetAttributes(&fa, reinterpret_cast<const void *>(&k_copy_bytes)));
  HIPCHK(hipFuncGetAttributes(&fa, reinterpret_cast<const void *>(&k_prepare)));
  HIPCHK(hipFuncGetAttributes(&fa, reinterpret_cast<const void *>(&k_spin)));
  HIPCHK(hipFuncGetAttributes(&fa, reinterpret_cast<const void *>(&k_nop)));
  choose_side(E, compute, copy);
  (void)scratch_of(E.device);  // the no-allocation entry point's scratch array, on this device
  for (int i = 0; i < events; ++i) {
    E.ev_sync();
    E.ev_time();
  }
  // error words and descriptor buffers for two calls (the pool hands out
  // the smallest buffer that is big enough)
  std::vector<std::pair<void *, size_t>> bufs;
  for (size_t bytes : {size_t(256), size_t(256), size_t(1) << 20, size_t(1) << 20}) {
    size_t cap = 0;
    bufs.push_back({E.pinned(bytes, &cap), cap});
  }
  std::lock_guard<std::mutex> g(g_pool_mu);
  auto &pool = g_pools[E.device].pinned;
  pool.insert(pool.end(), bufs.begin(), bufs.end());
}

void exec_launches(const Plan &P, std::vector<atp_launch> &out) {
  out.clear();
  if (P.exec) out = static_cast<const Exec *>(P.exec)->last_launches;
}

}  // namespace atp
