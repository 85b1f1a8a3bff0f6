// exec.hip — executor of the reshard library (Sec. III-C physical stage on
// one GPU): uploads the plan's descriptors into the caller's staging
// buffer, launches the prepare and repack kernels level by level on the
// compute stream, lands the missing bytes from the pinned host buffer on the
// copy stream (directly, or through the landing ring plus a scatter kernel),
// reads dropped outbound bytes out before an in-place overwrite, and orders
// the three with HIP events.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <chrono>
#include <map>
#include <mutex>
#include <cstring>
#include <string>
#include <vector>

#include "exec.h"
#include "kernels.h"
#include "plan.h"

namespace atp {
namespace {

void hip_check(hipError_t e, const char *what) {
  if (e != hipSuccess) throw Error(ATP_EHIP, std::string(what) + ": " + hipGetErrorString(e));
}
#define HIPCHK(x) hip_check((x), #x)

uint64_t magic_of(uint64_t d) {
  if (d <= 1) return 0;
  unsigned __int128 m = ((((unsigned __int128)1) << 64) + d - 1) / d;  // ceil(2^64 / d)
  return uint64_t(m);
}

struct CallState {
  bool pending = false;
  Desc *desc_host = nullptr;  // pinned copy of the descriptors
  size_t desc_cap = 0;
  int32_t *err_host = nullptr;  // pinned error word
  hipEvent_t start = nullptr;  // marks the caller's work queued before the call
  hipEvent_t tail_compute = nullptr, tail_copy = nullptr, tail_d2h = nullptr;
  hipEvent_t tail_late_copy = nullptr, tail_late_comp = nullptr;
  hipEvent_t rep0 = nullptr, rep1 = nullptr, h2d0 = nullptr, h2d1 = nullptr, d2h0 = nullptr, d2h1 = nullptr;
  struct LaunchRec {
    int kind, level;
    uint64_t bytes;
    hipEvent_t e0, e1;
  };
  std::vector<LaunchRec> launches;
  uint64_t h2d_bytes = 0, d2h_bytes = 0, scatter_bytes = 0, repack_bytes = 0;
};

// Process-wide recycling of HIP objects per device.  Each plan owns what it
// takes until it is freed; creating events, streams and pinned buffers for
// every plan would otherwise cost tens of milliseconds per reshard.
struct DevicePool {
  std::vector<hipEvent_t> sync_ev, time_ev;
  std::vector<hipStream_t> streams;
  std::vector<std::pair<void *, size_t>> pinned;
};
std::mutex g_pool_mu;
std::map<int, DevicePool> g_pools;

struct Exec {
  int device = -1;
  int grid_max = 2048;
  hipStream_t d2h = nullptr;    // outbound reads (in place)
  hipStream_t copy2 = nullptr;  // in-place weight landings that wait for levels / outbound reads
  hipStream_t comp2 = nullptr;  // in-place weight levels and scatters
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
      if (!e) HIPCHK(hipEventCreate(&e));
      time_pool.push_back(e);
    }
    return time_pool[time_used++];
  }
  hipStream_t stream() {
    {
      std::lock_guard<std::mutex> g(g_pool_mu);
      auto &v = g_pools[device].streams;
      if (!v.empty()) {
        hipStream_t s = v.back();
        v.pop_back();
        return s;
      }
    }
    hipStream_t s;
    HIPCHK(hipStreamCreateWithFlags(&s, hipStreamNonBlocking));  // default priority
    return s;
  }
  void *pinned(size_t bytes, size_t *cap) {
    {
      std::lock_guard<std::mutex> g(g_pool_mu);
      auto &v = g_pools[device].pinned;
      for (size_t i = 0; i < v.size(); ++i)
        if (v[i].second >= bytes) {
          void *p = v[i].first;
          *cap = v[i].second;
          v.erase(v.begin() + long(i));
          return p;
        }
    }
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
    for (hipStream_t st : {d2h, copy2, comp2})
      if (st) pl.streams.push_back(st);
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
                   uint64_t stage_bytes) {
  int64_t nb = kvcall ? P.kv.num_blocks : 0, live = kvcall ? P.kv.live_blocks : 0;
  for (const Fam &f : c.fams) {
    for (int side = 0; side < 2; ++side) {
      uint32_t slot = (f.flags >> (side == 0 ? DF_SRC_SHIFT : DF_DST_SHIFT)) & 3;
      uint64_t e = extent(f, side == 0, nb, live);
      uint64_t lim = slot == BUF_IN ? in_bytes : slot == BUF_OUT ? out_bytes : stage_bytes;
      if (e > lim) throw Error(ATP_ECAPACITY, "a copy would run past the end of a buffer");
    }
    uint64_t lines = uint64_t(kvcall ? std::max<int64_t>(nb, f.o_end - f.o_begin) : f.o_end - f.o_begin) * f.rows;
    if (lines * (f.run / 16 + 1) >= (uint64_t(1) << 32)) throw Error(ATP_EINVAL, "copy family too large");
  }
}

void launch_copy(Exec &E, const Launch &L, const Desc *dev_desc, const int64_t *dev_prefix, char *b0, char *b1,
                 char *b2, const int32_t *live, hipStream_t s) {
  // one workgroup per tile, or a fixed persistent grid
  uint64_t cap = ATP_PERSIST ? uint64_t(E.grid_max) : (uint64_t(1) << 30);
  uint64_t g = std::min<uint64_t>(std::max<uint64_t>(L.tiles_max, 1), cap);
  if (L.aligned)
    hipLaunchKernelGGL(k_copy16, dim3(unsigned(g)), dim3(kThreads), 0, s, dev_desc, dev_prefix, L.d0, L.d1, b0, b1,
                       b2, live);
  else
    hipLaunchKernelGGL(k_copy_bytes, dim3(unsigned(g)), dim3(kThreads), 0, s, dev_desc, dev_prefix, L.d0, L.d1, b0,
                       b1, b2, live);
  HIPCHK(hipGetLastError());
}

}  // namespace

void exec_call(Plan &P, bool kvcall, void *arena, uint64_t arena_bytes, void *new_arena, uint64_t new_bytes,
               const void *inflow_host, uint64_t inflow_bytes, void *outbound_host, uint64_t outbound_bytes,
               const int32_t *table, int64_t n_entries, void *staging, uint64_t staging_bytes, hipStream_t compute,
               hipStream_t copy) {
  CallPlan &c = kvcall ? P.k : P.w;
  Exec &E = exec_of(P);
  CallState &cs = kvcall ? E.k : E.w;
  if (cs.pending) throw Error(ATP_ESTATE, "reshard called again before atp_sync");
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
                staging_bytes);

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

  // every stream starts after what the caller already queued on `compute`
  // The other call of a weights + KV pair may already be pending: its
  // start event marks the caller's prior work, so this call's landings
  // need not wait for that call's own kernels.
  CallState &other = kvcall ? E.w : E.k;
  hipEvent_t start = other.pending && other.start ? other.start : nullptr;
  if (!start) {
    start = E.ev_sync();
    HIPCHK(hipEventRecord(start, compute));
  }
  cs.start = start;
  HIPCHK(hipStreamWaitEvent(copy, start, 0));

  // landings that depend on nothing go first, so that the link is busy at once
  cs.h2d0 = E.ev_time();
  HIPCHK(hipEventRecord(cs.h2d0, copy));
  for (const HostCopy &h : c.directs)
    if (h.gate_pos == 0 && h.gate_level < 0) {
      HIPCHK(hipMemcpyAsync(b_out + h.dev_off, host_in + h.host_off, h.bytes, hipMemcpyHostToDevice, copy));
      cs.h2d_bytes += h.bytes;
    }

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

  // ---- outbound (in place): read before overwrite ---------------------------------
  // issued in the plan's order (by the first level that overwrites them);
  // pos_ev[k] fires when the first k + 1 of them have finished
  std::vector<hipEvent_t> out_ev(c.outbound.size(), nullptr), pos_ev;
  if (do_out && !kvcall) {
    if (!E.d2h) E.d2h = E.stream();
    HIPCHK(hipStreamWaitEvent(E.d2h, start, 0));
    cs.d2h0 = E.ev_time();
    HIPCHK(hipEventRecord(cs.d2h0, E.d2h));
    for (int o : c.out_order) {
      const HostCopy &h = c.outbound[o];
      if (h.rows <= 1)
        HIPCHK(hipMemcpyAsync(host_out + h.host_off, b_in + h.dev_off, h.bytes, hipMemcpyDeviceToHost, E.d2h));
      else
        HIPCHK(hipMemcpy2DAsync(host_out + h.host_off, h.run, b_in + h.dev_off, h.dev_pitch, h.run, h.rows,
                                hipMemcpyDeviceToHost, E.d2h));
      out_ev[o] = E.ev_sync();
      HIPCHK(hipEventRecord(out_ev[o], E.d2h));
      pos_ev.push_back(out_ev[o]);
      cs.d2h_bytes += h.bytes;
    }
    cs.d2h1 = E.ev_time();
    HIPCHK(hipEventRecord(cs.d2h1, E.d2h));
  }

  // In place, the weight levels wait for outbound reads; that work and
  // everything after it (ring landings, scatters, gated landings) runs on
  // two library streams so that it does not hold up the caller's streams,
  // and with them the other call's work.
  const bool split = do_out && !kvcall;
  hipStream_t late_copy = copy, late_comp = compute;
  if (split) {
    if (!E.copy2) E.copy2 = E.stream();
    if (!E.comp2) E.comp2 = E.stream();
    late_copy = E.copy2;
    late_comp = E.comp2;
    hipEvent_t prepared = E.ev_sync();
    HIPCHK(hipEventRecord(prepared, compute));
    HIPCHK(hipStreamWaitEvent(late_comp, prepared, 0));
    HIPCHK(hipStreamWaitEvent(late_copy, start, 0));
  }

  // ---- repack levels ---------------------------------------------------------------
  std::vector<hipEvent_t> level_end(std::max(c.n_levels, 1), nullptr);
  cs.rep0 = E.ev_time();
  HIPCHK(hipEventRecord(cs.rep0, late_comp));
  for (size_t i = 0; i < c.levels.size(); ++i) {
    const Launch &L = c.levels[i];
    for (int o : L.wait_outbound)
      if (out_ev[o]) HIPCHK(hipStreamWaitEvent(late_comp, out_ev[o], 0));
    CallState::LaunchRec r{kvcall ? 1 : 0, L.level, L.bytes, E.ev_time(), E.ev_time()};
    HIPCHK(hipEventRecord(r.e0, late_comp));
    launch_copy(E, L, dev_desc, dev_prefix, b_in, b_out, b_st, dev_live, late_comp);
    HIPCHK(hipEventRecord(r.e1, late_comp));
    cs.launches.push_back(r);
    cs.repack_bytes += 2 * L.bytes;
    bool last_of_level = i + 1 == c.levels.size() || c.levels[i + 1].level != L.level;
    if (last_of_level) {
      level_end[L.level] = E.ev_sync();
      HIPCHK(hipEventRecord(level_end[L.level], late_comp));
    }
  }
  cs.rep1 = E.ev_time();
  HIPCHK(hipEventRecord(cs.rep1, late_comp));  // also: prepare and every level are done

  // KV outbound gathered into staging at level 0: copy it out after that level
  if (do_out && kvcall) {
    if (!E.d2h) E.d2h = E.stream();
    if (level_end[0]) HIPCHK(hipStreamWaitEvent(E.d2h, level_end[0], 0));
    cs.d2h0 = E.ev_time();
    HIPCHK(hipEventRecord(cs.d2h0, E.d2h));
    for (size_t o = 0; o < c.outbound.size(); ++o) {
      const HostCopy &h = c.outbound[o];
      HIPCHK(hipMemcpyAsync(host_out + h.host_off, b_st + h.dev_off, h.bytes, hipMemcpyDeviceToHost, E.d2h));
      cs.d2h_bytes += h.bytes;
    }
    cs.d2h1 = E.ev_time();
    HIPCHK(hipEventRecord(cs.d2h1, E.d2h));
  }

  // ---- inflow ------------------------------------------------------------------------
  auto gate_out = [&](hipStream_t s, int gate_pos) {
    if (gate_pos > 0 && gate_pos <= int(pos_ev.size())) HIPCHK(hipStreamWaitEvent(s, pos_ev[gate_pos - 1], 0));
  };
  auto direct = [&](const HostCopy &h, hipStream_t s) {
    if (h.gate_level >= 0 && level_end[h.gate_level]) HIPCHK(hipStreamWaitEvent(s, level_end[h.gate_level], 0));
    gate_out(s, h.gate_pos);
    HIPCHK(hipMemcpyAsync(b_out + h.dev_off, host_in + h.host_off, h.bytes, hipMemcpyHostToDevice, s));
    cs.h2d_bytes += h.bytes;
  };
  // (ungated landings were issued first) those waiting for levels only
  for (const HostCopy &h : c.directs)
    if (h.gate_pos == 0 && h.gate_level >= 0) direct(h, late_copy);
  // ring: H2D into a slot, scatter from it after every level (and after the
  // outbound reads the chunk overwrites)
  std::vector<hipEvent_t> slot_free(c.chunks.size(), nullptr);
  for (size_t i = 0; i < c.chunks.size(); ++i) {
    const Chunk &ch = c.chunks[i];
    hipStream_t cs_copy = late_copy, cs_comp = late_comp;  // scatters after every level
    if (i >= size_t(c.n_slots) && slot_free[i - c.n_slots])
      HIPCHK(hipStreamWaitEvent(cs_copy, slot_free[i - c.n_slots], 0));
    for (const HostCopy &h : ch.copies) {
      HIPCHK(hipMemcpyAsync(b_st + h.dev_off, host_in + h.host_off, h.bytes, hipMemcpyHostToDevice, cs_copy));
      cs.h2d_bytes += h.bytes;
    }
    hipEvent_t landed = E.ev_sync();
    HIPCHK(hipEventRecord(landed, cs_copy));
    HIPCHK(hipStreamWaitEvent(cs_comp, landed, 0));
    gate_out(cs_comp, ch.gate_pos);
    for (const Launch &L : ch.scatters) {
      CallState::LaunchRec r{2, -1, L.bytes, E.ev_time(), E.ev_time()};
      HIPCHK(hipEventRecord(r.e0, cs_comp));
      launch_copy(E, L, dev_desc, dev_prefix, b_in, b_out, b_st, dev_live, cs_comp);
      HIPCHK(hipEventRecord(r.e1, cs_comp));
      cs.launches.push_back(r);
      cs.scatter_bytes += L.bytes;
    }
    slot_free[i] = E.ev_sync();
    HIPCHK(hipEventRecord(slot_free[i], cs_comp));
  }
  for (const HostCopy &h : c.directs)
    if (h.gate_pos > 0) direct(h, late_copy);
  cs.h2d1 = E.ev_time();
  HIPCHK(hipEventRecord(cs.h2d1, late_copy));

  // ---- tails ----------------------------------------------------------------------
  HIPCHK(hipMemcpyAsync(cs.err_host, dev_err, sizeof(int32_t), hipMemcpyDeviceToHost, compute));
  cs.tail_compute = E.ev_sync();
  HIPCHK(hipEventRecord(cs.tail_compute, compute));
  cs.tail_copy = E.ev_sync();
  HIPCHK(hipEventRecord(cs.tail_copy, copy));
  cs.tail_d2h = cs.tail_late_copy = cs.tail_late_comp = nullptr;
  if (do_out) {
    cs.tail_d2h = E.ev_sync();
    HIPCHK(hipEventRecord(cs.tail_d2h, E.d2h));
  }
  if (split) {
    // the late streams are not joined back into the caller's streams (that
    // would hold up the other call's work); atp_sync waits for them
    cs.tail_late_copy = E.ev_sync();
    HIPCHK(hipEventRecord(cs.tail_late_copy, late_copy));
    cs.tail_late_comp = E.ev_sync();
    HIPCHK(hipEventRecord(cs.tail_late_comp, late_comp));
  }
  cs.pending = true;
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
  double h2d_ms = 0, rep_ms = 0;
  hipEvent_t h2d_first = nullptr, h2d_last = nullptr;  // union span of both calls
  for (int which = 0; which < 2; ++which) {
    CallState &cs = which == 0 ? E.w : E.k;
    if (!cs.pending) continue;
    for (hipEvent_t e : {cs.tail_compute, cs.tail_copy, cs.tail_d2h, cs.tail_late_copy, cs.tail_late_comp}) {
      if (!e) continue;
      hipError_t err = hipEventSynchronize(e);
      if (err != hipSuccess && rc == ATP_OK) {
        rc = ATP_EHIP;
        msg = std::string("reshard failed on the GPU: ") + hipGetErrorString(err);
      }
    }
    cs.pending = false;
    if (*cs.err_host && rc == ATP_OK) {
      rc = ATP_EINVAL;
      msg = "block table invalid:";
      if (*cs.err_host & ERR_BAD_BLOCK) msg += " a block id is >= num_blocks;";
      if (*cs.err_host & ERR_LIVE_COUNT) msg += " the number of distinct live blocks differs from kv.live_blocks;";
    }
    // busy time of the repack kernels (levels), and the span they cover
    double busy = 0;
    for (const auto &L : cs.launches)
      if (L.kind != 2) busy += ms(L.e0, L.e1);
    (which == 0 ? t.repack_w_ms : t.repack_kv_ms) = busy;
    t.repack_span_ms += ms(cs.rep0, cs.rep1);
    rep_ms += busy;
    h2d_first = h2d_first ? h2d_first : cs.h2d0;
    if (cs.h2d1) h2d_last = cs.h2d1;
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
    for (CallState *c : {&E->w, &E->k})
      if (c->pending)
        for (hipEvent_t e : {c->tail_compute, c->tail_copy, c->tail_d2h, c->tail_late_copy, c->tail_late_comp})
          if (e) (void)hipEventSynchronize(e);
    delete E;
    P.exec = nullptr;
  }
}

void exec_launches(const Plan &P, std::vector<atp_launch> &out) {
  out.clear();
  if (P.exec) out = static_cast<const Exec *>(P.exec)->last_launches;
}

}  // namespace atp
