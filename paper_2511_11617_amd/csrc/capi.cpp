// capi.cpp — the extern "C" boundary of the reshard library: argument
// marshalling, error codes and the thread-local error message.  All work
// happens in plan.cpp (host planning) and exec.hip (GPU execution).
#include <algorithm>
#include <climits>
#include <cstring>
#include <functional>
#include <string>

#include "../../include/atp.h"
#include "exec.h"
#include "kvbudget.h"
#include "loader.h"
#include "plan.h"
#include "state.h"

struct atp_plan_obj {
  atp::Plan *p;
};

struct atp_st_obj {
  atp::StFiles *f;
};

struct atp_state_obj {
  atp::StateConn *c;
};

namespace {
thread_local std::string g_err;

int fail(int code, const std::string &m) {
  g_err = m;
  return code;
}

template <class F>
int guard(F &&f) {
  try {
    return f();
  } catch (const atp::Error &e) {
    return fail(e.code, e.what());
  } catch (const std::bad_alloc &) {
    return fail(ATP_ECAPACITY, "host allocation failed");
  } catch (const std::exception &e) {
    return fail(ATP_EINVAL, e.what());
  }
}

template <class T, class Src>
int copy_out(const Src &src, T *out, int32_t cap, int32_t *n) {
  if (!n) return fail(ATP_EINVAL, "n is NULL");
  *n = int32_t(src.size());
  if (out) {
    if (cap < *n) return fail(ATP_ECAPACITY, "output array too small");
    for (size_t i = 0; i < src.size(); ++i) out[i] = src[i];
  }
  return ATP_OK;
}
}  // namespace

extern "C" {

const char *atp_last_error(void) { return g_err.c_str(); }

int atp_plan(const atp_problem *problem, atp_plan_t **out) {
  return guard([&]() -> int {
    if (!out) return fail(ATP_EINVAL, "out is NULL");
    atp::Plan *p = atp::make_plan(problem);
    *out = new atp_plan_obj{p};
    return ATP_OK;
  });
}

void atp_plan_free(atp_plan_t *plan) {
  if (!plan) return;
  try {
    atp::exec_free(*plan->p);
  } catch (...) {
  }
  delete plan->p;
  delete plan;
}

int atp_reshard_weights(atp_plan_t *plan, void *arena, uint64_t arena_bytes, void *new_arena,
                        uint64_t new_arena_bytes, const void *inflow_host, uint64_t inflow_bytes,
                        void *outbound_host, uint64_t outbound_bytes, void *staging, uint64_t staging_bytes,
                        atp_stream compute, atp_stream copy) {
  return guard([&]() -> int {
    if (!plan) return fail(ATP_EINVAL, "plan is NULL");
    atp::exec_call(*plan->p, false, arena, arena_bytes, new_arena, new_arena_bytes, inflow_host, inflow_bytes,
                   outbound_host, outbound_bytes, nullptr, 0, staging, staging_bytes,
                   static_cast<hipStream_t>(compute), static_cast<hipStream_t>(copy));
    return ATP_OK;
  });
}

int atp_reshard_kv(atp_plan_t *plan, void *kv_arena, uint64_t kv_bytes, void *new_kv_arena, uint64_t new_kv_bytes,
                   const int32_t *block_table, int32_t n_seq, int32_t max_blocks, const void *inflow_host,
                   uint64_t inflow_bytes, void *outbound_host, uint64_t outbound_bytes, void *staging,
                   uint64_t staging_bytes, atp_stream compute, atp_stream copy) {
  return guard([&]() -> int {
    if (!plan) return fail(ATP_EINVAL, "plan is NULL");
    if (!plan->p->has_kv) return fail(ATP_EINVAL, "the problem has no KV cache");
    if (n_seq <= 0 || max_blocks <= 0) return fail(ATP_EINVAL, "block table must have positive size");
    atp::exec_call(*plan->p, true, kv_arena, kv_bytes, new_kv_arena, new_kv_bytes, inflow_host, inflow_bytes,
                   outbound_host, outbound_bytes, block_table, int64_t(n_seq) * max_blocks, staging, staging_bytes,
                   static_cast<hipStream_t>(compute), static_cast<hipStream_t>(copy));
    return ATP_OK;
  });
}

int atp_reshard_kv_noalloc(atp_plan_t *plan, void *kv_arena, uint64_t kv_bytes, void *new_kv_arena,
                           uint64_t new_kv_bytes, const int32_t *block_table, int32_t n_seq, int32_t max_blocks,
                           const void *inflow_host, uint64_t inflow_bytes, void *outbound_host,
                           uint64_t outbound_bytes, atp_stream compute, atp_stream copy) {
  return guard([&]() -> int {
    if (!plan) return fail(ATP_EINVAL, "plan is NULL");
    if (!plan->p->has_kv) return fail(ATP_EINVAL, "the problem has no KV cache");
    if (n_seq <= 0 || max_blocks <= 0) return fail(ATP_EINVAL, "block table must have positive size");
    atp::exec_call(*plan->p, true, kv_arena, kv_bytes, new_kv_arena, new_kv_bytes, inflow_host, inflow_bytes,
                   outbound_host, outbound_bytes, block_table, int64_t(n_seq) * max_blocks, nullptr, 0,
                   static_cast<hipStream_t>(compute), static_cast<hipStream_t>(copy), nullptr, true);
    return ATP_OK;
  });
}

uint64_t atp_scratch_bytes(void) { return atp::scratch_bytes(); }

int atp_sync(atp_plan_t *plan, atp_timing *out) {
  return guard([&]() -> int {
    if (!plan) return fail(ATP_EINVAL, "plan is NULL");
    return atp::exec_sync(*plan->p, out);
  });
}

int atp_warmup(atp_stream compute, atp_stream copy, int32_t events) {
  return guard([&]() -> int {
    atp::exec_warmup(compute, copy, events);
    return ATP_OK;
  });
}

int atp_plan_stats(const atp_plan_t *plan, atp_stats *out) {
  if (!plan || !out) return fail(ATP_EINVAL, "NULL argument");
  *out = plan->p->stats;
  return ATP_OK;
}

int atp_plan_tasks(const atp_plan_t *plan, int32_t space, atp_task *out, int32_t cap, int32_t *n) {
  if (!plan) return fail(ATP_EINVAL, "plan is NULL");
  if (space < 0 || space >= int32_t(plan->p->sp.size())) return fail(ATP_EINVAL, "bad space");
  return copy_out(plan->p->sp[space].tasks, out, cap, n);
}

int atp_plan_ranges(const atp_plan_t *plan, int32_t space, atp_range *out, int32_t cap, int32_t *n) {
  if (!plan) return fail(ATP_EINVAL, "plan is NULL");
  if (space < 0 || space >= int32_t(plan->p->sp.size())) return fail(ATP_EINVAL, "bad space");
  std::vector<atp_range> r;
  for (const atp::Rng &x : plan->p->sp[space].new_r) r.push_back({x.b, x.e});
  return copy_out(r, out, cap, n);
}

int atp_plan_old_ranges(const atp_plan_t *plan, int32_t space, atp_range *out, int32_t cap, int32_t *n) {
  if (!plan) return fail(ATP_EINVAL, "plan is NULL");
  if (space < 0 || space >= int32_t(plan->p->sp.size())) return fail(ATP_EINVAL, "bad space");
  std::vector<atp_range> r;
  for (const atp::Rng &x : plan->p->sp[space].old_r) r.push_back({x.b, x.e});
  return copy_out(r, out, cap, n);
}

int atp_plan_owner(const atp_plan_t *plan, int32_t *owner, int32_t cap, int32_t *n) {
  if (!plan) return fail(ATP_EINVAL, "plan is NULL");
  std::vector<int32_t> o(plan->p->owner.begin(), plan->p->owner.end());
  return copy_out(o, owner, cap, n);
}

int atp_plan_layout(const atp_plan_t *plan, int32_t t, uint64_t *old_offset, uint64_t *new_offset,
                    uint64_t *new_bytes) {
  if (!plan) return fail(ATP_EINVAL, "plan is NULL");
  if (t < 0 || t >= int32_t(plan->p->tp.size())) return fail(ATP_EINVAL, "bad tensor index");
  const atp::TensorPlan &tp = plan->p->tp[t];
  if (old_offset) *old_offset = tp.old_off;
  if (new_offset) *new_offset = tp.new_off;
  if (new_bytes) *new_bytes = tp.new_bytes;
  return ATP_OK;
}

int atp_plan_segments(const atp_plan_t *plan, int32_t which, atp_segment *out, int32_t cap, int32_t *n) {
  if (!plan) return fail(ATP_EINVAL, "plan is NULL");
  const atp::Plan &P = *plan->p;
  switch (which) {
    case ATP_SEG_INFLOW_W: return copy_out(P.w.seg_in, out, cap, n);
    case ATP_SEG_OUTBOUND_W: return copy_out(P.w.seg_out, out, cap, n);
    case ATP_SEG_INFLOW_KV: return copy_out(P.k.seg_in, out, cap, n);
    case ATP_SEG_OUTBOUND_KV: return copy_out(P.k.seg_out, out, cap, n);
    default: return fail(ATP_EINVAL, "bad segment kind");
  }
}

int atp_plan_launches(const atp_plan_t *plan, atp_launch *out, int32_t cap, int32_t *n) {
  if (!plan) return fail(ATP_EINVAL, "plan is NULL");
  std::vector<atp_launch> v;
  atp::exec_launches(*plan->p, v);
  return copy_out(v, out, cap, n);
}

int atp_plan_copies(const atp_plan_t *plan, int32_t which, atp_copy *out, int32_t cap, int32_t *n) {
  if (!plan) return fail(ATP_EINVAL, "plan is NULL");
  const atp::Plan &P = *plan->p;
  if (which != 0 && which != 1) return fail(ATP_EINVAL, "which must be 0 (weights) or 1 (KV)");
  const atp::CallPlan &c = which ? P.k : P.w;
  auto buf_of = [&](uint32_t slot) {
    if (slot == atp::BUF_STAGE) return int32_t(ATP_BUF_STAGING);
    if (slot == atp::BUF_OUT) return int32_t(P.inplace ? ATP_BUF_OLD : ATP_BUF_NEW);
    return int32_t(ATP_BUF_OLD);
  };
  auto dev_copy = [&](const atp::Fam &f, int op, int level) {
    atp_copy x{};
    x.op = op;
    x.level = level;
    x.src_buf = buf_of((f.flags >> atp::DF_SRC_SHIFT) & 3);
    x.dst_buf = buf_of((f.flags >> atp::DF_DST_SHIFT) & 3);
    x.flags = ((f.flags & atp::DF_SRC_IND) ? ATP_COPY_SRC_INDEXED : 0) |
              ((f.flags & atp::DF_DST_IND) ? ATP_COPY_DST_INDEXED : 0) |
              ((f.flags & atp::DF_BLOCKRANGE) ? ATP_COPY_BLOCK_RANGE : 0);
    x.src_off = f.src_off;
    x.dst_off = f.dst_off;
    x.src_pitch = f.src_pitch;
    x.dst_pitch = f.dst_pitch;
    x.src_stride = f.src_ostride;
    x.dst_stride = f.dst_ostride;
    x.item_begin = f.o_begin;
    x.item_end = f.o_end;
    x.run = f.run;
    x.rows = f.rows;
    return x;
  };
  auto host_copy = [&](const atp::HostCopy &h, int op, int level, bool to_host) {
    atp_copy x{};
    x.op = op;
    x.level = level;
    int32_t dev = h.dev_buf == atp::BUF_STAGE ? int32_t(ATP_BUF_STAGING) : buf_of(uint32_t(h.dev_buf));
    x.src_buf = to_host ? dev : int32_t(ATP_BUF_INFLOW);
    x.dst_buf = to_host ? int32_t(ATP_BUF_OUTBOUND) : dev;
    x.src_off = to_host ? h.dev_off : h.host_off;
    x.dst_off = to_host ? h.host_off : h.dev_off;
    uint64_t run = h.rows > 1 ? h.run : h.bytes;
    x.src_stride = to_host ? h.dev_pitch : run;
    x.dst_stride = to_host ? run : run;
    x.item_begin = 0;
    x.item_end = int64_t(h.rows > 1 ? h.rows : 1);
    x.run = run;
    x.rows = 1;
    return x;
  };
  std::vector<atp_copy> v;
  // outbound reads first, in the order the executor issues them (by the
  // level that needs them); each must finish before that level
  if (P.inplace) {
    std::vector<int> need(c.outbound.size(), INT32_MAX);
    for (const atp::Launch &L : c.levels)
      for (int o : L.wait_outbound) need[o] = std::min(need[o], L.level);
    for (int o : c.out_order)
      if (c.outbound[o].dev_buf != atp::BUF_STAGE)
        v.push_back(host_copy(c.outbound[o], ATP_COPY_D2H, need[o] == INT32_MAX ? -1 : need[o], true));
  }
  for (const atp::Launch &L : c.levels)
    for (int d = L.d0; d < L.d1; ++d) v.push_back(dev_copy(c.fams[d], ATP_COPY_REPACK, L.level));
  if (P.inplace)  // outbound gathered into staging at level 0 (KV)
    for (const atp::HostCopy &h : c.outbound)
      if (h.dev_buf == atp::BUF_STAGE) v.push_back(host_copy(h, ATP_COPY_D2H, 1, true));
  for (const atp::HostCopy &h : c.directs) {
    atp_copy x = host_copy(h, ATP_COPY_H2D, h.gate_level, false);
    x.after_d2h = h.gate_pos;
    v.push_back(x);
  }
  // inflow the copy kernel reads from the host buffer: in place after the
  // last level and after every outbound read of the call, out of place at
  // any time
  int32_t n_d2h = 0;
  for (const atp_copy &x : v) n_d2h += x.op == ATP_COPY_D2H && x.src_buf != ATP_BUF_STAGING;
  for (const atp::Launch &L : c.host_reads)
    for (int d = L.d0; d < L.d1; ++d) {
      atp_copy x = dev_copy(c.fams[d], ATP_COPY_H2D, P.inplace && c.n_levels > 0 ? c.n_levels - 1 : -1);
      x.src_buf = ATP_BUF_INFLOW;
      x.after_d2h = n_d2h;
      v.push_back(x);
    }
  for (const atp::Chunk &ch : c.chunks) {
    for (const atp::HostCopy &h : ch.copies) v.push_back(host_copy(h, ATP_COPY_H2D_RING, -1, false));
    for (const atp::Launch &L : ch.scatters)
      for (int d = L.d0; d < L.d1; ++d) v.push_back(dev_copy(c.fams[d], ATP_COPY_SCATTER, -1));
  }
  return copy_out(v, out, cap, n);
}

int atp_partition(int64_t total, int32_t parts, int32_t rule, atp_range *out) {
  return guard([&]() -> int {
    if (!out) return fail(ATP_EINVAL, "out is NULL");
    std::vector<atp::Rng> r;
    atp::partition(total, parts, rule, r);
    for (int i = 0; i < parts; ++i) out[i] = {r[i].b, r[i].e};
    return ATP_OK;
  });
}

int atp_st_open(const char *const *paths, int32_t n_paths, atp_st_t **out) {
  return guard([&]() -> int {
    if (!out) return fail(ATP_EINVAL, "out is NULL");
    atp::StFiles *f = atp::st_open(paths, n_paths);
    *out = new atp_st_obj{f};
    return ATP_OK;
  });
}

void atp_st_close(atp_st_t *st) {
  if (!st) return;
  delete st->f;
  delete st;
}

int atp_st_find(const atp_st_t *st, const char *name, atp_st_tensor *out) {
  return guard([&]() -> int {
    if (!st || !name || !out) return fail(ATP_EINVAL, "st, name or out is NULL");
    auto it = st->f->map.find(name);
    if (it == st->f->map.end()) return fail(ATP_EINVAL, std::string("no tensor named '") + name + "'");
    const atp::StTensor &t = it->second;
    atp_st_tensor o{};
    o.file = t.file;
    o.elem_bytes = t.elem_bytes;
    o.ndim = int32_t(t.shape.size());
    for (size_t i = 0; i < t.shape.size() && i < 8; ++i) o.shape[i] = int64_t(t.shape[i]);
    o.offset = t.begin;
    o.bytes = t.end - t.begin;
    *out = o;
    return ATP_OK;
  });
}

int atp_load_weights(const atp_plan_t *plan, const atp_st_t *st, const char *const *names, int32_t n_names,
                     void *inflow_host, uint64_t inflow_bytes, int32_t n_threads, atp_load_stats *stats) {
  return guard([&]() -> int {
    if (!plan || !st) return fail(ATP_EINVAL, "plan or st is NULL");
    atp::load_weights(*plan->p, *st->f, names, n_names, inflow_host, inflow_bytes, n_threads, stats);
    return ATP_OK;
  });
}

int atp_load_reshard_weights(atp_plan_t *plan, const atp_st_t *st, const char *const *names, int32_t n_names,
                             void *arena, uint64_t arena_bytes, void *new_arena, uint64_t new_arena_bytes,
                             void *inflow_host, uint64_t inflow_bytes, void *outbound_host, uint64_t outbound_bytes,
                             void *staging, uint64_t staging_bytes, atp_stream compute, atp_stream copy,
                             int32_t n_threads, atp_load_stats *stats) {
  return guard([&]() -> int {
    if (!plan || !st) return fail(ATP_EINVAL, "plan or st is NULL");
    // checks the names and builds the reads before anything starts
    atp::LoadJob job(*plan->p, *st->f, names, n_names, inflow_host, inflow_bytes, n_threads);
    job.start();
    const std::function<void(uint64_t)> await = [&job](uint64_t end) { job.await(end); };
    atp::exec_call(*plan->p, false, arena, arena_bytes, new_arena, new_arena_bytes, inflow_host, inflow_bytes,
                   outbound_host, outbound_bytes, nullptr, 0, staging, staging_bytes,
                   static_cast<hipStream_t>(compute), static_cast<hipStream_t>(copy), &await);
    try {
      job.finish(stats);
    } catch (...) {
      // a read failed after the reshard was enqueued over the partly read
      // buffer: let it drain before the caller may free anything
      try {
        atp::exec_sync(*plan->p, nullptr);
      } catch (...) {
      }
      throw;
    }
    return ATP_OK;
  });
}

int atp_load_reshard_weights_async(atp_plan_t *plan, const atp_st_t *st, const char *const *names,
                                   int32_t n_names, void *arena, uint64_t arena_bytes, void *new_arena,
                                   uint64_t new_arena_bytes, void *inflow_host, uint64_t inflow_bytes,
                                   void *outbound_host, uint64_t outbound_bytes, void *staging, uint64_t staging_bytes,
                                   atp_stream compute, atp_stream copy, int32_t n_threads) {
  return guard([&]() -> int {
    if (!plan || !st) return fail(ATP_EINVAL, "plan or st is NULL");
    atp::Plan *P = plan->p;
    // checks the names and builds the reads before anything starts; the job
    // lives until atp_sync has issued every piece (or the plan is freed)
    auto job = std::make_shared<atp::LoadJob>(*P, *st->f, names, n_names, inflow_host, inflow_bytes, n_threads);
    job->start();
    P->load_stats_valid = false;
    const std::function<void(uint64_t)> await = [job](uint64_t end) { job->await(end); };
    atp::exec_call(*P, false, arena, arena_bytes, new_arena, new_arena_bytes, inflow_host, inflow_bytes,
                   outbound_host, outbound_bytes, nullptr, 0, staging, staging_bytes,
                   static_cast<hipStream_t>(compute), static_cast<hipStream_t>(copy), &await, false, true,
                   [job, P]() {
                     job->finish(&P->load_stats);
                     P->load_stats_valid = true;
                   });
    return ATP_OK;
  });
}

int atp_plan_load_stats(const atp_plan_t *plan, atp_load_stats *out) {
  if (!plan || !out) return fail(ATP_EINVAL, "NULL argument");
  if (!plan->p->load_stats_valid) return fail(ATP_ESTATE, "no synced atp_load_reshard_weights_async on this plan");
  *out = plan->p->load_stats;
  return ATP_OK;
}

int atp_kv_evict_lru(const int32_t *table, int32_t n_seq, int32_t max_blocks, int64_t num_blocks,
                     const int64_t *last_use, uint64_t block_bytes, uint64_t budget_bytes, int32_t compact,
                     int32_t *keep, int32_t *new_table, atp_evict_stats *stats) {
  return guard([&]() -> int {
    atp::evict_lru(table, n_seq, max_blocks, num_blocks, last_use, block_bytes, budget_bytes, compact != 0, keep,
                   new_table, stats);
    return ATP_OK;
  });
}

int atp_daemon_serve(const char *socket_path, int32_t device) {
  return guard([&]() -> int { return atp::daemon_serve(socket_path, device); });
}

int atp_state_connect(const char *socket_path, atp_state_t **out) {
  return guard([&]() -> int {
    if (!out) return fail(ATP_EINVAL, "out is NULL");
    *out = new atp_state_obj{atp::state_connect(socket_path)};
    return ATP_OK;
  });
}

void atp_state_disconnect(atp_state_t *s) {
  if (!s) return;
  atp::state_disconnect(s->c);
  delete s;
}

int atp_state_alloc(atp_state_t *s, const char *name, uint64_t bytes, void **dev_ptr) {
  return guard([&]() -> int {
    if (!s || !dev_ptr) return fail(ATP_EINVAL, "state or dev_ptr is NULL");
    *dev_ptr = atp::state_alloc(*s->c, name, bytes);
    return ATP_OK;
  });
}

int atp_state_open(atp_state_t *s, const char *name, void **dev_ptr, uint64_t *bytes) {
  return guard([&]() -> int {
    if (!s || !dev_ptr) return fail(ATP_EINVAL, "state or dev_ptr is NULL");
    *dev_ptr = atp::state_open(*s->c, name, bytes);
    return ATP_OK;
  });
}

int atp_state_release(atp_state_t *s, void *dev_ptr) {
  return guard([&]() -> int {
    if (!s) return fail(ATP_EINVAL, "state is NULL");
    atp::state_release(*s->c, dev_ptr);
    return ATP_OK;
  });
}

int atp_state_free(atp_state_t *s, const char *name) {
  return guard([&]() -> int {
    if (!s) return fail(ATP_EINVAL, "state is NULL");
    atp::state_free(*s->c, name);
    return ATP_OK;
  });
}

int atp_state_put(atp_state_t *s, const char *name, const void *data, uint64_t bytes) {
  return guard([&]() -> int {
    if (!s) return fail(ATP_EINVAL, "state is NULL");
    atp::state_put(*s->c, name, data, bytes);
    return ATP_OK;
  });
}

int atp_state_get(atp_state_t *s, const char *name, void *data, uint64_t cap, uint64_t *bytes) {
  return guard([&]() -> int {
    if (!s) return fail(ATP_EINVAL, "state is NULL");
    uint64_t n = 0;
    try {
      n = atp::state_get(*s->c, name, data, cap);
    } catch (const atp::Error &e) {
      if (e.code == ATP_ECAPACITY && bytes) *bytes = atp::state_get(*s->c, name, nullptr, 0);
      throw;
    }
    if (bytes) *bytes = n;
    return ATP_OK;
  });
}

int atp_state_list(atp_state_t *s, char *text, uint64_t cap, uint64_t *bytes) {
  return guard([&]() -> int {
    if (!s) return fail(ATP_EINVAL, "state is NULL");
    std::string t = atp::state_list(*s->c);
    if (bytes) *bytes = t.size() + 1;
    if (text) {
      if (cap < t.size() + 1) return fail(ATP_ECAPACITY, "text buffer too small");
      memcpy(text, t.c_str(), t.size() + 1);
    }
    return ATP_OK;
  });
}

int atp_state_shutdown(atp_state_t *s) {
  return guard([&]() -> int {
    if (!s) return fail(ATP_EINVAL, "state is NULL");
    atp::state_shutdown(*s->c);
    return ATP_OK;
  });
}

}  // extern "C"
