// plan.cpp — host planner: partitions (Alg. 1 floor rule, Sec. III-B
// unequal widths), the CMM loop (Alg. 1), Eq. 1 statistics, lowering of
// this GPU's share to copy families, the in-place hazard scheduler and the
// landing-ring chunking (Sec. III-C execution scheduler, pre-allocation).
#include "plan.h"

#include <algorithm>
#include <chrono>
#include <cstring>
#include <functional>
#include <memory>
#include <numeric>

namespace atp {
namespace {

[[noreturn]] void fail(int code, const std::string &m) { throw Error(code, m); }

uint64_t align_up(uint64_t x, uint64_t a) { return (x + a - 1) / a * a; }

// ---- interval sets (sorted, disjoint) --------------------------------------
using Set = std::vector<Rng>;

Set set_inter(const Set &s, Rng r) {
  Set out;
  for (const Rng &x : s) {
    int64_t lo = std::max(x.b, r.b), hi = std::min(x.e, r.e);
    if (lo < hi) out.push_back({lo, hi});
  }
  return out;
}

Set set_sub(const Set &s, Rng r) {
  Set out;
  for (const Rng &x : s) {
    if (x.e <= r.b || x.b >= r.e) {
      out.push_back(x);
      continue;
    }
    if (x.b < r.b) out.push_back({x.b, r.b});
    if (x.e > r.e) out.push_back({r.e, x.e});
  }
  return out;
}

int64_t measure(const Set &s) {
  int64_t m = 0;
  for (const Rng &x : s) m += x.e - x.b;
  return m;
}

Set union_of(std::vector<Rng> v) {
  std::sort(v.begin(), v.end(), [](Rng a, Rng b) { return a.b < b.b || (a.b == b.b && a.e < b.e); });
  Set out;
  for (const Rng &x : v) {
    if (x.b >= x.e) continue;
    if (!out.empty() && x.b <= out.back().e)
      out.back().e = std::max(out.back().e, x.e);
    else
      out.push_back(x);
  }
  return out;
}

int64_t overlap(Rng a, Rng b) { return std::max<int64_t>(0, std::min(a.e, b.e) - std::max(a.b, b.b)); }

uint64_t tensor_unit_bytes(const atp_tensor &t) {
  return uint64_t(t.kind == ATP_ROWS ? t.unit * t.cols : t.rows * t.unit) * uint64_t(t.elem_bytes);
}

uint64_t shard_bytes(const atp_tensor &t, Rng r) { return uint64_t(r.e - r.b) * tensor_unit_bytes(t); }

}  // namespace

// ---- partitions --------------------------------------------------------------
void partition(int64_t H, int M, int rule, std::vector<Rng> &out) {
  if (M <= 0 || H < 0) fail(ATP_EINVAL, "partition: bad size");
  out.assign(M, {0, 0});
  if (rule == ATP_RULE_FLOOR) {
    // Alg. 1: target j covers [floor(j H / M), floor((j + 1) H / M))
    for (int j = 0; j < M; ++j) {
      __int128 lo = (__int128)j * H / M, hi = (__int128)(j + 1) * H / M;
      out[j] = {int64_t(lo), int64_t(hi)};
    }
  } else if (rule == ATP_RULE_CEIL_FIRST) {
    // Sec. III-B: ceil(H/M) wide shards first, then floor(H/M)
    int64_t q = H / M, r = H % M, at = 0;
    for (int j = 0; j < M; ++j) {
      int64_t w = q + (j < r ? 1 : 0);
      out[j] = {at, at + w};
      at += w;
    }
  } else {
    fail(ATP_EINVAL, "partition: rule must be FLOOR or CEIL_FIRST");
  }
}

namespace {

// ---- problem intake ------------------------------------------------------------
// The n ranges of one side (old or new) of space s from a rule other than GQA.
void ranges_by_rule(int s, const char *side, int rule, int64_t H, int n, const atp_range *given,
                    const int64_t *widths, std::vector<Rng> &out) {
  const std::string where = "space " + std::to_string(s) + ": " + side;
  if (rule == ATP_RULE_EXPLICIT) {
    if (!given) fail(ATP_EINVAL, where + " ranges missing");
    out.resize(n);
    for (int j = 0; j < n; ++j) out[j] = {given[j].begin, given[j].end};
  } else if (rule == ATP_RULE_FLOOR || rule == ATP_RULE_CEIL_FIRST) {
    partition(H, n, rule, out);
  } else if (rule == ATP_RULE_WIDTHS) {
    if (!widths) fail(ATP_EINVAL, where + " widths missing");
    out.resize(n);
    int64_t at = 0;
    for (int j = 0; j < n; ++j) {
      if (widths[j] < 0 || widths[j] > H - at) fail(ATP_EINVAL, where + " widths must add up to total_units");
      out[j] = {at, at + widths[j]};
      at += widths[j];
    }
    if (at != H) fail(ATP_EINVAL, where + " widths must add up to total_units");
  } else {
    fail(ATP_EINVAL, where + " unknown rule");
  }
}

// Every range inside [0, H) and together covering it.
void check_cover(int s, const char *side, int64_t H, const std::vector<Rng> &r) {
  const std::string where = "space " + std::to_string(s) + ": " + side;
  for (size_t j = 0; j < r.size(); ++j)
    if (r[j].b < 0 || r[j].e < r[j].b || r[j].e > H)
      fail(ATP_EINVAL, where + " range " + std::to_string(j) + " out of bounds");
  Set u = union_of(r);
  if (u.size() != 1 || u[0].b != 0 || u[0].e != H) fail(ATP_EINVAL, where + " ranges do not cover [0, H)");
}

void resolve_spaces(Plan &P) {
  const atp_problem &p = P.prob;
  if (p.n_spaces <= 0 || !p.spaces) fail(ATP_EINVAL, "no partition spaces");
  P.sp.resize(p.n_spaces);
  int N = p.spaces[0].old_tp, M = p.spaces[0].new_tp;
  if (N <= 0 || M <= 0) fail(ATP_EINVAL, "old_tp and new_tp must be positive");
  for (int s = 0; s < p.n_spaces; ++s) {
    const atp_space &in = p.spaces[s];
    SpacePlan &sp = P.sp[s];
    if (in.old_tp != N || in.new_tp != M) fail(ATP_EINVAL, "every space must have the same old_tp and new_tp");
    if (in.total_units <= 0) fail(ATP_EINVAL, "space " + std::to_string(s) + ": total_units must be positive");
    sp.H = in.total_units;
    sp.N = N;
    sp.M = M;
  }
  // old ranges (rank order) and new ranges (target order): rule-based first,
  // then those that follow a query-head space (GQA)
  for (int side = 0; side < 2; ++side) {
    const bool old_side = side == 0;
    const char *name = old_side ? "old" : "new";
    for (int pass = 0; pass < 2; ++pass) {
      for (int s = 0; s < p.n_spaces; ++s) {
        const atp_space &in = p.spaces[s];
        SpacePlan &sp = P.sp[s];
        const int rule = old_side ? in.old_rule : in.new_rule;
        const bool gqa = rule == ATP_RULE_GQA;
        if ((pass == 0) == gqa) continue;
        std::vector<Rng> &out = old_side ? sp.old_r : sp.new_r;
        const int n = old_side ? N : M;
        if (!gqa) {
          ranges_by_rule(s, name, rule, sp.H, n, old_side ? in.old_ranges : in.new_ranges,
                         old_side ? in.old_widths : in.new_widths, out);
        } else {
          int q = in.gqa_space;
          if (q < 0 || q >= p.n_spaces || q == s ||
              (old_side ? p.spaces[q].old_rule : p.spaces[q].new_rule) == ATP_RULE_GQA)
            fail(ATP_EINVAL, "space " + std::to_string(s) + ": bad gqa_space");
          if (in.gqa_group <= 0) fail(ATP_EINVAL, "space " + std::to_string(s) + ": gqa_group must be positive");
          const int64_t g = in.gqa_group;
          const std::vector<Rng> &qr = old_side ? P.sp[q].old_r : P.sp[q].new_r;
          out.resize(n);
          for (int j = 0; j < n; ++j) out[j] = {qr[j].b / g, std::min<int64_t>(sp.H, (qr[j].e + g - 1) / g)};
        }
        check_cover(s, name, sp.H, out);
        if (old_side) {
          // Alg. 1: H is the largest end of any range, dead ranks included
          int64_t maxe = 0;
          for (const Rng &r : out) maxe = std::max(maxe, r.e);
          if (maxe != sp.H)
            fail(ATP_EINVAL, "space " + std::to_string(s) + ": total_units must equal the largest old range end");
        }
      }
    }
  }
}

void resolve_ranks(Plan &P) {
  const atp_problem &p = P.prob;
  int N = P.sp[0].N, M = P.sp[0].M;
  std::vector<char> dead(N, 0);
  if (p.n_failed < 0 || (p.n_failed > 0 && !p.failed)) fail(ATP_EINVAL, "bad failed list");
  for (int k = 0; k < p.n_failed; ++k) {
    int r = p.failed[k];
    if (r < 0 || r >= N) fail(ATP_EINVAL, "failed rank out of range");
    if (dead[r]) fail(ATP_EINVAL, "failed rank listed twice");
    dead[r] = 1;
    P.failed.push_back(r);
  }
  std::vector<int> alive;
  for (int i = 0; i < N; ++i)
    if (!dead[i]) alive.push_back(i);
  if (int(alive.size()) != M)
    fail(ATP_EINVAL, "new_tp must equal the number of surviving ranks (" + std::to_string(alive.size()) + ")");
  if (p.self_old_rank < 0 || p.self_old_rank >= N || dead[p.self_old_rank])
    fail(ATP_EINVAL, "self_old_rank must be a surviving rank");
  P.self_old = p.self_old_rank;

  int assign = p.flags & 0xF;
  if (assign == ATP_ASSIGN_INORDER) {
    // reading of Alg. 1: target j is hosted by the j-th survivor in rank order
    P.owner = alive;
  } else if (assign == ATP_ASSIGN_MAXRETAIN) {
    if (M > 10) fail(ATP_EINVAL, "MAXRETAIN searches M! permutations; M must be <= 10");
    std::vector<int> perm = alive, best;
    __int128 best_v = -1;
    do {
      __int128 v = 0;
      for (int j = 0; j < M; ++j)
        for (const SpacePlan &sp : P.sp)
          v += (__int128)sp.unit_bytes * overlap(sp.old_r[perm[j]], sp.new_r[j]);
      if (v > best_v) {
        best_v = v;
        best = perm;
      }
    } while (std::next_permutation(perm.begin(), perm.end()));
    P.owner = best;
  } else {
    fail(ATP_EINVAL, "unknown assignment flag");
  }
  P.self_new = int(std::find(P.owner.begin(), P.owner.end(), P.self_old) - P.owner.begin());
}

void resolve_tensors(Plan &P) {
  const atp_problem &p = P.prob;
  if (p.n_tensors < 0 || (p.n_tensors > 0 && !p.tensors)) fail(ATP_EINVAL, "bad tensor list");
  bool any_auto = false, any_explicit = false;
  for (int i = 0; i < p.n_tensors; ++i) {
    const atp_tensor &t = p.tensors[i];
    if (t.space < 0 || t.space >= p.n_spaces) fail(ATP_EINVAL, "tensor " + std::to_string(i) + ": bad space");
    if (t.kind != ATP_ROWS && t.kind != ATP_COLS) fail(ATP_EINVAL, "tensor " + std::to_string(i) + ": bad kind");
    if (t.elem_bytes <= 0 || t.rows <= 0 || t.cols <= 0 || t.unit <= 0)
      fail(ATP_EINVAL, "tensor " + std::to_string(i) + ": sizes must be positive");
    int64_t dim = t.kind == ATP_ROWS ? t.rows : t.cols;
    if (dim != t.unit * P.sp[t.space].H)
      fail(ATP_EINVAL, "tensor " + std::to_string(i) + ": sharded dimension must be unit * total_units");
    (t.old_offset == ATP_OFFSET_AUTO ? any_auto : any_explicit) = true;
  }
  if (any_auto && any_explicit) fail(ATP_EINVAL, "old offsets must be all explicit or all ATP_OFFSET_AUTO");
  for (const SpacePlan &sp : P.sp) (void)sp;
  for (int i = 0; i < p.n_tensors; ++i) P.sp[p.tensors[i].space].unit_bytes += tensor_unit_bytes(p.tensors[i]);
  P.tp.resize(p.n_tensors);
  uint64_t at_old = 0;
  for (int i = 0; i < p.n_tensors; ++i) {
    TensorPlan &tp = P.tp[i];
    tp.t = p.tensors[i];
    tp.old_r = P.sp[tp.t.space].old_r[P.self_old];
    tp.old_bytes = shard_bytes(tp.t, tp.old_r);
    if (any_auto) {
      tp.old_off = at_old;
      at_old = align_up(at_old + tp.old_bytes, 256);
    } else {
      tp.old_off = tp.t.old_offset;
      at_old = std::max(at_old, align_up(tp.old_off + tp.old_bytes, 256));
    }
  }
  // explicit old shards must not overlap
  if (any_explicit) {
    std::vector<std::pair<uint64_t, uint64_t>> iv;
    for (const TensorPlan &tp : P.tp)
      if (tp.old_bytes) iv.push_back({tp.old_off, tp.old_off + tp.old_bytes});
    std::sort(iv.begin(), iv.end());
    for (size_t i = 1; i < iv.size(); ++i)
      if (iv[i].first < iv[i - 1].second) fail(ATP_EINVAL, "old shards overlap");
  }
  P.w.old_bytes = at_old;
}

void resolve_kv(Plan &P) {
  const atp_problem &p = P.prob;
  P.has_kv = p.kv != nullptr;
  if (!P.has_kv) return;
  P.kv = *p.kv;
  const atp_kv &kv = P.kv;
  if (kv.space < 0 || kv.space >= p.n_spaces) fail(ATP_EINVAL, "kv: bad space");
  if (kv.num_layers <= 0 || kv.block_tokens <= 0 || kv.head_dim <= 0 || kv.elem_bytes <= 0 || kv.num_blocks <= 0)
    fail(ATP_EINVAL, "kv: sizes must be positive");
  if (kv.live_blocks < 0 || kv.live_blocks > kv.num_blocks) fail(ATP_EINVAL, "kv: live_blocks out of range");
  if (kv.num_blocks >= (int64_t(1) << 31)) fail(ATP_EINVAL, "kv: num_blocks must fit int32");
  if (kv.layout != ATP_KV_HEAD_MAJOR && kv.layout != ATP_KV_TOKEN_MAJOR) fail(ATP_EINVAL, "kv: bad layout");
  P.sp[kv.space].unit_bytes += uint64_t(kv.num_layers) * 2 * uint64_t(kv.live_blocks) * kv.block_tokens *
                               uint64_t(kv.head_dim) * kv.elem_bytes;
}

// ---- Alg. 1 ------------------------------------------------------------------------
void run_cmm(Plan &P) {
  bool greedy = P.flags & ATP_PLAN_GREEDY, full = P.flags & ATP_PLAN_FULL;
  if (greedy && full) fail(ATP_EINVAL, "GREEDY and FULL are exclusive");
  std::vector<char> dead(P.sp[0].N, 0);
  for (int r : P.failed) dead[r] = 1;
  for (SpacePlan &sp : P.sp) {
    sp.tasks.clear();
    for (int j = 0; j < sp.M; ++j) {
      int host = P.owner[j];
      Set tar;
      if (sp.new_r[j].b < sp.new_r[j].e) tar.push_back(sp.new_r[j]);
      // sources: the target's host first, then the other ranks ascending
      std::vector<int> order{host};
      for (int i = 0; i < sp.N; ++i)
        if (i != host) order.push_back(i);
      for (int i : order) {
        if (dead[i] || full) continue;
        if (greedy && i != host) continue;  // Sec. V Greedy: no cross-device fill
        Set inter = set_inter(tar, sp.old_r[i]);
        if (inter.empty()) continue;
        for (const Rng &x : inter)
          sp.tasks.push_back({i == host ? ATP_KEEP : ATP_P2P, i, j, host, x.b, x.e});
        tar = set_sub(tar, sp.old_r[i]);
      }
      for (const Rng &x : tar) sp.tasks.push_back({ATP_RELOAD, -1, j, host, x.b, x.e});
    }
  }
}

void global_stats(Plan &P) {
  std::vector<char> dead(P.sp[0].N, 0);
  for (int r : P.failed) dead[r] = 1;
  atp_stats &st = P.stats;
  for (const SpacePlan &sp : P.sp) {
    for (const atp_task &t : sp.tasks) {
      uint64_t b = uint64_t(t.end - t.begin) * sp.unit_bytes;
      if (t.kind == ATP_KEEP) st.global_keep += b;
      else if (t.kind == ATP_P2P) st.global_p2p += b;
      else st.global_reload += b;
    }
    // Eq. 1: per target, its size minus what surviving sources cover
    int64_t minr = 0;
    for (int j = 0; j < sp.M; ++j) {
      std::vector<Rng> cov;
      for (int i = 0; i < sp.N; ++i) {
        if (dead[i]) continue;
        Rng a = sp.old_r[i], t = sp.new_r[j];
        int64_t lo = std::max(a.b, t.b), hi = std::min(a.e, t.e);
        if (lo < hi) cov.push_back({lo, hi});
      }
      minr += (sp.new_r[j].e - sp.new_r[j].b) - measure(union_of(cov));
    }
    st.reload_min += uint64_t(minr) * sp.unit_bytes;
  }
}

// ---- lowering ------------------------------------------------------------------------
constexpr uint64_t kMaxRun = uint64_t(1) << 30;

uint32_t bufs(uint32_t src, uint32_t dst) { return (src << DF_SRC_SHIFT) | (dst << DF_DST_SHIFT); }

// Contiguous copy of `len` bytes, split so that every run fits 32 bits.
void push_contig(std::vector<Fam> &out, uint64_t src, uint64_t dst, uint64_t len, uint32_t flags) {
  while (len) {
    uint64_t n = std::min(len, kMaxRun);
    Fam f;
    f.src_off = src;
    f.dst_off = dst;
    f.run = n;
    f.flags = flags;
    out.push_back(f);
    src += n;
    dst += n;
    len -= n;
  }
}

// The rectangle of units [a, b) of tensor `tp` in a shard that starts at
// unit r0, seen as a copy family on one side (the other side is set later).
struct Rect {
  uint64_t off, run, items, pitch;  // items lines of `run` bytes at `pitch`
};

Rect rect_of(const TensorPlan &tp, uint64_t shard_off, Rng shard, int64_t a, int64_t b) {
  const atp_tensor &t = tp.t;
  uint64_t eb = t.elem_bytes;
  if (t.kind == ATP_ROWS) {
    uint64_t ub = uint64_t(t.unit) * t.cols * eb;
    return {shard_off + uint64_t(a - shard.b) * ub, uint64_t(b - a) * ub, 1, 0};
  }
  uint64_t cb = uint64_t(t.unit) * eb;
  uint64_t pitch = uint64_t(shard.e - shard.b) * cb;
  return {shard_off + uint64_t(a - shard.b) * cb, uint64_t(b - a) * cb, uint64_t(t.rows), pitch};
}

// Copy between two rectangles of equal shape -> families.
void push_rect_copy(std::vector<Fam> &out, const Rect &s, const Rect &d, uint32_t flags) {
  if (s.items == 1 || (s.run == s.pitch && d.run == d.pitch)) {
    push_contig(out, s.off, d.off, s.run * s.items, flags);
    return;
  }
  Fam f;
  f.src_off = s.off;
  f.dst_off = d.off;
  f.src_ostride = s.pitch;
  f.dst_ostride = d.pitch;
  f.o_begin = 0;
  f.o_end = int64_t(s.items);
  f.run = s.run;
  f.flags = flags;
  if (f.run > kMaxRun) fail(ATP_EINVAL, "a single row is larger than 1 GiB");
  out.push_back(f);
}

struct Pending {  // inflow / outbound piece before scheduling
  Fam fam;            // device-side family; host side is packed
  uint64_t host_off;  // packed position
  bool contiguous;
};

void lower_weights(Plan &P, std::vector<Fam> &retained, std::vector<Pending> &inflow,
                   std::vector<Pending> &outbound) {
  CallPlan &c = P.w;
  uint32_t rflags = bufs(BUF_IN, BUF_OUT);
  uint64_t cur_in = 0, cur_out = 0;
  // new packed layout (pre-allocation pass of Sec. III-C)
  uint64_t at = 0;
  for (TensorPlan &tp : P.tp) {
    tp.new_r = P.sp[tp.t.space].new_r[P.self_new];
    tp.new_bytes = shard_bytes(tp.t, tp.new_r);
    tp.new_off = at;
    at = align_up(at + tp.new_bytes, 256);
  }
  c.new_bytes = at;
  for (int ti = 0; ti < int(P.tp.size()); ++ti) {
    TensorPlan &tp = P.tp[ti];
    const SpacePlan &sp = P.sp[tp.t.space];
    uint64_t ub = tensor_unit_bytes(tp.t);
    for (const atp_task &x : sp.tasks) {
      if (x.dst != P.self_new) continue;
      Rect d = rect_of(tp, tp.new_off, tp.new_r, x.begin, x.end);
      if (x.kind == ATP_KEEP) {
        Rect s = rect_of(tp, tp.old_off, tp.old_r, x.begin, x.end);
        push_rect_copy(retained, s, d, rflags);
        c.retained += uint64_t(x.end - x.begin) * ub;
      } else {
        uint64_t bytes = uint64_t(x.end - x.begin) * ub;
        Rect h{cur_in, d.run, d.items, d.run};
        std::vector<Fam> tmp;
        push_rect_copy(tmp, h, d, bufs(BUF_STAGE, BUF_OUT));
        uint64_t hoff = cur_in;
        for (Fam &f : tmp) {
          Pending pd{f, hoff, f.o_end - f.o_begin == 1};
          hoff += f.bytes();
          inflow.push_back(pd);
        }
        atp_segment sg{ti, tp.t.layer, 0, x.kind, x.begin, x.end, cur_in, bytes};
        c.seg_in.push_back(sg);
        cur_in += bytes;
      }
    }
    // dropped outbound: what peers take from this GPU and it does not keep
    for (const atp_task &x : sp.tasks) {
      if (x.kind != ATP_P2P || x.src != P.self_old) continue;
      Set rest = set_sub({{x.begin, x.end}}, tp.new_r);
      for (const Rng &r : rest) {
        uint64_t bytes = uint64_t(r.e - r.b) * ub;
        Rect s = rect_of(tp, tp.old_off, tp.old_r, r.b, r.e);
        Rect h{cur_out, s.run, s.items, s.run};
        std::vector<Fam> tmp;
        push_rect_copy(tmp, s, h, bufs(BUF_IN, BUF_STAGE));
        uint64_t hoff = cur_out;
        for (Fam &f : tmp) {
          outbound.push_back({f, hoff, f.o_end - f.o_begin == 1});
          hoff += f.bytes();
        }
        atp_segment sg{ti, tp.t.layer, 0, ATP_P2P, r.b, r.e, cur_out, bytes};
        c.seg_out.push_back(sg);
        cur_out += bytes;
      }
    }
  }
  c.inflow = cur_in;
  c.outbound_bytes = cur_out;
}

void lower_kv(Plan &P, std::vector<Fam> &retained, std::vector<Pending> &inflow, std::vector<Pending> &outbound) {
  CallPlan &c = P.k;
  const atp_kv &kv = P.kv;
  const SpacePlan &sp = P.sp[kv.space];
  Rng ho = sp.old_r[P.self_old], hn = sp.new_r[P.self_new];
  uint64_t eb = kv.elem_bytes, bt = kv.block_tokens, hd = kv.head_dim;
  uint64_t nb = kv.num_blocks, live = kv.live_blocks;
  bool tok = kv.layout == ATP_KV_TOKEN_MAJOR;
  // compact: the new planes hold the live blocks only, each at its rank
  const bool compact = P.flags & ATP_KV_COMPACT;
  const uint64_t nb_new = compact ? live : nb;
  const uint32_t dst_ind = compact ? 0u : uint32_t(DF_DST_IND);
  uint64_t hb = bt * hd * eb;                  // one head of one block
  uint64_t obs = uint64_t(ho.e - ho.b) * hb;   // old block bytes
  uint64_t nbs = uint64_t(hn.e - hn.b) * hb;   // new block bytes
  c.old_bytes = uint64_t(kv.num_layers) * 2 * nb * obs;
  c.new_bytes = uint64_t(kv.num_layers) * 2 * nb_new * nbs;
  // a head range [a, b) of a block, in a block whose heads start at h0
  auto side = [&](uint64_t base, uint64_t block_bytes, int64_t h0, int64_t nh, int64_t a, int64_t b, Fam &f,
                  bool src) {
    uint64_t off, run, rows, pitch;
    if (!tok) {
      off = base + uint64_t(a - h0) * hb;
      run = uint64_t(b - a) * hb;
      rows = 1;
      pitch = 0;
    } else {
      off = base + uint64_t(a - h0) * hd * eb;
      run = uint64_t(b - a) * hd * eb;
      rows = bt;
      pitch = uint64_t(nh) * hd * eb;
    }
    f.run = run;
    f.rows = rows;
    if (src) {
      f.src_off = off;
      f.src_pitch = pitch;
      f.src_ostride = block_bytes;
    } else {
      f.dst_off = off;
      f.dst_pitch = pitch;
      f.dst_ostride = block_bytes;
    }
  };
  uint64_t cur_in = 0, cur_out = 0;
  for (int l = 0; l < kv.num_layers; ++l) {
    for (int which = 0; which < 2; ++which) {
      uint64_t g = uint64_t(l) * 2 + which;
      uint64_t obase = g * nb * obs, nbase = g * nb_new * nbs;
      for (const atp_task &x : sp.tasks) {
        if (x.dst != P.self_new) continue;
        Fam f;
        side(nbase, nbs, hn.b, hn.e - hn.b, x.begin, x.end, f, false);
        uint64_t bytes = live * f.rows * f.run;
        if (x.kind == ATP_KEEP) {
          side(obase, obs, ho.b, ho.e - ho.b, x.begin, x.end, f, true);
          f.flags = bufs(BUF_IN, BUF_OUT) | DF_SRC_IND | dst_ind;
          if (P.inplace) {
            f.flags |= DF_BLOCKRANGE;
            f.o_begin = 0;
            f.o_end = int64_t(nb);
          } else {
            f.o_begin = 0;
            f.o_end = int64_t(live);
          }
          if (live) retained.push_back(f);
          c.retained += bytes;
        } else {
          f.src_off = cur_in;
          f.src_pitch = f.run;
          f.src_ostride = f.rows * f.run;
          f.o_begin = 0;
          f.o_end = int64_t(live);
          f.flags = bufs(BUF_STAGE, BUF_OUT) | dst_ind;
          if (live) inflow.push_back({f, cur_in, false});
          atp_segment sg{-1, l, which, x.kind, x.begin, x.end, cur_in, bytes};
          c.seg_in.push_back(sg);
          cur_in += bytes;
        }
      }
      for (const atp_task &x : sp.tasks) {
        if (x.kind != ATP_P2P || x.src != P.self_old) continue;
        Set rest = set_sub({{x.begin, x.end}}, hn);
        for (const Rng &r : rest) {
          Fam f;
          side(obase, obs, ho.b, ho.e - ho.b, r.b, r.e, f, true);
          uint64_t bytes = live * f.rows * f.run;
          f.dst_off = cur_out;
          f.dst_pitch = f.run;
          f.dst_ostride = f.rows * f.run;
          f.o_begin = 0;
          f.o_end = int64_t(live);
          f.flags = bufs(BUF_IN, BUF_STAGE) | DF_SRC_IND;
          if (live) outbound.push_back({f, cur_out, false});
          atp_segment sg{-1, l, which, ATP_P2P, r.b, r.e, cur_out, bytes};
          c.seg_out.push_back(sg);
          cur_out += bytes;
        }
      }
    }
  }
  c.inflow = cur_in;
  c.outbound_bytes = cur_out;
}

// ---- spans and in-place scheduling ---------------------------------------------------
struct Span {
  uint64_t lo, hi;  // [lo, hi)
};

Span src_span(const Fam &f, int64_t p0, int64_t p1) {
  uint64_t lo = f.src_off + uint64_t(p0 - (f.flags & DF_BLOCKRANGE ? 0 : f.o_begin)) * f.src_ostride;
  uint64_t hi = f.src_off + uint64_t(p1 - 1 - (f.flags & DF_BLOCKRANGE ? 0 : f.o_begin)) * f.src_ostride +
                (f.rows - 1) * f.src_pitch + f.run;
  return {lo, hi};
}

Span dst_span(const Fam &f, int64_t p0, int64_t p1) {
  uint64_t lo = f.dst_off + uint64_t(p0 - (f.flags & DF_BLOCKRANGE ? 0 : f.o_begin)) * f.dst_ostride;
  uint64_t hi = f.dst_off + uint64_t(p1 - 1 - (f.flags & DF_BLOCKRANGE ? 0 : f.o_begin)) * f.dst_ostride +
                (f.rows - 1) * f.dst_pitch + f.run;
  return {lo, hi};
}

bool spans_meet(Span a, Span b) { return a.lo < b.hi && b.lo < a.hi; }

// A family restricted to outer items [p0, p1) (same coordinates as o_begin).
Fam sub_fam(const Fam &f, int64_t p0, int64_t p1) {
  Fam g = f;
  if (f.flags & (DF_BLOCKRANGE | DF_SRC_IND | DF_DST_IND)) {
    // indexed sides use absolute positions; only the range changes
    g.o_begin = p0;
    g.o_end = p1;
    return g;
  }
  g.src_off = f.src_off + uint64_t(p0 - f.o_begin) * f.src_ostride;
  g.dst_off = f.dst_off + uint64_t(p0 - f.o_begin) * f.dst_ostride;
  g.o_begin = 0;
  g.o_end = p1 - p0;
  return g;
}

// True when every byte of the family would be copied onto itself.
bool is_identity(const Fam &f) {
  if (f.rows > 1 && f.src_pitch != f.dst_pitch) return false;
  if (f.flags & DF_BLOCKRANGE) {
    // items are absolute block ids: item p sits at off + p * stride
    if (f.o_end - f.o_begin == 1)
      return f.src_off + uint64_t(f.o_begin) * f.src_ostride == f.dst_off + uint64_t(f.o_begin) * f.dst_ostride;
    return f.src_off == f.dst_off && f.src_ostride == f.dst_ostride;
  }
  return f.src_off == f.dst_off && (f.o_end - f.o_begin <= 1 || f.src_ostride == f.dst_ostride);
}

constexpr uint64_t kSplitLine = 64 * 1024;
constexpr uint64_t kRingSlots = 4, kRingSlotMax = 256ull << 20;  // landing ring of the in-place KV inflow
// Tail staging (schedule): the cost of one more level (its launch and the gap
// before the next, measured at 15-20 us for small levels on the MI355X), the
// copy rate of the extra staging traffic (bytes of traffic per second), and
// the most bytes routed that way.
constexpr double kLevelCost = 15e-6;
constexpr double kTailRate = 6e12;
constexpr uint64_t kTailMax = 256ull << 20;
constexpr uint64_t kDirectMin = 32ull << 20;  // smallest inflow gap landed directly
constexpr size_t kMaxPieces = 1u << 20;

struct Node {
  enum Kind { NORMAL, STAGED, GATHER } kind = NORMAL;
  Fam fam;             // arena -> arena (NORMAL / STAGED) or arena -> staging (GATHER)
  uint64_t stage_off = 0;
  int level = -1;      // NORMAL, GATHER; for STAGED: level of the write half
  int out_index = -1;  // GATHER: index into outbound pending list
};

// Split a retained family until no piece writes over its own source.
void split_family(const Fam &f, std::vector<Node> &nodes, std::vector<Fam> &to_stage, size_t &budget) {
  std::function<void(const Fam &, int64_t, int64_t)> rec = [&](const Fam &g, int64_t p0, int64_t p1) {
    Fam piece = sub_fam(g, p0, p1);
    if (is_identity(piece)) return;  // bytes that stay where they are
    Span s = src_span(g, p0, p1), d = dst_span(g, p0, p1);
    if (!spans_meet(s, d)) {
      if (nodes.size() >= kMaxPieces) fail(ATP_ECAPACITY, "in-place schedule needs too many pieces");
      Node n;
      n.fam = piece;
      nodes.push_back(n);
      return;
    }
    if (p1 - p0 > 1 && budget > 0) {
      --budget;
      int64_t mid = p0 + (p1 - p0) / 2;
      rec(g, mid, p1);
      rec(g, p0, mid);
      return;
    }
    if (p1 - p0 == 1 && piece.rows == 1 && piece.run > 2 * kSplitLine && budget > 0 &&
        !(g.flags & (DF_SRC_IND | DF_DST_IND))) {
      // one long line: view it as lines of kSplitLine bytes and split those
      uint64_t n = piece.run / kSplitLine;
      Fam lines = piece;
      lines.run = kSplitLine;
      lines.src_ostride = lines.dst_ostride = kSplitLine;
      lines.o_begin = 0;
      lines.o_end = int64_t(n);
      rec(lines, 0, int64_t(n));
      uint64_t rest = piece.run - n * kSplitLine;
      if (rest) {
        Fam tail = piece;
        tail.src_off += n * kSplitLine;
        tail.dst_off += n * kSplitLine;
        tail.run = rest;
        rec(tail, 0, 1);
      }
      return;
    }
    to_stage.push_back(piece);
  };
  rec(f, f.o_begin, f.o_end);
}

// Overlap queries of read spans.
struct SpanIndex {
  std::vector<Span> sp;
  std::vector<int> id;
  std::vector<uint64_t> maxhi;
  void build() {
    std::vector<int> ord(sp.size());
    std::iota(ord.begin(), ord.end(), 0);
    std::sort(ord.begin(), ord.end(), [&](int a, int b) { return sp[a].lo < sp[b].lo; });
    std::vector<Span> s2;
    std::vector<int> i2;
    for (int o : ord) {
      s2.push_back(sp[o]);
      i2.push_back(id[o]);
    }
    sp.swap(s2);
    id.swap(i2);
    maxhi.resize(sp.size());
    uint64_t m = 0;
    for (size_t i = 0; i < sp.size(); ++i) maxhi[i] = m = std::max(m, sp[i].hi);
  }
  template <class F>
  void query(Span q, F &&fn) const {
    // last index with lo < q.hi
    size_t hi = std::lower_bound(sp.begin(), sp.end(), q.hi, [](const Span &s, uint64_t v) { return s.lo < v; }) -
                sp.begin();
    for (size_t i = hi; i-- > 0;) {
      if (maxhi[i] <= q.lo) break;
      if (sp[i].hi > q.lo) fn(id[i]);
    }
  }
};

// ---- descriptors, launches and ring ------------------------------------------------
bool fam_aligned(const Fam &f) {
  return f.src_off % 16 == 0 && f.dst_off % 16 == 0 && f.run % 16 == 0 && f.src_pitch % 16 == 0 &&
         f.dst_pitch % 16 == 0 && f.src_ostride % 16 == 0 && f.dst_ostride % 16 == 0;
}

// Tiles of a family whose DF_ALIGNED / DF_WIDE flags are set.
uint64_t fam_tiles(const Fam &f, int64_t items_hint) {
  uint64_t lines = uint64_t(items_hint) * f.rows;
  if (f.flags & DF_ALIGNED) {
    uint64_t chunks = lines * (f.run / 16);
    return (chunks + uint64_t(tile_chunks(f.flags)) - 1) / uint64_t(tile_chunks(f.flags));
  }
  return lines * ((f.run + kSegBytes - 1) / kSegBytes);
}

// Emit launches for a group of families: aligned ones first (with wide
// tiles, if `allow_wide`, for short KV lines), then the 2-byte-granular ones.
// Families are appended to c.fams; every family of a launch has the same
// DF_ALIGNED and DF_WIDE flags.
void emit_group(CallPlan &c, std::vector<Fam> group, int level, int kind, std::vector<Launch> &out,
                int64_t live_hint, bool allow_wide) {
  for (Fam &f : group) {
    f.flags &= ~(DF_ALIGNED | DF_WIDE);
    if (!fam_aligned(f)) continue;
    f.flags |= DF_ALIGNED;
    if (allow_wide && f.run <= kWideMaxRun && (f.flags & (DF_SRC_IND | DF_DST_IND | DF_BLOCKRANGE)))
      f.flags |= DF_WIDE;
  }
  for (int pass = 0; pass < 3; ++pass) {
    Launch L;
    L.level = level;
    L.kind = kind;
    L.aligned = pass < 2;
    L.wide = pass == 1;
    L.d0 = int(c.fams.size());
    for (const Fam &f : group) {
      if (((f.flags & DF_ALIGNED) != 0) != L.aligned || ((f.flags & DF_WIDE) != 0) != L.wide) continue;
      int64_t items = (f.flags & DF_BLOCKRANGE) ? std::min<int64_t>(f.o_end - f.o_begin, live_hint)
                                                : f.o_end - f.o_begin;
      L.bytes += uint64_t(items) * f.rows * f.run;
      L.tiles_max += fam_tiles(f, items);
      c.fams.push_back(f);
    }
    L.d1 = int(c.fams.size());
    if (L.d1 > L.d0) out.push_back(L);
  }
}

void schedule(Plan &P, CallPlan &c, std::vector<Fam> &retained, std::vector<Pending> &inflow,
              std::vector<Pending> &outbound, bool kvcall) {
  int64_t live_hint = kvcall ? P.kv.live_blocks : INT64_MAX;
  uint64_t cap = P.prob.staging_cap ? P.prob.staging_cap : UINT64_MAX;
  // staging header: meta, descriptors and prefix sums are sized after the
  // schedule; reserve the ring and staged bytes first
  std::vector<Node> nodes;
  std::vector<Fam> to_stage;
  uint64_t stage_bytes = 0;
  auto moved_of = [&](const Node &x) {
    return uint64_t(std::min<int64_t>(x.fam.o_end - x.fam.o_begin, live_hint)) * x.fam.rows * x.fam.run;
  };

  if (!P.inplace) {
    for (Fam &f : retained) {
      Node n;
      n.fam = f;
      n.level = 0;
      nodes.push_back(n);
      c.moved += uint64_t(std::min<int64_t>(f.o_end - f.o_begin, live_hint)) * f.rows * f.run;
    }
  } else {
    for (Fam &f : retained) {
      size_t budget = 4096;
      split_family(f, nodes, to_stage, budget);
    }
    for (Node &n : nodes) c.moved += moved_of(n);
    for (Fam &f : to_stage) {
      Node n;
      n.kind = Node::STAGED;
      n.fam = f;
      nodes.push_back(n);
      c.moved += f.bytes();
    }
    // KV outbound (indexed blocks) is gathered into staging at level 0
    if (kvcall) {
      for (size_t i = 0; i < outbound.size(); ++i) {
        Node n;
        n.kind = Node::GATHER;
        n.fam = outbound[i].fam;
        n.out_index = int(i);
        nodes.push_back(n);
      }
    }
  }

  // Staging room for the tail of the level chain (below): what the cap
  // leaves after the pieces already staged, the KV outbound gathered there,
  // the landing ring at its full size and the descriptor and block-list
  // area, at most kTailMax.
  uint64_t tail_room = 0;
  if (P.inplace && !(P.prob.flags & ATP_NO_TAIL_STAGING)) {
    uint64_t used = 0;
    for (const Node &x : nodes)
      if (x.kind != Node::NORMAL) used += align_up(x.kind == Node::GATHER ? x.fam.bytes() : moved_of(x), 256);
    if (kvcall) {
      uint64_t ring_in = 0;
      for (const Pending &pd : inflow) ring_in += pd.fam.bytes();
      used += std::min<uint64_t>(kRingSlots * kRingSlotMax, align_up(ring_in, 256));
      used += uint64_t(P.kv.num_blocks) * 12 + 1024;
    }
    used += (uint64_t(nodes.size()) * 2 + outbound.size() + inflow.size() + 64) * (sizeof(Desc) + 8) + (1u << 20);
    tail_room = used < cap ? std::min<uint64_t>(cap - used, kTailMax) : 0;
  }

  // ---- in-place dependency graph --------------------------------------------------
  // R(A) -> W(B) edge when B writes over bytes A reads (A != B).  Readers:
  // NORMAL (src), STAGED (src, at level 0), GATHER (src, level 0).  Writers:
  // NORMAL (dst), STAGED (dst, the write half).
  int n = int(nodes.size());
  std::vector<std::vector<int>> preds(n);
  std::vector<Span> rspan(n), wspan(n);
  auto node_items = [&](const Node &x) { return std::pair<int64_t, int64_t>(x.fam.o_begin, x.fam.o_end); };
  if (P.inplace && n) {
    SpanIndex idx;
    for (int i = 0; i < n; ++i) {
      auto it = node_items(nodes[i]);
      if (it.second <= it.first) continue;
      rspan[i] = src_span(nodes[i].fam, it.first, it.second);
      if (nodes[i].kind == Node::GATHER) {
        // indexed source over live-list positions: any block of the pool
        const Fam &f = nodes[i].fam;
        uint64_t nb = uint64_t(P.kv.num_blocks);
        rspan[i] = {f.src_off, f.src_off + (nb - 1) * f.src_ostride + (f.rows - 1) * f.src_pitch + f.run};
      } else {
        wspan[i] = dst_span(nodes[i].fam, it.first, it.second);
      }
      idx.sp.push_back(rspan[i]);
      idx.id.push_back(i);
    }
    idx.build();
    for (int b = 0; b < n; ++b) {
      if (nodes[b].kind == Node::GATHER) continue;
      auto it = node_items(nodes[b]);
      if (it.second <= it.first) continue;
      idx.query(wspan[b], [&](int a) {
        if (a != b) preds[b].push_back(a);
      });
    }
    // levels by longest path; STAGED and GATHER reads sit at level 0 and
    // do not propagate (their readers are done before anything writes)
    auto solve = [&](std::vector<int> &lvl) -> bool {
      lvl.assign(n, -1);
      std::vector<int> indeg(n, 0);
      std::vector<std::vector<int>> succ(n);
      for (int b = 0; b < n; ++b)
        for (int a : preds[b])
          if (nodes[a].kind == Node::NORMAL) {
            succ[a].push_back(b);
            indeg[b]++;
          }
      std::vector<int> q;
      for (int i = 0; i < n; ++i)
        if (indeg[i] == 0) q.push_back(i);
      std::vector<int> base(n, 0);
      for (int b = 0; b < n; ++b)
        for (int a : preds[b])
          if (nodes[a].kind != Node::NORMAL) base[b] = std::max(base[b], 1);
      for (int i = 0; i < n; ++i)
        if (nodes[i].kind == Node::STAGED) base[i] = std::max(base[i], 1);  // write half after its read
      size_t head = 0;
      int done = 0;
      while (head < q.size()) {
        int a = q[head++];
        ++done;
        int la = nodes[a].kind == Node::GATHER ? 0 : base[a];
        lvl[a] = la;
        for (int b : succ[a]) {
          base[b] = std::max(base[b], la + 1);
          if (--indeg[b] == 0) q.push_back(b);
        }
      }
      return done == n;
    };
    std::vector<int> lvl;
    int rounds = 0;
    while (!solve(lvl)) {
      // cycle: route the smallest unresolved NORMAL node of each strongly
      // connected component through staging
      if (++rounds > 10000) fail(ATP_ECAPACITY, "in-place schedule: too many cycles");
      // Tarjan over the unresolved NORMAL subgraph (edges a -> b: b waits a)
      std::vector<std::vector<int>> succ(n);
      for (int b = 0; b < n; ++b)
        if (lvl[b] < 0 && nodes[b].kind == Node::NORMAL)
          for (int a : preds[b])
            if (lvl[a] < 0 && nodes[a].kind == Node::NORMAL) succ[a].push_back(b);
      std::vector<int> index(n, -1), low(n, 0), comp(n, -1), st;
      std::vector<char> on(n, 0);
      int counter = 0, ncomp = 0;
      std::function<void(int)> strong = [&](int v) {
        index[v] = low[v] = counter++;
        st.push_back(v);
        on[v] = 1;
        for (int w : succ[v]) {
          if (index[w] < 0) {
            strong(w);
            low[v] = std::min(low[v], low[w]);
          } else if (on[w]) {
            low[v] = std::min(low[v], index[w]);
          }
        }
        if (low[v] == index[v]) {
          for (;;) {
            int w = st.back();
            st.pop_back();
            on[w] = 0;
            comp[w] = ncomp;
            if (w == v) break;
          }
          ++ncomp;
        }
      };
      for (int v = 0; v < n; ++v)
        if (lvl[v] < 0 && nodes[v].kind == Node::NORMAL && index[v] < 0) strong(v);
      std::vector<int> size(ncomp, 0), pick(ncomp, -1);
      for (int v = 0; v < n; ++v)
        if (comp[v] >= 0) size[comp[v]]++;
      bool changed = false;
      for (int v = 0; v < n; ++v) {
        int cpt = comp[v];
        if (cpt < 0) continue;
        bool self_loop = false;
        for (int w : succ[v]) self_loop |= (w == v);
        if (size[cpt] < 2 && !self_loop) continue;
        if (pick[cpt] < 0 || nodes[v].fam.bytes() < nodes[pick[cpt]].fam.bytes()) pick[cpt] = v;
      }
      for (int cpt = 0; cpt < ncomp; ++cpt)
        if (pick[cpt] >= 0) {
          nodes[pick[cpt]].kind = Node::STAGED;
          changed = true;
        }
      if (!changed) fail(ATP_ECAPACITY, "in-place schedule: unresolvable order");
    }
    // The tail of the level chain through staging.  A shard that grows on
    // its own arena gives a chain of levels in which each level writes where
    // the next one reads, each moving about half as much as the one before;
    // the last levels move little, yet each costs a launch and the gap
    // before the next one.  The nodes of levels k and above are staged
    // instead: their reads join level 0 and their writes the level after
    // the last level that reads their destination, so no level above k
    // remains.  Every byte so routed is read and written once more.  k
    // maximises the levels saved times kLevelCost less that extra traffic
    // at kTailRate, within the room the staging cap leaves.
    if (tail_room > 0) {
      int nl = 0;
      for (int i = 0; i < n; ++i)
        if (nodes[i].kind == Node::NORMAL) nl = std::max(nl, lvl[i] + 1);
      std::vector<uint64_t> suffix(size_t(nl) + 1, 0);  // bytes moved by NORMAL nodes of levels >= l
      for (int i = 0; i < n; ++i)
        if (nodes[i].kind == Node::NORMAL) suffix[size_t(lvl[i])] += moved_of(nodes[i]);
      for (int l = nl - 1; l >= 0; --l) suffix[size_t(l)] += suffix[size_t(l) + 1];
      int best_k = nl;
      double best_gain = 0;
      for (int k = 1; k + 1 < nl; ++k) {
        if (suffix[size_t(k)] > tail_room) continue;
        const double gain = double(nl - k - 1) * kLevelCost - 2.0 * double(suffix[size_t(k)]) / kTailRate;
        if (gain > best_gain) {
          best_gain = gain;
          best_k = k;
        }
      }
      if (best_k < nl) {
        for (int i = 0; i < n; ++i)
          if (nodes[i].kind == Node::NORMAL && lvl[i] >= best_k) {
            nodes[i].kind = Node::STAGED;
            c.tail += moved_of(nodes[i]);
          }
        // fewer NORMAL nodes cannot close a cycle
        if (!solve(lvl)) fail(ATP_ECAPACITY, "in-place schedule: unresolvable order after staging the tail");
      }
    }
    for (int i = 0; i < n; ++i) nodes[i].level = lvl[i];
  }

  // staged bytes (packed, 256-aligned pieces)
  for (Node &x : nodes) {
    if (x.kind == Node::STAGED || x.kind == Node::GATHER) {
      x.stage_off = stage_bytes;
      uint64_t b = uint64_t(std::min<int64_t>(x.fam.o_end - x.fam.o_begin, live_hint)) * x.fam.rows * x.fam.run;
      if (x.kind == Node::GATHER) b = x.fam.bytes();
      stage_bytes = align_up(stage_bytes + b, 256);
      if (x.kind == Node::STAGED) c.staged += b;
    }
  }

  // ---- launches per level -------------------------------------------------------------
  int maxl = 0;
  for (Node &x : nodes) maxl = std::max(maxl, x.level);
  c.n_levels = nodes.empty() ? 0 : maxl + 1;
  std::vector<std::vector<Fam>> per_level(c.n_levels);
  for (Node &x : nodes) {
    if (x.kind == Node::NORMAL) {
      per_level[x.level].push_back(x.fam);
    } else if (x.kind == Node::GATHER) {
      Fam g = x.fam;  // dst offset re-based into the staged area later
      g.dst_off = x.stage_off;
      per_level[0].push_back(g);
    } else {  // STAGED: read half at level 0, write half at x.level
      Fam r = x.fam, w = x.fam;
      bool blk = x.fam.flags & DF_BLOCKRANGE;
      uint64_t item = x.fam.rows * x.fam.run;
      r.flags = (r.flags & ~(3u << DF_DST_SHIFT) & ~DF_DST_IND) | (BUF_STAGE << DF_DST_SHIFT);
      r.dst_off = x.stage_off;
      r.dst_pitch = x.fam.run;
      r.dst_ostride = item;
      w.flags = (w.flags & ~(3u << DF_SRC_SHIFT) & ~DF_SRC_IND) | (BUF_STAGE << DF_SRC_SHIFT);
      w.src_off = x.stage_off;
      w.src_pitch = x.fam.run;
      w.src_ostride = item;
      (void)blk;  // block ranges: the packed side counts from the first live block
      per_level[0].push_back(r);
      per_level[x.level].push_back(w);
    }
  }
  // outbound copies that later writers depend on (weights, in place)
  std::vector<int> needed_by(outbound.size(), INT32_MAX);
  if (P.inplace && !kvcall) {
    SpanIndex widx;
    for (int i = 0; i < n; ++i) {
      if (nodes[i].kind == Node::GATHER) continue;
      widx.sp.push_back(wspan[i]);
      widx.id.push_back(i);
    }
    widx.build();
    for (size_t o = 0; o < outbound.size(); ++o) {
      const Fam &f = outbound[o].fam;
      Span s = src_span(f, f.o_begin, f.o_end);
      widx.query(s, [&](int b) { needed_by[o] = std::min(needed_by[o], nodes[b].level); });
    }
  }
  for (int l = 0; l < c.n_levels; ++l) {
    size_t before = c.levels.size();
    emit_group(c, per_level[l], l, 0, c.levels, live_hint, true);
    if (P.inplace && !kvcall && c.levels.size() > before) {
      for (size_t o = 0; o < outbound.size(); ++o)
        if (needed_by[o] == l) c.levels[before].wait_outbound.push_back(int(o));
    }
  }
  // outbound issue order: by the first level that overwrites it
  std::vector<int> pos(outbound.size(), 0);
  c.out_order.resize(outbound.size());
  std::iota(c.out_order.begin(), c.out_order.end(), 0);
  std::stable_sort(c.out_order.begin(), c.out_order.end(),
                   [&](int a, int b) { return needed_by[a] < needed_by[b]; });
  for (size_t k = 0; k < c.out_order.size(); ++k) pos[c.out_order[k]] = int(k);
  // outbound host copies
  for (size_t o = 0; o < outbound.size(); ++o) {
    const Pending &pd = outbound[o];
    HostCopy h;
    h.host_off = pd.host_off;
    h.bytes = pd.fam.bytes();
    if (kvcall) {
      // gathered into staging at level 0, then one linear copy
      h.dev_buf = BUF_STAGE;
      for (Node &x : nodes)
        if (x.kind == Node::GATHER && x.out_index == int(o)) h.dev_off = x.stage_off;
      h.rows = 1;
      h.run = h.bytes;
      h.gate_level = 0;
    } else {
      h.dev_buf = BUF_IN;
      h.dev_off = pd.fam.src_off;
      h.rows = uint64_t(pd.fam.o_end - pd.fam.o_begin);
      h.run = pd.fam.run;
      h.dev_pitch = pd.fam.src_ostride;
    }
    c.outbound.push_back(h);
  }
  if (P.inplace && !kvcall && !c.out_order.empty()) {
    // the copy kernel reads them out: arena (slot IN) -> pinned outbound
    // buffer (slot OUT of those launches), packed row after row
    c.out_d0 = int(c.fams.size());
    for (int o : c.out_order) {
      const HostCopy &h = c.outbound[size_t(o)];
      Fam f;
      f.src_off = h.dev_off;
      f.src_ostride = h.dev_pitch;
      f.dst_off = h.host_off;
      f.dst_ostride = h.run;
      f.o_begin = 0;
      f.o_end = int64_t(h.rows);
      f.run = h.run;
      f.rows = 1;
      f.flags = bufs(BUF_IN, BUF_OUT);
      const bool al = fam_aligned(f);
      if (al) f.flags |= DF_ALIGNED;
      c.out_aligned.push_back(al);
      c.out_tiles.push_back(fam_tiles(f, f.o_end));
      c.fams.push_back(f);
    }
  }

  // ---- inflow: direct copies (contiguous) and ring chunks (strided) --------------------
  SpanIndex ridx;  // readers of the old arena, for gating direct landings
  SpanIndex oidx;  // outbound sources
  if (P.inplace) {
    for (int i = 0; i < n; ++i) {
      ridx.sp.push_back(rspan[i]);
      ridx.id.push_back(i);
    }
    ridx.build();
    if (!kvcall) {
      for (size_t o = 0; o < outbound.size(); ++o) {
        const Fam &f = outbound[o].fam;
        oidx.sp.push_back(src_span(f, f.o_begin, f.o_end));
        oidx.id.push_back(int(o));
      }
      oidx.build();
    }
  }
  // outbound copies a landing on `d` must wait for: the first k in issue order
  auto out_gate = [&](Span d) {
    int k = 0;
    if (P.inplace && !kvcall) oidx.query(d, [&](int o) { k = std::max(k, pos[o] + 1); });
    return k;
  };
  std::vector<const Pending *> ring;  // through the landing ring
  std::vector<Fam> host_pieces;       // read by the copy kernel from the host buffer
  uint64_t ring_total = 0, max_item = 0;
  for (const Pending &pd : inflow) {
    // Only large contiguous gaps land directly on the DMA engine, each copy
    // command and each event between them costing it tens of microseconds.
    // Every other piece is read by the copy kernel straight from the pinned
    // host buffer into its final place: out of place from the start, beside
    // the repack (the two write disjoint bytes); in place, for the weights,
    // after the last level, since a copy command that waits for a level or
    // an outbound read holds up every later host-to-device copy on the DMA
    // engine.  The in-place KV landings go through the landing ring, whose
    // copies wait only for their slot's previous scatter and land while the
    // KV levels run.
    if (pd.contiguous && pd.fam.bytes() >= kDirectMin) {
      HostCopy h;
      h.host_off = pd.host_off;
      h.dev_off = pd.fam.dst_off;
      h.bytes = pd.fam.bytes();
      h.dev_buf = BUF_OUT;
      if (P.inplace) {
        Span d{h.dev_off, h.dev_off + h.bytes};
        ridx.query(d, [&](int a) {
          int l = nodes[a].kind == Node::NORMAL ? nodes[a].level : 0;
          h.gate_level = std::max(h.gate_level, l);
        });
        h.gate_pos = out_gate(d);
      }
      if (!P.inplace || (h.gate_level < 0 && h.gate_pos == 0)) {
        c.directs.push_back(h);
        continue;
      }
    }
    if (!(P.inplace && kvcall)) {
      Fam f = pd.fam;  // source side: packed host offsets
      f.flags = (f.flags & ~(3u << DF_SRC_SHIFT)) | (BUF_IN << DF_SRC_SHIFT);
      host_pieces.push_back(f);
    } else {
      // the KV call in place: nothing here is read by an outbound copy (KV
      // outbound is gathered at level 0), and the scatters run after every
      // level
      const Fam &f = pd.fam;
      ring.push_back(&pd);
      ring_total += f.bytes();
      max_item = std::max<uint64_t>(max_item, f.rows * f.run);
    }
  }
  // level: in place after the last level, out of place at any time (-1)
  // host reads keep the narrow tile: more bytes in flight over PCIe would
  // slow the repack beside them
  if (!host_pieces.empty())
    emit_group(c, host_pieces, P.inplace ? c.n_levels : -1, 4, c.host_reads, live_hint, false);

  uint64_t slot = 0;
  if (!ring.empty()) {
    // Up to 4 slots of 256 MiB, no more than the ring's bytes fill.  Every
    // copy command, and the event between it and its scatter, costs the DMA
    // engine tens of microseconds, so few large copies keep the link full:
    // the 80-layer TP 8->7 reshard in place took 1019.6 ms with 256 MiB
    // slots, 1023.4 with 128 and 1031.6 with 64.
    const uint64_t item = align_up(max_item, 256);
    auto slots_for = [&](uint64_t s) { return std::min<uint64_t>(kRingSlots, (ring_total + s - 1) / s); };
    slot = std::max<uint64_t>(std::min<uint64_t>(kRingSlotMax, align_up(ring_total, 256)), item);
    // respect the staging cap: shrink slots if needed
    while (slots_for(slot) * slot + stage_bytes + (1u << 20) > cap && slot / 2 >= item && slot > (4u << 20))
      slot = align_up(slot / 2, 256);
    c.n_slots = int(slots_for(slot));
  }
  c.ring_slot = slot;

  // chunking: whole items of ring families, in host-buffer order
  if (!ring.empty()) {
    Chunk ch;
    uint64_t fill = 0;
    int next_slot = 0;
    std::vector<Fam> pieces;
    auto flush = [&]() {
      if (pieces.empty()) return;
      ch.slot = next_slot;
      next_slot = (next_slot + 1) % c.n_slots;
      emit_group(c, pieces, -1, 2, ch.scatters, live_hint, true);
      c.chunks.push_back(ch);
      pieces.clear();
      ch = Chunk();
      fill = 0;
    };
    for (const Pending *pd : ring) {
      const Fam &f = pd->fam;
      uint64_t item = f.rows * f.run;
      int64_t k = f.o_begin;
      while (k < f.o_end) {
        int64_t room = int64_t((slot - fill) / item);
        if (room <= 0) {
          flush();
          continue;
        }
        int64_t k1 = std::min<int64_t>(f.o_end, k + room);
        // host copy of items [k, k1) into the slot at `fill`
        uint64_t hoff = pd->host_off + uint64_t(k - f.o_begin) * item;
        uint64_t bytes = uint64_t(k1 - k) * item;
        if (!ch.copies.empty() && ch.copies.back().host_off + ch.copies.back().bytes == hoff &&
            ch.copies.back().dev_off + ch.copies.back().bytes == fill)
          ch.copies.back().bytes += bytes;
        else {
          HostCopy h;
          h.host_off = hoff;
          h.dev_off = fill;  // within the slot; re-based at execution
          h.bytes = bytes;
          h.dev_buf = BUF_STAGE;
          ch.copies.push_back(h);
        }
        Fam s = f;
        s.o_begin = k;
        s.o_end = k1;
        s.src_off = fill;  // relative to the slot; re-based below
        s.src_pitch = f.run;
        s.src_ostride = item;
        // the source side counts from the piece's first item
        if (!(s.flags & DF_DST_IND)) {
          s.dst_off = f.dst_off + uint64_t(k - f.o_begin) * f.dst_ostride;
          s.o_begin = 0;
          s.o_end = k1 - k;
        }
        pieces.push_back(s);
        fill = align_up(fill + bytes, 256);
        k = k1;
      }
    }
    flush();
  }

  // ---- staging layout ------------------------------------------------------------------
  uint64_t nd = c.fams.size();
  uint64_t at = 0;
  c.off_meta = at;
  at += 256;
  c.off_desc = at;
  at = align_up(at + nd * sizeof(Desc), 256);
  c.off_prefix = at;
  at = align_up(at + (nd + 1) * 8, 256);
  if (kvcall) {
    uint64_t nb = P.kv.num_blocks;
    c.off_kvflags = at;
    at = align_up(at + nb * 4, 256);
    c.off_kvpref = at;
    at = align_up(at + (nb + 1) * 4, 256);
    c.off_kvlive = at;
    at = align_up(at + nb * 4, 256);
  }
  c.off_ring = at;
  at += uint64_t(c.n_slots) * c.ring_slot;
  c.off_stage = at;
  at += stage_bytes;
  c.staging_need = align_up(at, 256);
  if (P.inplace && c.staging_need > cap)
    fail(ATP_ECAPACITY, std::string(kvcall ? "KV" : "weights") + " in-place schedule needs " +
                            std::to_string(c.staging_need) + " staging bytes, cap is " + std::to_string(cap));
  // re-base staging offsets now that the layout is known: staged pieces
  // live in the stage area, ring pieces in their slot
  for (Chunk &ch : c.chunks) {
    uint64_t base = c.off_ring + uint64_t(ch.slot) * c.ring_slot;
    for (HostCopy &h : ch.copies) h.dev_off += base;
    for (Launch &L : ch.scatters)
      for (int d = L.d0; d < L.d1; ++d) c.fams[d].src_off += base;
  }
  for (Launch &L : c.levels)
    for (int d = L.d0; d < L.d1; ++d) {
      Fam &f = c.fams[d];
      if (((f.flags >> DF_SRC_SHIFT) & 3) == BUF_STAGE) f.src_off += c.off_stage;
      if (((f.flags >> DF_DST_SHIFT) & 3) == BUF_STAGE) f.dst_off += c.off_stage;
    }
  for (HostCopy &h : c.outbound)
    if (h.dev_buf == BUF_STAGE) h.dev_off += c.off_stage;
}

}  // namespace

Plan *make_plan(const atp_problem *p) {
  auto t0 = std::chrono::steady_clock::now();
  if (!p) fail(ATP_EINVAL, "problem is NULL");
  std::unique_ptr<Plan> P(new Plan());
  P->prob = *p;
  P->flags = p->flags;
  P->inplace = p->flags & ATP_INPLACE;
  // the in-place schedule relies on block ids that stay put
  if (P->inplace && (p->flags & ATP_KV_COMPACT)) fail(ATP_EINVAL, "ATP_KV_COMPACT needs an out-of-place reshard");
  resolve_spaces(*P);
  if (p->self_old_rank < 0 || p->self_old_rank >= P->sp[0].N) fail(ATP_EINVAL, "self_old_rank out of range");
  P->self_old = p->self_old_rank;  // shard geometry below is this rank's
  resolve_tensors(*P);
  resolve_kv(*P);
  resolve_ranks(*P);
  run_cmm(*P);
  global_stats(*P);

  std::vector<Fam> ret_w, ret_k;
  std::vector<Pending> in_w, in_k, out_w, out_k;
  lower_weights(*P, ret_w, in_w, out_w);
  schedule(*P, P->w, ret_w, in_w, out_w, false);
  if (P->has_kv) {
    lower_kv(*P, ret_k, in_k, out_k);
    schedule(*P, P->k, ret_k, in_k, out_k, true);
  }

  atp_stats &st = P->stats;
  st.self_new_rank = P->self_new;
  st.n_levels_w = P->w.n_levels;
  st.n_levels_kv = P->k.n_levels;
  st.n_desc_w = int(P->w.fams.size());
  st.n_desc_kv = int(P->k.fams.size());
  st.old_arena_bytes = P->w.old_bytes;
  st.new_arena_bytes = P->w.new_bytes;
  st.old_kv_bytes = P->k.old_bytes;
  st.new_kv_bytes = P->k.new_bytes;
  st.retained_w = P->w.retained;
  st.inflow_w = P->w.inflow;
  st.outbound_w = P->w.outbound_bytes;
  st.retained_kv = P->k.retained;
  st.inflow_kv = P->k.inflow;
  st.outbound_kv = P->k.outbound_bytes;
  st.moved_w = P->w.moved;
  st.moved_kv = P->k.moved;
  st.staged_w = P->w.staged;
  st.staged_kv = P->k.staged;
  st.tail_w = P->w.tail;
  st.tail_kv = P->k.tail;
  st.staging_w = P->w.staging_need;
  st.staging_kv = P->has_kv ? P->k.staging_need : 0;
  P->plan_ms = std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - t0).count();
  return P.release();
}

}  // namespace atp
