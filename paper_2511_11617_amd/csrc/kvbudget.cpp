// kvbudget.cpp — KV budget under recovery (Sec. III-A, state management):
// sessions carry a last-use time; when the KV the new layout needs exceeds
// the budget, the least recently used sessions are released one at a time
// until it fits.  Blocks are reference-counted over sessions, so a block
// shared by several sessions is freed only with the last of them.
#include "kvbudget.h"

#include <algorithm>
#include <numeric>
#include <vector>

namespace atp {

void evict_lru(const int32_t *table, int32_t n_seq, int32_t max_blocks, int64_t num_blocks,
               const int64_t *last_use, uint64_t block_bytes, uint64_t budget_bytes, bool compact,
               int32_t *keep, int32_t *new_table, atp_evict_stats *st) {
  if (n_seq < 0 || max_blocks < 0 || num_blocks < 0) throw Error(ATP_EINVAL, "negative table size");
  const size_t entries = size_t(n_seq) * size_t(max_blocks);
  if (entries && (!table || !new_table)) throw Error(ATP_EINVAL, "table or new_table is NULL");
  if (n_seq && (!last_use || !keep)) throw Error(ATP_EINVAL, "last_use or keep is NULL");
  std::vector<int32_t> ref(size_t(num_blocks), 0);
  int64_t live = 0;
  for (size_t i = 0; i < entries; ++i) {
    int32_t p = table[i];
    if (p < -1 || p >= num_blocks) throw Error(ATP_EINVAL, "block id outside [-1, num_blocks)");
    if (p >= 0 && ref[size_t(p)]++ == 0) ++live;
  }
  auto demand = [&](int64_t n) { return (unsigned __int128)uint64_t(n) * block_bytes; };
  const int64_t live0 = live;
  std::vector<int32_t> order(static_cast<size_t>(n_seq));
  std::iota(order.begin(), order.end(), 0);
  std::stable_sort(order.begin(), order.end(), [&](int32_t a, int32_t b) { return last_use[a] < last_use[b]; });
  std::vector<int32_t> kept(size_t(n_seq), 1);
  int32_t evicted = 0;
  for (int32_t s : order) {
    if (demand(live) <= budget_bytes) break;
    kept[size_t(s)] = 0;
    ++evicted;
    for (int32_t b = 0; b < max_blocks; ++b) {
      int32_t p = table[size_t(s) * size_t(max_blocks) + size_t(b)];
      if (p >= 0 && --ref[size_t(p)] == 0) --live;
    }
  }
  // rank of each kept block among the kept ids (compact numbering)
  std::vector<int32_t> rank;
  if (compact) {
    rank.assign(size_t(num_blocks), -1);
    int32_t r = 0;
    for (int64_t p = 0; p < num_blocks; ++p)
      if (ref[size_t(p)] > 0) rank[size_t(p)] = r++;
  }
  for (int32_t s = 0; s < n_seq; ++s) {
    keep[s] = kept[size_t(s)];
    for (int32_t b = 0; b < max_blocks; ++b) {
      size_t i = size_t(s) * size_t(max_blocks) + size_t(b);
      int32_t p = table[i];
      new_table[i] = (!kept[size_t(s)] || p < 0) ? -1 : (compact ? rank[size_t(p)] : p);
    }
  }
  if (st) {
    st->kept_sessions = n_seq - evicted;
    st->evicted_sessions = evicted;
    st->live_before = live0;
    st->live_after = live;
    st->demand_before = uint64_t(std::min<unsigned __int128>(demand(live0), UINT64_MAX));
    st->demand_after = uint64_t(std::min<unsigned __int128>(demand(live), UINT64_MAX));
  }
}

}  // namespace atp
