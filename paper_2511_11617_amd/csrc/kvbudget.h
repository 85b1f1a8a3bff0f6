// kvbudget.h — KV budget under recovery (Sec. III-A): least-recently-used
// session eviction and the compact renumbering of the block table.
#pragma once

#include <cstdint>

#include "plan.h"

namespace atp {

// Throws Error(ATP_EINVAL) on a malformed table.
void evict_lru(const int32_t *table, int32_t n_seq, int32_t max_blocks, int64_t num_blocks,
               const int64_t *last_use, uint64_t block_bytes, uint64_t budget_bytes, bool compact,
               int32_t *keep, int32_t *new_table, atp_evict_stats *stats);

}  // namespace atp
