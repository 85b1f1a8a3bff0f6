// exec.h — executor entry points (exec.hip), called by the C ABI layer.
#pragma once
#include <hip/hip_runtime_api.h>

#include <functional>
#include <vector>

#include "plan.h"

namespace atp {

// Enqueue one reshard call (weights: kvcall = false).  Throws Error.  With
// `await`, the host calls it with the end of each inflow piece's bytes in
// the inflow buffer before issuing that piece, and it returns once those
// bytes are there (the inflow buffer is still being filled).  With
// `on_scratch`, the call runs on the device's scratch array instead of
// `staging` and allocates nothing: events, pinned buffers and the side
// stream must come from what atp_warmup pooled (ATP_ESTATE otherwise).
// With `defer` (a weights call with `await`), the call returns once the work
// that needs no inflow byte is queued; exec_sync issues the awaited pieces
// (keeping a copy of `await`), then runs `after_issue` (which may throw: the
// error is then exec_sync's, after everything queued has drained).
void exec_call(Plan &P, bool kvcall, void *arena, uint64_t arena_bytes, void *new_arena, uint64_t new_bytes,
               const void *inflow_host, uint64_t inflow_bytes, void *outbound_host, uint64_t outbound_bytes,
               const int32_t *table, int64_t n_entries, void *staging, uint64_t staging_bytes, hipStream_t compute,
               hipStream_t copy, const std::function<void(uint64_t)> *await = nullptr, bool on_scratch = false,
               bool defer = false, std::function<void()> after_issue = {});
// Bytes of the scratch array (the no-allocation entry point's limit).
uint64_t scratch_bytes();
int exec_sync(Plan &P, atp_timing *out);
void exec_free(Plan &P);
void exec_launches(const Plan &P, std::vector<atp_launch> &out);
void exec_warmup(void *compute, void *copy, int events);

}  // namespace atp
