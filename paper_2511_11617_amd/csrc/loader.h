// loader.h — range-read reload source (Sec. IV loader): opened safetensors
// files and the fill of a plan's packed weight inflow buffer.
#pragma once

#include <cstdint>
#include <memory>
#include <string>
#include <unordered_map>
#include <vector>

#include "plan.h"

namespace atp {

struct StTensor {
  int file = 0;
  int elem_bytes = 0;
  std::vector<uint64_t> shape;
  uint64_t begin = 0, end = 0;  // absolute byte range in the file
};

struct StFiles {
  std::vector<std::string> paths;
  std::vector<int> fds;
  std::unordered_map<std::string, StTensor> map;
  ~StFiles();
};

// Opens and validates every file; throws Error(ATP_EINVAL) on any problem.
StFiles *st_open(const char *const *paths, int n);

// Reads exactly the intervals of the plan's weight inflow segments into
// `inflow` (packing order of the plan); throws Error on failure.
void load_weights(const Plan &P, const StFiles &S, const char *const *names, int n_names, void *inflow,
                  uint64_t inflow_bytes, int n_threads, atp_load_stats *stats);

}  // namespace atp
