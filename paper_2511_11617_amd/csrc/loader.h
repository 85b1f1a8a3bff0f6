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

// The same reads run on background threads, with the byte prefix of the
// buffer they have completed observable: a reshard can issue each inflow
// piece as soon as the bytes under it have landed.  The constructor checks
// the names and builds the reads (throws Error, nothing started); start()
// launches the threads; await(end) blocks until [0, end) is read or a read
// failed; finish() joins them and throws Error if a read failed.  The
// destructor stops and joins threads still running.
class LoadJob {
 public:
  LoadJob(const Plan &P, const StFiles &S, const char *const *names, int n_names, void *inflow,
          uint64_t inflow_bytes, int n_threads);
  ~LoadJob();
  void start();
  void await(uint64_t end);
  void finish(atp_load_stats *stats);

  struct Impl;

 private:
  std::unique_ptr<Impl> impl_;
};

}  // namespace atp
