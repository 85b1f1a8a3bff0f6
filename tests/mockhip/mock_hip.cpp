// mock_hip.cpp — a host-only stand-in for the HIP runtime calls libatp.so
// makes (test infrastructure: tests/test_exec_replay.py preloads it into a
// child process on a machine without a GPU, so that the executor's host
// logic runs for real).
//   * Device memory is address ranges only (never dereferenced); pinned
//     buffers up to 256 MiB are real host memory (the executor writes its
//     descriptors and reads its error word there), larger ones ranges too.
//   * Every copy must lie inside one allocation, with the right host/device
//     sides for its direction; every event and stream must exist when used;
//     launches need a non-empty grid.  A violation prints MOCKHIP FAULT and
//     aborts the process.
//   * Kernels are counted, not run; events time 0.125 ms.
#include <hip/hip_runtime_api.h>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <map>
#include <mutex>
#include <set>
#include <vector>

namespace {
std::mutex mu;
struct Alloc { uintptr_t b, e; bool host; bool real; };
std::map<uintptr_t, Alloc> allocs;  // by base
uintptr_t next_dev = uintptr_t(1) << 44, next_fake_host = uintptr_t(3) << 44;
std::set<void *> events, streams;
std::set<void *> recorded;
long launches = 0, copies = 0, waits = 0;
dim3 cfg_grid, cfg_block;
size_t cfg_shmem;
hipStream_t cfg_stream;
hipError_t last = hipSuccess;

void die(const char *what, const void *p, size_t n) {
  fprintf(stderr, "MOCKHIP FAULT: %s at %p (+%zu)\n", what, p, n);
  abort();
}
const Alloc *find(const void *p, size_t n) {
  uintptr_t a = uintptr_t(p);
  auto it = allocs.upper_bound(a);
  if (it == allocs.begin()) return nullptr;
  --it;
  if (a >= it->second.b && a + n <= it->second.e) return &it->second;
  return nullptr;
}
}  // namespace

extern "C" {
hipError_t hipGetDevice(int *d) { *d = 0; return hipSuccess; }
hipError_t hipSetDevice(int) { return hipSuccess; }
hipError_t hipDeviceGetAttribute(int *v, hipDeviceAttribute_t, int) { *v = 256; return hipSuccess; }
hipError_t hipEventCreate(hipEvent_t *e) { std::lock_guard<std::mutex> g(mu); *e = (hipEvent_t)malloc(64); events.insert(*e); return hipSuccess; }
hipError_t hipEventCreateWithFlags(hipEvent_t *e, unsigned) { return hipEventCreate(e); }
hipError_t hipEventDestroy(hipEvent_t e) { std::lock_guard<std::mutex> g(mu); events.erase(e); free(e); return hipSuccess; }
hipError_t hipEventRecord(hipEvent_t e, hipStream_t s) {
  std::lock_guard<std::mutex> g(mu);
  if (!events.count(e)) die("record of an unknown event", e, 0);
  if (s && !streams.count(s)) die("record on an unknown stream", s, 0);
  recorded.insert(e);
  return hipSuccess;
}
hipError_t hipEventSynchronize(hipEvent_t e) { std::lock_guard<std::mutex> g(mu); if (!events.count(e)) die("sync of an unknown event", e, 0); return hipSuccess; }
hipError_t hipEventElapsedTime(float *ms, hipEvent_t a, hipEvent_t b) {
  std::lock_guard<std::mutex> g(mu);
  if (!events.count(a) || !events.count(b)) die("elapsed of an unknown event", a, 0);
  if (!recorded.count(a) || !recorded.count(b)) return hipErrorNotReady;
  *ms = 0.125f;
  return hipSuccess;
}
hipError_t hipStreamCreateWithFlags(hipStream_t *s, unsigned) { std::lock_guard<std::mutex> g(mu); *s = (hipStream_t)malloc(64); streams.insert(*s); return hipSuccess; }
hipError_t hipStreamWaitEvent(hipStream_t s, hipEvent_t e, unsigned) {
  std::lock_guard<std::mutex> g(mu);
  if (s && !streams.count(s)) die("wait on an unknown stream", s, 0);
  if (!events.count(e)) die("wait for an unknown event", e, 0);
  ++waits;
  return hipSuccess;
}
hipError_t hipStreamSynchronize(hipStream_t) { return hipSuccess; }
hipError_t hipDeviceSynchronize(void) { return hipSuccess; }
hipError_t hipMalloc(void **p, size_t n) {
  std::lock_guard<std::mutex> g(mu);
  uintptr_t b = next_dev;
  next_dev += (n + 0xFFFFF) & ~uintptr_t(0xFFFFF);
  next_dev += 1 << 20;
  allocs[b] = {b, b + n, false, false};
  *p = (void *)b;
  return hipSuccess;
}
hipError_t hipHostMalloc(void **p, size_t n, unsigned) {
  std::lock_guard<std::mutex> g(mu);
  uintptr_t b;
  bool real = n <= (size_t(1) << 28);
  if (real) {
    void *q = nullptr;
    if (posix_memalign(&q, 4096, n)) return hipErrorOutOfMemory;
    memset(q, 0, n);
    b = uintptr_t(q);
  } else {
    b = next_fake_host;
    next_fake_host += ((n + 0xFFFFF) & ~uintptr_t(0xFFFFF)) + (1 << 20);
  }
  allocs[b] = {b, b + n, true, real};
  *p = (void *)b;
  return hipSuccess;
}
hipError_t hipFree(void *p) { std::lock_guard<std::mutex> g(mu); allocs.erase(uintptr_t(p)); return hipSuccess; }
hipError_t hipHostFree(void *p) {
  std::lock_guard<std::mutex> g(mu);
  auto it = allocs.find(uintptr_t(p));
  if (it != allocs.end() && it->second.real) free(p);
  allocs.erase(uintptr_t(p));
  return hipSuccess;
}
hipError_t hipPointerGetAttributes(hipPointerAttribute_t *a, const void *p) {
  std::lock_guard<std::mutex> g(mu);
  const Alloc *x = find(p, 1);
  memset(a, 0, sizeof(*a));
  if (!x) { last = hipErrorInvalidValue; return hipErrorInvalidValue; }
  a->type = x->host ? hipMemoryTypeHost : hipMemoryTypeDevice;
  a->hostPointer = x->host ? (void *)p : nullptr;
  a->devicePointer = (void *)p;
  return hipSuccess;
}
hipError_t hipMemcpyAsync(void *d, const void *s, size_t n, hipMemcpyKind k, hipStream_t st) {
  std::lock_guard<std::mutex> g(mu);
  if (st && !streams.count(st)) die("copy on an unknown stream", st, 0);
  const Alloc *xd = find(d, n), *xs = find(s, n);
  if (!xd) die("copy destination outside every allocation", d, n);
  if (!xs) die("copy source outside every allocation", s, n);
  if (k == hipMemcpyHostToDevice && (!xs->host || xd->host)) die("H2D copy with wrong sides", d, n);
  if (k == hipMemcpyDeviceToHost && (xs->host || !xd->host)) die("D2H copy with wrong sides", d, n);
  if (xd->host && xd->real && xs->host && xs->real) memcpy(d, s, n);
  ++copies;
  return hipSuccess;
}
hipError_t hipLaunchKernel(const void *, dim3 g, dim3 b, void **, size_t, hipStream_t s) {
  std::lock_guard<std::mutex> lk(mu);
  if (s && !streams.count(s)) die("launch on an unknown stream", s, 0);
  if (g.x == 0 || b.x == 0) die("empty launch", nullptr, 0);
  ++launches;
  return hipSuccess;
}
hipError_t __hipPushCallConfiguration(dim3 g, dim3 b, size_t sh, hipStream_t s) {
  cfg_grid = g; cfg_block = b; cfg_shmem = sh; cfg_stream = s; return hipSuccess;
}
hipError_t __hipPopCallConfiguration(dim3 *g, dim3 *b, size_t *sh, hipStream_t *s) {
  *g = cfg_grid; *b = cfg_block; *sh = cfg_shmem; *s = cfg_stream; return hipSuccess;
}
void **__hipRegisterFatBinary(const void *) { static void *h[1]; return h; }
void __hipRegisterFunction(void **, const void *, char *, const char *, unsigned int, void *, void *, void *, void *, int *) {}
void __hipRegisterVar(void **, void *, char *, const char *, int, size_t, int, int) {}
void __hipUnregisterFatBinary(void **) {}
hipError_t hipFuncGetAttributes(hipFuncAttributes *a, const void *) { memset(a, 0, sizeof(*a)); return hipSuccess; }
hipError_t hipGetSymbolAddress(void **p, const void *) {
  static void *sym = nullptr;
  if (!sym) (void)hipMalloc(&sym, size_t(64) << 20);
  *p = sym;
  return hipSuccess;
}
hipError_t hipGetLastError(void) { hipError_t e = last; last = hipSuccess; return e; }
const char *hipGetErrorString(hipError_t e) { return e == hipSuccess ? "no error" : "mock error"; }
hipError_t hipIpcGetMemHandle(hipIpcMemHandle_t *, void *) { return hipErrorNotSupported; }
hipError_t hipIpcOpenMemHandle(void **, hipIpcMemHandle_t, unsigned) { return hipErrorNotSupported; }
hipError_t hipIpcCloseMemHandle(void *) { return hipErrorNotSupported; }
// statistics for the driver
long mock_launches(void) { return launches; }
long mock_copies(void) { return copies; }
long mock_waits(void) { return waits; }
int mock_streams(void) { return int(streams.size()); }
}
