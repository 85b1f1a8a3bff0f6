// state.h — state plane of the reshard library (Sec. III-A): a long-lived
// daemon owns the device memory that holds the weights and the KV cache and
// hands inference processes IPC handles to it; host metadata the recovery
// needs (block tables, per-session recency) is kept by the daemon as well.
// A crashed inference process therefore leaves both in place, and a fresh
// process maps them again before it reshards.
#pragma once

#include <stdint.h>

#include <map>
#include <string>

namespace atp {

// A shared region must stay under 2 GiB: opening a larger IPC allocation
// has not returned on the machines this was built for.
constexpr uint64_t kMaxRegion = (uint64_t(2) << 30) - (uint64_t(1) << 20);

int daemon_serve(const char *socket_path, int device);

struct StateConn {
  int fd = -1;
  std::map<void *, std::string> mapped;  // regions this client opened
};

StateConn *state_connect(const char *socket_path);
void state_disconnect(StateConn *c);
void *state_alloc(StateConn &c, const char *name, uint64_t bytes);
void *state_open(StateConn &c, const char *name, uint64_t *bytes);
void state_release(StateConn &c, void *ptr);
void state_free(StateConn &c, const char *name);
void state_put(StateConn &c, const char *name, const void *data, uint64_t bytes);
uint64_t state_get(StateConn &c, const char *name, void *data, uint64_t cap);
std::string state_list(StateConn &c);
void state_shutdown(StateConn &c);

}  // namespace atp
