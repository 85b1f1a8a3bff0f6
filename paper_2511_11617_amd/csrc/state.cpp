// state.cpp — state plane of Sec. III-A on one node.
//
// The daemon is the owner of the GPU memory that holds the model's weights
// and KV cache: it allocates a region on request, exports an IPC handle to
// it, and keeps it until it is freed or the daemon shuts down.  Inference
// processes map the regions through those handles and read and write them.
// The daemon also stores named host blobs (block tables, per-session
// recency for the KV budget of the recovery).  It does no computation and
// talks to its clients over a Unix socket with one request at a time per
// client; a client that disappears (a crashed inference process) is simply
// dropped, its regions stay.
//
// Wire format (native endianness, one host): a request is ReqHdr, the name,
// then `payload` bytes; the answer is RepHdr, an error message of msg_len
// bytes, then `payload` bytes.
#include "state.h"

#include <errno.h>
#include <poll.h>
#include <string.h>
#include <sys/socket.h>
#include <sys/un.h>
#include <unistd.h>

#include <hip/hip_runtime_api.h>

#include <new>
#include <string>
#include <vector>

#include "plan.h"  // Error

namespace atp {
namespace {

enum : uint32_t { OP_ALLOC = 1, OP_OPEN, OP_FREE, OP_PUT, OP_GET, OP_LIST, OP_PING, OP_SHUTDOWN };

struct ReqHdr {
  uint32_t op, name_len;
  uint64_t arg, payload;
};
struct RepHdr {
  int32_t status;
  uint32_t msg_len;
  uint64_t value, payload;
};

constexpr uint32_t kMaxName = 4096;
constexpr uint64_t kMaxBlob = uint64_t(1) << 32;

bool write_all(int fd, const void *p, size_t n) {
  const char *b = static_cast<const char *>(p);
  while (n) {
    ssize_t k = send(fd, b, n, MSG_NOSIGNAL);
    if (k < 0 && errno == EINTR) continue;
    if (k <= 0) return false;
    b += k;
    n -= size_t(k);
  }
  return true;
}

bool read_all(int fd, void *p, size_t n) {
  char *b = static_cast<char *>(p);
  while (n) {
    ssize_t k = recv(fd, b, n, 0);
    if (k < 0 && errno == EINTR) continue;
    if (k <= 0) return false;
    b += k;
    n -= size_t(k);
  }
  return true;
}

sockaddr_un address(const char *path) {
  if (!path || !*path) throw Error(ATP_EINVAL, "socket path is empty");
  sockaddr_un a{};
  a.sun_family = AF_UNIX;
  if (strlen(path) >= sizeof(a.sun_path)) throw Error(ATP_EINVAL, std::string("socket path too long: ") + path);
  strcpy(a.sun_path, path);
  return a;
}

// A failed call also stays the thread's last HIP error, which the caller's
// next launch check (torch's, say) would report as its own: the error is
// reported here, so it is cleared.
void hip_ok(hipError_t e, const char *what) {
  if (e == hipSuccess) return;
  (void)hipGetLastError();
  throw Error(ATP_EHIP, std::string(what) + ": " + hipGetErrorString(e));
}

struct Region {
  void *ptr = nullptr;
  uint64_t bytes = 0;
  hipIpcMemHandle_t handle{};
};

struct Daemon {
  int device = 0;
  bool device_ready = false;
  std::map<std::string, Region> regions;
  std::map<std::string, std::vector<char>> blobs;

  void ensure_device() {
    if (device_ready) return;
    hip_ok(hipSetDevice(device), "hipSetDevice");
    device_ready = true;
  }

  // Handle one request of client `fd`; false when the client is gone.
  bool serve_one(int fd, bool &stop) {
    ReqHdr h{};
    if (!read_all(fd, &h, sizeof h)) return false;
    RepHdr r{ATP_OK, 0, 0, 0};
    std::string msg;
    std::vector<char> out;
    if (h.name_len > kMaxName || h.payload > kMaxBlob) {
      r.status = ATP_EINVAL;
      msg = "request too large";
      r.msg_len = uint32_t(msg.size());
      write_all(fd, &r, sizeof r) && write_all(fd, msg.data(), msg.size());
      return false;  // the stream cannot be resynchronised
    }
    std::string name(h.name_len, '\0');
    std::vector<char> payload;
    try {
      payload.resize(h.payload);
    } catch (const std::bad_alloc &) {
      return false;
    }
    if (!read_all(fd, &name[0], name.size()) || !read_all(fd, payload.data(), payload.size())) return false;
    try {
      switch (h.op) {
        case OP_ALLOC: {
          if (name.empty()) throw Error(ATP_EINVAL, "region name is empty");
          if (regions.count(name)) throw Error(ATP_EINVAL, "region '" + name + "' exists");
          if (h.arg == 0 || h.arg > kMaxRegion)
            throw Error(ATP_EINVAL, "region '" + name + "': size must be 1 byte to 2 GiB - 1 MiB");
          ensure_device();
          Region g;
          g.bytes = h.arg;
          hip_ok(hipMalloc(&g.ptr, g.bytes), "hipMalloc");
          hipError_t e = hipIpcGetMemHandle(&g.handle, g.ptr);
          if (e != hipSuccess) {
            (void)hipFree(g.ptr);
            hip_ok(e, "hipIpcGetMemHandle");
          }
          regions[name] = g;
          r.value = g.bytes;
          out.assign(reinterpret_cast<const char *>(&g.handle), reinterpret_cast<const char *>(&g.handle) + sizeof g.handle);
          break;
        }
        case OP_OPEN: {
          auto it = regions.find(name);
          if (it == regions.end()) throw Error(ATP_EINVAL, "no region '" + name + "'");
          r.value = it->second.bytes;
          const Region &g = it->second;
          out.assign(reinterpret_cast<const char *>(&g.handle), reinterpret_cast<const char *>(&g.handle) + sizeof g.handle);
          break;
        }
        case OP_FREE: {
          auto it = regions.find(name);
          if (it == regions.end()) throw Error(ATP_EINVAL, "no region '" + name + "'");
          hip_ok(hipFree(it->second.ptr), "hipFree");
          regions.erase(it);
          break;
        }
        case OP_PUT:
          if (name.empty()) throw Error(ATP_EINVAL, "blob name is empty");
          blobs[name].swap(payload);
          break;
        case OP_GET: {
          auto it = blobs.find(name);
          if (it == blobs.end()) throw Error(ATP_EINVAL, "no blob '" + name + "'");
          out = it->second;
          r.value = out.size();
          break;
        }
        case OP_LIST: {
          std::string t;
          for (const auto &g : regions) t += "region " + g.first + " " + std::to_string(g.second.bytes) + "\n";
          for (const auto &b : blobs) t += "blob " + b.first + " " + std::to_string(b.second.size()) + "\n";
          out.assign(t.begin(), t.end());
          r.value = regions.size();
          break;
        }
        case OP_PING:
          r.value = regions.size();
          break;
        case OP_SHUTDOWN:
          stop = true;
          break;
        default:
          throw Error(ATP_EINVAL, "unknown request " + std::to_string(h.op));
      }
    } catch (const Error &e) {
      r.status = e.code;
      msg = e.what();
      out.clear();
    } catch (const std::bad_alloc &) {
      r.status = ATP_ECAPACITY;
      msg = "daemon out of host memory";
      out.clear();
    }
    r.msg_len = uint32_t(msg.size());
    r.payload = out.size();
    return write_all(fd, &r, sizeof r) && write_all(fd, msg.data(), msg.size()) &&
           write_all(fd, out.data(), out.size());
  }

  void release_all() {
    if (device_ready)
      for (auto &g : regions) (void)hipFree(g.second.ptr);
    regions.clear();
    blobs.clear();
  }
};

std::vector<char> call(StateConn &c, uint32_t op, const std::string &name, uint64_t arg, const void *data,
                       uint64_t n, uint64_t *value) {
  if (c.fd < 0) throw Error(ATP_ESTATE, "not connected");
  ReqHdr h{op, uint32_t(name.size()), arg, n};
  if (name.size() > kMaxName) throw Error(ATP_EINVAL, "name too long");
  if (n > kMaxBlob) throw Error(ATP_EINVAL, "blob larger than 4 GiB");
  if (!write_all(c.fd, &h, sizeof h) || !write_all(c.fd, name.data(), name.size()) || !write_all(c.fd, data, n))
    throw Error(ATP_ESTATE, "lost the connection to the state daemon");
  RepHdr r{};
  if (!read_all(c.fd, &r, sizeof r)) throw Error(ATP_ESTATE, "lost the connection to the state daemon");
  std::string msg(r.msg_len, '\0');
  std::vector<char> out(r.payload);
  if (!read_all(c.fd, &msg[0], msg.size()) || !read_all(c.fd, out.data(), out.size()))
    throw Error(ATP_ESTATE, "lost the connection to the state daemon");
  if (r.status != ATP_OK) throw Error(r.status, "state daemon: " + msg);
  if (value) *value = r.value;
  return out;
}

void *map_handle(StateConn &c, const std::string &name, const std::vector<char> &h) {
  if (h.size() != sizeof(hipIpcMemHandle_t)) throw Error(ATP_EINVAL, "malformed IPC handle from the daemon");
  hipIpcMemHandle_t handle;
  memcpy(&handle, h.data(), sizeof handle);
  void *p = nullptr;
  hip_ok(hipIpcOpenMemHandle(&p, handle, hipIpcMemLazyEnablePeerAccess), "hipIpcOpenMemHandle");
  c.mapped[p] = name;
  return p;
}

}  // namespace

int daemon_serve(const char *path, int device) {
  sockaddr_un a = address(path);
  // refuse a path another daemon still answers on; remove a stale socket
  {
    int probe = socket(AF_UNIX, SOCK_STREAM | SOCK_CLOEXEC, 0);
    if (probe < 0) throw Error(ATP_EINVAL, std::string("socket: ") + strerror(errno));
    bool live = connect(probe, reinterpret_cast<sockaddr *>(&a), sizeof a) == 0;
    close(probe);
    if (live) throw Error(ATP_EINVAL, std::string("a state daemon already serves ") + path);
    unlink(path);
  }
  int ls = socket(AF_UNIX, SOCK_STREAM | SOCK_CLOEXEC, 0);
  if (ls < 0) throw Error(ATP_EINVAL, std::string("socket: ") + strerror(errno));
  if (bind(ls, reinterpret_cast<sockaddr *>(&a), sizeof a) != 0 || listen(ls, 64) != 0) {
    std::string e = strerror(errno);
    close(ls);
    throw Error(ATP_EINVAL, std::string("cannot listen on ") + path + ": " + e);
  }
  Daemon D;
  D.device = device;
  std::vector<pollfd> fds{{ls, POLLIN, 0}};
  bool stop = false;
  while (!stop) {
    int k = poll(fds.data(), fds.size(), -1);
    if (k < 0) {
      if (errno == EINTR) continue;
      break;
    }
    for (size_t i = 1; i < fds.size();) {
      if (fds[i].revents & (POLLIN | POLLHUP | POLLERR)) {
        if (!D.serve_one(fds[i].fd, stop)) {
          close(fds[i].fd);
          fds.erase(fds.begin() + long(i));
          continue;
        }
        if (stop) break;
      }
      ++i;
    }
    if (!stop && (fds[0].revents & POLLIN)) {
      int cfd = accept4(ls, nullptr, nullptr, SOCK_CLOEXEC);
      if (cfd >= 0) fds.push_back({cfd, POLLIN, 0});
    }
  }
  for (size_t i = 1; i < fds.size(); ++i) close(fds[i].fd);
  close(ls);
  unlink(path);
  D.release_all();
  return ATP_OK;
}

StateConn *state_connect(const char *path) {
  sockaddr_un a = address(path);
  int fd = socket(AF_UNIX, SOCK_STREAM | SOCK_CLOEXEC, 0);
  if (fd < 0) throw Error(ATP_EINVAL, std::string("socket: ") + strerror(errno));
  if (connect(fd, reinterpret_cast<sockaddr *>(&a), sizeof a) != 0) {
    std::string e = strerror(errno);
    close(fd);
    throw Error(ATP_EINVAL, std::string("no state daemon at ") + path + ": " + e);
  }
  StateConn *c = new StateConn();
  c->fd = fd;
  return c;
}

void state_disconnect(StateConn *c) {
  if (!c) return;
  for (auto &m : c->mapped) (void)hipIpcCloseMemHandle(m.first);
  if (c->fd >= 0) close(c->fd);
  delete c;
}

void *state_alloc(StateConn &c, const char *name, uint64_t bytes) {
  std::string n = name ? name : "";
  return map_handle(c, n, call(c, OP_ALLOC, n, bytes, nullptr, 0, nullptr));
}

void *state_open(StateConn &c, const char *name, uint64_t *bytes) {
  std::string n = name ? name : "";
  uint64_t v = 0;
  std::vector<char> h = call(c, OP_OPEN, n, 0, nullptr, 0, &v);
  void *p = map_handle(c, n, h);
  if (bytes) *bytes = v;
  return p;
}

void state_release(StateConn &c, void *ptr) {
  auto it = c.mapped.find(ptr);
  if (it == c.mapped.end()) throw Error(ATP_EINVAL, "pointer is not a region this client opened");
  hip_ok(hipIpcCloseMemHandle(ptr), "hipIpcCloseMemHandle");
  c.mapped.erase(it);
}

void state_free(StateConn &c, const char *name) {
  std::string n = name ? name : "";
  for (auto it = c.mapped.begin(); it != c.mapped.end();) {  // unmap our own view first
    if (it->second == n) {
      (void)hipIpcCloseMemHandle(it->first);
      it = c.mapped.erase(it);
    } else {
      ++it;
    }
  }
  call(c, OP_FREE, n, 0, nullptr, 0, nullptr);
}

void state_put(StateConn &c, const char *name, const void *data, uint64_t bytes) {
  if (bytes && !data) throw Error(ATP_EINVAL, "data is NULL");
  call(c, OP_PUT, name ? name : "", 0, data, bytes, nullptr);
}

uint64_t state_get(StateConn &c, const char *name, void *data, uint64_t cap) {
  std::vector<char> b = call(c, OP_GET, name ? name : "", 0, nullptr, 0, nullptr);
  if (data) {
    if (cap < b.size()) throw Error(ATP_ECAPACITY, "blob '" + std::string(name) + "' needs " + std::to_string(b.size()) + " bytes");
    memcpy(data, b.data(), b.size());
  }
  return b.size();
}

std::string state_list(StateConn &c) {
  std::vector<char> b = call(c, OP_LIST, "", 0, nullptr, 0, nullptr);
  return std::string(b.begin(), b.end());
}

void state_shutdown(StateConn &c) { call(c, OP_SHUTDOWN, "", 0, nullptr, 0, nullptr); }

}  // namespace atp
