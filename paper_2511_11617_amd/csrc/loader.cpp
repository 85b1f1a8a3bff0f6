// loader.cpp — range-read reload source (Sec. IV, the loader of the
// implementation): parses the headers of safetensors files (per-tensor dtype,
// shape and data offsets) and fills a plan's packed weight inflow buffer by
// reading only the byte intervals the plan lands on this GPU, with pread
// from a pool of host threads.
//
// safetensors layout: an 8-byte little-endian header length N, N bytes of
// JSON mapping each tensor name to {"dtype", "shape", "data_offsets":
// [begin, end)} (offsets relative to the byte after the header), then the
// data.  An optional "__metadata__" entry holds string pairs.
#include "loader.h"

#include <fcntl.h>
#include <sys/stat.h>
#include <unistd.h>

#include <algorithm>
#include <atomic>
#include <cctype>
#include <cerrno>
#include <chrono>
#include <condition_variable>
#include <cstring>
#include <memory>
#include <mutex>
#include <thread>

namespace atp {
namespace {

[[noreturn]] void fail(const std::string &m) { throw Error(ATP_EINVAL, m); }

constexpr uint64_t kMaxHeader = 256ull << 20;  // larger headers are rejected
constexpr uint64_t kPiece = 16ull << 20;       // largest single read

int dtype_bytes(const std::string &d) {
  static const std::pair<const char *, int> tab[] = {
      {"BOOL", 1}, {"U8", 1},  {"I8", 1},  {"F8_E4M3", 1}, {"F8_E5M2", 1}, {"I16", 2}, {"U16", 2}, {"F16", 2},
      {"BF16", 2}, {"I32", 4}, {"U32", 4}, {"F32", 4},     {"I64", 8},     {"U64", 8}, {"F64", 8}};
  for (const auto &e : tab)
    if (d == e.first) return e.second;
  return 0;
}

// A strict reader for the JSON subset safetensors headers use; any other
// value (true/false/null, floats, nested objects) is skipped where allowed.
class Json {
 public:
  Json(const char *b, const char *e, const std::string &where) : p_(b), e_(e), where_(where) {}

  void ws() {
    while (p_ < e_ && (*p_ == ' ' || *p_ == '\t' || *p_ == '\n' || *p_ == '\r')) ++p_;
  }
  bool peek(char c) {
    ws();
    return p_ < e_ && *p_ == c;
  }
  void expect(char c) {
    ws();
    if (p_ >= e_ || *p_ != c) bad(std::string("expected '") + c + "'");
    ++p_;
  }
  bool at_end() {
    ws();
    return p_ >= e_;
  }
  std::string str() {
    expect('"');
    std::string out;
    while (true) {
      if (p_ >= e_) bad("unterminated string");
      char c = *p_++;
      if (c == '"') break;
      if (static_cast<unsigned char>(c) < 0x20) bad("control character in string");
      if (c != '\\') {
        out += c;
        continue;
      }
      if (p_ >= e_) bad("unterminated escape");
      char x = *p_++;
      switch (x) {
        case '"': out += '"'; break;
        case '\\': out += '\\'; break;
        case '/': out += '/'; break;
        case 'b': out += '\b'; break;
        case 'f': out += '\f'; break;
        case 'n': out += '\n'; break;
        case 'r': out += '\r'; break;
        case 't': out += '\t'; break;
        case 'u': {
          uint32_t cp = hex4();
          if (cp >= 0xD800 && cp < 0xDC00) {  // surrogate pair
            if (e_ - p_ < 6 || p_[0] != '\\' || p_[1] != 'u') bad("lone surrogate");
            p_ += 2;
            uint32_t lo = hex4();
            if (lo < 0xDC00 || lo >= 0xE000) bad("bad surrogate pair");
            cp = 0x10000 + ((cp - 0xD800) << 10) + (lo - 0xDC00);
          }
          utf8(cp, out);
          break;
        }
        default: bad("bad escape");
      }
    }
    return out;
  }
  uint64_t uint() {
    ws();
    if (p_ >= e_ || *p_ < '0' || *p_ > '9') bad("expected a non-negative integer");
    uint64_t v = 0;
    while (p_ < e_ && *p_ >= '0' && *p_ <= '9') {
      uint64_t d = uint64_t(*p_++ - '0');
      if (v > (UINT64_MAX - d) / 10) bad("integer overflow");
      v = v * 10 + d;
    }
    if (p_ < e_ && (*p_ == '.' || *p_ == 'e' || *p_ == 'E')) bad("expected an integer");
    return v;
  }
  std::vector<uint64_t> uints() {
    std::vector<uint64_t> v;
    expect('[');
    if (peek(']')) {
      ++p_;
      return v;
    }
    while (true) {
      v.push_back(uint());
      if (peek(',')) {
        ++p_;
        continue;
      }
      expect(']');
      return v;
    }
  }
  void skip(int depth = 0) {
    if (depth > 64) bad("nesting too deep");
    ws();
    if (p_ >= e_) bad("unexpected end");
    char c = *p_;
    if (c == '"') {
      str();
    } else if (c == '{' || c == '[') {
      char close = c == '{' ? '}' : ']';
      ++p_;
      if (peek(close)) {
        ++p_;
        return;
      }
      while (true) {
        if (c == '{') {
          str();
          expect(':');
        }
        skip(depth + 1);
        if (peek(',')) {
          ++p_;
          continue;
        }
        expect(close);
        return;
      }
    } else {
      const char *s = p_;
      while (p_ < e_ && (std::isalnum(static_cast<unsigned char>(*p_)) || *p_ == '-' || *p_ == '+' || *p_ == '.'))
        ++p_;
      if (p_ == s) bad("unexpected character");
    }
  }
  [[noreturn]] void bad(const std::string &m) { fail(where_ + ": malformed header: " + m); }

 private:
  uint32_t hex4() {
    if (e_ - p_ < 4) bad("short \\u escape");
    uint32_t v = 0;
    for (int i = 0; i < 4; ++i) {
      char c = *p_++;
      v <<= 4;
      if (c >= '0' && c <= '9') v |= uint32_t(c - '0');
      else if (c >= 'a' && c <= 'f') v |= uint32_t(c - 'a' + 10);
      else if (c >= 'A' && c <= 'F') v |= uint32_t(c - 'A' + 10);
      else bad("bad hex digit");
    }
    return v;
  }
  static void utf8(uint32_t cp, std::string &o) {
    if (cp < 0x80) {
      o += char(cp);
    } else if (cp < 0x800) {
      o += char(0xC0 | (cp >> 6));
      o += char(0x80 | (cp & 0x3F));
    } else if (cp < 0x10000) {
      o += char(0xE0 | (cp >> 12));
      o += char(0x80 | ((cp >> 6) & 0x3F));
      o += char(0x80 | (cp & 0x3F));
    } else {
      o += char(0xF0 | (cp >> 18));
      o += char(0x80 | ((cp >> 12) & 0x3F));
      o += char(0x80 | ((cp >> 6) & 0x3F));
      o += char(0x80 | (cp & 0x3F));
    }
  }
  const char *p_, *e_;
  std::string where_;
};

// pread all of [off, off + n) into dst; false on EOF or an error.
bool read_all(int fd, uint64_t off, char *dst, uint64_t n) {
  while (n) {
    ssize_t r = ::pread(fd, dst, size_t(std::min<uint64_t>(n, 1ull << 30)), off_t(off));
    if (r < 0) {
      if (errno == EINTR) continue;
      return false;
    }
    if (r == 0) return false;
    dst += r;
    off += uint64_t(r);
    n -= uint64_t(r);
  }
  return true;
}

void parse_file(StFiles &S, int fi) {
  const std::string &path = S.paths[fi];
  int fd = S.fds[fi];
  struct stat stt {};
  if (fstat(fd, &stt) != 0) fail(path + ": cannot stat");
  uint64_t size = uint64_t(stt.st_size);
  unsigned char hl[8];
  if (size < 8 || !read_all(fd, 0, reinterpret_cast<char *>(hl), 8)) fail(path + ": shorter than a safetensors header");
  uint64_t n = 0;
  for (int i = 7; i >= 0; --i) n = (n << 8) | hl[i];
  if (n > kMaxHeader || n > size - 8) fail(path + ": header length " + std::to_string(n) + " does not fit the file");
  std::string head(size_t(n), '\0');
  if (!read_all(fd, 8, head.data(), n)) fail(path + ": cannot read the header");
  uint64_t data0 = 8 + n, data_bytes = size - data0;
  Json j(head.data(), head.data() + head.size(), path);
  j.expect('{');
  bool first = true;
  while (!j.peek('}')) {
    if (!first) j.expect(',');
    first = false;
    std::string name = j.str();
    j.expect(':');
    if (name == "__metadata__") {
      j.skip();
      continue;
    }
    std::string dtype;
    std::vector<uint64_t> shape, offs;
    bool has_dtype = false, has_shape = false, has_offs = false;
    j.expect('{');
    bool f2 = true;
    while (!j.peek('}')) {
      if (!f2) j.expect(',');
      f2 = false;
      std::string k = j.str();
      j.expect(':');
      if (k == "dtype") {
        dtype = j.str();
        has_dtype = true;
      } else if (k == "shape") {
        shape = j.uints();
        has_shape = true;
      } else if (k == "data_offsets") {
        offs = j.uints();
        has_offs = true;
      } else {
        j.skip();
      }
    }
    j.expect('}');
    if (!has_dtype || !has_shape || !has_offs) fail(path + ": tensor '" + name + "' lacks dtype, shape or data_offsets");
    int eb = dtype_bytes(dtype);
    if (!eb) fail(path + ": tensor '" + name + "' has unknown dtype " + dtype);
    if (offs.size() != 2 || offs[0] > offs[1] || offs[1] > data_bytes)
      fail(path + ": tensor '" + name + "' data_offsets outside the data");
    unsigned __int128 count = 1;
    for (uint64_t d : shape) {
      count *= d;
      if (count > (unsigned __int128)UINT64_MAX) fail(path + ": tensor '" + name + "' is too large");
    }
    if (count * unsigned(eb) != (unsigned __int128)(offs[1] - offs[0]))
      fail(path + ": tensor '" + name + "' size does not match its shape and dtype");
    StTensor t;
    t.file = fi;
    t.elem_bytes = eb;
    t.shape.assign(shape.begin(), shape.end());
    t.begin = data0 + offs[0];
    t.end = data0 + offs[1];
    if (!S.map.emplace(name, t).second) fail(path + ": tensor '" + name + "' appears twice");
  }
  j.expect('}');
  if (!j.at_end()) j.bad("trailing bytes after the header object");
}

struct ReadOp {
  int fd;
  uint64_t off;
  char *dst;
  uint64_t bytes;
};

}  // namespace

StFiles::~StFiles() {
  for (int fd : fds)
    if (fd >= 0) ::close(fd);
}

StFiles *st_open(const char *const *paths, int n) {
  if (n <= 0 || !paths) fail("no files");
  std::unique_ptr<StFiles> S(new StFiles());
  for (int i = 0; i < n; ++i) {
    if (!paths[i]) fail("file path is NULL");
    S->paths.push_back(paths[i]);
    int fd = ::open(paths[i], O_RDONLY | O_CLOEXEC);
    if (fd < 0) fail(std::string(paths[i]) + ": " + std::strerror(errno));
    S->fds.push_back(fd);
    parse_file(*S, i);
  }
  return S.release();
}

// ---- reads -------------------------------------------------------------------------

struct LoadJob::Impl {
  std::vector<ReadOp> ops;  // in buffer order: ops [0, k) cover [0, ops[k].dst - base)
  char *base = nullptr;
  uint64_t bytes = 0, tensor_bytes = 0;
  int threads = 1;
  size_t batch = 1, n_batches = 0;
  std::atomic<size_t> next{0};
  std::atomic<bool> bad{false};
  std::mutex mu;
  std::condition_variable cv;
  std::vector<char> done;   // per batch, under mu
  size_t front = 0;         // first batch not done, under mu
  uint64_t ready = 0;       // buffer prefix read, under mu
  bool failed = false;      // under mu
  std::vector<std::thread> pool;
  std::chrono::steady_clock::time_point t0;
  double read_ms = 0;
  // duplicates of the files' descriptors, so that the reads never depend
  // on the caller keeping the opened files (a closed descriptor's number
  // may already name another file)
  std::unordered_map<int, int> own_fd;
  int fd_of(int fd) {
    auto it = own_fd.find(fd);
    if (it != own_fd.end()) return it->second;
    int d = ::dup(fd);
    if (d < 0) throw Error(ATP_EINVAL, std::string("cannot duplicate a file descriptor: ") + strerror(errno));
    own_fd[fd] = d;
    return d;
  }
  ~Impl() {
    for (auto &kv : own_fd) ::close(kv.second);
  }

  void batch_done(size_t b, bool ok) {
    std::lock_guard<std::mutex> g(mu);
    if (!ok) {
      failed = true;
      ready = bytes;  // wake every waiter
    } else {
      done[b] = 1;
      while (front < n_batches && done[front]) ++front;
      if (!failed) ready = front < n_batches ? uint64_t(ops[front * batch].dst - base) : bytes;
    }
    cv.notify_all();
  }
  void work() {
    while (!bad.load(std::memory_order_relaxed)) {
      size_t i0 = next.fetch_add(batch);
      if (i0 >= ops.size()) return;
      size_t i1 = std::min(ops.size(), i0 + batch);
      bool ok = true;
      for (size_t i = i0; i < i1 && ok; ++i) ok = read_all(ops[i].fd, ops[i].off, ops[i].dst, ops[i].bytes);
      if (!ok) bad = true;
      batch_done(i0 / batch, ok);
    }
  }
  void join() {
    for (auto &th : pool) th.join();
    pool.clear();
  }
};

LoadJob::LoadJob(const Plan &P, const StFiles &S, const char *const *names, int n_names, void *inflow,
                 uint64_t inflow_bytes, int n_threads)
    : impl_(new Impl()) {
  const CallPlan &c = P.w;
  Impl &J = *impl_;
  if (n_names != int(P.tp.size())) fail("one tensor name per problem tensor is needed");
  if (!names) fail("names is NULL");
  if (inflow_bytes != c.inflow || (c.inflow && !inflow)) fail("inflow buffer must hold exactly " + std::to_string(c.inflow) + " bytes");
  // tensors named by the plan, checked against the problem's shapes
  std::vector<const StTensor *> ft(P.tp.size(), nullptr);
  for (size_t i = 0; i < P.tp.size(); ++i) {
    if (!names[i]) fail("tensor name " + std::to_string(i) + " is NULL");
    auto it = S.map.find(names[i]);
    if (it == S.map.end()) fail(std::string("tensor '") + names[i] + "' is in none of the files");
    const atp_tensor &t = P.tp[i].t;
    const StTensor &f = it->second;
    if (f.elem_bytes != t.elem_bytes) fail(std::string("tensor '") + names[i] + "' has another element size than the problem");
    if (f.shape.size() != 2 || f.shape[0] != uint64_t(t.rows) || f.shape[1] != uint64_t(t.cols))
      fail(std::string("tensor '") + names[i] + "' has another shape than the problem's [rows, cols]");
    ft[i] = &f;
    J.tensor_bytes += f.end - f.begin;
  }
  // the byte intervals of every inflow segment, in buffer order
  std::vector<ReadOp> &ops = J.ops;
  char *base = static_cast<char *>(inflow);
  J.base = base;
  J.bytes = c.inflow;
  for (const atp_segment &s : c.seg_in) {
    const atp_tensor &t = P.tp[size_t(s.tensor)].t;
    const StTensor &f = *ft[size_t(s.tensor)];
    const int fd = J.fd_of(S.fds[size_t(f.file)]);
    const uint64_t eb = uint64_t(t.elem_bytes), a = uint64_t(s.unit_begin) * uint64_t(t.unit),
                   b = uint64_t(s.unit_end) * uint64_t(t.unit);
    char *dst = base + s.host_offset;
    uint64_t got = 0;
    auto add = [&](uint64_t off, uint64_t n) {
      // merge with the previous read when both file and buffer continue it
      if (!ops.empty()) {
        ReadOp &q = ops.back();
        if (q.fd == fd && q.off + q.bytes == off && q.dst + q.bytes == dst + got && q.bytes + n <= kPiece) {
          q.bytes += n;
          got += n;
          return;
        }
      }
      while (n) {
        uint64_t k = std::min(n, kPiece);
        ops.push_back({fd, off, dst + got, k});
        off += k;
        got += k;
        n -= k;
      }
    };
    if (t.kind == ATP_ROWS) {
      // rows [a, b) of the [rows, cols] tensor: one interval
      add(f.begin + a * uint64_t(t.cols) * eb, (b - a) * uint64_t(t.cols) * eb);
    } else {
      // columns [a, b): one interval per row, packed row after row
      for (int64_t r = 0; r < t.rows; ++r) add(f.begin + (uint64_t(r) * uint64_t(t.cols) + a) * eb, (b - a) * eb);
    }
    if (got != s.bytes) throw Error(ATP_EINVAL, "inflow segment size disagrees with its tensor");
  }
  // balanced byte batches, taken in buffer order by a pool of threads
  unsigned hw = std::max(1u, std::thread::hardware_concurrency());
  J.threads = n_threads > 0 ? n_threads : int(std::min(16u, hw));
  J.threads = std::max(1, std::min<int>(J.threads, int(std::max<size_t>(ops.size(), 1))));
  J.batch = std::max<size_t>(1, ops.size() / (size_t(J.threads) * 64));
  J.n_batches = (ops.size() + J.batch - 1) / J.batch;
  J.done.assign(J.n_batches, 0);
  J.ready = ops.empty() ? J.bytes : 0;
}

LoadJob::~LoadJob() {
  if (impl_) {
    impl_->bad = true;  // stop taking batches
    impl_->join();
  }
}

void LoadJob::start() {
  Impl &J = *impl_;
  J.t0 = std::chrono::steady_clock::now();
  for (int i = 0; i < J.threads; ++i) J.pool.emplace_back([&J]() { J.work(); });
}

void LoadJob::await(uint64_t end) {
  Impl &J = *impl_;
  std::unique_lock<std::mutex> g(J.mu);
  J.cv.wait(g, [&]() { return J.ready >= std::min(end, J.bytes) || J.failed; });
}

void LoadJob::finish(atp_load_stats *st) {
  Impl &J = *impl_;
  J.join();
  J.read_ms = std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - J.t0).count();
  if (J.failed) fail("a range read failed (file shorter than its header says, or an I/O error)");
  if (st) {
    st->read_ms = J.read_ms;
    st->bytes = J.bytes;
    st->reads = J.ops.size();
    st->tensor_bytes = J.tensor_bytes;
    st->threads = J.threads;
  }
}

void load_weights(const Plan &P, const StFiles &S, const char *const *names, int n_names, void *inflow,
                  uint64_t inflow_bytes, int n_threads, atp_load_stats *st) {
  LoadJob job(P, S, names, n_names, inflow, inflow_bytes, n_threads);
  job.start();
  job.finish(st);
}

}  // namespace atp
