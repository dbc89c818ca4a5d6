// Local request server and client (paper §2.3: the module's model interface
// sends its inputs to an inference server and blocks until the outputs come
// back; many client processes share one GPU, and the server merges their
// requests into larger batches).  The transport here is a Unix-domain stream
// socket on one machine; the classification behind it is the library's own.
//
// Wire format (host byte order, both ends on one machine):
//   request   32-byte header {magic "PIDQ", kind, plane, 0, n, id} + payload
//             kind 1: hits, int32 [n][2] = (wire, tick) on `plane`, or
//                     [n][3] = (plane, wire, tick) when plane < 0
//             kind 2: pre-cut patches, fp32 [n][48][48]
//   response  32-byte header {magic "PIDR", status, n, id, server_ns} and, when
//             status is POINTID_OK, fp32 scores [n][4]
// A connection carries one request at a time (the client blocks, as the
// paper's module does).  The server runs one thread per connection with its
// own HIP stream, pinned staging buffer and device buffers: payload -> device,
// classification (hits through the library's dynamic batcher when it is on,
// so concurrent clients share launches; patches by pointid_classify_patches),
// scores -> host -> socket.
#include <fcntl.h>
#include <poll.h>
#include <sys/socket.h>
#include <sys/un.h>
#include <unistd.h>

#include <atomic>
#include <cerrno>
#include <chrono>
#include <cstring>
#include <memory>
#include <mutex>
#include <new>
#include <string>
#include <system_error>
#include <thread>
#include <vector>

#include "internal.h"
#include "pointid.h"

namespace {

constexpr uint32_t kReqMagic = 0x51444950u;    // "PIDQ"
constexpr uint32_t kRespMagic = 0x52444950u;   // "PIDR"
constexpr uint32_t kKindHits = 1, kKindPatches = 2;
// Per-request limits, which bound the buffers a client can make the server
// allocate: 4,194,304 hits (48 MiB) or 65,536 patches (576 MiB).
constexpr int64_t kMaxRequest = int64_t(1) << 22;
constexpr int64_t kMaxPatches = int64_t(1) << 16;
constexpr size_t kPatchBytes = sizeof(float) * 48 * 48;

struct ReqHeader {
  uint32_t magic, kind;
  int32_t plane, reserved;
  int64_t n;
  uint64_t id;
};
struct RespHeader {
  uint32_t magic;
  int32_t status;
  int64_t n;
  uint64_t id;
  int64_t server_ns;
};
static_assert(sizeof(ReqHeader) == 32 && sizeof(RespHeader) == 32, "wire headers are 32 bytes");

bool read_all(int fd, void* p, size_t n) {
  char* c = static_cast<char*>(p);
  while (n > 0) {
    const ssize_t r = recv(fd, c, n, 0);
    if (r < 0 && errno == EINTR) continue;
    if (r <= 0) return false;
    c += r;
    n -= (size_t)r;
  }
  return true;
}

bool write_all(int fd, const void* p, size_t n) {
  const char* c = static_cast<const char*>(p);
  while (n > 0) {
    const ssize_t r = send(fd, c, n, MSG_NOSIGNAL);
    if (r < 0 && errno == EINTR) continue;
    if (r <= 0) return false;
    c += r;
    n -= (size_t)r;
  }
  return true;
}

int fail_io(const std::string& what) {
  return pointid::set_error(POINTID_EIO, what + ": " + std::strerror(errno));
}

bool make_address(const char* path, sockaddr_un* a) {
  if (!path || std::strlen(path) >= sizeof(a->sun_path) || path[0] == 0) return false;
  std::memset(a, 0, sizeof(*a));
  a->sun_family = AF_UNIX;
  std::strncpy(a->sun_path, path, sizeof(a->sun_path) - 1);
  return true;
}

// Device and pinned host buffers of one connection, grown on demand.
struct Buffers {
  void* host = nullptr;
  size_t host_cap = 0;
  void* in = nullptr;
  size_t in_cap = 0;
  float* out = nullptr;
  size_t out_cap = 0;

  hipError_t ensure(size_t host_b, size_t in_b, size_t out_b) {
    hipError_t e = hipSuccess;
    if (host_b > host_cap) {
      if (host) (void)hipHostFree(host);
      host = nullptr;
      host_cap = 0;
      if ((e = hipHostMalloc(&host, host_b)) != hipSuccess) return e;
      host_cap = host_b;
    }
    if (in_b > in_cap) {
      if (in) (void)hipFree(in);
      in = nullptr;
      in_cap = 0;
      if ((e = hipMalloc(&in, in_b)) != hipSuccess) return e;
      in_cap = in_b;
    }
    if (out_b > out_cap) {
      if (out) (void)hipFree(out);
      out = nullptr;
      out_cap = 0;
      if ((e = hipMalloc((void**)&out, out_b)) != hipSuccess) return e;
      out_cap = out_b;
    }
    return e;
  }
  void release() {
    if (host) (void)hipHostFree(host);
    if (in) (void)hipFree(in);
    if (out) (void)hipFree(out);
    host = in = nullptr;
    out = nullptr;
  }
};

}  // namespace

// One connection: its socket, its thread, and whether the thread has ended.
struct Conn {
  int fd = -1;
  std::thread th;
  std::atomic<bool> done{false};
};

struct pointid_server_s {
  pointid_handle h = nullptr;
  int device = 0;
  std::vector<pointid_plane> planes;
  pointid_batcher batcher = nullptr;
  std::string path;
  int listen_fd = -1;
  int wake[2] = {-1, -1};
  std::thread acceptor;
  std::mutex mu;
  std::vector<std::unique_ptr<Conn>> conns;
  std::atomic<bool> stopping{false};

  void accept_loop();
  void serve(Conn* c);
  int handle_request(int fd, const ReqHeader& q, Buffers& buf, hipStream_t s, std::string* err);
};

int pointid_server_s::handle_request(int fd, const ReqHeader& q, Buffers& buf, hipStream_t s,
                                     std::string* err) {
  const bool hits = q.kind == kKindHits;
  const int stride = q.plane >= 0 ? 2 : 3;
  const size_t in_b = hits ? sizeof(int32_t) * stride * (size_t)q.n : kPatchBytes * (size_t)q.n;
  const size_t out_b = 16 * (size_t)q.n;
  hipError_t e = buf.ensure(in_b > out_b ? in_b : out_b, in_b, out_b);
  if (e != hipSuccess) {
    *err = std::string("server buffers: ") + hipGetErrorString(e);
    // the payload must still be consumed to keep the stream in step
    std::vector<char> sink(1 << 16);
    for (size_t left = in_b; left > 0;) {
      const size_t k = left < sink.size() ? left : sink.size();
      if (!read_all(fd, sink.data(), k)) return POINTID_EIO;
      left -= k;
    }
    return POINTID_ENOMEM;
  }
  if (!read_all(fd, buf.host, in_b)) return POINTID_EIO;
  if ((e = hipMemcpyAsync(buf.in, buf.host, in_b, hipMemcpyHostToDevice, s)) != hipSuccess) {
    *err = std::string("copy to device: ") + hipGetErrorString(e);
    return POINTID_EHIP;
  }
  int rc = POINTID_OK;
  if (!hits) {
    rc = pointid_classify_patches(h, static_cast<const float*>(buf.in), q.n, buf.out, s);
  } else if (batcher) {
    // the batcher's own stream reads the hits: they must be on the device first
    if ((e = hipStreamSynchronize(s)) != hipSuccess) {
      *err = std::string("copy to device: ") + hipGetErrorString(e);
      return POINTID_EHIP;
    }
    pointid_request r;
    r.hits = static_cast<const int32_t*>(buf.in);
    r.n_hits = q.n;
    r.plane = q.plane;
    r.scores = buf.out;
    uint64_t ticket = 0;
    rc = pointid_batcher_submit(batcher, &r, s, &ticket);
    if (rc == POINTID_OK) rc = pointid_batcher_wait(batcher, ticket);
  } else if (q.plane >= 0) {
    const pointid_plane& p = planes[q.plane];
    rc = pointid_classify(h, p.image, p.n_wires, p.n_ticks, static_cast<const int32_t*>(buf.in),
                          q.n, buf.out, s);
  } else {
    rc = pointid_classify_planes(h, planes.data(), (int32_t)planes.size(),
                                 static_cast<const int32_t*>(buf.in), q.n, buf.out, s);
  }
  if (rc != POINTID_OK) {
    *err = pointid_last_error();
    return rc;
  }
  if ((e = hipMemcpyAsync(buf.host, buf.out, out_b, hipMemcpyDeviceToHost, s)) == hipSuccess)
    e = hipStreamSynchronize(s);
  if (e != hipSuccess) {
    *err = std::string("copy to host: ") + hipGetErrorString(e);
    return POINTID_EHIP;
  }
  return POINTID_OK;
}

void pointid_server_s::serve(Conn* conn) {
  const int fd = conn->fd;
  (void)hipSetDevice(device);
  hipStream_t s = nullptr;
  const bool stream_ok = hipStreamCreate(&s) == hipSuccess;
  Buffers buf;
  for (;;) {
    ReqHeader q;
    if (!read_all(fd, &q, sizeof(q))) break;
    const auto t0 = std::chrono::steady_clock::now();
    RespHeader r{kRespMagic, POINTID_OK, q.n, q.id, 0};
    std::string err;
    bool keep = true;
    if (q.magic != kReqMagic || (q.kind != kKindHits && q.kind != kKindPatches) || q.n < 0 ||
        q.n > (q.kind == kKindPatches ? kMaxPatches : kMaxRequest)) {
      r.status = POINTID_EINVAL;        // the payload length is unknown: drop the connection
      keep = false;
    } else if (q.kind == kKindHits && (q.plane >= (int32_t)planes.size() || planes.empty())) {
      r.status = POINTID_EINVAL;
      keep = false;
    } else if (!stream_ok) {
      r.status = POINTID_EHIP;
      keep = false;
    } else if (q.n > 0) {
      r.status = handle_request(fd, q, buf, s, &err);
      if (r.status == POINTID_EIO) break;
    }
    r.server_ns = std::chrono::duration_cast<std::chrono::nanoseconds>(
                      std::chrono::steady_clock::now() - t0).count();
    if (!write_all(fd, &r, sizeof(r))) break;
    if (r.status == POINTID_OK && q.n > 0 && !write_all(fd, buf.host, 16 * (size_t)q.n)) break;
    if (!keep) break;
  }
  buf.release();
  if (s) (void)hipStreamDestroy(s);
  shutdown(fd, SHUT_RDWR);
  conn->done.store(true);
}

void pointid_server_s::accept_loop() {
  for (;;) {
    pollfd p[2] = {{listen_fd, POLLIN, 0}, {wake[0], POLLIN, 0}};
    const int k = poll(p, 2, -1);
    if (k < 0 && errno == EINTR) continue;
    if (k < 0 || stopping.load() || (p[1].revents & POLLIN)) break;
    if (!(p[0].revents & POLLIN)) continue;
    const int fd = accept(listen_fd, nullptr, nullptr);
    if (fd < 0) continue;
    std::lock_guard<std::mutex> g(mu);
    if (stopping.load()) {
      close(fd);
      break;
    }
    // connections whose clients have gone: join their threads, close their sockets
    for (size_t i = 0; i < conns.size();) {
      if (conns[i]->done.load()) {
        conns[i]->th.join();
        close(conns[i]->fd);
        conns[i] = std::move(conns.back());
        conns.pop_back();
      } else {
        ++i;
      }
    }
    // a connection the server cannot take (no memory or thread) is closed,
    // which the client sees as a dropped connection
    try {
      auto c = std::make_unique<Conn>();
      c->fd = fd;
      Conn* raw = c.get();
      conns.reserve(conns.size() + 1);
      c->th = std::thread(&pointid_server_s::serve, this, raw);
      conns.push_back(std::move(c));
    } catch (const std::exception&) {
      close(fd);
    }
  }
}

struct pointid_client_s {
  int fd = -1;
  uint64_t next_id = 1;
};

namespace {

int client_call(pointid_client c, uint32_t kind, int32_t plane, const void* payload,
                size_t payload_b, int64_t n, float* scores, int64_t* server_ns) {
  ReqHeader q{kReqMagic, kind, plane, 0, n, c->next_id++};
  if (!write_all(c->fd, &q, sizeof(q)) || !write_all(c->fd, payload, payload_b))
    return fail_io("send to server");
  RespHeader r;
  if (!read_all(c->fd, &r, sizeof(r))) return fail_io("receive from server");
  if (r.magic != kRespMagic || r.id != q.id || r.n != n)
    return pointid::set_error(POINTID_EIO, "malformed response from server");
  if (server_ns) *server_ns = r.server_ns;
  if (r.status != POINTID_OK)
    return pointid::set_error(r.status, "server rejected the request (status " +
                                            std::to_string(r.status) + ")");
  if (n > 0 && !read_all(c->fd, scores, 16 * (size_t)n)) return fail_io("receive from server");
  return POINTID_OK;
}

}  // namespace

extern "C" {

int pointid_server_start(pointid_handle h, const pointid_plane* planes, int32_t n_planes,
                         const char* socket_path, int32_t max_requests, int32_t max_delay_us,
                         pointid_server* out) {
  using pointid::set_error;
  if (!out) return set_error(POINTID_EINVAL, "out is NULL");
  *out = nullptr;
  if (!h) return set_error(POINTID_EINVAL, "handle is NULL");
  if (n_planes < 0 || n_planes > POINTID_MAX_PLANES)
    return set_error(POINTID_EINVAL, "n_planes must be in [0, 64]");
  if (n_planes > 0 && !planes) return set_error(POINTID_EINVAL, "planes is NULL");
  for (int i = 0; i < n_planes; ++i)
    if (!planes[i].image || planes[i].n_wires <= 0 || planes[i].n_ticks <= 0)
      return set_error(POINTID_EINVAL, "plane " + std::to_string(i) + " is invalid");
  if (max_requests < 0 || max_delay_us < 0)
    return set_error(POINTID_EINVAL, "max_requests and max_delay_us must be >= 0");
  sockaddr_un addr;
  if (!make_address(socket_path, &addr))
    return set_error(POINTID_EINVAL, "socket_path is NULL, empty or too long");
  auto* s = new (std::nothrow) pointid_server_s();
  if (!s) return set_error(POINTID_ENOMEM, "host allocation failed");
  s->h = h;
  s->device = pointid::handle_device(h);
  s->planes.assign(planes, planes + n_planes);
  s->path = socket_path;
  if (max_requests > 0 && n_planes > 0) {
    const int rc = pointid_batcher_create(h, planes, n_planes, max_requests, max_delay_us,
                                          &s->batcher);
    if (rc != POINTID_OK) {
      delete s;
      return rc;
    }
  }
  int rc = POINTID_OK;
  s->listen_fd = socket(AF_UNIX, SOCK_STREAM | SOCK_CLOEXEC, 0);
  if (s->listen_fd < 0) {
    rc = fail_io("socket");
  } else if (bind(s->listen_fd, reinterpret_cast<sockaddr*>(&addr), sizeof(addr)) != 0) {
    rc = fail_io(std::string("bind ") + socket_path);
  } else if (listen(s->listen_fd, 256) != 0) {
    rc = fail_io("listen");
  } else if (pipe2(s->wake, O_CLOEXEC) != 0) {
    rc = fail_io("pipe");
  }
  if (rc != POINTID_OK) {
    if (s->listen_fd >= 0) close(s->listen_fd);
    if (s->batcher) (void)pointid_batcher_destroy(s->batcher);
    delete s;
    return rc;
  }
  try {
    s->acceptor = std::thread(&pointid_server_s::accept_loop, s);
  } catch (const std::system_error& x) {
    close(s->listen_fd);
    close(s->wake[0]);
    close(s->wake[1]);
    unlink(s->path.c_str());
    if (s->batcher) (void)pointid_batcher_destroy(s->batcher);
    delete s;
    return set_error(POINTID_ENOMEM, std::string("server thread: ") + x.what());
  }
  *out = s;
  return POINTID_OK;
}

int pointid_server_stop(pointid_server s) {
  if (!s) return POINTID_OK;
  s->stopping.store(true);
  const char x = 1;
  (void)!write(s->wake[1], &x, 1);
  if (s->acceptor.joinable()) s->acceptor.join();
  {
    std::lock_guard<std::mutex> g(s->mu);
    for (auto& c : s->conns) shutdown(c->fd, SHUT_RDWR);     // a blocked read returns
  }
  for (auto& c : s->conns) {
    if (c->th.joinable()) c->th.join();
    close(c->fd);
  }
  if (s->batcher) (void)pointid_batcher_destroy(s->batcher);
  close(s->listen_fd);
  close(s->wake[0]);
  close(s->wake[1]);
  unlink(s->path.c_str());
  delete s;
  return POINTID_OK;
}

int pointid_client_connect(const char* socket_path, pointid_client* out) {
  using pointid::set_error;
  if (!out) return set_error(POINTID_EINVAL, "out is NULL");
  *out = nullptr;
  sockaddr_un addr;
  if (!make_address(socket_path, &addr))
    return set_error(POINTID_EINVAL, "socket_path is NULL, empty or too long");
  const int fd = socket(AF_UNIX, SOCK_STREAM | SOCK_CLOEXEC, 0);
  if (fd < 0) return fail_io("socket");
  if (connect(fd, reinterpret_cast<sockaddr*>(&addr), sizeof(addr)) != 0) {
    const int rc = fail_io(std::string("connect ") + socket_path);
    close(fd);
    return rc;
  }
  auto* c = new (std::nothrow) pointid_client_s();
  if (!c) {
    close(fd);
    return set_error(POINTID_ENOMEM, "host allocation failed");
  }
  c->fd = fd;
  *out = c;
  return POINTID_OK;
}

int pointid_client_classify(pointid_client c, int32_t plane, const int32_t* hits, int64_t n_hits,
                            float* scores, int64_t* server_ns) {
  using pointid::set_error;
  if (!c) return set_error(POINTID_EINVAL, "client is NULL");
  if (n_hits < 0 || n_hits > kMaxRequest)
    return set_error(POINTID_EINVAL, "n_hits must be in [0, 4194304]");
  if (n_hits > 0 && (!hits || !scores)) return set_error(POINTID_EINVAL, "NULL pointer");
  const size_t b = sizeof(int32_t) * (plane >= 0 ? 2 : 3) * (size_t)n_hits;
  return client_call(c, kKindHits, plane, hits, b, n_hits, scores, server_ns);
}

int pointid_client_classify_patches(pointid_client c, const float* patches, int64_t n,
                                    float* scores, int64_t* server_ns) {
  using pointid::set_error;
  if (!c) return set_error(POINTID_EINVAL, "client is NULL");
  if (n < 0 || n > kMaxPatches) return set_error(POINTID_EINVAL, "n must be in [0, 65536]");
  if (n > 0 && (!patches || !scores)) return set_error(POINTID_EINVAL, "NULL pointer");
  return client_call(c, kKindPatches, -1, patches, kPatchBytes * (size_t)n, n, scores, server_ns);
}

int pointid_client_close(pointid_client c) {
  if (!c) return POINTID_OK;
  close(c->fd);
  delete c;
  return POINTID_OK;
}

}  // extern "C"
