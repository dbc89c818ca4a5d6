// C ABI of libpointid (declared in include/pointid.h): argument validation,
// weight upload, device scratch from a per-handle cache, launch sequencing.
// Every call only enqueues work on the caller's stream.
#include "pointid.h"

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "internal.h"

using namespace pointid;

// Per-handle cache of device scratch buffers, reused across calls.  A call
// takes one buffer big enough for all its scratch and records an event on its
// stream after enqueueing its work; the next user of the buffer either runs on
// the same stream (stream order protects it) or finds that event complete, and
// only when neither is possible waits for it on its own stream.  Buffers are
// allocated only when no free one fits, so steady-state calls allocate nothing.
struct ScratchPool {
  struct Entry {
    void* ptr = nullptr;
    size_t bytes = 0;
    hipEvent_t done = nullptr;     // recorded after the last user's work
    hipStream_t last = nullptr;    // stream of the last user
    bool used = false;             // `done` has been recorded
    bool busy = false;             // taken by a call being enqueued
  };
  std::mutex mu;
  std::vector<Entry> entries;
};

struct pointid_s {
  int device;
  int precision;
  DeviceWeights w;     // device pointers into `blob`
  void* blob;          // one allocation holding every parameter tensor
  ScratchPool* scratch;
};

namespace {

thread_local std::string g_err;

int fail(int code, const std::string& msg) {
  g_err = msg;
  return code;
}

int hip_fail(hipError_t e, const char* what) {
  g_err = std::string(what) + ": " + hipGetErrorString(e);
  return (e == hipErrorOutOfMemory || e == hipErrorMemoryAllocation) ? POINTID_ENOMEM
                                                                      : POINTID_EHIP;
}

// Makes `dev` current for the scope of a call and restores the caller's device.
class DeviceScope {
 public:
  explicit DeviceScope(int dev) {
    if (hipGetDevice(&old_) != hipSuccess) old_ = -1;
    if (old_ != dev) err_ = hipSetDevice(dev);
  }
  ~DeviceScope() {
    if (old_ >= 0 && err_ == hipSuccess) (void)hipSetDevice(old_);
  }
  hipError_t error() const { return err_; }

 private:
  int old_ = -1;
  hipError_t err_ = hipSuccess;
};

// ---- optional per-kernel timing (pointid_timing_*)
//
// The timed kernels of one call form a chain on its stream: the first is timed
// from an event recorded on the stream just before it, and every kernel
// carries a stop event on its own dispatch (hipExtLaunchKernel); a kernel's
// time runs from the end of the one before it (or that first event) to its
// own end, the launch gap in between charged to it.  A stop event on a
// dispatch adds nothing to the stream; a recorded event leaves a gap of about
// 3.5 us (one per call), and a start event on the dispatch about 5 us and
// 10-20 us of host time.
// Events are reference counted: a record holds its two, and the chain holds
// its last stop event until the next kernel has taken it as its start.
struct TimingRec {
  const char* name;
  hipEvent_t a, b;
};
struct Timing {
  std::atomic<bool> on{false};
  std::mutex mu;
  std::vector<TimingRec> pending;
  std::map<std::string, std::pair<double, int64_t>> total;
  std::map<hipEvent_t, int> refs;
  // with mu held
  void hold(hipEvent_t e) { ++refs[e]; }
  void release(hipEvent_t e) {
    auto it = refs.find(e);
    if (it == refs.end() || --it->second > 0) return;
    refs.erase(it);
    (void)hipEventDestroy(e);
  }
};
Timing& timing() {
  static Timing t;
  return t;
}

// The calling thread's chain; a call's workspace opens it (nested workspaces
// share it).
struct TimingChain {
  int depth = 0;
  hipStream_t stream = nullptr;
  hipEvent_t last = nullptr;                 // held by the chain
};
TimingChain& timing_chain() {
  static thread_local TimingChain c;
  return c;
}
class ChainScope {
 public:
  ChainScope() { ++timing_chain().depth; }
  ~ChainScope() {
    TimingChain& c = timing_chain();
    if (--c.depth > 0 || !c.last) return;
    std::lock_guard<std::mutex> g(timing().mu);
    timing().release(c.last);
    c.last = nullptr;
  }
};

// Times the one launch in its scope while timing is enabled.
class KernelTimer {
 public:
  KernelTimer(const char* name, hipStream_t s) : name_(name), s_(s) {
    Timing& T = timing();
    if (!T.on.load(std::memory_order_relaxed)) return;
    if (hipEventCreate(&b_) != hipSuccess) return;
    TimingChain& c = timing_chain();
    std::lock_guard<std::mutex> g(T.mu);
    if (c.depth > 0 && c.last && c.stream == s) {
      a_ = c.last;                           // the previous kernel's end
    } else if (hipEventCreate(&a_) != hipSuccess) {
      (void)hipEventDestroy(b_);
      return;
    } else if (hipEventRecord(a_, s) != hipSuccess) {
      (void)hipEventDestroy(a_);
      (void)hipEventDestroy(b_);
      return;
    }
    T.hold(a_);
    T.hold(b_);
    LaunchEvents& ev = launch_events();
    ev.start = nullptr;
    ev.stop = b_;
    active_ = true;
  }
  ~KernelTimer() {
    if (!active_) return;
    LaunchEvents& ev = launch_events();
    const bool launched = ev.stop == nullptr;   // the launch took the events
    ev = LaunchEvents();
    Timing& T = timing();
    std::lock_guard<std::mutex> g(T.mu);
    if (!launched) {                         // nothing was launched (an empty call)
      T.release(a_);
      T.release(b_);
      return;
    }
    TimingChain& c = timing_chain();
    if (c.depth > 0) {
      if (c.last) T.release(c.last);
      c.last = b_;
      c.stream = s_;
      T.hold(b_);
    }
    T.pending.push_back({name_, a_, b_});
  }

 private:
  const char* name_;
  hipStream_t s_;
  hipEvent_t a_{}, b_{};
  bool active_ = false;
};

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

constexpr size_t kScratchAlign = 256;
constexpr size_t kMaxScratchBuffers = 512;
size_t pad256(size_t b) { return (b + kScratchAlign - 1) / kScratchAlign * kScratchAlign; }

// One call's scratch: a buffer of the handle's ScratchPool, handed back (with
// its event recorded on the call's stream) when the scope ends.
class Workspace {
 public:
  Workspace(ScratchPool* pool, hipStream_t s) : pool_(pool), s_(s) {}
  // A caller-provided buffer of `cap` bytes instead of the pool: reserve only
  // checks the size, and nothing is allocated or recorded.
  Workspace(void* base, size_t cap) : pool_(nullptr), s_(nullptr) {
    fixed_ = true;
    base_ = static_cast<char*>(base);
    cap_ = cap;
  }
  ~Workspace() {
    if (idx_ < 0) return;
    hipError_t e = recorded_ ? hipSuccess : hipEventRecord(done_, s_);
    // without the event, the next user could not tell when this call's work
    // is done: wait for it here (an error path only)
    if (e != hipSuccess) (void)hipStreamSynchronize(s_);
    std::lock_guard<std::mutex> g(pool_->mu);
    ScratchPool::Entry& en = pool_->entries[idx_];
    en.busy = false;
    en.last = s_;
    en.used = (e == hipSuccess);
  }

  // Takes a buffer of at least `bytes` for this call.
  hipError_t reserve(size_t bytes) {
    if (fixed_) return bytes <= cap_ ? hipSuccess : hipErrorInvalidValue;
    std::unique_lock<std::mutex> g(pool_->mu);
    std::vector<ScratchPool::Entry>& v = pool_->entries;
    int same = -1, ready = -1, any = -1;
    for (int i = 0; i < (int)v.size(); ++i) {
      const ScratchPool::Entry& en = v[i];
      if (en.busy || !en.ptr || en.bytes < bytes) continue;   // (empty slots are skipped)
      if (en.last == s_ || !en.used) {
        if (same < 0 || en.bytes < v[same].bytes) same = i;
      } else if (hipEventQuery(en.done) == hipSuccess) {
        if (ready < 0 || en.bytes < v[ready].bytes) ready = i;
      } else if (any < 0 || en.bytes < v[any].bytes) {
        any = i;
      }
    }
    int pick = same >= 0 ? same : ready;
    if (pick < 0 && (v.size() >= kMaxScratchBuffers)) pick = any;
    if (pick >= 0) {
      take(pick);
      const bool wait = v[pick].used && v[pick].last != s_ && pick != ready;
      g.unlock();
      return wait ? hipStreamWaitEvent(s_, done_, 0) : hipSuccess;
    }
    // a new buffer, sized to the next power of two (at least 4 MiB) so that
    // requests of varying size share buffers; past 1 GiB to the next 256 MiB,
    // so that a very large call does not reserve up to twice its need.  It
    // takes the slot of a buffer pointid_trim freed, if there is one.
    int slot = -1;
    for (int i = 0; i < (int)v.size() && slot < 0; ++i)
      if (!v[i].ptr && !v[i].busy) slot = i;
    if (slot < 0) {
      v.emplace_back();
      slot = (int)v.size() - 1;
    }
    v[slot] = ScratchPool::Entry();
    v[slot].busy = true;
    g.unlock();
    size_t cap = size_t(4) << 20;
    while (cap < bytes && cap < (size_t(1) << 30)) cap <<= 1;
    if (cap < bytes) cap = (bytes + (size_t(256) << 20) - 1) & ~((size_t(256) << 20) - 1);
    void* p = nullptr;
    hipEvent_t ev = nullptr;
    hipError_t e = hipEventCreateWithFlags(&ev, hipEventDisableTiming);
    if (e == hipSuccess) e = hipMalloc(&p, cap);
    g.lock();
    if (e != hipSuccess) {
      if (ev) (void)hipEventDestroy(ev);
      v[slot] = ScratchPool::Entry();            // empty, free: skipped by later calls
      return e;
    }
    v[slot].ptr = p;
    v[slot].bytes = cap;
    v[slot].done = ev;
    take(slot);
    return hipSuccess;
  }

  // Lets the calling thread's next launch record the completion event at the
  // end of its kernel (no packet of its own on the stream); false for a
  // caller's buffer, which has no event.
  bool attach_done() {
    if (fixed_ || idx_ < 0) return false;
    LaunchEvents& ev = launch_events();
    if (ev.stop) return false;
    ev.stop = done_;
    return true;
  }
  void mark_recorded() { recorded_ = true; }

  // Carves the next piece (256-byte aligned) out of the reserved buffer.
  hipError_t get(size_t bytes, void** out) {
    *out = nullptr;
    if (bytes == 0) return hipSuccess;
    if ((idx_ < 0 && !fixed_) || used_ + pad256(bytes) > cap_) return hipErrorInvalidValue;
    *out = base_ + used_;
    used_ += pad256(bytes);
    return hipSuccess;
  }

 private:
  void take(int i) {                           // with pool_->mu held
    ScratchPool::Entry& en = pool_->entries[i];
    en.busy = true;
    idx_ = i;
    base_ = static_cast<char*>(en.ptr);
    cap_ = en.bytes;
    done_ = en.done;
  }

  ChainScope chain_;                           // the call's timed kernels
  ScratchPool* pool_;
  hipStream_t s_;
  bool fixed_ = false;
  bool recorded_ = false;
  int idx_ = -1;
  char* base_ = nullptr;
  size_t cap_ = 0, used_ = 0;
  hipEvent_t done_ = nullptr;
};

// Scope of a call's last launch: the launch also records the workspace's
// completion event.
class EndsCall {
 public:
  explicit EndsCall(Workspace& ws) : ws_(ws), on_(ws.attach_done()) {}
  ~EndsCall() {
    if (on_) launch_events().stop = nullptr;
  }
  void launched(hipError_t e) {
    if (on_ && e == hipSuccess && launch_events().stop == nullptr) ws_.mark_recorded();
  }

 private:
  Workspace& ws_;
  bool on_;
};

// Pre-cut fp32 batches up to this size are rounded to 16 bits inside the
// fused kernel (measured crossover: about 4,096 patches).
constexpr int64_t kInKernelCast = 4096;

// Scratch bytes of one call: 16-bit or fp32 patches (when the call makes
// them) and the FC1 split-K partials.
size_t scratch_bytes(int precision, int64_t n, bool makes_patches) {
  const bool half = precision != POINTID_FP32;
  size_t b = 0;
  if (makes_patches) b += pad256((half ? 2 : 4) * (size_t)n * kPatchPix);
  const int S = precision == POINTID_FP8 ? conv_fc1_8_splits()
                : half ? conv_fc1_16_splits() : conv_fc1_f32_splits();
  b += pad256(sizeof(float) * (size_t)S * n * kFc1Out);
  return b;
}

// fp32 handles: patches (fp32 [n][2304]) -> scores, or into the outputs of the
// requests of `reqs` when it is given.
int run_network_fp32(pointid_handle h, const float* patches, int64_t n, float* scores,
                     hipStream_t stream, Workspace& ws, const RequestTable* reqs = nullptr) {
  const int S = conv_fc1_f32_splits();
  float* part = nullptr;
  hipError_t e = ws.get(sizeof(float) * (size_t)S * n * kFc1Out, (void**)&part);
  if (e != hipSuccess) return hip_fail(e, "workspace (FC1 partials)");
  {
    KernelTimer kt("conv_fc1_f32", stream);
    e = launch_conv_fc1_f32(patches, n, 0, n, h->w.conv_w, h->w.conv_b, h->w.fc1_wt, part, stream);
  }
  if (e != hipSuccess) return hip_fail(e, "conv_fc1_f32 launch");
  {
    KernelTimer kt("tail", stream);
    EndsCall end(ws);
    e = reqs ? launch_tail_requests(part, S, h->w, *reqs, stream)
             : launch_tail(part, S, n, h->w, scores, stream);
    end.launched(e);
  }
  if (e != hipSuccess) return hip_fail(e, "tail launch");
  return POINTID_OK;
}

// Element type of the patches a handle's network reads: 8-bit handles run
// their conv on fp16 patches.
int patch_dtype(int precision) { return precision == POINTID_FP8 ? POINTID_FP16 : precision; }

// 16-bit and 8-bit handles: patches (bf16 or fp16 [n][2304], or fp32 when
// f32_in, rounded by the fused 16-bit kernel) -> scores.
int run_network_16(pointid_handle h, const void* patches, bool f32_in, int64_t n, float* scores,
                   hipStream_t stream, Workspace& ws, const RequestTable* reqs = nullptr) {
  const bool fp8 = h->precision == POINTID_FP8;
  const int S = fp8 ? conv_fc1_8_splits() : conv_fc1_16_splits();
  float* part = nullptr;
  hipError_t e = ws.get(sizeof(float) * (size_t)S * n * kFc1Out, (void**)&part);
  if (e != hipSuccess) return hip_fail(e, "workspace (FC1 partials)");
  if (fp8 && f32_in) return fail(POINTID_EUNSUPPORTED, "8-bit handles read 16-bit patches");
  if (fp8) {
    KernelTimer kt("conv_fc1_8", stream);
    e = launch_conv_fc1_8(static_cast<const uint16_t*>(patches), n, 0, n, h->w.fc1_frag8,
                          h->w.conv_frag, part, stream);
  } else {
    KernelTimer kt("conv_fc1_16", stream);
    e = launch_conv_fc1_16(h->precision == POINTID_FP16, patches, f32_in, n, 0, n, h->w.fc1_frag,
                           h->w.conv_frag, part, stream);
  }
  if (e != hipSuccess) return hip_fail(e, "conv_fc1 launch");
  {
    KernelTimer kt("tail", stream);
    EndsCall end(ws);
    e = reqs ? launch_tail_requests(part, S, h->w, *reqs, stream)
             : launch_tail(part, S, n, h->w, scores, stream);
    end.launched(e);
  }
  if (e != hipSuccess) return hip_fail(e, "tail launch");
  return POINTID_OK;
}

// The hit paths: gather, then the network.  Scratch comes from the handle's
// pool, or, when `fixed` is given, from that buffer (already sized).
int classify_hits(pointid_handle h, const PlaneTable& planes, const int32_t* hits,
                  int stride, int64_t n, float* scores, void* stream_, int tick_div = 1,
                  Workspace* fixed = nullptr) {
  hipStream_t stream = static_cast<hipStream_t>(stream_);
  DeviceScope dev(h->device);
  if (dev.error() != hipSuccess) return hip_fail(dev.error(), "hipSetDevice");
  Workspace pooled(h->scratch, stream);
  Workspace& ws = fixed ? *fixed : pooled;
  hipError_t e = ws.reserve(scratch_bytes(h->precision, n, true));
  if (e != hipSuccess) return hip_fail(e, "scratch buffer");
  const bool half = h->precision != POINTID_FP32;
  void* patches = nullptr;
  e = ws.get((half ? 2 : 4) * (size_t)n * kPatchPix, &patches);
  if (e != hipSuccess) return hip_fail(e, "workspace (patches)");
  {
    KernelTimer kt("gather", stream);
    e = launch_gather(planes, hits, stride, n, patches, patch_dtype(h->precision), stream, tick_div);
  }
  if (e != hipSuccess) return hip_fail(e, "gather launch");
  if (half) return run_network_16(h, patches, false, n, scores, stream, ws);
  return run_network_fp32(h, static_cast<const float*>(patches), n, scores, stream, ws);
}

int check_planes(const pointid_plane* planes, int32_t n_planes, PlaneTable* t) {
  if (!planes) return fail(POINTID_EINVAL, "planes is NULL");
  if (n_planes < 1 || n_planes > kMaxPlanes)
    return fail(POINTID_EINVAL, "n_planes must be in [1, 64]");
  std::memset(t, 0, sizeof(*t));
  t->n = n_planes;
  for (int i = 0; i < n_planes; ++i) {
    if (!planes[i].image) return fail(POINTID_EINVAL, "plane " + std::to_string(i) + " image is NULL");
    if (planes[i].n_wires <= 0 || planes[i].n_ticks <= 0)
      return fail(POINTID_EINVAL, "plane " + std::to_string(i) + " has a non-positive size");
    t->p[i].image = planes[i].image;
    t->p[i].n_wires = planes[i].n_wires;
    t->p[i].n_ticks = planes[i].n_ticks;
  }
  return POINTID_OK;
}

// One batch of at most kMaxRequests non-empty requests: their hits are
// gathered into one patch buffer and classified together; the tail writes
// every patch's scores into its request's output.
int classify_request_batch(pointid_handle h, const PlaneTable& planes, const RequestTable& reqs,
                           hipStream_t stream) {
  const int64_t n = reqs.start[reqs.n];
  if (n == 0) return POINTID_OK;
  Workspace ws(h->scratch, stream);
  hipError_t e = ws.reserve(scratch_bytes(h->precision, n, true));
  if (e != hipSuccess) return hip_fail(e, "scratch buffer");
  const bool half = h->precision != POINTID_FP32;
  void* patches = nullptr;
  e = ws.get((half ? 2 : 4) * (size_t)n * kPatchPix, &patches);
  if (e != hipSuccess) return hip_fail(e, "workspace (patches)");
  {
    KernelTimer kt("gather", stream);
    e = launch_gather_requests(planes, reqs, patches, patch_dtype(h->precision), stream);
  }
  if (e != hipSuccess) return hip_fail(e, "gather launch");
  if (half) return run_network_16(h, patches, false, n, nullptr, stream, ws, &reqs);
  return run_network_fp32(h, static_cast<const float*>(patches), n, nullptr, stream, ws, &reqs);
}

// ---- scratch for pointid_classify_planes_noalloc: a fixed device array,
// sized for kNoAllocMaxHits hits at any precision (fp32 patches and the
// split-K partials of both fused kernels, 8 splits each).  Every GPU the
// library runs on holds its own copy until the process ends.  In host code
// the array's name is no device address: the address comes from
// hipGetSymbolAddress, once per device, and only that address is used.
constexpr int64_t kNoAllocMaxHits = 8192;
constexpr size_t kNoAllocBytes =
    ((size_t)kNoAllocMaxHits * kPatchPix * 4 + kScratchAlign - 1) / kScratchAlign * kScratchAlign +
    ((size_t)8 * kNoAllocMaxHits * kFc1Out * 4 + kScratchAlign - 1) / kScratchAlign * kScratchAlign;
static __device__ __align__(256) unsigned char scratch[kNoAllocBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// The device address of `scratch` on the current device `dev`, looked up on
// the first call there.
hipError_t noalloc_scratch(int dev, void** out) {
  *out = nullptr;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> g(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}

}  // namespace

namespace pointid {
LaunchEvents& launch_events() {
  static thread_local LaunchEvents ev;
  return ev;
}
int set_error(int code, const std::string& msg) { return fail(code, msg); }
int handle_device(pointid_handle h) { return h->device; }
}  // namespace pointid

extern "C" {

const char* pointid_last_error(void) { return g_err.c_str(); }

const char* pointid_version(void) { return "libpointid 0.1 (gfx950)"; }

int pointid_timing_enable(int on) {
  timing().on.store(on != 0);
  return POINTID_OK;
}

int pointid_timing_reset(void) {
  Timing& T = timing();
  std::lock_guard<std::mutex> g(T.mu);
  for (TimingRec& r : T.pending) {
    (void)hipEventSynchronize(r.b);
    T.release(r.a);
    T.release(r.b);
  }
  T.pending.clear();
  T.total.clear();
  return POINTID_OK;
}

int pointid_timing_query(const char* kernel, double* total_ms, int64_t* launches) {
  if (!kernel || !total_ms || !launches) return fail(POINTID_EINVAL, "NULL argument");
  Timing& T = timing();
  std::lock_guard<std::mutex> g(T.mu);
  int rc = POINTID_OK;
  for (TimingRec& r : T.pending) {
    float ms = 0.f;
    hipError_t e = hipEventSynchronize(r.b);
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, r.a, r.b);
    if (e != hipSuccess) rc = hip_fail(e, "timing event");
    auto& slot = T.total[r.name];
    slot.first += ms;
    slot.second += 1;
  }
  for (TimingRec& r : T.pending) {
    T.release(r.a);
    T.release(r.b);
  }
  T.pending.clear();
  auto it = T.total.find(kernel);
  *total_ms = it == T.total.end() ? 0.0 : it->second.first;
  *launches = it == T.total.end() ? 0 : it->second.second;
  return rc;
}

int pointid_create(const pointid_weights* w, int precision, int device,
                   pointid_handle* out) {
  if (!out) return fail(POINTID_EINVAL, "out is NULL");
  *out = nullptr;
  if (!w) return fail(POINTID_EINVAL, "weights is NULL");
  const float* members[] = {w->conv_w, w->conv_b, w->fc1_w, w->fc1_b, w->fc2_w,
                            w->fc2_b,  w->cls_w,  w->cls_b, w->mic_w, w->mic_b};
  for (const float* m : members)
    if (!m) return fail(POINTID_EINVAL, "a weight pointer is NULL");
  if (precision != POINTID_FP32 && precision != POINTID_BF16 && precision != POINTID_FP16 &&
      precision != POINTID_FP8)
    return fail(POINTID_EUNSUPPORTED,
                "precision must be POINTID_FP32, POINTID_BF16, POINTID_FP16 or POINTID_FP8");
  int count = 0;
  if (hipGetDeviceCount(&count) != hipSuccess || count <= 0)
    return fail(POINTID_ENODEV, "no HIP device visible");
  if (device < 0 || device >= count)
    return fail(POINTID_ENODEV, "device ordinal out of range");
  hipDeviceProp_t prop;
  hipError_t e = hipGetDeviceProperties(&prop, device);
  if (e != hipSuccess) return hip_fail(e, "hipGetDeviceProperties");
  if (std::strncmp(prop.gcnArchName, "gfx950", 6) != 0)
    return fail(POINTID_ENODEV, std::string("device is ") + prop.gcnArchName + ", library is built for gfx950");
  DeviceScope dev(device);
  if (dev.error() != hipSuccess) return hip_fail(dev.error(), "hipSetDevice");

  auto* hnd = new (std::nothrow) pointid_s();
  if (!hnd) return fail(POINTID_ENOMEM, "host allocation failed");
  hnd->device = device;
  hnd->precision = precision;
  hnd->w.precision = precision;
  const bool half = precision != POINTID_FP32;
  const bool fp8 = precision == POINTID_FP8;
  // 8-bit handles: per FC1 output n the exponent k_n, the largest with
  // max |W1[.][n]| 2^k_n <= 448 = (7/8) 2^9 (with max = f 2^e, f in [1/2, 1):
  // 9 - e when f <= 7/8, else 8 - e; 0 for a column of zeros), and 2^-k_n
  std::vector<int> fc1_exp(fp8 ? kFc1Out : 0);
  std::vector<float> fc1_scale(fp8 ? kFc1Out : 0);
  if (fp8) {
    std::vector<float> mx(kFc1Out, 0.f);
    for (int64_t k = 0; k < kFc1In; ++k)
      for (int o = 0; o < kFc1Out; ++o) mx[o] = std::max(mx[o], std::fabs(w->fc1_w[k * kFc1Out + o]));
    for (int o = 0; o < kFc1Out; ++o) {
      int e2 = 0;
      const float f = std::frexp(mx[o], &e2);
      fc1_exp[o] = mx[o] > 0.f ? (f <= 0.875f ? 9 - e2 : 8 - e2) : 0;
      fc1_scale[o] = std::ldexp(1.0f, -fc1_exp[o]);
    }
  }

  // one device allocation for every tensor the handle keeps
  struct Piece { const void* src; size_t bytes; const void** dst; };
  std::vector<Piece> pieces = {
      {w->conv_w, sizeof(float) * kCh * kK * kK, (const void**)&hnd->w.conv_w},
      {w->conv_b, sizeof(float) * kCh, (const void**)&hnd->w.conv_b},
      {w->fc1_b, sizeof(float) * kFc1Out, (const void**)&hnd->w.fc1_b},
      {w->fc2_w, sizeof(float) * kFc1Out * kFc2Out, (const void**)&hnd->w.fc2_w},
      {w->fc2_b, sizeof(float) * kFc2Out, (const void**)&hnd->w.fc2_b},
      {w->cls_w, sizeof(float) * kFc2Out * kNcls, (const void**)&hnd->w.cls_w},
      {w->cls_b, sizeof(float) * kNcls, (const void**)&hnd->w.cls_b},
      {w->mic_w, sizeof(float) * kFc2Out, (const void**)&hnd->w.mic_w},
      {w->mic_b, sizeof(float), (const void**)&hnd->w.mic_b},
  };
  const int* fc1_exp_dev = nullptr;
  if (fp8) {
    pieces.push_back({nullptr, (size_t)kConvFrags * 16, (const void**)&hnd->w.conv_frag});
    pieces.push_back({nullptr, (size_t)kFc1Frag8Bytes, (const void**)&hnd->w.fc1_frag8});
    pieces.push_back({fc1_scale.data(), sizeof(float) * kFc1Out, (const void**)&hnd->w.fc1_scale});
    pieces.push_back({fc1_exp.data(), sizeof(int) * kFc1Out, (const void**)&fc1_exp_dev});
  } else if (half) {
    pieces.push_back({nullptr, (size_t)kConvFrags * 16, (const void**)&hnd->w.conv_frag});
    pieces.push_back({nullptr, (size_t)kFc1Frags * 16, (const void**)&hnd->w.fc1_frag});
  } else {
    pieces.push_back({nullptr, sizeof(float) * kFc1In * kFc1Out, (const void**)&hnd->w.fc1_wt});
  }
  size_t total = 0;
  std::vector<size_t> offs;
  for (const Piece& p : pieces) {
    offs.push_back(total);
    total += (p.bytes + 255) & ~size_t(255);
  }
  e = hipMalloc(&hnd->blob, total);
  if (e != hipSuccess) {
    delete hnd;
    return hip_fail(e, "hipMalloc(weights)");
  }
  for (size_t i = 0; i < pieces.size(); ++i) {
    char* d = static_cast<char*>(hnd->blob) + offs[i];
    *pieces[i].dst = d;
    if (!pieces[i].src) continue;            // filled on the device below
    e = hipMemcpy(d, pieces[i].src, pieces[i].bytes, hipMemcpyHostToDevice);
    if (e != hipSuccess) {
      (void)hipFree(hnd->blob);
      delete hnd;
      return hip_fail(e, "hipMemcpy(weights)");
    }
  }
  {
    // FC1 is rearranged on the device from a temporary fp32 copy: 16-bit
    // fragments for the MFMA kernel, or the transposed fp32 matrix
    float* w1 = nullptr;
    e = hipMalloc(&w1, sizeof(float) * kFc1In * kFc1Out);
    if (e == hipSuccess)
      e = hipMemcpy(w1, w->fc1_w, sizeof(float) * kFc1In * kFc1Out, hipMemcpyHostToDevice);
    if (e == hipSuccess && fp8) {
      e = launch_pack_conv_fp16(hnd->w.conv_w, hnd->w.conv_b, const_cast<uint4*>(hnd->w.conv_frag),
                                nullptr);
      if (e == hipSuccess)
        e = launch_pack_fc1_8(w1, fc1_exp_dev, const_cast<uint8_t*>(hnd->w.fc1_frag8), nullptr);
    }
    if (e == hipSuccess && half && !fp8)
      e = launch_pack_16(precision == POINTID_FP16, hnd->w.conv_w, hnd->w.conv_b, w1,
                         const_cast<uint4*>(hnd->w.conv_frag), const_cast<uint4*>(hnd->w.fc1_frag),
                         nullptr);
    if (e == hipSuccess && !half)
      e = launch_transpose_w1(w1, const_cast<float*>(hnd->w.fc1_wt), nullptr);
    if (e == hipSuccess) e = hipDeviceSynchronize();
    if (w1) (void)hipFree(w1);
    if (e != hipSuccess) {
      (void)hipFree(hnd->blob);
      delete hnd;
      return hip_fail(e, "weight packing");
    }
  }
  hnd->scratch = new (std::nothrow) ScratchPool();
  if (!hnd->scratch) {
    (void)hipFree(hnd->blob);
    delete hnd;
    return fail(POINTID_ENOMEM, "host allocation failed");
  }
  *out = hnd;
  return POINTID_OK;
}

int pointid_destroy(pointid_handle h) {
  if (!h) return POINTID_OK;
  {
    DeviceScope dev(h->device);
    (void)hipDeviceSynchronize();
    if (h->blob) (void)hipFree(h->blob);
    if (h->scratch) {
      for (ScratchPool::Entry& en : h->scratch->entries) {
        if (en.ptr) (void)hipFree(en.ptr);
        if (en.done) (void)hipEventDestroy(en.done);
      }
      delete h->scratch;
    }
  }
  delete h;
  return POINTID_OK;
}

int pointid_trim(pointid_handle h, uint64_t keep_bytes, uint64_t* cached_bytes) {
  if (!h) return fail(POINTID_EINVAL, "handle is NULL");
  DeviceScope dev(h->device);
  if (dev.error() != hipSuccess) return hip_fail(dev.error(), "hipSetDevice");
  ScratchPool* pool = h->scratch;
  std::lock_guard<std::mutex> g(pool->mu);
  std::vector<ScratchPool::Entry>& v = pool->entries;
  uint64_t total = 0;
  for (const ScratchPool::Entry& en : v) total += en.bytes;
  // idle buffers, largest first: not being taken by a call, and their last
  // user's work done (or never used)
  std::vector<int> idle;
  for (int i = 0; i < (int)v.size(); ++i) {
    const ScratchPool::Entry& en = v[i];
    if (!en.ptr || en.busy) continue;
    if (!en.used || hipEventQuery(en.done) == hipSuccess) idle.push_back(i);
  }
  std::sort(idle.begin(), idle.end(), [&](int a, int b) { return v[a].bytes > v[b].bytes; });
  int rc = POINTID_OK;
  for (int i : idle) {
    if (total <= keep_bytes) break;
    ScratchPool::Entry& en = v[i];
    const hipError_t e = hipFree(en.ptr);
    if (e != hipSuccess) {
      rc = hip_fail(e, "hipFree(scratch)");
      break;
    }
    if (en.done) (void)hipEventDestroy(en.done);
    total -= en.bytes;
    en = ScratchPool::Entry();              // an empty slot, reused by the next allocation
  }
  if (cached_bytes) *cached_bytes = total;
  return rc;
}

int pointid_precision(pointid_handle h) {
  if (!h) return fail(POINTID_EINVAL, "handle is NULL");
  return h->precision;
}

int pointid_classify(pointid_handle h, const float* image, int32_t n_wires,
                     int32_t n_ticks, const int32_t* hits, int64_t n_hits,
                     float* scores, void* stream) {
  if (!h) return fail(POINTID_EINVAL, "handle is NULL");
  if (n_hits < 0) return fail(POINTID_EINVAL, "n_hits is negative");
  if (n_wires <= 0 || n_ticks <= 0) return fail(POINTID_EINVAL, "n_wires and n_ticks must be positive");
  if (n_hits == 0) return POINTID_OK;
  if (!image || !hits || !scores) return fail(POINTID_EINVAL, "NULL device pointer");
  if (!aligned16(scores)) return fail(POINTID_EINVAL, "scores must be 16-byte aligned");
  PlaneTable t;
  std::memset(&t, 0, sizeof(t));
  t.n = 1;
  t.p[0] = {image, n_wires, n_ticks};
  return classify_hits(h, t, hits, 2, n_hits, scores, stream);
}

int pointid_classify_planes(pointid_handle h, const pointid_plane* planes, int32_t n_planes,
                            const int32_t* hits, int64_t n_hits, float* scores,
                            void* stream) {
  if (!h) return fail(POINTID_EINVAL, "handle is NULL");
  if (n_hits < 0) return fail(POINTID_EINVAL, "n_hits is negative");
  PlaneTable t;
  int rc = check_planes(planes, n_planes, &t);
  if (rc != POINTID_OK) return rc;
  if (n_hits == 0) return POINTID_OK;
  if (!hits || !scores) return fail(POINTID_EINVAL, "NULL device pointer");
  if (!aligned16(scores)) return fail(POINTID_EINVAL, "scores must be 16-byte aligned");
  return classify_hits(h, t, hits, 3, n_hits, scores, stream);
}

int pointid_classify_planes_noalloc(pointid_handle h, const pointid_plane* planes, int32_t n_planes,
                                    const int32_t* hits, int64_t n_hits, float* scores,
                                    void* stream) {
  if (!h) return fail(POINTID_EINVAL, "handle is NULL");
  if (n_hits < 0) return fail(POINTID_EINVAL, "n_hits is negative");
  if (n_hits > kNoAllocMaxHits)
    return fail(POINTID_EINVAL, "n_hits " + std::to_string(n_hits) +
                                    " exceeds the no-alloc scratch, which holds at most " +
                                    std::to_string(kNoAllocMaxHits) + " hits");
  PlaneTable t;
  int rc = check_planes(planes, n_planes, &t);
  if (rc != POINTID_OK) return rc;
  if (n_hits == 0) return POINTID_OK;
  if (!hits || !scores) return fail(POINTID_EINVAL, "NULL device pointer");
  if (!aligned16(scores)) return fail(POINTID_EINVAL, "scores must be 16-byte aligned");
  DeviceScope dev(h->device);
  if (dev.error() != hipSuccess) return hip_fail(dev.error(), "hipSetDevice");
  void* base = nullptr;
  const hipError_t e = noalloc_scratch(h->device, &base);
  if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
  // every byte of scratch a call reads was written earlier in the same call
  // (patches by the gather, partials by the fused kernel), so nothing needs
  // clearing between calls
  Workspace ws(base, kNoAllocBytes);
  return classify_hits(h, t, hits, 3, n_hits, scores, stream, 1, &ws);
}

int pointid_classify_planes_ds(pointid_handle h, const pointid_plane* planes, int32_t n_planes,
                               int32_t ticks_per_column, const int32_t* hits, int64_t n_hits,
                               float* scores, void* stream_) {
  if (!h) return fail(POINTID_EINVAL, "handle is NULL");
  if (n_hits < 0) return fail(POINTID_EINVAL, "n_hits is negative");
  if (ticks_per_column < 1) return fail(POINTID_EINVAL, "ticks_per_column must be >= 1");
  PlaneTable t;
  int rc = check_planes(planes, n_planes, &t);
  if (rc != POINTID_OK) return rc;
  if (n_hits == 0) return POINTID_OK;
  if (!hits || !scores) return fail(POINTID_EINVAL, "NULL device pointer");
  if (!aligned16(scores)) return fail(POINTID_EINVAL, "scores must be 16-byte aligned");
  hipStream_t stream = static_cast<hipStream_t>(stream_);
  DeviceScope dev(h->device);
  if (dev.error() != hipSuccess) return hip_fail(dev.error(), "hipSetDevice");
  // the binned planes live in a scratch buffer of their own until the
  // classification below has been enqueued after the binning
  PlaneTable binned = t;
  size_t bytes = 0;
  for (int i = 0; i < t.n; ++i) {
    binned.p[i].n_ticks = (int32_t)(((int64_t)t.p[i].n_ticks + ticks_per_column - 1) / ticks_per_column);
    bytes += pad256(sizeof(float) * (size_t)t.p[i].n_wires * (size_t)binned.p[i].n_ticks);
  }
  Workspace ws(h->scratch, stream);
  hipError_t e = ws.reserve(bytes);
  if (e != hipSuccess) return hip_fail(e, "scratch buffer");
  for (int i = 0; i < t.n; ++i) {
    void* p = nullptr;
    e = ws.get(sizeof(float) * (size_t)t.p[i].n_wires * (size_t)binned.p[i].n_ticks, &p);
    if (e != hipSuccess) return hip_fail(e, "workspace (binned planes)");
    binned.p[i].image = static_cast<const float*>(p);
  }
  {
    KernelTimer kt("bin_ticks", stream);
    e = launch_bin_ticks(t, binned, ticks_per_column, stream);
  }
  if (e != hipSuccess) return hip_fail(e, "tick binning launch");
  return classify_hits(h, binned, hits, 3, n_hits, scores, stream, ticks_per_column);
}

int pointid_classify_requests(pointid_handle h, const pointid_plane* planes, int32_t n_planes,
                              const pointid_request* requests, int32_t n_requests,
                              void* stream_) {
  if (!h) return fail(POINTID_EINVAL, "handle is NULL");
  if (n_requests < 0) return fail(POINTID_EINVAL, "n_requests is negative");
  PlaneTable t;
  int rc = check_planes(planes, n_planes, &t);
  if (rc != POINTID_OK) return rc;
  if (n_requests == 0) return POINTID_OK;
  if (!requests) return fail(POINTID_EINVAL, "requests is NULL");
  int64_t total = 0;
  for (int32_t r = 0; r < n_requests; ++r) {
    const pointid_request& q = requests[r];
    const std::string at = "request " + std::to_string(r) + ": ";
    if (q.n_hits < 0) return fail(POINTID_EINVAL, at + "n_hits is negative");
    if (q.plane >= n_planes) return fail(POINTID_EINVAL, at + "plane index out of range");
    if (q.n_hits == 0) continue;
    if (!q.hits || !q.scores) return fail(POINTID_EINVAL, at + "NULL device pointer");
    if (!aligned16(q.scores)) return fail(POINTID_EINVAL, at + "scores must be 16-byte aligned");
    total += q.n_hits;
  }
  if (total == 0) return POINTID_OK;
  hipStream_t stream = static_cast<hipStream_t>(stream_);
  DeviceScope dev(h->device);
  if (dev.error() != hipSuccess) return hip_fail(dev.error(), "hipSetDevice");
  RequestTable tab;
  std::memset(&tab, 0, sizeof(tab));
  for (int32_t r = 0; r <= n_requests; ++r) {
    // flush a full table, and the last one
    if (r == n_requests || tab.n == kMaxRequests) {
      if (tab.n > 0) {
        rc = classify_request_batch(h, t, tab, stream);
        if (rc != POINTID_OK) return rc;
      }
      std::memset(&tab, 0, sizeof(tab));
      if (r == n_requests) break;
    }
    const pointid_request& q = requests[r];
    if (q.n_hits == 0) continue;
    tab.hits[tab.n] = q.hits;
    tab.scores[tab.n] = q.scores;
    tab.plane[tab.n] = q.plane < 0 ? -1 : q.plane;
    tab.start[tab.n + 1] = tab.start[tab.n] + q.n_hits;
    ++tab.n;
  }
  return POINTID_OK;
}

int pointid_classify_patches(pointid_handle h, const float* patches, int64_t n,
                             float* scores, void* stream_) {
  if (!h) return fail(POINTID_EINVAL, "handle is NULL");
  if (n < 0) return fail(POINTID_EINVAL, "n is negative");
  if (n == 0) return POINTID_OK;
  if (!patches || !scores) return fail(POINTID_EINVAL, "NULL device pointer");
  if (!aligned16(scores) || !aligned16(patches))
    return fail(POINTID_EINVAL, "patches and scores must be 16-byte aligned");
  hipStream_t stream = static_cast<hipStream_t>(stream_);
  DeviceScope dev(h->device);
  if (dev.error() != hipSuccess) return hip_fail(dev.error(), "hipSetDevice");
  // 16-bit handles: up to kInKernelCast patches the fused kernel rounds the
  // fp32 rows itself (one launch fewer, which is what a small batch pays for);
  // above, a separate cast writes 16-bit patches, whose rows the fused kernel
  // then reads at half the bytes
  const bool half = h->precision != POINTID_FP32;
  const bool cast = half && (n > kInKernelCast || h->precision == POINTID_FP8);
  Workspace ws(h->scratch, stream);
  hipError_t e = ws.reserve(scratch_bytes(h->precision, n, cast));
  if (e != hipSuccess) return hip_fail(e, "scratch buffer");
  if (!half) return run_network_fp32(h, patches, n, scores, stream, ws);
  if (!cast) return run_network_16(h, patches, true, n, scores, stream, ws);
  uint16_t* pb = nullptr;
  e = ws.get(2 * (size_t)n * kPatchPix, (void**)&pb);
  if (e != hipSuccess) return hip_fail(e, "workspace (16-bit patches)");
  {
    KernelTimer kt("patches_to_16", stream);
    e = launch_patches_to_16(patch_dtype(h->precision) == POINTID_FP16, patches, n, pb, stream);
  }
  if (e != hipSuccess) return hip_fail(e, "16-bit cast launch");
  return run_network_16(h, pb, false, n, scores, stream, ws);
}

int pointid_gather(const float* image, int32_t n_wires, int32_t n_ticks,
                   const int32_t* hits, int64_t n_hits, void* patches_out,
                   int out_dtype, void* stream) {
  if (n_hits < 0) return fail(POINTID_EINVAL, "n_hits is negative");
  if (n_wires <= 0 || n_ticks <= 0) return fail(POINTID_EINVAL, "n_wires and n_ticks must be positive");
  if (out_dtype != POINTID_FP32 && out_dtype != POINTID_BF16 && out_dtype != POINTID_FP16)
    return fail(POINTID_EUNSUPPORTED, "out_dtype must be POINTID_FP32, POINTID_BF16 or POINTID_FP16");
  if (n_hits == 0) return POINTID_OK;
  if (!image || !hits || !patches_out) return fail(POINTID_EINVAL, "NULL device pointer");
  if (!aligned16(patches_out)) return fail(POINTID_EINVAL, "patches_out must be 16-byte aligned");
  PlaneTable t;
  std::memset(&t, 0, sizeof(t));
  t.n = 1;
  t.p[0] = {image, n_wires, n_ticks};
  hipError_t e = launch_gather(t, hits, 2, n_hits, patches_out, out_dtype,
                               static_cast<hipStream_t>(stream));
  return e == hipSuccess ? POINTID_OK : hip_fail(e, "gather launch");
}

int pointid_gather_planes(const pointid_plane* planes, int32_t n_planes, const int32_t* hits,
                          int64_t n_hits, void* patches_out, int out_dtype, void* stream) {
  if (n_hits < 0) return fail(POINTID_EINVAL, "n_hits is negative");
  if (out_dtype != POINTID_FP32 && out_dtype != POINTID_BF16 && out_dtype != POINTID_FP16)
    return fail(POINTID_EUNSUPPORTED, "out_dtype must be POINTID_FP32, POINTID_BF16 or POINTID_FP16");
  PlaneTable t;
  int rc = check_planes(planes, n_planes, &t);
  if (rc != POINTID_OK) return rc;
  if (n_hits == 0) return POINTID_OK;
  if (!hits || !patches_out) return fail(POINTID_EINVAL, "NULL device pointer");
  if (!aligned16(patches_out)) return fail(POINTID_EINVAL, "patches_out must be 16-byte aligned");
  hipError_t e = launch_gather(t, hits, 3, n_hits, patches_out, out_dtype,
                               static_cast<hipStream_t>(stream));
  return e == hipSuccess ? POINTID_OK : hip_fail(e, "gather launch");
}


int pointid_downsample(const float* image, int32_t n_wires, int32_t n_ticks,
                       int32_t ticks_per_column, float* out, void* stream) {
  if (n_wires <= 0 || n_ticks <= 0) return fail(POINTID_EINVAL, "n_wires and n_ticks must be positive");
  if (ticks_per_column < 1) return fail(POINTID_EINVAL, "ticks_per_column must be >= 1");
  if (!image || !out) return fail(POINTID_EINVAL, "NULL device pointer");
  PlaneTable in, o;
  std::memset(&in, 0, sizeof(in));
  std::memset(&o, 0, sizeof(o));
  in.n = o.n = 1;
  in.p[0] = {image, n_wires, n_ticks};
  o.p[0] = {out, n_wires, (int32_t)(((int64_t)n_ticks + ticks_per_column - 1) / ticks_per_column)};
  hipError_t e = launch_bin_ticks(in, o, ticks_per_column, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? POINTID_OK : hip_fail(e, "tick binning launch");
}

int pointid_find_hits(pointid_handle h, const pointid_plane* planes, int32_t n_planes,
                      float threshold, int32_t* hits_out, int64_t capacity, int64_t* n_found,
                      void* stream_) {
  if (!h) return fail(POINTID_EINVAL, "handle is NULL");
  if (capacity < 0) return fail(POINTID_EINVAL, "capacity is negative");
  PlaneTable t;
  int rc = check_planes(planes, n_planes, &t);
  if (rc != POINTID_OK) return rc;
  if (!n_found) return fail(POINTID_EINVAL, "n_found is NULL");
  if ((reinterpret_cast<uintptr_t>(n_found) & 7) != 0)
    return fail(POINTID_EINVAL, "n_found must be 8-byte aligned");
  if (capacity > 0 && !hits_out) return fail(POINTID_EINVAL, "hits_out is NULL");
  HitSteps st;
  std::memset(&st, 0, sizeof(st));
  hit_steps(t, &st);
  hipStream_t stream = static_cast<hipStream_t>(stream_);
  DeviceScope dev(h->device);
  if (dev.error() != hipSuccess) return hip_fail(dev.error(), "hipSetDevice");
  const size_t mask_bytes = 4 * sizeof(uint64_t) * (size_t)st.step0[st.n];
  const size_t count_bytes = sizeof(int32_t) * (size_t)st.workers;
  const size_t off_bytes = sizeof(int64_t) * (size_t)st.workers;
  Workspace ws(h->scratch, stream);
  hipError_t e = ws.reserve(pad256(mask_bytes) + pad256(count_bytes) + pad256(off_bytes));
  if (e != hipSuccess) return hip_fail(e, "scratch buffer");
  uint64_t* mask = nullptr;
  int32_t* counts = nullptr;
  int64_t* offsets = nullptr;
  e = ws.get(mask_bytes, (void**)&mask);
  if (e == hipSuccess) e = ws.get(count_bytes, (void**)&counts);
  if (e == hipSuccess) e = ws.get(off_bytes, (void**)&offsets);
  if (e != hipSuccess) return hip_fail(e, "workspace (hit finding)");
  {
    KernelTimer kt("hits_mask", stream);
    e = launch_hits_mask(t, st, threshold, mask, counts, stream);
  }
  if (e != hipSuccess) return hip_fail(e, "hit mask launch");
  {
    KernelTimer kt("hits_scan", stream);
    e = launch_hits_scan(counts, st.workers, offsets, n_found, stream);
  }
  if (e != hipSuccess) return hip_fail(e, "hit scan launch");
  {
    KernelTimer kt("hits_emit", stream);
    e = launch_hits_emit(t, st, mask, counts, offsets, hits_out, capacity, stream);
  }
  if (e != hipSuccess) return hip_fail(e, "hit emit launch");
  return POINTID_OK;
}

}  // extern "C"
