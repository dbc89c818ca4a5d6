// Dynamic batching of classification requests (paper §2.3: the inference
// server combines requests from many clients into larger batches; §3.2
// measures the gain) over one handle and one set of resident planes.
//
// Host threads submit requests and later wait for them.  A submit records an
// event on the submitter's stream; a launcher thread takes the pending
// requests in arrival order, makes the batcher's own stream wait for each
// one's event (so the work the submitter enqueued before it -- the hits'
// producer, the scores buffer's previous user -- comes first), and issues them
// as one pointid_classify_requests call on that stream when max_requests are
// pending or the oldest has waited max_delay_us; up to kMaxInFlight batches
// run at once.  A completion thread waits for each batch's event in
// launch order and wakes the requests' waiters.  Every request gets the scores
// (bit for bit) it would get alone: batching only changes which launch
// classifies it.
#include <chrono>
#include <condition_variable>
#include <deque>
#include <mutex>
#include <new>
#include <string>
#include <system_error>
#include <thread>
#include <vector>

#include "internal.h"
#include "pointid.h"

namespace {

constexpr size_t kMaxInFlight = 4;
using Clock = std::chrono::steady_clock;

struct Pending {
  pointid_request req;
  uint64_t ticket;
  Clock::time_point arrived;
  hipEvent_t ready;     // recorded on the submitter's stream at submit
};

struct Flight {
  hipEvent_t done;      // recorded after the batch's kernels (if launched)
  uint64_t first, last; // tickets of the batch
  int status;           // launch status
  std::string msg;
};

struct Failure {
  uint64_t first, last;
  int status;
  std::string msg;
};

}  // namespace

struct pointid_batcher_s {
  pointid_handle h = nullptr;
  int device = 0;
  std::vector<pointid_plane> planes;
  int max_requests = 1;
  std::chrono::microseconds max_delay{0};
  hipStream_t stream = nullptr;
  std::vector<hipEvent_t> free_events;
  std::vector<hipEvent_t> free_ready;  // submit events no pending request holds

  std::mutex mu;
  std::condition_variable cv_work;   // launcher: new requests, or stop
  std::condition_variable cv_flight; // launcher: room in flight; completer: a new batch
  std::condition_variable cv_done;   // waiters
  std::deque<Pending> pending;
  std::deque<Flight> flight;
  std::vector<Failure> failures;
  uint64_t next_ticket = 1;
  uint64_t done_upto = 0;            // every ticket <= done_upto is finished
  bool stop = false;
  bool launcher_done = false;
  std::thread launcher, completer;

  void launch_loop();
  void complete_loop();
};

void pointid_batcher_s::launch_loop() {
  (void)hipSetDevice(device);
  std::unique_lock<std::mutex> lk(mu);
  for (;;) {
    cv_work.wait(lk, [&] { return stop || !pending.empty(); });
    if (pending.empty()) break;                         // stop, nothing left
    // fill the batch until it is full or its oldest request is due
    const Clock::time_point due = pending.front().arrived + max_delay;
    while (!stop && (int)pending.size() < max_requests && Clock::now() < due)
      cv_work.wait_until(lk, due);
    cv_flight.wait(lk, [&] { return flight.size() < kMaxInFlight; });
    std::vector<pointid_request> batch;
    std::vector<hipEvent_t> ready;
    const uint64_t first = pending.front().ticket;
    uint64_t last = first;
    while (!pending.empty() && (int)batch.size() < max_requests) {
      batch.push_back(pending.front().req);
      ready.push_back(pending.front().ready);
      last = pending.front().ticket;
      pending.pop_front();
    }
    hipEvent_t ev = free_events.back();
    free_events.pop_back();
    lk.unlock();
    Flight f{ev, first, last, POINTID_OK, {}};
    // the batch starts after what each submitter enqueued before its submit;
    // a wait takes the event's state when it is enqueued, so the event can be
    // recorded again at once
    for (hipEvent_t r : ready) {
      const hipError_t e = hipStreamWaitEvent(stream, r, 0);
      if (e != hipSuccess && f.status == POINTID_OK) {
        f.status = POINTID_EHIP;
        f.msg = std::string("batch wait for a submitter's stream: ") + hipGetErrorString(e);
      }
    }
    if (f.status == POINTID_OK)
      f.status = pointid_classify_requests(h, planes.data(), (int32_t)planes.size(), batch.data(),
                                           (int32_t)batch.size(), stream);
    if (f.status == POINTID_OK) {
      const hipError_t e = hipEventRecord(ev, stream);
      if (e != hipSuccess) {
        f.status = POINTID_EHIP;
        f.msg = std::string("batch event: ") + hipGetErrorString(e);
      }
    } else if (f.msg.empty()) {
      f.msg = pointid_last_error();
    }
    lk.lock();
    for (hipEvent_t r : ready) free_ready.push_back(r);
    flight.push_back(std::move(f));
    cv_flight.notify_all();
  }
  launcher_done = true;
  cv_flight.notify_all();
}

void pointid_batcher_s::complete_loop() {
  (void)hipSetDevice(device);
  std::unique_lock<std::mutex> lk(mu);
  for (;;) {
    cv_flight.wait(lk, [&] { return !flight.empty() || launcher_done; });
    if (flight.empty()) break;                          // launcher finished, all drained
    Flight f = flight.front();
    lk.unlock();
    int status = f.status;
    std::string msg = f.msg;
    if (status == POINTID_OK) {
      const hipError_t e = hipEventSynchronize(f.done);
      if (e != hipSuccess) {
        status = POINTID_EHIP;
        msg = std::string("batch: ") + hipGetErrorString(e);
      }
    }
    lk.lock();
    flight.pop_front();
    free_events.push_back(f.done);
    if (status != POINTID_OK) failures.push_back({f.first, f.last, status, msg});
    done_upto = f.last;
    cv_done.notify_all();
    cv_flight.notify_all();
  }
}

extern "C" {

int pointid_batcher_create(pointid_handle h, const pointid_plane* planes, int32_t n_planes,
                           int32_t max_requests, int32_t max_delay_us, pointid_batcher* out) {
  using namespace pointid;
  if (!out) return set_error(POINTID_EINVAL, "out is NULL");
  *out = nullptr;
  if (!h) return set_error(POINTID_EINVAL, "handle is NULL");
  if (!planes) return set_error(POINTID_EINVAL, "planes is NULL");
  if (n_planes < 1 || n_planes > kMaxPlanes)
    return set_error(POINTID_EINVAL, "n_planes must be in [1, 64]");
  for (int32_t i = 0; i < n_planes; ++i)
    if (!planes[i].image || planes[i].n_wires <= 0 || planes[i].n_ticks <= 0)
      return set_error(POINTID_EINVAL, "plane " + std::to_string(i) + " is invalid");
  if (max_requests < 1 || max_requests > 4096)
    return set_error(POINTID_EINVAL, "max_requests must be in [1, 4096]");
  if (max_delay_us < 0) return set_error(POINTID_EINVAL, "max_delay_us is negative");
  auto* b = new (std::nothrow) pointid_batcher_s;
  if (!b) return set_error(POINTID_ENOMEM, "host allocation failed");
  b->h = h;
  b->device = handle_device(h);
  b->planes.assign(planes, planes + n_planes);
  b->max_requests = max_requests;
  b->max_delay = std::chrono::microseconds(max_delay_us);
  int prev = 0;
  hipError_t e = hipGetDevice(&prev);
  if (e == hipSuccess) e = hipSetDevice(b->device);
  if (e == hipSuccess) e = hipStreamCreateWithFlags(&b->stream, hipStreamNonBlocking);
  for (size_t i = 0; e == hipSuccess && i < kMaxInFlight; ++i) {
    hipEvent_t ev = nullptr;
    e = hipEventCreateWithFlags(&ev, hipEventDisableTiming);
    if (e == hipSuccess) b->free_events.push_back(ev);
  }
  (void)hipSetDevice(prev);
  if (e != hipSuccess) {
    for (hipEvent_t ev : b->free_events) (void)hipEventDestroy(ev);
    if (b->stream) (void)hipStreamDestroy(b->stream);
    delete b;
    return set_error(POINTID_EHIP, std::string("batcher stream/events: ") + hipGetErrorString(e));
  }
  try {
    b->launcher = std::thread([b] { b->launch_loop(); });
    b->completer = std::thread([b] { b->complete_loop(); });
  } catch (const std::system_error& x) {
    // the launcher ends at once on stop with nothing pending
    if (b->launcher.joinable()) {
      {
        std::lock_guard<std::mutex> lk(b->mu);
        b->stop = true;
      }
      b->cv_work.notify_all();
      b->launcher.join();
    }
    for (hipEvent_t ev : b->free_events) (void)hipEventDestroy(ev);
    (void)hipStreamDestroy(b->stream);
    delete b;
    return set_error(POINTID_ENOMEM, std::string("batcher threads: ") + x.what());
  }
  *out = b;
  return POINTID_OK;
}

int pointid_batcher_destroy(pointid_batcher b) {
  if (!b) return POINTID_OK;
  {
    std::lock_guard<std::mutex> lk(b->mu);
    b->stop = true;
  }
  b->cv_work.notify_all();
  b->launcher.join();
  b->completer.join();
  for (hipEvent_t ev : b->free_events) (void)hipEventDestroy(ev);
  for (hipEvent_t ev : b->free_ready) (void)hipEventDestroy(ev);   // every request was launched
  (void)hipStreamDestroy(b->stream);
  delete b;
  return POINTID_OK;
}

int pointid_batcher_submit(pointid_batcher b, const pointid_request* req, void* stream,
                           uint64_t* ticket) {
  using namespace pointid;
  if (!b || !req || !ticket) return set_error(POINTID_EINVAL, "NULL batcher, request or ticket");
  if (req->n_hits < 0) return set_error(POINTID_EINVAL, "n_hits is negative");
  if (req->plane >= (int32_t)b->planes.size())
    return set_error(POINTID_EINVAL, "plane index out of range");
  if (req->n_hits > 0) {
    if (!req->hits || !req->scores) return set_error(POINTID_EINVAL, "NULL device pointer");
    if (reinterpret_cast<uintptr_t>(req->scores) & 15)
      return set_error(POINTID_EINVAL, "scores must be 16-byte aligned");
  }
  // an event marking the submitter's stream here: taken from the pool, or new
  hipEvent_t ready = nullptr;
  {
    std::lock_guard<std::mutex> lk(b->mu);
    if (b->stop) return set_error(POINTID_EINVAL, "batcher is being destroyed");
    if (!b->free_ready.empty()) {
      ready = b->free_ready.back();
      b->free_ready.pop_back();
    }
  }
  hipError_t e = hipSuccess;
  if (!ready) {
    int prev = 0;
    e = hipGetDevice(&prev);
    if (e == hipSuccess && prev != b->device) e = hipSetDevice(b->device);
    if (e == hipSuccess) e = hipEventCreateWithFlags(&ready, hipEventDisableTiming);
    if (prev != b->device) (void)hipSetDevice(prev);
  }
  if (e == hipSuccess) e = hipEventRecord(ready, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) {
    if (ready) {
      std::lock_guard<std::mutex> lk(b->mu);
      b->free_ready.push_back(ready);
    }
    return set_error(POINTID_EHIP, std::string("submit event: ") + hipGetErrorString(e));
  }
  {
    std::lock_guard<std::mutex> lk(b->mu);
    if (b->stop) {
      b->free_ready.push_back(ready);
      return set_error(POINTID_EINVAL, "batcher is being destroyed");
    }
    try {
      b->pending.push_back({*req, b->next_ticket, Clock::now(), ready});
    } catch (const std::bad_alloc&) {
      b->free_ready.push_back(ready);
      return set_error(POINTID_ENOMEM, "host allocation failed");
    }
    *ticket = b->next_ticket++;
  }
  b->cv_work.notify_one();
  return POINTID_OK;
}

int pointid_batcher_wait(pointid_batcher b, uint64_t ticket) {
  using namespace pointid;
  if (!b) return set_error(POINTID_EINVAL, "batcher is NULL");
  std::unique_lock<std::mutex> lk(b->mu);
  if (ticket == 0 || ticket >= b->next_ticket)
    return set_error(POINTID_EINVAL, "unknown ticket");
  b->cv_done.wait(lk, [&] { return b->done_upto >= ticket; });
  for (const Failure& f : b->failures)
    if (ticket >= f.first && ticket <= f.last) return set_error(f.status, f.msg);
  return POINTID_OK;
}

}  // extern "C"
