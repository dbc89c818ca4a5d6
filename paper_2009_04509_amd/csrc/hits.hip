// Hit finding on deconvolved plane images (paper §2.1: the reconstruction
// finds wire hits on the deconvolved waveforms before they are classified; the
// paper names no algorithm).  A tick t of a wire's waveform x is a hit when
//   x[t] > threshold,  x[t] > x[t-1]  and  x[t] >= x[t+1],
// where ticks outside the waveform count as minus infinity, so a plateau gives
// one hit at its first tick.  Comparisons are exact fp32 comparisons, so the
// result is bit-exact.  Hits come out as (plane, wire, tick) in plane, then
// wire, then tick order: the same order on every run, whatever the launch.
//
// The waveforms are cut into steps of 256 ticks (one wire each), numbered in
// output order, and every wave ("worker") owns one contiguous range of steps,
// so all workers have the same amount of image to read whatever the plane
// shapes.  Three launches, each a plain pass (no atomics, no waits between
// blocks):
//   mask   per step, 4 consecutive ticks per lane (one 16-byte load), the
//          neighbours from the adjacent lanes and, at the step's two ends,
//          one extra value; the step's hit bits are stored as 4 ballots
//          (32 B) and the worker's hit count at the end;
//   scan   one block: exclusive prefix sum of the worker counts -> each
//          worker's first output index, and the total;
//   emit   one block per worker with hits, its waves splitting the worker's
//          steps: each step's output index comes from a prefix sum of the
//          steps' hit counts across lanes; a hit is ranked within its step by
//          the set bits of the lanes below it, and the step's (plane, wire,
//          tick) rows are staged in LDS and stored as contiguous dwords.
// The image is read once (the bits are 1/32 of it), so the whole call is bound
// by HBM reads of the image.
#include "pointid.h"
#include "internal.h"

namespace pointid {
namespace {

constexpr int kMaskWaves = 4;             // workers per mask block
constexpr int kUnroll = 8;                // steps whose loads are in flight together
constexpr int kEmitWaves = 4;             // waves sharing one worker's steps in the emit

// Position of a step: plane p, wire `row`, step s along the wire, with plane
// p's sizes and the wire's first tick cached (reloaded only when the cursor
// enters the next plane).
struct Cursor {
  int p, row, s;
  int per_row, n_wires, T;
  const float* x;                                // tick 0 of wire `row`
};

__device__ __forceinline__ void enter_plane(const PlaneTable& planes, const HitSteps& st,
                                            Cursor& c) {
  c.per_row = st.per_row[c.p];
  c.n_wires = planes.p[c.p].n_wires;
  c.T = planes.p[c.p].n_ticks;
  c.x = planes.p[c.p].image + (int64_t)c.row * c.T;
}

__device__ __forceinline__ Cursor locate(const PlaneTable& planes, const HitSteps& st, int64_t g) {
  int p = 0, hi = st.n - 1;                      // last plane starting at or before g
  while (p < hi) {
    const int mid = (p + hi + 1) >> 1;
    if (st.step0[mid] <= g) p = mid;
    else hi = mid - 1;
  }
  const int64_t local = g - st.step0[p];
  const int64_t per_row = st.per_row[p];
  Cursor c;
  c.p = p;
  c.row = (int)(local / per_row);
  c.s = (int)(local - (int64_t)c.row * per_row);
  enter_plane(planes, st, c);
  return c;
}

__device__ __forceinline__ void advance(const PlaneTable& planes, const HitSteps& st, Cursor& c) {
  if (++c.s == c.per_row) {
    c.s = 0;
    c.x += c.T;
    if (++c.row == c.n_wires) {
      c.row = 0;
      if (++c.p < st.n) enter_plane(planes, st, c);
    }
  }
}

template <bool kVec>
__global__ __launch_bounds__(64 * kMaskWaves) void hits_mask_kernel(PlaneTable planes, HitSteps st,
                                                                    float thr,
                                                                    uint64_t* __restrict__ mask,
                                                                    int32_t* __restrict__ counts) {
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int64_t w = (int64_t)blockIdx.x * kMaskWaves + wave;
  if (w >= st.workers) return;                           // wave-uniform
  const float ninf = -__builtin_huge_valf();
  const int64_t total = st.step0[st.n];
  int64_t g = w * st.per;
  const int64_t end = g + st.per < total ? g + st.per : total;
  Cursor c = locate(planes, st, g);
  int32_t count = 0;
  for (; g < end; g += kUnroll) {
    float v[kUnroll][4], edge[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const bool live = g + u < end;                     // wave-uniform
      const int64_t T = c.T;
      const float* x = c.x;
      const int64_t t0 = (int64_t)c.s * kHitStep + 4 * lane;
      if constexpr (kVec) {
        if (live && t0 < T) {                             // T % 4 == 0: all 4 inside
          const float4 q = *reinterpret_cast<const float4*>(x + t0);
          v[u][0] = q.x;
          v[u][1] = q.y;
          v[u][2] = q.z;
          v[u][3] = q.w;
        } else {
          v[u][0] = v[u][1] = v[u][2] = v[u][3] = ninf;
        }
      } else {
#pragma unroll
        for (int j = 0; j < 4; ++j) v[u][j] = (live && t0 + j < T) ? x[t0 + j] : ninf;
      }
      // lane 0 needs the tick before the step, lane 63 the tick after it
      const int64_t te = lane == 0 ? (int64_t)c.s * kHitStep - 1 : ((int64_t)c.s + 1) * kHitStep;
      edge[u] = (live && (lane == 0 || lane == 63) && te >= 0 && te < T) ? x[te] : ninf;
      if (live) advance(planes, st, c);
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      if (g + u >= end) break;                           // wave-uniform
      float before = __shfl_up(v[u][3], 1);
      float after = __shfl_down(v[u][0], 1);
      if (lane == 0) before = edge[u];
      if (lane == 63) after = edge[u];
      const float* a = v[u];
      const uint64_t b0 = __ballot(a[0] > thr && a[0] > before && a[0] >= a[1]);
      const uint64_t b1 = __ballot(a[1] > thr && a[1] > a[0] && a[1] >= a[2]);
      const uint64_t b2 = __ballot(a[2] > thr && a[2] > a[1] && a[2] >= a[3]);
      const uint64_t b3 = __ballot(a[3] > thr && a[3] > a[2] && a[3] >= after);
      count += __popcll(b0) + __popcll(b1) + __popcll(b2) + __popcll(b3);
      if (lane < 4) mask[(g + u) * 4 + lane] = lane == 0 ? b0 : lane == 1 ? b1 : lane == 2 ? b2 : b3;
    }
  }
  if (lane == 0) counts[w] = count;
}

constexpr int kScanThreads = 1024;
constexpr int kScanPer = kHitMaxWorkers / kScanThreads;   // counts per thread

__global__ __launch_bounds__(kScanThreads) void hits_scan_kernel(const int32_t* __restrict__ counts,
                                                                 int32_t n,
                                                                 int64_t* __restrict__ offsets,
                                                                 int64_t* __restrict__ total) {
  __shared__ int64_t wsum[kScanThreads / 64];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int i0 = tid * kScanPer;
  int64_t v[kScanPer];
  int64_t s = 0;
#pragma unroll
  for (int k = 0; k < kScanPer; ++k) {
    v[k] = i0 + k < n ? counts[i0 + k] : 0;
    s += v[k];
  }
  int64_t x = s;                                          // inclusive scan over the wave
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const int64_t y = __shfl_up(x, d);
    if (lane >= d) x += y;
  }
  if (lane == 63) wsum[wave] = x;
  __syncthreads();
  if (wave == 0) {                                        // inclusive scan of the wave sums
    int64_t y = lane < kScanThreads / 64 ? wsum[lane] : 0;
#pragma unroll
    for (int d = 1; d < kScanThreads / 64; d <<= 1) {
      const int64_t z = __shfl_up(y, d);
      if (lane >= d) y += z;
    }
    if (lane < kScanThreads / 64) wsum[lane] = y;
  }
  __syncthreads();
  int64_t run = x - s + (wave > 0 ? wsum[wave - 1] : 0);
#pragma unroll
  for (int k = 0; k < kScanPer; ++k) {
    if (i0 + k < n) offsets[i0 + k] = run;
    run += v[k];
  }
  if (tid == 0) *total = wsum[kScanThreads / 64 - 1];
}

__device__ __forceinline__ uint64_t lane_word(uint64_t v, int l) {
  const uint32_t lo = __builtin_amdgcn_readlane((int)(uint32_t)v, l);
  const uint32_t hi = __builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), l);
  return ((uint64_t)hi << 32) | lo;
}

// Inclusive prefix sum over the 64 lanes.
__device__ __forceinline__ int wave_incl_scan(int x, int lane) {
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const int y = __shfl_up(x, d);
    if (lane >= d) x += y;
  }
  return x;
}

// Keeps the compiler from moving LDS accesses across this point.  A wave's
// LDS instructions execute in issue order, so a lane reading what another lane
// of the same wave wrote earlier needs no wait (the waves of an emit block
// never share LDS).
__device__ __forceinline__ void wave_lds_order() {
  __builtin_amdgcn_wave_barrier();
  asm volatile("" ::: "memory");
}

// One block per worker; its kEmitWaves waves split the worker's steps into
// consecutive ranges.  A wave takes its first output index from the worker's
// offset plus the hits of the worker's steps before its range, and each
// step's from a prefix sum of the steps' counts across lanes (64 steps per
// pass), so the steps do not wait on each other.
__global__ __launch_bounds__(64 * kEmitWaves) void hits_emit_kernel(PlaneTable planes, HitSteps st,
                                                                    const uint64_t* __restrict__ mask,
                                                                    const int32_t* __restrict__ counts,
                                                                    const int64_t* __restrict__ offsets,
                                                                    int32_t* __restrict__ hits,
                                                                    int64_t capacity) {
  __shared__ int32_t stage_all[kEmitWaves][3 * kHitStep];
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int64_t w = blockIdx.x;
  int32_t* stage = stage_all[wave];
  if (counts[w] == 0) return;
  int64_t base = offsets[w];
  if (base >= capacity) return;
  const int64_t total = st.step0[st.n];
  const int64_t g0 = w * st.per;
  const int64_t g1 = g0 + st.per < total ? g0 + st.per : total;
  const int64_t share = (g1 - g0 + kEmitWaves - 1) / kEmitWaves;
  const int64_t a = g0 + wave * share;
  const int64_t b = a + share < g1 ? a + share : g1;
  if (a >= b) return;                                    // wave-uniform
  const uint4* m4 = reinterpret_cast<const uint4*>(mask);   // 2 per step
  auto step_hits = [&](int64_t g, uint4& lo, uint4& hi) {
    lo = m4[2 * g];
    hi = m4[2 * g + 1];
    return __popc(lo.x) + __popc(lo.y) + __popc(lo.z) + __popc(lo.w) + __popc(hi.x) +
           __popc(hi.y) + __popc(hi.z) + __popc(hi.w);
  };
  for (int64_t c = g0; c < a; c += 64) {                 // hits of the steps before the range
    uint4 lo, hi;
    const int n = c + lane < a ? step_hits(c + lane, lo, hi) : 0;
    base += __builtin_amdgcn_readlane(wave_incl_scan(n, lane), 63);
  }
  Cursor cur = locate(planes, st, a);
  for (int64_t c = a; c < b && base < capacity; c += 64) {
    const int nst = (int)(b - c < 64 ? b - c : 64);
    uint4 lo = make_uint4(0, 0, 0, 0), hi = lo;
    const int n = lane < nst ? step_hits(c + lane, lo, hi) : 0;
    const int incl = wave_incl_scan(n, lane);
    const uint64_t mw[4] = {((uint64_t)lo.y << 32) | lo.x, ((uint64_t)lo.w << 32) | lo.z,
                            ((uint64_t)hi.y << 32) | hi.x, ((uint64_t)hi.w << 32) | hi.z};
    for (int k = 0; k < nst; ++k) {
      const int nk = __builtin_amdgcn_readlane(n, k);
      const int64_t bk = base + __builtin_amdgcn_readlane(incl, k) - nk;
      if (bk >= capacity) break;                         // wave-uniform
      if (nk > 0) {
        const uint64_t ws[4] = {lane_word(mw[0], k), lane_word(mw[1], k), lane_word(mw[2], k),
                                lane_word(mw[3], k)};
        // hits of the lanes below this one come first (their ticks are lower)
        uint32_t pos = 0;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          pos = __builtin_amdgcn_mbcnt_lo((uint32_t)ws[j], pos);
          pos = __builtin_amdgcn_mbcnt_hi((uint32_t)(ws[j] >> 32), pos);
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          if ((ws[j] >> lane) & 1) {
            stage[3 * pos] = cur.p;
            stage[3 * pos + 1] = cur.row;
            stage[3 * pos + 2] = cur.s * kHitStep + 4 * lane + j;
            ++pos;
          }
        }
        wave_lds_order();
        const int lim = 3 * (int)(nk < capacity - bk ? nk : capacity - bk);
        int32_t* o = hits + 3 * bk;
        for (int i = lane; i < lim; i += 256) {          // 4 LDS reads in flight
          int32_t v[4];
#pragma unroll
          for (int u = 0; u < 4; ++u) v[u] = i + 64 * u < lim ? stage[i + 64 * u] : 0;
#pragma unroll
          for (int u = 0; u < 4; ++u)
            if (i + 64 * u < lim) o[i + 64 * u] = v[u];
        }
        wave_lds_order();
      }
      advance(planes, st, cur);
    }
    base += __builtin_amdgcn_readlane(incl, nst - 1);
  }
}

}  // namespace

void hit_steps(const PlaneTable& planes, HitSteps* st) {
  st->n = planes.n;
  st->step0[0] = 0;
  for (int i = 0; i < planes.n; ++i) {
    st->per_row[i] = (int32_t)(((int64_t)planes.p[i].n_ticks + kHitStep - 1) / kHitStep);
    st->step0[i + 1] = st->step0[i] + (int64_t)planes.p[i].n_wires * st->per_row[i];
  }
  const int64_t total = st->step0[planes.n];
  st->per = (total + kHitMaxWorkers - 1) / kHitMaxWorkers;
  st->workers = (int32_t)((total + st->per - 1) / st->per);
}

hipError_t launch_hits_mask(const PlaneTable& planes, const HitSteps& st, float threshold,
                            uint64_t* mask, int32_t* counts, hipStream_t stream) {
  if (st.workers <= 0) return hipSuccess;
  bool vec = true;
  for (int i = 0; i < planes.n; ++i)
    vec = vec && (reinterpret_cast<uintptr_t>(planes.p[i].image) & 15) == 0 &&
          planes.p[i].n_ticks % 4 == 0;
  const dim3 grid((unsigned)((st.workers + kMaskWaves - 1) / kMaskWaves));
  if (vec)
    return launch_kernel(hits_mask_kernel<true>, grid, dim3(64 * kMaskWaves), 0, stream, planes, st,
                         threshold, mask, counts);
  return launch_kernel(hits_mask_kernel<false>, grid, dim3(64 * kMaskWaves), 0, stream, planes, st,
                       threshold, mask, counts);
}

hipError_t launch_hits_scan(const int32_t* counts, int32_t n, int64_t* offsets, int64_t* total,
                            hipStream_t stream) {
  if (n > kHitMaxWorkers) return hipErrorInvalidValue;
  return launch_kernel(hits_scan_kernel, dim3(1), dim3(kScanThreads), 0, stream, counts, n, offsets,
                       total);
}

hipError_t launch_hits_emit(const PlaneTable& planes, const HitSteps& st, const uint64_t* mask,
                            const int32_t* counts, const int64_t* offsets, int32_t* hits,
                            int64_t capacity, hipStream_t stream) {
  if (st.workers <= 0 || capacity <= 0) return hipSuccess;
  return launch_kernel(hits_emit_kernel, dim3((unsigned)st.workers), dim3(64 * kEmitWaves), 0, stream,
                       planes, st, mask, counts, offsets, hits, capacity);
}

}  // namespace pointid
