// Hit finding on deconvolved plane images (paper §2.1: the reconstruction
// finds wire hits on the deconvolved waveforms before they are classified; the
// paper names no algorithm).  A tick t of a wire's waveform x is a hit when
//   x[t] > threshold,  x[t] > x[t-1]  and  x[t] >= x[t+1],
// where ticks outside the waveform count as minus infinity, so a plateau gives
// one hit at its first tick.  Comparisons are exact fp32 comparisons, so the
// result is bit-exact.  Hits come out as (plane, wire, tick) in plane, then
// wire, then tick order: the same order on every run, whatever the launch.
//
// Three launches, each a plain pass (no atomics, no waits between blocks):
//   mask   one wave per wire (row): reads the row once, 256 ticks per step
//          (4 consecutive ticks per lane, neighbours from the adjacent lanes
//          and, at a step's ends, one extra value), writes the step's hit bits
//          as 4 ballots (32 B) and the row's hit count;
//   scan   one block: exclusive prefix sum of the row counts in row order
//          -> each row's first output index, and the total;
//   emit   one wave per row with hits: expands the bits into (plane, wire,
//          tick) at the row's offset, each lane placing its hits by the count
//          of set bits of the lanes below it.
// The image is read once (the mask is 1/32 of its size), so the pass is bound
// by HBM reads of the image.
#include "pointid.h"
#include "internal.h"

namespace pointid {
namespace {

constexpr int kRowWaves = 4;              // rows per block (one wave each)
constexpr int kStep = 256;                // ticks per wave step
constexpr int kUnroll = 4;                // steps whose loads are in flight together

__device__ __forceinline__ int plane_of(const HitRows& rows, int64_t r) {
  int p = 0;                              // last plane starting at or before r (scalar)
  for (int q = 1; q < rows.n; ++q)
    if (rows.row0[q] <= r) p = q;
  return p;
}

__device__ __forceinline__ uint64_t ballot(bool b) { return __ballot(b); }

// Hits of one row of T ticks at x (kVec: x and T allow 16-byte loads).
template <bool kVec>
__device__ __forceinline__ void mask_row(const float* __restrict__ x, int64_t T, float thr,
                                         uint64_t* __restrict__ mask, int32_t* __restrict__ count_out,
                                         int lane) {
  const float ninf = -__builtin_huge_valf();
  const int64_t steps = (T + kStep - 1) / kStep;
  int32_t count = 0;
  for (int64_t s0 = 0; s0 < steps; s0 += kUnroll) {
    float v[kUnroll][4], edge[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int64_t t0 = (s0 + u) * kStep + 4 * lane;
      if constexpr (kVec) {
        if (t0 < T) {                       // T % 4 == 0: the 4 ticks are all inside
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
        for (int j = 0; j < 4; ++j) v[u][j] = (t0 + j < T) ? x[t0 + j] : ninf;
      }
      // lane 0 needs the tick before the step, lane 63 the tick after it
      const int64_t te = lane == 0 ? (s0 + u) * kStep - 1 : (s0 + u + 1) * kStep;
      edge[u] = ((lane == 0 || lane == 63) && te >= 0 && te < T) ? x[te] : ninf;
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      if (s0 + u >= steps) break;           // wave-uniform
      float before = __shfl_up(v[u][3], 1);
      float after = __shfl_down(v[u][0], 1);
      if (lane == 0) before = edge[u];
      if (lane == 63) after = edge[u];
      const float* a = v[u];
      const uint64_t b0 = ballot(a[0] > thr && a[0] > before && a[0] >= a[1]);
      const uint64_t b1 = ballot(a[1] > thr && a[1] > a[0] && a[1] >= a[2]);
      const uint64_t b2 = ballot(a[2] > thr && a[2] > a[1] && a[2] >= a[3]);
      const uint64_t b3 = ballot(a[3] > thr && a[3] > a[2] && a[3] >= after);
      count += __popcll(b0) + __popcll(b1) + __popcll(b2) + __popcll(b3);
      if (lane < 4) {
        const uint64_t w = lane == 0 ? b0 : lane == 1 ? b1 : lane == 2 ? b2 : b3;
        mask[(s0 + u) * 4 + lane] = w;
      }
    }
  }
  if (lane == 0) *count_out = count;
}

__global__ __launch_bounds__(256) void hits_mask_kernel(PlaneTable planes, HitRows rows, float thr,
                                                        uint64_t* __restrict__ mask,
                                                        int64_t mask_stride,
                                                        int32_t* __restrict__ counts) {
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int64_t r = (int64_t)blockIdx.x * kRowWaves + wave;
  if (r >= rows.row0[rows.n]) return;                    // wave-uniform
  const int p = plane_of(rows, r);
  const PlaneDesc d = planes.p[p];
  const int64_t T = d.n_ticks;
  const float* x = d.image + (r - rows.row0[p]) * T;
  uint64_t* m = mask + r * mask_stride;
  const bool vec = ((reinterpret_cast<uintptr_t>(d.image) & 15) == 0) && (T % 4 == 0);
  if (vec)
    mask_row<true>(x, T, thr, m, counts + r, lane);
  else
    mask_row<false>(x, T, thr, m, counts + r, lane);
}

constexpr int kScanThreads = 1024;

__global__ __launch_bounds__(kScanThreads) void hits_scan_kernel(const int32_t* __restrict__ counts,
                                                                 int64_t n_rows,
                                                                 int64_t* __restrict__ offsets,
                                                                 int64_t* __restrict__ total) {
  __shared__ int64_t part[kScanThreads];
  const int tid = threadIdx.x;
  const int64_t per = (n_rows + kScanThreads - 1) / kScanThreads;
  const int64_t lo = tid * per < n_rows ? tid * per : n_rows;
  const int64_t hi = lo + per < n_rows ? lo + per : n_rows;
  int64_t s = 0;
  for (int64_t r = lo; r < hi; ++r) s += counts[r];
  part[tid] = s;
  __syncthreads();
  for (int d = 1; d < kScanThreads; d <<= 1) {           // inclusive scan of the partials
    const int64_t add = tid >= d ? part[tid - d] : 0;
    __syncthreads();
    part[tid] += add;
    __syncthreads();
  }
  int64_t run = part[tid] - s;
  for (int64_t r = lo; r < hi; ++r) {
    offsets[r] = run;
    run += counts[r];
  }
  if (tid == kScanThreads - 1) *total = part[tid];
}

__global__ __launch_bounds__(256) void hits_emit_kernel(HitRows rows,
                                                        const uint64_t* __restrict__ mask,
                                                        int64_t mask_stride,
                                                        const int32_t* __restrict__ counts,
                                                        const int64_t* __restrict__ offsets,
                                                        int32_t* __restrict__ hits,
                                                        int64_t capacity) {
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int64_t r = (int64_t)blockIdx.x * kRowWaves + wave;
  if (r >= rows.row0[rows.n]) return;                    // wave-uniform
  if (counts[r] == 0) return;
  int64_t base = offsets[r];
  if (base >= capacity) return;
  const int p = plane_of(rows, r);
  const int32_t wire = (int32_t)(r - rows.row0[p]);
  const int64_t steps = ((int64_t)rows.n_ticks[p] + kStep - 1) / kStep;
  const uint64_t* m = mask + r * mask_stride;
  for (int64_t s = 0; s < steps && base < capacity; ++s) {
    const uint64_t w0 = m[4 * s], w1 = m[4 * s + 1], w2 = m[4 * s + 2], w3 = m[4 * s + 3];
    const int64_t n = __popcll(w0) + __popcll(w1) + __popcll(w2) + __popcll(w3);
    if (n == 0) continue;
    // hits of the lanes below this one come first (their ticks are lower)
    uint32_t below = 0;
    below = __builtin_amdgcn_mbcnt_lo((uint32_t)w0, below);
    below = __builtin_amdgcn_mbcnt_hi((uint32_t)(w0 >> 32), below);
    below = __builtin_amdgcn_mbcnt_lo((uint32_t)w1, below);
    below = __builtin_amdgcn_mbcnt_hi((uint32_t)(w1 >> 32), below);
    below = __builtin_amdgcn_mbcnt_lo((uint32_t)w2, below);
    below = __builtin_amdgcn_mbcnt_hi((uint32_t)(w2 >> 32), below);
    below = __builtin_amdgcn_mbcnt_lo((uint32_t)w3, below);
    below = __builtin_amdgcn_mbcnt_hi((uint32_t)(w3 >> 32), below);
    int64_t idx = base + below;
    const uint64_t ws[4] = {w0, w1, w2, w3};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      if ((ws[j] >> lane) & 1) {
        if (idx < capacity) {
          int32_t* o = hits + 3 * idx;
          o[0] = p;
          o[1] = wire;
          o[2] = (int32_t)(s * kStep + 4 * lane + j);
        }
        ++idx;
      }
    }
    base += n;
  }
}

}  // namespace

int64_t hits_mask_stride(const PlaneTable& planes) {
  int64_t steps = 0;
  for (int i = 0; i < planes.n; ++i) {
    const int64_t s = ((int64_t)planes.p[i].n_ticks + kStep - 1) / kStep;
    if (s > steps) steps = s;
  }
  return 4 * steps;
}

void hit_rows(const PlaneTable& planes, HitRows* rows) {
  rows->n = planes.n;
  rows->row0[0] = 0;
  for (int i = 0; i < planes.n; ++i) {
    rows->row0[i + 1] = rows->row0[i] + planes.p[i].n_wires;
    rows->n_ticks[i] = planes.p[i].n_ticks;
  }
}

hipError_t launch_hits_mask(const PlaneTable& planes, const HitRows& rows, float threshold,
                            uint64_t* mask, int64_t mask_stride, int32_t* counts,
                            hipStream_t stream) {
  const int64_t n = rows.row0[rows.n];
  if (n <= 0) return hipSuccess;
  const dim3 grid((unsigned)((n + kRowWaves - 1) / kRowWaves));
  hits_mask_kernel<<<grid, dim3(64 * kRowWaves), 0, stream>>>(planes, rows, threshold, mask,
                                                               mask_stride, counts);
  return hipGetLastError();
}

hipError_t launch_hits_scan(const int32_t* counts, int64_t n_rows, int64_t* offsets,
                            int64_t* total, hipStream_t stream) {
  hits_scan_kernel<<<dim3(1), dim3(kScanThreads), 0, stream>>>(counts, n_rows, offsets, total);
  return hipGetLastError();
}

hipError_t launch_hits_emit(const HitRows& rows, const uint64_t* mask, int64_t mask_stride,
                            const int32_t* counts, const int64_t* offsets, int32_t* hits,
                            int64_t capacity, hipStream_t stream) {
  const int64_t n = rows.row0[rows.n];
  if (n <= 0 || capacity <= 0) return hipSuccess;
  const dim3 grid((unsigned)((n + kRowWaves - 1) / kRowWaves));
  hits_emit_kernel<<<grid, dim3(64 * kRowWaves), 0, stream>>>(rows, mask, mask_stride, counts,
                                                               offsets, hits, capacity);
  return hipGetLastError();
}

}  // namespace pointid
