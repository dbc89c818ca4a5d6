// Split-K reduction of FC1 and the rest of the network (paper §2.2):
// h1 = ReLU(b1 + sum of the FC1 partial sums [x 2^-k_n on 8-bit handles]), h2 = ReLU(b2 + h1 W2), then the
// softmax branch (3 outputs) and the sigmoid (Michel) branch (1 output), in fp32.
//
// A block of 256 threads handles 8 patches, one per group of 32 lanes.
//   1. Each thread owns one float4 column slice of one patch row; it issues the
//      loads of all 8 splits' partials at once (coalesced 512 B rows) and adds
//      them in ascending split order, adds b1, applies ReLU and stores h1 in LDS.
//   2. W2 (16 KB) is staged once per block through LDS into registers: lane j
//      of a group keeps column j and forms h2[j] from h1 broadcast out of LDS,
//      as two half sums (inputs 0-63, then 64-127) added in that order.  The
//      four head inputs are reduced across the 32 lanes by a fixed butterfly.
// 80 VGPRs, so 6 waves share a SIMD: 8-patch blocks keep more of the
// partials' loads in flight than 32-patch blocks with half the splits' loads
// at once (event, 50,000 patches: 42.3 against 47.5 us).
// Every patch is computed by the same instruction sequence whatever its
// position, so results do not depend on the batch or the hit order.
#include "internal.h"

namespace pointid {
namespace {

constexpr int kRows = 8;                    // patches per block, one per 32 lanes
constexpr int kSplitsInFlight = 8;          // splits whose loads are issued together
constexpr int kPitch = kFc1Out + 4;        // LDS row pitch (floats)
typedef float vec4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(1))) vec4 global_float4;

__device__ __forceinline__ float sum32(float v) {
#pragma unroll
  for (int m = 16; m >= 1; m >>= 1) v += __shfl_xor(v, m, 32);
  return v;
}

__device__ __forceinline__ void add4(float4& a, const float4& v) {
  a.x += v.x;
  a.y += v.y;
  a.z += v.z;
  a.w += v.w;
}

// Where patch p's 4 scores go: a score array [n][4] ...
struct PlainOut {
  float* scores;
  __device__ float* row(int64_t p) const { return scores + 4 * p; }
};
// ... or the output of the request holding it (a uniform scan of the table, so
// every table read is scalar).
struct RequestOut {
  RequestTable tab;
  __device__ float* row(int64_t p) const {
    float* d = tab.scores[0] + 4 * (p - tab.start[0]);
    for (int k = 1; k < tab.n; ++k)
      if (p >= tab.start[k]) d = tab.scores[k] + 4 * (p - tab.start[k]);
    return d;
  }
};

template <class Out>
__global__ __launch_bounds__(256) void tail_kernel(const float* __restrict__ part, int splits,
                                                   int64_t n, DeviceWeights w, Out out) {
  constexpr int kBlockRows = kRows;
  constexpr int kMaxSplits = kSplitsInFlight;
  __shared__ __attribute__((aligned(16))) float H[kBlockRows][kPitch];
  __shared__ __attribute__((aligned(16))) float W2s[kFc1Out * kFc2Out];
  // output rows, kept as global-address-space pointers so that the stores
  // are global (not flat) stores
  __shared__ global_float4* dst[kBlockRows];
  const int tid = threadIdx.x;
  const int64_t p0 = (int64_t)blockIdx.x * kBlockRows;
  if (tid < kBlockRows && p0 + tid < n) dst[tid] = reinterpret_cast<global_float4*>(reinterpret_cast<uintptr_t>(out.row(p0 + tid)));
  // W2 (16 KiB) into LDS: 4 float4 per thread, coalesced
  for (int i = tid; i < kFc1Out * kFc2Out / 4; i += 256)
    reinterpret_cast<float4*>(W2s)[i] = reinterpret_cast<const float4*>(w.fc2_w)[i];

  // ---- 1. fixed-order split-K reduction, + b1, ReLU
  {
    const int c4 = tid & 31;                 // float4 column
    const int r0 = tid >> 5;                 // rows r0, r0 + 8, ...
    float4 acc[kBlockRows / 8];
#pragma unroll
    for (int k = 0; k < kBlockRows / 8; ++k) acc[k] = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int s0 = 0; s0 < splits; s0 += kMaxSplits) {
      float4 v[kMaxSplits][kBlockRows / 8];
#pragma unroll
      for (int s = 0; s < kMaxSplits; ++s) {
        const float4* src =
            reinterpret_cast<const float4*>(part + ((int64_t)(s0 + s) * n + p0) * kFc1Out);
#pragma unroll
        for (int k = 0; k < kBlockRows / 8; ++k) {
          const int r = r0 + 8 * k;
          v[s][k] = (s0 + s < splits && p0 + r < n) ? src[r * (kFc1Out / 4) + c4]
                                                     : make_float4(0.f, 0.f, 0.f, 0.f);
        }
      }
#pragma unroll
      for (int s = 0; s < kMaxSplits; ++s)
#pragma unroll
        for (int k = 0; k < kBlockRows / 8; ++k) add4(acc[k], v[s][k]);
    }
    const float4 b = reinterpret_cast<const float4*>(w.fc1_b)[c4];
    if (w.fc1_scale) {                       // 8-bit handles: the sums times 2^-k_n (exact)
      const float4 sc = reinterpret_cast<const float4*>(w.fc1_scale)[c4];
#pragma unroll
      for (int k = 0; k < kBlockRows / 8; ++k)
        acc[k] = make_float4(acc[k].x * sc.x, acc[k].y * sc.y, acc[k].z * sc.z, acc[k].w * sc.w);
    }
#pragma unroll
    for (int k = 0; k < kBlockRows / 8; ++k) {
      const int r = r0 + 8 * k;
      *reinterpret_cast<float4*>(&H[r][4 * c4]) =
          make_float4(fmaxf(acc[k].x + b.x, 0.f), fmaxf(acc[k].y + b.y, 0.f),
                      fmaxf(acc[k].z + b.z, 0.f), fmaxf(acc[k].w + b.w, 0.f));
    }
  }
  __syncthreads();

  // ---- 2. FC2 + heads
  const int j = tid & 31;
  const float b2 = w.fc2_b[j];
  const float c0 = w.cls_w[j * 3 + 0], c1 = w.cls_w[j * 3 + 1], c2 = w.cls_w[j * 3 + 2];
  const float mw = w.mic_w[j];
  const float cb0 = w.cls_b[0], cb1 = w.cls_b[1], cb2 = w.cls_b[2], mb = w.mic_b[0];
  auto finish = [&](int r, float h, bool writer) {
    h = fmaxf(h + b2, 0.f);
    const float z0 = sum32(h * c0) + cb0;
    const float z1 = sum32(h * c1) + cb1;
    const float z2 = sum32(h * c2) + cb2;
    const float q = sum32(h * mw) + mb;
    if (writer) {
      const float zm = fmaxf(z0, fmaxf(z1, z2));
      const float e0 = expf(z0 - zm), e1 = expf(z1 - zm), e2 = expf(z2 - zm);
      const float inv = 1.f / (e0 + e1 + e2);
      const float eq = expf(-fabsf(q));
      const float sig = (q >= 0.f) ? 1.f / (1.f + eq) : eq / (1.f + eq);
      *dst[r] = (vec4){e0 * inv, e1 * inv, e2 * inv, sig};
    }
  };
  {
    // 8 groups of 32 lanes, lane j holding column j of W2
    const int grp = tid >> 5;
    float wc[kFc1Out];
#pragma unroll
    for (int i = 0; i < kFc1Out; ++i) wc[i] = W2s[i * kFc2Out + j];
    for (int r = grp; r < kBlockRows; r += 8) {
      if (p0 + r >= n) break;
      float h0 = 0.f, h1 = 0.f;
#pragma unroll
      for (int i = 0; i < kFc1Out / 2; ++i) h0 = fmaf(H[r][i], wc[i], h0);
#pragma unroll
      for (int i = kFc1Out / 2; i < kFc1Out; ++i) h1 = fmaf(H[r][i], wc[i], h1);
      finish(r, h0 + h1, j == 0);
    }
  }
}

}  // namespace

hipError_t launch_tail(const float* part, int splits, int64_t n, const DeviceWeights& w,
                       float* scores, hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  if (splits < 1) return hipErrorInvalidValue;
  return launch_kernel(tail_kernel<PlainOut>, dim3((unsigned)((n + kRows - 1) / kRows)), dim3(256), 0,
                       stream, part, splits, n, w, PlainOut{scores});
}

hipError_t launch_tail_requests(const float* part, int splits, const DeviceWeights& w,
                                const RequestTable& reqs, hipStream_t stream) {
  if (reqs.n < 1 || reqs.n > kMaxRequests) return hipErrorInvalidValue;
  const int64_t n = reqs.start[reqs.n];
  if (n <= 0) return hipSuccess;
  if (splits < 1) return hipErrorInvalidValue;
  return launch_kernel(tail_kernel<RequestOut>, dim3((unsigned)((n + kRows - 1) / kRows)), dim3(256), 0,
                       stream, part, splits, n, w, RequestOut{reqs});
}

}  // namespace pointid
