// fp32 conv and FC1 on the vector ALUs (paper §2.2), unfused: the conv writes
// the 44x44x48 maps of a chunk of patches to device memory (channels-last),
// then FC1 reads them back as a [n][92928] matrix.  Plain LDS-tiled kernels,
// exact fp32 arithmetic with fp32 accumulation.
#include "internal.h"

namespace pointid {
namespace {

// ---------------------------------------------------------------- conv
// One block per patch.  The patch and the 48x25 filters sit in LDS; each
// thread computes all 48 channels of one map position at a time from the 25
// taps held in registers, and writes them as 12 contiguous float4.
__global__ __launch_bounds__(256) void conv_fp32_kernel(const float* __restrict__ patches,
                                                        const float* __restrict__ conv_w,
                                                        const float* __restrict__ conv_b,
                                                        float* __restrict__ act) {
  __shared__ float P[kPatchPix];
  __shared__ float K[kCh * kK * kK];
  __shared__ float B[kCh];
  const int64_t pid = blockIdx.x;
  const float* src = patches + pid * kPatchPix;
  for (int i = threadIdx.x; i < kPatchPix; i += 256) P[i] = src[i];
  for (int i = threadIdx.x; i < kCh * kK * kK; i += 256) K[i] = conv_w[i];
  if (threadIdx.x < kCh) B[threadIdx.x] = conv_b[threadIdx.x];
  __syncthreads();
  float* dst = act + pid * (int64_t)kFc1In;
  for (int p = threadIdx.x; p < kPos; p += 256) {
    const int y = p / kFm, x = p - (p / kFm) * kFm;
    float tap[kK * kK];
#pragma unroll
    for (int u = 0; u < kK; ++u)
#pragma unroll
      for (int v = 0; v < kK; ++v) tap[u * kK + v] = P[(y + u) * kPatch + x + v];
    float4* o = reinterpret_cast<float4*>(dst + (int64_t)p * kCh);
#pragma unroll 1
    for (int k4 = 0; k4 < kCh / 4; ++k4) {
      float r[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int k = k4 * 4 + q;
        float s = B[k];
#pragma unroll
        for (int j = 0; j < kK * kK; ++j) s = fmaf(K[k * kK * kK + j], tap[j], s);
        r[q] = fmaxf(s, 0.f);
      }
      o[k4] = make_float4(r[0], r[1], r[2], r[3]);
    }
  }
}

// ---------------------------------------------------------------- FC1
// Tile: 64 rows x 128 outputs per block, K step 32, split-K over gridDim.y.
// Thread (ty, tx) owns rows ty*4..+3 and outputs tx*8..+7.
constexpr int kTM = 64;
constexpr int kTK = 32;

__global__ __launch_bounds__(256) void fc1_fp32_kernel(const float* __restrict__ act,
                                                       int64_t n,
                                                       const float* __restrict__ w1,
                                                       int64_t k_per_split,
                                                       float* __restrict__ part,
                                                       int64_t row0, int64_t n_total) {
  __shared__ float As[kTK][kTM + 4];
  __shared__ float Ws[kTK][kFc1Out];
  const int tid = threadIdx.x;
  const int ty = tid >> 4, tx = tid & 15;
  const int64_t m0 = (int64_t)blockIdx.x * kTM;
  const int s = blockIdx.y;
  const int64_t k0 = (int64_t)s * k_per_split;
  float acc[4][8];
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int b = 0; b < 8; ++b) acc[a][b] = 0.f;

  for (int64_t kk = 0; kk < k_per_split; kk += kTK) {
    // A tile 64 x 32: thread loads 8 values, k fastest (coalesced)
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int idx = tid + q * 256;
      const int r = idx >> 5, c = idx & 31;
      const int64_t m = m0 + r;
      As[c][r] = (m < n) ? act[m * kFc1In + k0 + kk + c] : 0.f;
    }
    // W tile 32 x 128
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      const int idx = tid + q * 256;
      const int r = idx >> 7, c = idx & 127;
      Ws[r][c] = w1[(k0 + kk + r) * kFc1Out + c];
    }
    __syncthreads();
#pragma unroll 4
    for (int k = 0; k < kTK; ++k) {
      float a[4], b[8];
#pragma unroll
      for (int q = 0; q < 4; ++q) a[q] = As[k][ty * 4 + q];
#pragma unroll
      for (int q = 0; q < 8; ++q) b[q] = Ws[k][tx * 8 + q];
#pragma unroll
      for (int p = 0; p < 4; ++p)
#pragma unroll
        for (int q = 0; q < 8; ++q) acc[p][q] = fmaf(a[p], b[q], acc[p][q]);
    }
    __syncthreads();
  }
  float* dst = part + ((int64_t)s * n_total + row0) * kFc1Out;
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    const int64_t m = m0 + ty * 4 + p;
    if (m < n) {
      float4* o = reinterpret_cast<float4*>(dst + m * kFc1Out + tx * 8);
      o[0] = make_float4(acc[p][0], acc[p][1], acc[p][2], acc[p][3]);
      o[1] = make_float4(acc[p][4], acc[p][5], acc[p][6], acc[p][7]);
    }
  }
}

}  // namespace

hipError_t launch_conv_fp32(const float* patches, int64_t n, const DeviceWeights& w,
                            float* act, hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  conv_fp32_kernel<<<dim3((unsigned)n), dim3(256), 0, stream>>>(patches, w.conv_w, w.conv_b, act);
  return hipGetLastError();
}

hipError_t launch_fc1_fp32(const float* act, int64_t n, int64_t row0, int64_t n_total,
                           const DeviceWeights& w, int splits, float* part,
                           hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  if (splits <= 0 || kFc1In % (splits * kTK) != 0) return hipErrorInvalidValue;
  const int64_t kps = kFc1In / splits;
  dim3 grid((unsigned)((n + kTM - 1) / kTM), (unsigned)splits);
  fc1_fp32_kernel<<<grid, dim3(256), 0, stream>>>(act, n, w.fc1_w, kps, part, row0, n_total);
  return hipGetLastError();
}

}  // namespace pointid
