// fp32 conv on the vector ALUs (paper §2.2), for the fp32 path: the conv
// writes the 44x44x48 maps of a chunk of patches to device memory
// (channels-last), and FC1 (fc1_f32.hip, fp32 MFMA) reads them back as a
// [n][92928] matrix.  Exact fp32 arithmetic.
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

}  // namespace

hipError_t launch_conv_fp32(const float* patches, int64_t n, const DeviceWeights& w,
                            float* act, hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  conv_fp32_kernel<<<dim3((unsigned)n), dim3(256), 0, stream>>>(patches, w.conv_w, w.conv_b, act);
  return hipGetLastError();
}

}  // namespace pointid
