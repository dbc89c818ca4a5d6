// Split-K reduction of FC1 and the rest of the network (paper §2.2):
// h1 = ReLU(b1 + sum_s part[s]), h2 = ReLU(b2 + h1 W2), then the softmax
// branch (3 outputs) and the sigmoid (Michel) branch (1 output), in fp32.
//
// One wavefront handles 64 patches.  The partials are summed in ascending
// split order by the thread that owns each element, so the result does not
// depend on scheduling.  W2 and the head weights are broadcast from LDS; each
// lane then evaluates one patch.
#include "internal.h"

namespace pointid {
namespace {

constexpr int kRows = 64;

__global__ __launch_bounds__(64) void tail_kernel(const float* __restrict__ part, int splits,
                                                  int64_t n, DeviceWeights w,
                                                  float* __restrict__ scores) {
  __shared__ float H[kRows][kFc1Out + 1];
  __shared__ float W2[kFc1Out][kFc2Out];
  __shared__ float Hd[kFc2Out][4];     // cls_w (3) | mic_w
  __shared__ float B1[kFc1Out];
  __shared__ float B2[kFc2Out];
  const int tid = threadIdx.x;
  const int64_t p0 = (int64_t)blockIdx.x * kRows;
  const int rows = (int)((n - p0) < kRows ? (n - p0) : kRows);

  for (int i = tid; i < kFc1Out * kFc2Out; i += 64) W2[i / kFc2Out][i % kFc2Out] = w.fc2_w[i];
  for (int i = tid; i < kFc1Out; i += 64) B1[i] = w.fc1_b[i];
  if (tid < kFc2Out) {
    B2[tid] = w.fc2_b[tid];
    Hd[tid][0] = w.cls_w[tid * 3 + 0];
    Hd[tid][1] = w.cls_w[tid * 3 + 1];
    Hd[tid][2] = w.cls_w[tid * 3 + 2];
    Hd[tid][3] = w.mic_w[tid];
  }
  __syncthreads();

  // fixed-order split-K reduction (each element owned by one thread)
  for (int idx = tid; idx < rows * kFc1Out; idx += 64) {
    const int r = idx >> 7, c = idx & 127;
    const float* src = part + (p0 + r) * kFc1Out + c;
    float s = src[0];
    for (int q = 1; q < splits; ++q) s += src[(int64_t)q * n * kFc1Out];
    H[r][c] = fmaxf(s + B1[c], 0.f);
  }
  __syncthreads();
  if (tid >= rows) return;

  float h2[kFc2Out];
#pragma unroll
  for (int j = 0; j < kFc2Out; ++j) h2[j] = 0.f;
  for (int i = 0; i < kFc1Out; ++i) {
    const float hv = H[tid][i];
#pragma unroll
    for (int j = 0; j < kFc2Out; ++j) h2[j] = fmaf(hv, W2[i][j], h2[j]);
  }
  float z0 = w.cls_b[0], z1 = w.cls_b[1], z2 = w.cls_b[2], q = w.mic_b[0];
#pragma unroll
  for (int j = 0; j < kFc2Out; ++j) {
    const float v = fmaxf(h2[j] + B2[j], 0.f);
    z0 = fmaf(v, Hd[j][0], z0);
    z1 = fmaf(v, Hd[j][1], z1);
    z2 = fmaf(v, Hd[j][2], z2);
    q = fmaf(v, Hd[j][3], q);
  }
  const float zm = fmaxf(z0, fmaxf(z1, z2));
  const float e0 = expf(z0 - zm), e1 = expf(z1 - zm), e2 = expf(z2 - zm);
  const float inv = 1.f / (e0 + e1 + e2);
  const float eq = expf(-fabsf(q));
  const float sig = (q >= 0.f) ? 1.f / (1.f + eq) : eq / (1.f + eq);
  reinterpret_cast<float4*>(scores)[p0 + tid] = make_float4(e0 * inv, e1 * inv, e2 * inv, sig);
}

}  // namespace

hipError_t launch_tail(const float* part, int splits, int64_t n, const DeviceWeights& w,
                       float* scores, hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  const int64_t blocks = (n + kRows - 1) / kRows;
  tail_kernel<<<dim3((unsigned)blocks), dim3(64), 0, stream>>>(part, splits, n, w, scores);
  return hipGetLastError();
}

}  // namespace pointid
