// Patch construction (paper §2.1): for hit (w, t) the 48x48 patch
// P[r][c] = image[w - 24 + r][t - 24 + c], zero outside the plane.
//
// One wavefront builds one patch in two phases through LDS:
//   1. stage: the 48 rows of the window are read as 13 aligned 16-byte chunks
//      per row (52 floats covering the 48 needed plus the 0-3 float misalignment
//      of the window start), zero-filled wherever a pixel is outside the plane;
//   2. emit: each lane reads 4 (fp32) or 8 (bf16) consecutive pixels of a patch
//      row from LDS at the row's misalignment offset and writes one aligned
//      16-byte store, so a wavefront writes 1 KiB of contiguous output per
//      instruction.
// Values are copied, never computed (bf16 / fp16 output is the
// round-to-nearest-even of the fp32 pixel), so the result is bit-exact.
#include "pointid.h"
#include "internal.h"
#include "op16.h"

namespace pointid {
namespace {

constexpr int kWaves = 4;                 // patches per block (one per wave)
constexpr int kChunks = 13;               // 16-byte chunks staged per row
constexpr int kStageCols = kChunks * 4;   // 52 floats

__device__ __forceinline__ int64_t mod4(int64_t x) { return ((x % 4) + 4) % 4; }

template <int kOut>
__global__ __launch_bounds__(256) void gather_kernel(PlaneTable planes,
                                                     const int32_t* __restrict__ hits,
                                                     int hit_stride, int64_t n,
                                                     void* __restrict__ out) {
  __shared__ __attribute__((aligned(16))) float stage[kWaves][kPatch][kStageCols];
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int64_t i = (int64_t)blockIdx.x * kWaves + wave;
  const bool active = i < n;

  int plane = 0, w = 0, t = 0;
  if (active) {
    const int32_t* h = hits + i * hit_stride;
    if (hit_stride == 3) {
      plane = h[0];
      w = h[1];
      t = h[2];
    } else {
      w = h[0];
      t = h[1];
    }
  }
  // one patch per wave: make the hit wave-uniform so plane lookups are scalar
  plane = __builtin_amdgcn_readfirstlane(plane);
  w = __builtin_amdgcn_readfirstlane(w);
  t = __builtin_amdgcn_readfirstlane(t);
  const bool plane_ok = active && plane >= 0 && plane < planes.n;
  const float* img = nullptr;
  int W = 0, T = 1;
  if (plane_ok) {
    img = planes.p[plane].image;
    W = planes.p[plane].n_wires;
    T = planes.p[plane].n_ticks;
  }
  const bool base_aligned = (reinterpret_cast<uintptr_t>(img) & 15) == 0;

  float(*st)[kStageCols] = stage[wave];
  // ---- stage
  for (int k = lane; k < kPatch * kChunks; k += 64) {
    const int r = k / kChunks;
    const int j = k - r * kChunks;
    const int wire = w - kHalf + r;
    float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
    if (plane_ok && wire >= 0 && wire < W) {
      const int64_t flat0 = (int64_t)wire * T + (t - kHalf);
      const int64_t tick0 = (int64_t)(t - kHalf) - mod4(flat0) + 4 * j;
      const float* rowp = img + (int64_t)wire * T;
      if (base_aligned && tick0 >= 0 && tick0 + 3 < T) {
        v = *reinterpret_cast<const float4*>(rowp + tick0);
      } else {
        float e[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int64_t tk = tick0 + q;
          e[q] = (tk >= 0 && tk < T) ? rowp[tk] : 0.f;
        }
        v = make_float4(e[0], e[1], e[2], e[3]);
      }
    }
    *reinterpret_cast<float4*>(&st[r][4 * j]) = v;
  }
  __syncthreads();
  if (!active) return;

  // ---- emit
  if constexpr (kOut == POINTID_FP32) {
    float4* o = reinterpret_cast<float4*>(static_cast<float*>(out) + i * kPatchPix);
    for (int k = lane; k < kPatch * 12; k += 64) {
      const int r = k / 12;
      const int c = (k - r * 12) * 4;
      const int wire = w - kHalf + r;
      const int off = (plane_ok && wire >= 0 && wire < W)
                          ? (int)mod4((int64_t)wire * T + (t - kHalf)) : 0;
      const float* s = &st[r][off + c];
      o[k] = make_float4(s[0], s[1], s[2], s[3]);
    }
  } else {
    uint4* o = reinterpret_cast<uint4*>(static_cast<uint16_t*>(out) + i * kPatchPix);
    for (int k = lane; k < kPatch * 6; k += 64) {
      const int r = k / 6;
      const int c = (k - r * 6) * 8;
      const int wire = w - kHalf + r;
      const int off = (plane_ok && wire >= 0 && wire < W)
                          ? (int)mod4((int64_t)wire * T + (t - kHalf)) : 0;
      const float* s = &st[r][off + c];
      using Op = Op16<kOut == POINTID_FP16>;
      o[k] = make_uint4(Op::pack(s[0], s[1]), Op::pack(s[2], s[3]), Op::pack(s[4], s[5]),
                        Op::pack(s[6], s[7]));
    }
  }
}

// Elementwise fp32 -> 16-bit (RNE) for pre-cut patches: 8 values per thread.
template <bool kFp16>
__global__ __launch_bounds__(256) void to_16_kernel(const float4* __restrict__ in, int64_t n8,
                                                    uint4* __restrict__ out) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n8) return;
  const float4 a = in[2 * i], b = in[2 * i + 1];
  using Op = Op16<kFp16>;
  out[i] = make_uint4(Op::pack(a.x, a.y), Op::pack(a.z, a.w), Op::pack(b.x, b.y),
                      Op::pack(b.z, b.w));
}

}  // namespace

hipError_t launch_patches_to_16(bool fp16, const float* in, int64_t n, uint16_t* out,
                                hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  const int64_t n8 = n * kPatchPix / 8;
  const dim3 grid((unsigned)((n8 + 255) / 256));
  if (fp16)
    to_16_kernel<true><<<grid, dim3(256), 0, stream>>>(reinterpret_cast<const float4*>(in), n8,
                                                      reinterpret_cast<uint4*>(out));
  else
    to_16_kernel<false><<<grid, dim3(256), 0, stream>>>(reinterpret_cast<const float4*>(in), n8,
                                                       reinterpret_cast<uint4*>(out));
  return hipGetLastError();
}

hipError_t launch_gather(const PlaneTable& planes, const int32_t* hits,
                         int hit_stride, int64_t n, void* out, int out_dtype,
                         hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  const dim3 grid((unsigned)((n + kWaves - 1) / kWaves));
  if (out_dtype == POINTID_BF16)
    gather_kernel<POINTID_BF16><<<grid, dim3(256), 0, stream>>>(planes, hits, hit_stride, n, out);
  else if (out_dtype == POINTID_FP16)
    gather_kernel<POINTID_FP16><<<grid, dim3(256), 0, stream>>>(planes, hits, hit_stride, n, out);
  else
    gather_kernel<POINTID_FP32><<<grid, dim3(256), 0, stream>>>(planes, hits, hit_stride, n, out);
  return hipGetLastError();
}

}  // namespace pointid
