// Repacking of the fp32 conv and FC1 weights into the 16-bit and 8-bit MFMA
// operand fragments read by the fused conv/FC1 kernels (layouts documented
// there), run once per handle at create time.  Rounding uses the same hardware RNE
// conversion as the kernel's activations.
#include "internal.h"
#include "op16.h"

namespace pointid {
namespace {

// conv tiles (shift, channel tile) feeding K=32 step q: slots 0-3 from the
// first, 4-7 from the second
__constant__ int kStepTiles[3][2][2] = {{{0, 0}, {0, 1}}, {{0, 2}, {1, 0}}, {{1, 1}, {1, 2}}};

// One thread per (fragment, lane): fragment f = (pair P, step q, output tile m).
template <bool kFp16>
__global__ __launch_bounds__(256) void pack_fc1_kernel(const float* __restrict__ w1,
                                                       uint4* __restrict__ out) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= kFc1Frags) return;
  const int lane = (int)(idx & 63);
  const int64_t f = idx >> 6;
  const int m = (int)(f % 8);
  const int q = (int)((f / 8) % 3);
  const int64_t P = f / 24;
  const int n = 16 * m + (lane & 15), g = lane >> 4;
  float v[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int s = kStepTiles[q][j >> 2][0], t = kStepTiles[q][j >> 2][1];
    const int64_t k = (2 * P + s) * kCh + 16 * t + 4 * g + (j & 3);
    v[j] = w1[k * kFc1Out + n];
  }
  using Op = Op16<kFp16>;
  out[idx] = make_uint4(Op::pack(v[0], v[1]), Op::pack(v[2], v[3]), Op::pack(v[4], v[5]),
                        Op::pack(v[6], v[7]));
}

// One thread per (shift s, channel tile t, lane): lane = (channel 16t + lane%16,
// slot group g); slot f = 8g + j < 30 is window pixel (f/6, f%6) and holds
// K[ch][f/6][f%6 - s] when that tap exists; slots 30 and 31 hold the bias
// split into a rounded high part and the rounded remainder.
template <bool kFp16>
__global__ __launch_bounds__(64) void pack_conv_kernel(const float* __restrict__ K,
                                                       const float* __restrict__ b,
                                                       uint4* __restrict__ out) {
  const int st = blockIdx.x;                 // s * 3 + t
  const int s = st / 3, t = st % 3;
  const int lane = threadIdx.x;
  const int ch = 16 * t + (lane & 15), g = lane >> 4;
  using Op = Op16<kFp16>;
  const uint32_t hi2 = Op::pack(b[ch], 0.f);
  const float hi = Op::value((uint16_t)(hi2 & 0xFFFFu));
  float v[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int f = 8 * g + j;
    if (f < 30) {
      const int u = f / 6, vv = f % 6 - s;
      v[j] = (vv >= 0 && vv < kK) ? K[ch * kK * kK + u * kK + vv] : 0.f;
    } else {
      v[j] = (f == 30) ? b[ch] : b[ch] - hi;
    }
  }
  out[st * 64 + lane] = make_uint4(Op::pack(v[0], v[1]), Op::pack(v[2], v[3]),
                                   Op::pack(v[4], v[5]), Op::pack(v[6], v[7]));
}

// One thread per (fragment, lane) of the 8-bit FC1 weights: fragment
// f = (pair P, output tile m), 1536 bytes: lane (r, g) holds, in dword d < 6,
// the inputs of conv tile (shift d / 3, channel tile d % 3) of pair P —
// byte e is input (2P + d / 3) * 48 + 16 (d % 3) + 4g + e of output 16m + r —
// dwords 0-3 at byte 16 lane, dwords 4-5 at byte 1024 + 8 lane.  Each weight
// is multiplied by 2^exp2[n] (exact) and rounded to e4m3 (nearest even; the
// exponent keeps every product within 448, the clamp only restates it).
__global__ __launch_bounds__(256) void pack_fc1_8_kernel(const float* __restrict__ w1,
                                                         const int* __restrict__ exp2,
                                                         uint8_t* __restrict__ out) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (int64_t)(kPos / 2) * 8 * 64) return;
  const int lane = (int)(idx & 63);
  const int64_t f = idx >> 6;
  const int m = (int)(f % 8);
  const int64_t P = f / 8;
  const int n = 16 * m + (lane & 15), g = lane >> 4;
  const int k = exp2[n];
  uint32_t d[6];
#pragma unroll
  for (int j = 0; j < 6; ++j) {
    const int s = j / 3, t = j % 3;
    const int64_t base = (2 * P + s) * kCh + 16 * t + 4 * g;
    float v[4];
#pragma unroll
    for (int e = 0; e < 4; ++e)
      v[e] = __builtin_amdgcn_fmed3f(ldexpf(w1[(base + e) * kFc1Out + n], k), -448.f, 448.f);
    const int lo = __builtin_amdgcn_cvt_pk_fp8_f32(v[0], v[1], 0, false);
    d[j] = (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(v[2], v[3], lo, true);
  }
  uint8_t* o = out + f * 1536;
  *reinterpret_cast<uint4*>(o + 16 * lane) = make_uint4(d[0], d[1], d[2], d[3]);
  *reinterpret_cast<uint2*>(o + 1024 + 8 * lane) = make_uint2(d[4], d[5]);
}

}  // namespace

hipError_t launch_pack_conv_fp16(const float* conv_w, const float* conv_b, uint4* conv_frag,
                                 hipStream_t stream) {
  return launch_kernel(pack_conv_kernel<true>, dim3(6), dim3(64), 0, stream, conv_w, conv_b, conv_frag);
}

hipError_t launch_pack_fc1_8(const float* fc1_w, const int* exp2, uint8_t* fc1_frag8,
                             hipStream_t stream) {
  const unsigned blocks = (unsigned)(((int64_t)(kPos / 2) * 8 * 64 + 255) / 256);
  return launch_kernel(pack_fc1_8_kernel, dim3(blocks), dim3(256), 0, stream, fc1_w, exp2, fc1_frag8);
}

hipError_t launch_pack_16(bool fp16, const float* conv_w, const float* conv_b,
                          const float* fc1_w, uint4* conv_frag, uint4* fc1_frag,
                          hipStream_t stream) {
  const unsigned blocks = (unsigned)((kFc1Frags + 255) / 256);
  hipError_t e;
  if (fp16) {
    e = launch_kernel(pack_conv_kernel<true>, dim3(6), dim3(64), 0, stream, conv_w, conv_b, conv_frag);
    if (e == hipSuccess)
      e = launch_kernel(pack_fc1_kernel<true>, dim3(blocks), dim3(256), 0, stream, fc1_w, fc1_frag);
  } else {
    e = launch_kernel(pack_conv_kernel<false>, dim3(6), dim3(64), 0, stream, conv_w, conv_b, conv_frag);
    if (e == hipSuccess)
      e = launch_kernel(pack_fc1_kernel<false>, dim3(blocks), dim3(256), 0, stream, fc1_w, fc1_frag);
  }
  return e;
}

}  // namespace pointid
