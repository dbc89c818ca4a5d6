// The fp32 path's conv and FC1 (paper §2.2) on fp32 MFMA.
//
// Conv: maps act[p][(y*44 + x)*48 + k] = ReLU(b_k + sum_{u,v} K[k][u][v] P[y+u][x+v])
// for a chunk of patches.  As in the 16-bit kernel, positions go in pairs
// (x, x+1), x even, whose 5x6 window (30 pixels) plus a bias slot fills a K=32
// operand, here 8 v_mfma_f32_16x16x4_f32 (slot f = 4i + g for MFMA i and lane
// group g).  A = filter (16 channels x 4 slots; the fragment for position
// x + s holds K[k][u][c - s] at slot f = 6u + c, and b_k at slot 30), B = window
// (4 slots x 16 patches), C = 16 channels x 16 patches of one position: 6 conv
// tiles (2 shifts x 3 channel tiles) per pair.  A block of 8 waves owns 16
// patches; wave w takes the pairs w, w + 8, ...; the filter fragments stay in
// registers and each lane writes its 4 channels of a tile as one 16-byte store.
//
// FC1: split-K partial products
//   part[s][row0 + p][o] = sum over split s of act[p][k] * W1[k][o],
// with the conv maps `act` [m][92928] (HWC flatten, written by the conv kernel)
// and the weights stored transposed, W1t[o][k] = W1[k][o].
//
// v_mfma_f32_16x16x4_f32 with A = W1t (16 outputs x 4 k), B = act (4 k x 16
// patches), C = outputs x patches.  For a block of 16 k, lane l (i = l % 16,
// g = l / 16) loads the 16 bytes W1t[o0 + i][k0 + 4g .. 4g + 3] and
// act[p0 + i][k0 + 4g .. 4g + 3]; MFMA j (j = 0..3) takes component j of both,
// so its K-slot g holds k0 + 4g + j in both operands.  Every (output, patch)
// sum runs over the split's k in the same order wherever the patch sits in the
// batch.
//
// A block of 4 waves owns 64 patches and one of `splits` contiguous k ranges
// (blockIdx % splits, so blocks on one XCD share a weight slice): wave w takes
// outputs 64 (w % 2) .. + 63 (4 tiles) and patches 32 (w / 2) .. + 31 (2 tiles),
// 8 accumulator tiles.  Loads run three 16-k blocks ahead of the MFMAs.
#include "internal.h"

namespace pointid {
namespace {

typedef float floatx4 __attribute__((ext_vector_type(4)));

// ---------------------------------------------------------------- conv
constexpr int kConvWaves = 8;
constexpr int kPairs = kPos / 2;              // 968
constexpr int kPairsPerRow = kFm / 2;         // 22

__global__ __launch_bounds__(kConvWaves * 64) void conv_f32_kernel(
    const float* __restrict__ patches, int64_t m, const float* __restrict__ conv_w,
    const float* __restrict__ conv_b, float* __restrict__ act) {
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int col = lane & 15, g = lane >> 4;
  const int64_t p = (int64_t)blockIdx.x * 16 + col;
  const float* src = patches + (p < m ? p : m - 1) * kPatchPix;   // past the end: the last patch, not stored
  // filter fragments fa[s * 3 + t][i]: channel 16 t + col, slot f = 4 i + g
  float fa[6][8];
#pragma unroll
  for (int s = 0; s < 2; ++s)
#pragma unroll
    for (int t = 0; t < 3; ++t)
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int f = 4 * i + g, ch = 16 * t + col;
        float v = 0.f;
        if (f < 30) {
          const int u = f / 6, c = f - (f / 6) * 6 - s;
          if (c >= 0 && c < kK) v = conv_w[ch * kK * kK + u * kK + c];
        } else if (f == 30) {
          v = conv_b[ch];
        }
        fa[s * 3 + t][i] = v;
      }
  // window slot f of this lane: pixel offset (f < 30) or a constant
  int woff[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int f = 4 * i + g;
    woff[i] = f < 30 ? (f / 6) * kPatch + f - (f / 6) * 6 : 0;
  }
  float* dst = act + p * kFc1In + 4 * g;
#pragma unroll 1
  for (int P = wave; P < kPairs; P += kConvWaves) {
    const int y = P / kPairsPerRow, x = 2 * (P - y * kPairsPerRow);
    const float* w0 = src + y * kPatch + x;
    float b[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int f = 4 * i + g;
      b[i] = f < 30 ? w0[woff[i]] : (f == 30 ? 1.f : 0.f);
    }
    floatx4 c[6];
#pragma unroll
    for (int k = 0; k < 6; ++k) c[k] = (floatx4){0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int k = 0; k < 6; ++k) c[k] = __builtin_amdgcn_mfma_f32_16x16x4f32(fa[k][i], b[i], c[k], 0, 0, 0);
    if (p < m) {
#pragma unroll
      for (int s = 0; s < 2; ++s)
#pragma unroll
        for (int t = 0; t < 3; ++t) {
          const floatx4 v = c[s * 3 + t];
          *reinterpret_cast<floatx4*>(dst + (y * kFm + x + s) * kCh + 16 * t) =
              (floatx4){fmaxf(v[0], 0.f), fmaxf(v[1], 0.f), fmaxf(v[2], 0.f), fmaxf(v[3], 0.f)};
        }
    }
  }
}

// ---------------------------------------------------------------- FC1
constexpr int kPB = 64;                      // patches per block
constexpr int kKB = kFc1In / 16;             // 5808 blocks of 16 k
constexpr int kDepth = 3;                    // load sets in flight
static_assert(kFc1In % 16 == 0, "whole 16-k blocks");

__global__ __launch_bounds__(256, 2) void fc1_f32_kernel(const float* __restrict__ act, int64_t m,
                                                         const float* __restrict__ w1t, int splits,
                                                         float* __restrict__ part, int64_t row0,
                                                         int64_t n_total) {
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int oh = wave & 1, pp = wave >> 1;
  const int i = lane & 15, g = lane >> 4;
  const int split = blockIdx.x % splits;
  const int64_t p_base = (int64_t)(blockIdx.x / splits) * kPB;
  const int kb0 = (int)((int64_t)kKB * split / splits);
  const int kb1 = (int)((int64_t)kKB * (split + 1) / splits);

  // Operands through buffer resources: a lane's row is a per-lane byte offset,
  // the 16-k block a scalar one (both fit 32 bits: the launch checks the sizes).
  // Patches past the end of the chunk read the last patch; their results are
  // not stored.
  const __amdgpu_buffer_rsrc_t wr = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<float*>(w1t), (short)0, (int)(sizeof(float) * kFc1Out * kFc1In), 0x00020000);
  const __amdgpu_buffer_rsrc_t ar = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<float*>(act), (short)0, (int)(sizeof(float) * m * kFc1In), 0x00020000);
  int woff[4], aoff[2];
#pragma unroll
  for (int t = 0; t < 4; ++t) woff[t] = ((64 * oh + 16 * t + i) * kFc1In + 4 * g) * 4;
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    int64_t p = p_base + 32 * pp + 16 * u + i;
    if (p > m - 1) p = m - 1;
    aoff[u] = (int)((p * kFc1In + 4 * g) * 4);
  }

  floatx4 acc[4][2];
#pragma unroll
  for (int t = 0; t < 4; ++t)
#pragma unroll
    for (int u = 0; u < 2; ++u) acc[t][u] = (floatx4){0.f, 0.f, 0.f, 0.f};

  floatx4 wa[kDepth][4], aa[kDepth][2];
  // 16-k block kb: 4 consecutive floats per lane at byte 64 kb of its row.
  // load_in_order: the same, volatile, so the compiler keeps program order.
  auto load = [&](int d, int kb) {
#pragma unroll
    for (int t = 0; t < 4; ++t)
      wa[d][t] = __builtin_bit_cast(floatx4, __builtin_amdgcn_raw_buffer_load_b128(wr, woff[t], kb * 64, 0));
#pragma unroll
    for (int u = 0; u < 2; ++u)
      aa[d][u] = __builtin_bit_cast(floatx4, __builtin_amdgcn_raw_buffer_load_b128(ar, aoff[u], kb * 64, 0));
  };
  constexpr int kVolatile = (int)(1u << 31);
  auto load_in_order = [&](int d, int kb) {
#pragma unroll
    for (int t = 0; t < 4; ++t)
      wa[d][t] = __builtin_bit_cast(floatx4, __builtin_amdgcn_raw_buffer_load_b128(wr, woff[t], kb * 64, kVolatile));
#pragma unroll
    for (int u = 0; u < 2; ++u)
      aa[d][u] = __builtin_bit_cast(floatx4, __builtin_amdgcn_raw_buffer_load_b128(ar, aoff[u], kb * 64, kVolatile));
  };
  auto step = [&](int d) {
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int t = 0; t < 4; ++t)
#pragma unroll
        for (int u = 0; u < 2; ++u)
          acc[t][u] = __builtin_amdgcn_mfma_f32_16x16x4f32(wa[d][t][j], aa[d][u][j], acc[t][u], 0, 0, 0);
  };

  // (a split holds a whole number of kDepth-block rounds, checked at launch,
  // so the loop body has no branch and the compiler can count the loads in
  // flight across iterations)
#pragma unroll
  for (int d = 0; d < kDepth; ++d) {
    // in the loop's order (set by set, each set as the loop issues it): the
    // loop's waits count the loads in flight on entry, so these must match
    // (volatile: the compiler keeps them in program order)
    load_in_order(d, kb0 + d);
    __builtin_amdgcn_sched_barrier(0);
  }
#pragma unroll 1
  for (int kb = kb0; kb < kb1; kb += kDepth) {
#pragma unroll
    for (int d = 0; d < kDepth; ++d) {
      step(d);
      load(d, kb + d + kDepth);
      // keep the loads here, kDepth blocks ahead of their MFMAs (left alone,
      // the scheduler sinks them to their use)
      __builtin_amdgcn_sched_barrier(0);
    }
  }

  // acc[t][u]: outputs 64 oh + 16 t + 4 g + e for patch 32 pp + 16 u + i
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const int64_t p = p_base + 32 * pp + 16 * u + i;
    if (p >= m) continue;
    float* dst = part + ((int64_t)split * n_total + row0 + p) * kFc1Out + 64 * oh + 4 * g;
#pragma unroll
    for (int t = 0; t < 4; ++t) *reinterpret_cast<floatx4*>(dst + 16 * t) = acc[t][u];
  }
}

// W1t[o][k] = W1[k][o]: 32 x 32 tiles through LDS, both sides coalesced.
__global__ __launch_bounds__(256) void transpose_w1_kernel(const float* __restrict__ w1,
                                                           float* __restrict__ w1t) {
  __shared__ float tile[32][33];
  const int k0 = blockIdx.x * 32, o0 = blockIdx.y * 32;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;   // 32 x 8
#pragma unroll
  for (int r = ty; r < 32; r += 8) tile[r][tx] = w1[(int64_t)(k0 + r) * kFc1Out + o0 + tx];
  __syncthreads();
#pragma unroll
  for (int r = ty; r < 32; r += 8) w1t[(int64_t)(o0 + r) * kFc1In + k0 + tx] = tile[tx][r];
}

}  // namespace

hipError_t launch_conv_f32(const float* patches, int64_t m, const DeviceWeights& w, float* act,
                           hipStream_t stream) {
  if (m <= 0) return hipSuccess;
  const int64_t blocks = (m + 15) / 16;
  conv_f32_kernel<<<dim3((unsigned)blocks), dim3(kConvWaves * 64), 0, stream>>>(patches, m, w.conv_w,
                                                                                 w.conv_b, act);
  return hipGetLastError();
}

hipError_t launch_transpose_w1(const float* w1, float* w1t, hipStream_t stream) {
  static_assert(kFc1In % 32 == 0 && kFc1Out % 32 == 0, "whole 32 x 32 tiles");
  transpose_w1_kernel<<<dim3(kFc1In / 32, kFc1Out / 32), dim3(256), 0, stream>>>(w1, w1t);
  return hipGetLastError();
}

hipError_t launch_fc1_f32(const float* act, int64_t m, int64_t row0, int64_t n_total,
                          const float* w1t, int splits, float* part, hipStream_t stream) {
  if (m <= 0) return hipSuccess;
  if (splits < 1 || kKB % splits != 0 || (kKB / splits) % kDepth != 0) return hipErrorInvalidValue;
  if ((double)m * kFc1In * sizeof(float) >= 2147483648.0) return hipErrorInvalidValue;  // 32-bit offsets
  const int64_t blocks = (m + kPB - 1) / kPB * splits;
  fc1_f32_kernel<<<dim3((unsigned)blocks), dim3(256), 0, stream>>>(act, m, w1t, splits, part, row0,
                                                                   n_total);
  return hipGetLastError();
}

}  // namespace pointid
