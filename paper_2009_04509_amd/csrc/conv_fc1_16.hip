// Fused conv 5x5 (1->48) + ReLU + FC1 (92928->128) on 16-bit MFMA (paper §2.2),
// with bf16 or fp16 operands and fp32 accumulation.
//
// FC1 is a skinny, very deep GEMM (M = patches, N = 128, K = 92,928) whose A
// operand — the conv maps, 185,856 B per patch in bf16 — would cost twice its
// size in HBM traffic if written out and read back.  Here the conv is FC1's
// operand producer: the maps exist only in registers.
//
// Work split.  A block owns 128 patches and one of kSplits contiguous ranges of
// map positions (split-K); blockIdx % 8 selects the range, so every block on one
// XCD reads the same 1/8 of the FC1 weights and that slice (2.97 MB) stays in
// the XCD's 4 MB L2.  Positions are taken in pairs (x, x+1) with x even: the
// 5x6 pixel window of a pair (30 values) fits one K=32 MFMA operand, shared by
// both positions.  The block's four waves take interleaved pairs; each wave
// accumulates all 128 outputs for all 128 patches (8 x 8 tiles of 16x16, 256
// accumulator registers), so an FC1 weight fragment fetched from L2 is used for
// 8 MFMAs and no weight goes through LDS.  LDS holds a ring of 8 patch rows
// (the 5 rows a map row needs, plus the next) for the block's 128 patches.
//
// Per pair and per 16-patch tile, v_mfma_f32_16x16x32_{bf16,f16}:
//   conv:  D[ch][patch] = sum_slot Kc[ch][slot] * Win[slot][patch]
//          slot f < 30 holds window pixel (u, c) = (f / 6, f % 6), rows y+u and
//          columns x+c; the filter fragment for position x+s holds K[ch][u][c-s].
//          Slots 30 and 31 hold 1.0 in the window and the conv bias split into
//          two 16-bit halves (hi + lo) in the filter, so the fp32 accumulator
//          adds the bias at about twice the operand precision.
//   ReLU + round to 16 bits (RNE) on the accumulator lanes, then the 16x16 result
//   tile is used directly as the B operand of FC1: a lane holds output rows
//   4g..4g+3 for one patch column, which is the B operand's K-slot group g.  Two
//   conv tiles make one K=32 FC1 step; the FC1 weights are repacked at create
//   time into the matching K order, one 1 KiB fragment per (pair, step, 16 outputs).
//   FC1:   acc[n][patch] += W1t[n][k] * maps[k][patch]
//
// The block's four partial sums are added in LDS in a fixed order and written
// as fp32 partials [split][patch][128]; the tail kernel adds the splits.
#include "internal.h"
#include "op16.h"

namespace pointid {
namespace {

constexpr int kWaves = 4;
constexpr int kBt = 112;                    // patches per block (7 MFMA tiles)
constexpr int kTiles = kBt / 16;            // 16-patch MFMA tiles per wave
constexpr int kPairsPerRow = kFm / 2;       // 22
constexpr int kRing = 8;                    // patch-row ring slots
constexpr int kRP = 26;                     // LDS row pitch, dwords (24 used)
constexpr int kSlot = kBt * kRP;            // dwords per ring slot
constexpr int kLdsDwords = 2 * 64 * 256;    // 128 KiB: ring (104 KiB) / reduction (128 KiB)
// One patch row (96 B) of each of the block's patches: kBt x 6 chunks of 16 B,
// at most 3 per thread.
constexpr int kRowChunks = kBt * 6;

__device__ __forceinline__ void row_load(const uint16_t* __restrict__ patches, int64_t n,
                                         int64_t p_base, int r, uint4 (&v)[3]) {
#pragma unroll
  for (int k = 0; k < 3; ++k) {
    const int c = threadIdx.x + 256 * k;
    const int p = c / 6, h = c - (c / 6) * 6;
    const int64_t gp = p_base + p;
    v[k] = (c < kRowChunks && gp < n)
               ? *reinterpret_cast<const uint4*>(patches + gp * kPatchPix + r * kPatch + h * 8)
               : make_uint4(0u, 0u, 0u, 0u);
  }
}

__device__ __forceinline__ void row_store(uint32_t* lds, int r, const uint4 (&v)[3]) {
  const int slot = r & (kRing - 1);
#pragma unroll
  for (int k = 0; k < 3; ++k) {
    const int c = threadIdx.x + 256 * k;
    if (c >= kRowChunks) break;
    const int p = c / 6, h = c - (c / 6) * 6;
    uint32_t* d = lds + slot * kSlot + p * kRP + h * 4;
    *reinterpret_cast<uint2*>(d) = make_uint2(v[k].x, v[k].y);
    *reinterpret_cast<uint2*>(d + 2) = make_uint2(v[k].z, v[k].w);
  }
}

template <bool kFp16, int kSplits>
__global__ __launch_bounds__(256, 1) void conv_fc1_16_kernel(
    const uint16_t* __restrict__ patches, int64_t n, const uint4* __restrict__ w1p,
    const uint4* __restrict__ convp, float* __restrict__ part, int64_t row0, int64_t n_total) {
  __shared__ __attribute__((aligned(16))) uint32_t lds[kLdsDwords];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int col = lane & 15;                 // MFMA column (patch within tile) / row
  const int grp = lane >> 4;                 // MFMA K-slot group
  const int split = blockIdx.x % kSplits;
  const int64_t p_base = (int64_t)(blockIdx.x / kSplits) * kBt;
  // split boundaries on whole steps of 4 pairs, so every wave runs `steps` pairs
  constexpr int kGroups = kPos / 2 / kWaves;            // 242
  const int G0 = (kGroups * split) / kSplits;
  const int steps = (kGroups * (split + 1)) / kSplits - G0;
  const int P0 = kWaves * G0;

  // conv filter fragments: [shift][channel tile]
  uint4 cw[2][3];
#pragma unroll
  for (int s = 0; s < 2; ++s)
#pragma unroll
    for (int t = 0; t < 3; ++t) cw[s][t] = convp[(s * 3 + t) * 64 + lane];

  // this lane's 4 window dwords: slot pair f = 8*grp + 2d -> pixel (u, c)
  int woff[4], wrow[4];
#pragma unroll
  for (int d = 0; d < 4; ++d) {
    int f = 8 * grp + 2 * d;
    if (f > 28) f = 28;                      // slots 30-31 are constants (masked below)
    wrow[d] = f / 6;
    woff[d] = (f % 6) / 2 + col * kRP;
  }
  const bool const_slot = (grp == 3);
  using Op = Op16<kFp16>;

  floatx4 acc[8][kTiles];
#pragma unroll
  for (int m = 0; m < 8; ++m)
#pragma unroll
    for (int i = 0; i < kTiles; ++i) acc[m][i] = (floatx4){0.f, 0.f, 0.f, 0.f};

  // ---- initial patch rows
  auto top_row = [&](int step) {             // highest input row needed by a step
    return (P0 + kWaves * step + kWaves - 1) / kPairsPerRow + kK - 1;
  };
  int loaded_hi = top_row(0);
  for (int r = P0 / kPairsPerRow; r <= loaded_hi; ++r) {
    uint4 v[3];
    row_load(patches, n, p_base, r, v);
    row_store(lds, r, v);
  }
  __syncthreads();

  const uint4* wl = w1p + lane;
  uint4 wcur[8];
#pragma unroll
  for (int m = 0; m < 8; ++m) wcur[m] = wl[(((P0 + wave) * 3 + 0) * 8 + m) * 64];

#pragma unroll 1
  for (int step = 0; step < steps; ++step) {
    // prefetch the patch row the next step adds (at most one; block-uniform)
    uint4 rv[3];
    const int next_hi = (step + 1 < steps) ? top_row(step + 1) : loaded_hi;
    const bool new_row = next_hi > loaded_hi;
    if (new_row) row_load(patches, n, p_base, next_hi, rv);

    const int P = P0 + kWaves * step + wave;
    const int y = P / kPairsPerRow;
    const int xh = P - y * kPairsPerRow;     // x / 2
    uint4 win[kTiles];
    {
      int base[4];
#pragma unroll
      for (int d = 0; d < 4; ++d) base[d] = ((y + wrow[d]) & (kRing - 1)) * kSlot + woff[d] + xh;
#pragma unroll
      for (int i = 0; i < kTiles; ++i) {
        const int o = i * 16 * kRP;
        win[i].x = lds[base[0] + o];
        win[i].y = lds[base[1] + o];
        win[i].z = lds[base[2] + o];
        const uint32_t w3 = lds[base[3] + o];
        win[i].w = const_slot ? Op::kOnes : w3;
      }
    }
#pragma unroll
    for (int q = 0; q < 3; ++q) {
      // prefetch the next FC1 weight step of this wave (clamped past the end)
      int Pn = (q < 2) ? P : P + kWaves;
      const int qn = (q < 2) ? q + 1 : 0;
      if (Pn > kPos / 2 - 1) Pn = kPos / 2 - 1;
      uint4 wnext[8];
#pragma unroll
      for (int m = 0; m < 8; ++m) wnext[m] = wl[((Pn * 3 + qn) * 8 + m) * 64];
      // conv tiles feeding this K=32 step: (shift, channel tile)
      const int sa = (q == 2) ? 1 : 0, ta = (q == 0) ? 0 : (q == 1 ? 2 : 1);
      const int sb = (q == 0) ? 0 : 1, tb = (q == 0) ? 1 : (q == 1 ? 0 : 2);
#pragma unroll
      for (int i = 0; i < kTiles; ++i) {
        const floatx4 z = {0.f, 0.f, 0.f, 0.f};
        const floatx4 ca = Op::mfma(cw[sa][ta], win[i], z);
        const floatx4 cb = Op::mfma(cw[sb][tb], win[i], z);
        const uint4 bf = make_uint4(relu2(Op::pack(ca[0], ca[1])), relu2(Op::pack(ca[2], ca[3])),
                                    relu2(Op::pack(cb[0], cb[1])), relu2(Op::pack(cb[2], cb[3])));
#pragma unroll
        for (int m = 0; m < 8; ++m) acc[m][i] = Op::mfma(wcur[m], bf, acc[m][i]);
      }
#pragma unroll
      for (int m = 0; m < 8; ++m) wcur[m] = wnext[m];
    }
    if (new_row) {
      row_store(lds, next_hi, rv);
      loaded_hi = next_hi;
    }
    __syncthreads();
  }

  // ---- fixed-order reduction of the four waves: (w0 + w2) + (w1 + w3)
  float* red = reinterpret_cast<float*>(lds);
  auto put = [&](int region) {
#pragma unroll
    for (int m = 0; m < 8; ++m)
#pragma unroll
      for (int i = 0; i < kTiles; ++i)
#pragma unroll
        for (int e = 0; e < 4; ++e)
          red[region * 16384 + ((m * kTiles + i) * 4 + e) * 64 + lane] = acc[m][i][e];
  };
  auto add = [&](int region) {
#pragma unroll
    for (int m = 0; m < 8; ++m)
#pragma unroll
      for (int i = 0; i < kTiles; ++i)
#pragma unroll
        for (int e = 0; e < 4; ++e)
          acc[m][i][e] += red[region * 16384 + ((m * kTiles + i) * 4 + e) * 64 + lane];
  };
  if (wave >= 2) put(wave - 2);
  __syncthreads();
  if (wave < 2) add(wave);
  __syncthreads();
  if (wave == 1) put(0);
  __syncthreads();
  if (wave != 0) return;
  add(0);

  // acc[m][i]: outputs 16m + 4*grp + e for patch 16i + col
  float* dst = part + ((int64_t)split * n_total + row0 + p_base) * kFc1Out;
#pragma unroll
  for (int i = 0; i < kTiles; ++i) {
    const int64_t p = (int64_t)i * 16 + col;
    if (p_base + p < n) {
#pragma unroll
      for (int m = 0; m < 8; ++m)
        *reinterpret_cast<floatx4*>(dst + p * kFc1Out + 16 * m + 4 * grp) = acc[m][i];
    }
  }
}

constexpr int kSplits16 = 8;

}  // namespace

int conv_fc1_16_splits() { return kSplits16; }

hipError_t launch_conv_fc1_16(bool fp16, const uint16_t* patches, int64_t n, int64_t row0,
                              int64_t n_total, const uint4* w1p, const uint4* convp,
                              float* part, hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  const int64_t tiles = (n + kBt - 1) / kBt;
  const dim3 grid((unsigned)(tiles * kSplits16));
  if (fp16)
    conv_fc1_16_kernel<true, kSplits16><<<grid, dim3(256), 0, stream>>>(
        patches, n, w1p, convp, part, row0, n_total);
  else
    conv_fc1_16_kernel<false, kSplits16><<<grid, dim3(256), 0, stream>>>(
        patches, n, w1p, convp, part, row0, n_total);
  return hipGetLastError();
}

}  // namespace pointid
