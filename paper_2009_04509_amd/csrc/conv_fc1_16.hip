// Fused conv 5x5 (1->48) + ReLU + FC1 (92928->128) on 16-bit MFMA (paper §2.2),
// with bf16 or fp16 operands and fp32 accumulation.
//
// FC1 is a skinny, very deep GEMM (M = patches, N = 128, K = 92,928) whose A
// operand — the conv maps, 185,856 B per patch in 16 bits — would cost twice its
// size in HBM traffic if written out and read back.  Here the conv is FC1's
// operand producer: the maps exist only in registers.
//
// Work split.  A block owns 96 patches and one of kSplits contiguous ranges of
// map positions (split-K); blockIdx % 8 selects the range, so every block on one
// XCD reads the same 1/8 of the FC1 weights and that slice (2.97 MB) stays in
// the XCD's 4 MB L2.  Positions are taken in pairs (x, x+1) with x even: the
// 5x6 pixel window of a pair (30 values) fits one K=32 MFMA operand, shared by
// both positions.  The block's 8 waves (2 per SIMD, so one wave's conversions
// overlap the other's MFMAs) form 4 position groups x 2 output halves: the two
// waves of a group take the same interleaved pairs and the same 96 patches, and
// each accumulates 64 of the 128 outputs (4 x 6 tiles of 16x16).  Both compute
// the conv of their pair; each FC1 weight fragment fetched from L2 feeds 6
// MFMAs and no weight goes through LDS.  LDS holds a ring of 8 patch rows (the 5
// rows a map row needs, plus the next) for the block's 96 patches.
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
// The four position groups' partial sums are added in LDS in a fixed order and
// written as fp32 partials [split][patch][128]; the tail kernel adds the splits.
#include "internal.h"
#include "op16.h"

namespace pointid {
namespace {

constexpr int kKGroups = 4;                   // position groups (interleaved pairs)
constexpr int kNHalves = 2;                   // output halves
constexpr int kWaves = kKGroups * kNHalves;   // 8
constexpr int kThreads = kWaves * 64;         // 512
constexpr int kMT = 8 / kNHalves;             // 16-output tiles per wave
constexpr int kBt = 96;                       // patches per block
constexpr int kTiles = kBt / 16;              // 16-patch MFMA tiles
constexpr int kPairsPerRow = kFm / 2;         // 22
constexpr int kRing = 8;                      // patch-row ring slots
constexpr int kRP = 26;                       // LDS row pitch, dwords (24 used)
constexpr int kSlot = kBt * kRP;              // dwords per ring slot
constexpr int kRegion = kMT * kTiles * 4 * 64;          // one wave's partial sums (floats)
constexpr int kLdsDwords = (kRing * kSlot > 4 * kRegion) ? kRing * kSlot : 4 * kRegion;

// One patch row (96 B) of each of the block's patches: kBt x 6 chunks of 16 B.
// Chunk c = tid, plus c = kThreads + tid for the first kRowExtra threads (whole
// waves, so no lane diverges).  Patches past the end of the batch are read from
// the last patch instead: their results are never stored.
constexpr int kRowChunks = kBt * 6;
constexpr int kRowExtra = kRowChunks - kThreads;
static_assert(kRowExtra > 0 && kRowExtra % 64 == 0 && kRowExtra <= kThreads, "row chunking");

__device__ __forceinline__ uint4 row_chunk_load(const uint16_t* __restrict__ patches, int64_t n,
                                                int64_t p_base, int r, int c) {
  typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
  const int p = c / 6, h = c - (c / 6) * 6;
  int64_t gp = p_base + p;
  gp = gp < n ? gp : n - 1;
  // streamed once per block: non-temporal, so it does not push the block's FC1
  // weight slice out of L2
  return __builtin_bit_cast(uint4, __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(
                                       patches + gp * kPatchPix + r * kPatch + h * 8)));
}

__device__ __forceinline__ void row_chunk_store(uint32_t* lds, int r, int c, const uint4& v) {
  const int p = c / 6, h = c - (c / 6) * 6;
  uint32_t* d = lds + (r & (kRing - 1)) * kSlot + p * kRP + h * 4;
  *reinterpret_cast<uint2*>(d) = make_uint2(v.x, v.y);
  *reinterpret_cast<uint2*>(d + 2) = make_uint2(v.z, v.w);
}

__device__ __forceinline__ void row_load(const uint16_t* __restrict__ patches, int64_t n,
                                         int64_t p_base, int r, bool extra, uint4 (&v)[2]) {
  v[0] = row_chunk_load(patches, n, p_base, r, threadIdx.x);
  if (extra) v[1] = row_chunk_load(patches, n, p_base, r, threadIdx.x + kThreads);
}

__device__ __forceinline__ void row_store(uint32_t* lds, int r, bool extra, const uint4 (&v)[2]) {
  row_chunk_store(lds, r, threadIdx.x, v[0]);
  if (extra) row_chunk_store(lds, r, threadIdx.x + kThreads, v[1]);
}

template <bool kFp16, int kSplits>
__global__ __launch_bounds__(kThreads, 1) void conv_fc1_16_kernel(
    const uint16_t* __restrict__ patches, int64_t n, const uint4* __restrict__ w1p,
    const uint4* __restrict__ convp, float* __restrict__ part, int64_t row0, int64_t n_total) {
  __shared__ __attribute__((aligned(16))) uint32_t lds[kLdsDwords];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int kg = wave % kKGroups;            // position group
  const int nh = wave / kKGroups;            // output half
  const bool extra = wave < kRowExtra / 64;  // wave-uniform
  const int col = lane & 15;                 // MFMA column (patch within tile) / row
  const int grp = lane >> 4;                 // MFMA K-slot group
  const int split = blockIdx.x % kSplits;
  const int64_t p_base = (int64_t)(blockIdx.x / kSplits) * kBt;
  // split boundaries on whole steps of kKGroups pairs: every wave runs `steps` pairs
  constexpr int kGroups = kPos / 2 / kKGroups;          // 242
  const int G0 = (kGroups * split) / kSplits;
  const int steps = (kGroups * (split + 1)) / kSplits - G0;
  const int P0 = kKGroups * G0;

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

  floatx4 acc[kMT][kTiles];
#pragma unroll
  for (int m = 0; m < kMT; ++m)
#pragma unroll
    for (int i = 0; i < kTiles; ++i) acc[m][i] = (floatx4){0.f, 0.f, 0.f, 0.f};

  // ---- initial patch rows
  auto top_row = [&](int step) {             // highest input row needed by a step
    return (P0 + kKGroups * step + kKGroups - 1) / kPairsPerRow + kK - 1;
  };
  int loaded_hi = top_row(0);
  for (int r = P0 / kPairsPerRow; r <= loaded_hi; ++r) {
    uint4 v[2];
    row_load(patches, n, p_base, r, extra, v);
    row_store(lds, r, extra, v);
  }
  __syncthreads();

  // FC1 fragments through a buffer resource: the fragment base is a scalar
  // offset and the output tiles are immediate offsets, so the loads need no
  // per-lane address arithmetic; reads past the end return 0.
  const __amdgpu_buffer_rsrc_t w1r = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint4*>(w1p), (short)0, (int)(kFc1Frags * 16), 0x00020000);
  const int voff = lane * 16 + nh * kMT * 1024;
  auto load_w = [&](int P, int q, uint4 (&w)[kMT]) {
    const int so = (P * 3 + q) * 8 * 1024;
#pragma unroll
    for (int m = 0; m < kMT; ++m)
      w[m] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(w1r, voff + m * 1024, so, 0));
  };
  uint4 wcur[kMT];
  load_w(P0 + kg, 0, wcur);

#pragma unroll 1
  for (int step = 0; step < steps; ++step) {
    // prefetch the patch row the next step adds (at most one; block-uniform)
    uint4 rv[2];
    const int next_hi = (step + 1 < steps) ? top_row(step + 1) : loaded_hi;
    const bool new_row = next_hi > loaded_hi;
    if (new_row) row_load(patches, n, p_base, next_hi, extra, rv);

    const int P = P0 + kKGroups * step + kg;
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
      // prefetch the next FC1 weight step of this wave (past the end reads 0)
      const int Pn = (q < 2) ? P : P + kKGroups;
      const int qn = (q < 2) ? q + 1 : 0;
      uint4 wnext[kMT];
      load_w(Pn, qn, wnext);
      // keep these loads here: the scheduler would otherwise sink them to their
      // use in the next step and expose the full memory latency
      __builtin_amdgcn_sched_barrier(0);
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
        for (int m = 0; m < kMT; ++m) acc[m][i] = Op::mfma(wcur[m], bf, acc[m][i]);
      }
#pragma unroll
      for (int m = 0; m < kMT; ++m) wcur[m] = wnext[m];
    }
    // The ring slot a new row overwrites held row next_hi - 8, which is below
    // every row the steps since the last barrier read, so waves may drift
    // apart between row loads; the barrier publishes the new row before any
    // wave's next step reads it.  (new_row is block-uniform.)
    if (new_row) {
      row_store(lds, next_hi, extra, rv);
      loaded_hi = next_hi;
      __syncthreads();
    }
  }
  __syncthreads();

  // ---- fixed-order reduction over position groups, per output half:
  //      (g0 + g2) + (g1 + g3)
  float* red = reinterpret_cast<float*>(lds);
  auto put = [&](int region) {
#pragma unroll
    for (int m = 0; m < kMT; ++m)
#pragma unroll
      for (int i = 0; i < kTiles; ++i)
#pragma unroll
        for (int e = 0; e < 4; ++e)
          red[region * kRegion + ((m * kTiles + i) * 4 + e) * 64 + lane] = acc[m][i][e];
  };
  auto add = [&](int region) {
#pragma unroll
    for (int m = 0; m < kMT; ++m)
#pragma unroll
      for (int i = 0; i < kTiles; ++i)
#pragma unroll
        for (int e = 0; e < 4; ++e)
          acc[m][i][e] += red[region * kRegion + ((m * kTiles + i) * 4 + e) * 64 + lane];
  };
  if (kg >= 2) put(nh * 2 + (kg - 2));
  __syncthreads();
  if (kg < 2) add(nh * 2 + kg);
  __syncthreads();
  if (kg == 1) put(nh);
  __syncthreads();
  if (kg != 0) return;
  add(nh);

  // acc[m][i]: outputs 16(nh*kMT + m) + 4*grp + e for patch 16i + col
  float* dst = part + ((int64_t)split * n_total + row0 + p_base) * kFc1Out;
#pragma unroll
  for (int i = 0; i < kTiles; ++i) {
    const int64_t p = (int64_t)i * 16 + col;
    if (p_base + p < n) {
#pragma unroll
      for (int m = 0; m < kMT; ++m)
        *reinterpret_cast<floatx4*>(dst + p * kFc1Out + 16 * (nh * kMT + m) + 4 * grp) = acc[m][i];
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
    conv_fc1_16_kernel<true, kSplits16><<<grid, dim3(kThreads), 0, stream>>>(
        patches, n, w1p, convp, part, row0, n_total);
  else
    conv_fc1_16_kernel<false, kSplits16><<<grid, dim3(kThreads), 0, stream>>>(
        patches, n, w1p, convp, part, row0, n_total);
  return hipGetLastError();
}

}  // namespace pointid
