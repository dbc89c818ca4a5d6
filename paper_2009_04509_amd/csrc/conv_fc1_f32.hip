// Fused conv 5x5 (1->48) + ReLU + FC1 (92928->128) in fp32 on the fp32 MFMA
// (v_mfma_f32_16x16x4_f32), paper §2.2: the fp32 path.  The conv maps exist
// only in registers, as in the 16-bit kernel (conv_fc1_16.hip), whose layout
// this kernel follows with fp32 operands.
//
// Work split.  A block owns 64 patches (4 MFMA patch tiles; 32 in the blocks
// that finish a small batch, see conv_fc1_f32_tiles) and one of 8
// contiguous ranges of map positions (split-K, blockIdx % 8, so the blocks on
// one XCD share a slice of the FC1 weights).  Positions go in pairs (x, x+1),
// x even; the 5x6 window of a pair (30 pixels), a constant 1.0 for the bias and
// a zero fill the K = 32 conv operand, taken as 8 MFMAs of K = 4 (slot
// f = 4i + g for MFMA i and lane group g).  Its 6 conv tiles (2 shifts x 3
// channel tiles of 16) are the pair's 6 K-steps.  8 waves = 4 position groups
// (interleaved pairs) x 2 output halves; the two waves of a group take the same
// pairs, each computes the conv of 2 of the 4 patch tiles, and they swap the
// ReLU'd conv tiles through LDS (double-buffered, one barrier per K-step).
//
// Per K-step q (shift s, channel tile t) and 16-patch tile:
//   conv:  C[ch][patch] = sum_f Kc[ch][f] * Win[f][patch] (8 MFMAs); lane
//          (col, g) ends with channels 16t + 4g + e, e = 0..3, of patch col;
//   FC1:   chunk e uses that value as B operand K-slot g, so K-slot g of chunk
//          e is FC1 input (y*44 + x + s)*48 + 16t + 4g + e, and the A operand of
//          lane (i, g) is W1t[o][that index] for output o = 16m + i: the lane's
//          16 B at W1t[o][... + 16t + 4g] are its A operands of the 4 chunks, so
//          the transposed fp32 weights are read as they are (no repacking).
// With 64-patch tiles: 80 MFMAs per wave and K-step (16 conv, 64 FC1) against
// 4 weight loads, 2 filter and 4 swap LDS accesses and a share of the window
// reads (half the MFMAs and swap accesses with 32-patch tiles).
//
// LDS (dwords): ring of 8 patch rows (patches x 52) | conv filter fragments
// [6 conv tiles][64 lanes][8] | swap buffers [2][8 waves][own tiles][64 lanes]
// x 4; the final reduction reuses it from the start.  The four position
// groups' partial sums are added in a fixed order ((g0 + g2) + (g1 + g3)), each
// group finishing a quarter of the tiles, and written as fp32 partials
// [split][patch][128] for the tail kernel: results do not depend on the batch
// or the hit order.
#include "internal.h"

namespace pointid {
namespace {

typedef float floatx4 __attribute__((ext_vector_type(4)));

constexpr int kGroups = 4;                    // position groups
constexpr int kHalves = 2;                    // output halves
constexpr int kWaves = kGroups * kHalves;     // 8
constexpr int kThreads = kWaves * 64;         // 512
constexpr int kMT = 8 / kHalves;              // 4 output tiles per wave
constexpr int kRing = 8;                      // patch-row ring slots
constexpr int kRP = 52;                       // LDS row pitch (dwords; 48 used)
constexpr int kPairsPerRow = kFm / 2;         // 22
constexpr int kPairs = kPos / 2;              // 968
constexpr int kPairGroups = kPairs / kGroups; // 242
constexpr int kPrologueRows = 2 + kK - 1;     // rows of the first two steps
constexpr int kQ = 6;                         // K-steps per pair (2 shifts x 3 channel tiles)
constexpr int kSplits = 8;
constexpr int kBigTile = 64;                  // patches per block (most blocks)
constexpr int kSmallTile = 32;                // patches per block (the last ones)
static_assert(kPairs % kGroups == 0, "whole pair groups");

// Layout of a block of kBt patches (LDS offsets in dwords).  A patch row (192
// B) of each of the block's patches is kBt x 12 chunks of 16 B: chunk c = tid
// for the first kRowMain threads, plus c = kThreads + tid for the first
// kRowExtra threads (whole waves, so no lane diverges).
template <int kBt>
struct Tile {
  static constexpr int kTiles = kBt / 16;                 // 16-patch MFMA tiles
  static constexpr int kOwn = kTiles / kHalves;           // tiles whose conv a wave computes
  static constexpr int kSlot = kBt * kRP;                 // dwords per ring slot
  static constexpr int kFiltOff = kRing * kSlot;
  static constexpr int kSwapOff = kFiltOff + kQ * 64 * 8;
  static constexpr int kSwapBuf = kWaves * kOwn * 64 * 4;
  static constexpr int kMain = kSwapOff + 2 * kSwapBuf;
  // the reduction: per output half, 3 tiles from the other groups per accumulator tile
  static constexpr int kRed = kHalves * kMT * kTiles * (kGroups - 1) * 64 * 4;
  static constexpr int kLds = kMain > kRed ? kMain : kRed;
  static constexpr int kRowChunks = kBt * 12;
  static constexpr int kRowMain = kRowChunks < kThreads ? kRowChunks : kThreads;
  static constexpr int kRowExtra = kRowChunks - kRowMain;
  static_assert(kTiles % kHalves == 0, "whole tiles per output half");
  static_assert(kLds * 4 <= 160 * 1024, "LDS");
  static_assert(kRowMain % 64 == 0 && kRowExtra % 64 == 0 && kRowExtra <= kThreads,
                "row chunking in whole waves");
};
static_assert(Tile<kBigTile>::kLds >= Tile<kSmallTile>::kLds, "LDS sized by the big tile");

__device__ __forceinline__ floatx4 mfma4(float a, float b, const floatx4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// chunk c (16 B) of row r of the block's patches; past the batch: the last patch
__device__ __forceinline__ float4 row_chunk(const float* __restrict__ patches, int64_t n,
                                            int64_t p_base, int r, int c) {
  const int p = c / 12, h = c - (c / 12) * 12;
  int64_t gp = p_base + p;
  gp = gp < n ? gp : n - 1;
  typedef float fx4 __attribute__((ext_vector_type(4)));
  const fx4 v = __builtin_nontemporal_load(
      reinterpret_cast<const fx4*>(patches + gp * kPatchPix + r * kPatch + 4 * h));
  return make_float4(v[0], v[1], v[2], v[3]);
}

template <int kBt>
__device__ __forceinline__ void row_store(float* lds, int r, int c, const float4& v) {
  const int p = c / 12, h = c - (c / 12) * 12;
  *reinterpret_cast<float4*>(lds + (r & (kRing - 1)) * Tile<kBt>::kSlot + p * kRP + 4 * h) = v;
}

// One block: patches p_base .. p_base + kBt - 1 (clamped to the batch) and
// position range `split`.
template <int kBt>
__device__ __forceinline__ void conv_fc1_f32_block(
    float* lds, int split, int64_t p_base, const float* __restrict__ patches, int64_t n,
    const float* __restrict__ conv_w, const float* __restrict__ conv_b,
    const float* __restrict__ w1t, float* __restrict__ part, int64_t row0, int64_t n_total) {
  using T = Tile<kBt>;
  constexpr int kTiles = T::kTiles, kOwn = T::kOwn, kSlot = T::kSlot;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int kg = wave % kGroups;             // position group
  const int nh = wave / kGroups;             // output half; also the half of the tiles it convolves
  const int partner = kg + kGroups * (1 - nh);
  const bool rmain = wave < T::kRowMain / 64;   // wave-uniform: a first row chunk
  const bool extra = wave < T::kRowExtra / 64;  // wave-uniform: a second row chunk
  const int col = lane & 15, grp = lane >> 4;
  const int G0 = (kPairGroups * split) / kSplits;
  const int steps = (kPairGroups * (split + 1)) / kSplits - G0;
  const int P0 = kGroups * G0;

  // ---- conv filter fragments: [conv tile q = 3s + t][lane][MFMA i]
  float* filt = lds + T::kFiltOff;
  for (int e = tid; e < kQ * 64 * 8; e += kThreads) {
    const int i = e & 7, l = (e >> 3) & 63, q = e >> 9;
    const int s = q / 3, t = q - 3 * (q / 3);
    const int ch = 16 * t + (l & 15), f = 4 * i + (l >> 4);
    float v = 0.f;
    if (f < 30) {
      const int u = f / 6, c = f - 6 * (f / 6) - s;
      if (c >= 0 && c < kK) v = conv_w[ch * kK * kK + u * kK + c];
    } else if (f == 30) {
      v = conv_b[ch];
    }
    filt[e] = v;
  }

  // ---- patch rows: the ring is filled two steps ahead of the step computed
  auto top_row = [&](int step) {
    int pl = P0 + kGroups * step + kGroups - 1;
    if (pl > kPairs - 1) pl = kPairs - 1;
    return pl / kPairsPerRow + kK - 1;
  };
  int loaded_hi = top_row(1);
  {
    const int r0 = P0 / kPairsPerRow;
    float4 v[kPrologueRows][2];
#pragma unroll
    for (int j = 0; j < kPrologueRows; ++j)
      if (r0 + j <= loaded_hi) {
        if (rmain) v[j][0] = row_chunk(patches, n, p_base, r0 + j, tid);
        if (extra) v[j][1] = row_chunk(patches, n, p_base, r0 + j, kThreads + tid);
      }
#pragma unroll
    for (int j = 0; j < kPrologueRows; ++j)
      if (r0 + j <= loaded_hi) {
        if (rmain) row_store<kBt>(lds, r0 + j, tid, v[j][0]);
        if (extra) row_store<kBt>(lds, r0 + j, kThreads + tid, v[j][1]);
      }
  }
  __syncthreads();

  // window of pair P for this wave's own tiles: slot f = 4i + grp of patch col
  const int wbase = col * kRP + nh * kOwn * 16 * kRP;
  auto read_win = [&](int P, float (&win)[kOwn][8]) {
    const int y = P / kPairsPerRow;
    const int x = 2 * (P - y * kPairsPerRow);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int f = 4 * i + grp;
      const int fc = f > 29 ? 29 : f;        // slots 30-31 are constants (set below)
      // ring slot (y + fc / 6) & 7, column x + fc % 6
      int a = (y & (kRing - 1)) * kSlot + (fc / 6) * kSlot + (fc % 6) + wbase + x;
      if (a >= kRing * kSlot) a -= kRing * kSlot;
#pragma unroll
      for (int j = 0; j < kOwn; ++j)
        win[j][i] = f < 30 ? lds[a + j * 16 * kRP] : (f == 30 ? 1.f : 0.f);
    }
  };
  auto conv = [&](int q, const float (&win)[kOwn][8], floatx4 (&out)[kOwn]) {
    const float4* fp = reinterpret_cast<const float4*>(filt + (q * 64 + lane) * 8);
    const float4 fa = fp[0], fb = fp[1];
    const float fr[8] = {fa.x, fa.y, fa.z, fa.w, fb.x, fb.y, fb.z, fb.w};
#pragma unroll
    for (int j = 0; j < kOwn; ++j) {
      floatx4 c = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int i = 0; i < 8; ++i) c = mfma4(fr[i], win[j][i], c);
      out[j] = (floatx4){fmaxf(c[0], 0.f), fmaxf(c[1], 0.f), fmaxf(c[2], 0.f), fmaxf(c[3], 0.f)};
    }
  };
  floatx4* swp = reinterpret_cast<floatx4*>(lds + T::kSwapOff);
  auto put = [&](int buf, const floatx4 (&v)[kOwn]) {
#pragma unroll
    for (int j = 0; j < kOwn; ++j) swp[((buf * kWaves + wave) * kOwn + j) * 64 + lane] = v[j];
  };
  auto get = [&](int buf, floatx4 (&v)[kOwn]) {
#pragma unroll
    for (int j = 0; j < kOwn; ++j) v[j] = swp[((buf * kWaves + partner) * kOwn + j) * 64 + lane];
  };

  // FC1 weights: W1t[o][k] through a buffer resource; the lane's row and
  // K-slot group are a per-lane offset, the pair and K-step a scalar one
  const __amdgpu_buffer_rsrc_t wr = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<float*>(w1t), (short)0, (int)(sizeof(float) * kFc1Out * kFc1In), 0x00020000);
  int voff[kMT];
#pragma unroll
  for (int m = 0; m < kMT; ++m) voff[m] = ((16 * (nh * kMT + m) + col) * kFc1In + 4 * grp) * 4;
  // K-step k of this wave: pair P0 + kGroups * (k / 6) + kg, conv tile k % 6
  auto load_w = [&](int k, floatx4 (&w)[kMT]) {
    const int P = P0 + kGroups * (k / kQ) + kg;
    const int q = k - kQ * (k / kQ);
    const int s = q / 3, t = q - 3 * (q / 3);
    const int y = P / kPairsPerRow;
    const int x = 2 * (P - y * kPairsPerRow);
    const int soff = (((y * kFm + x + s) * kCh) + 16 * t) * 4;
#pragma unroll
    for (int m = 0; m < kMT; ++m)
      w[m] = __builtin_bit_cast(floatx4, __builtin_amdgcn_raw_buffer_load_b128(wr, voff[m], soff, 0));
  };

  floatx4 acc[kMT][kTiles];                  // [m][own tiles, then the partner's]
#pragma unroll
  for (int m = 0; m < kMT; ++m)
#pragma unroll
    for (int j = 0; j < kTiles; ++j) acc[m][j] = (floatx4){0.f, 0.f, 0.f, 0.f};

  const int K = steps * kQ;
  floatx4 w[3][kMT], own[kOwn], oth[kOwn], nxt[kOwn];
  float win[kOwn][8];
  load_w(0, w[0]);
  if (K > 1) load_w(1, w[1]);
  read_win(P0 + kg, win);
  conv(0, win, own);
  put(0, own);
  __syncthreads();

  // a new patch row two steps ahead, at most one per step (block-uniform):
  // loaded in the step's first K-step, stored in its third.  A step's 6
  // K-steps are unrolled, so the weight ring slot (k % 3) and the swap buffer
  // (k % 2) are compile-time indices: K-step k = 6 step + q has q % 3 and q % 2.
#pragma unroll 1
  for (int step = 0; step < steps; ++step) {
    float4 rv[2];
    const int want_hi = top_row(step + 2);
    const bool new_row = want_hi > loaded_hi;
    if (new_row) {
      if (rmain) rv[0] = row_chunk(patches, n, p_base, want_hi, tid);
      if (extra) rv[1] = row_chunk(patches, n, p_base, want_hi, kThreads + tid);
    }
#pragma unroll
    for (int q = 0; q < kQ; ++q) {
      const int k = step * kQ + q;
      get(q & 1, oth);
      if (k + 2 < K) load_w(k + 2, w[(q + 2) % 3]);
      // conv of the next K-step (the next pair's window when it starts a pair)
      const bool more = k + 1 < K;
      if (more) {
        if (q == kQ - 1) {
          // the current pair's window was last used by the previous K-step
          read_win(P0 + kGroups * (step + 1) + kg, win);
          conv(0, win, nxt);
        } else {
          conv(q + 1, win, nxt);
        }
      }
      // FC1 of this K-step
#pragma unroll
      for (int e = 0; e < 4; ++e)
#pragma unroll
        for (int m = 0; m < kMT; ++m) {
#pragma unroll
          for (int j = 0; j < kOwn; ++j) acc[m][j] = mfma4(w[q % 3][m][e], own[j][e], acc[m][j]);
#pragma unroll
          for (int j = 0; j < kOwn; ++j)
            acc[m][kOwn + j] = mfma4(w[q % 3][m][e], oth[j][e], acc[m][kOwn + j]);
        }
      if (more) {
        put((q + 1) & 1, nxt);
#pragma unroll
        for (int j = 0; j < kOwn; ++j) own[j] = nxt[j];
      }
      if (q == 2 && new_row) {
        // the slot it overwrites held a row below every row still read; the
        // barrier publishes it before the step that first needs it
        if (rmain) row_store<kBt>(lds, want_hi, tid, rv[0]);
        if (extra) row_store<kBt>(lds, want_hi, kThreads + tid, rv[1]);
        loaded_hi = want_hi;
      }
      __syncthreads();
    }
  }

  // ---- fixed-order reduction over the position groups: (g0 + g2) + (g1 + g3),
  // each position group finishing a quarter of its output half's accumulator
  // tiles after one barrier (the four waves of a half hold the same tiles)
  constexpr int kSlots = kMT * kTiles;
  constexpr int kPer = kSlots / kGroups;
  static_assert(kSlots % kGroups == 0, "whole quarters");
  floatx4* red = reinterpret_cast<floatx4*>(lds);
  auto entry = [&](int q, int src) { return ((nh * kSlots + q) * (kGroups - 1) + src) * 64 + lane; };
  auto tile_acc = [&](auto qc) -> floatx4& {
    constexpr int q = decltype(qc)::value;
    return acc[q / kTiles][q % kTiles];
  };
  static_for<kSlots>([&](auto qc) {
    constexpr int o = decltype(qc)::value / kPer;
    if (kg != o) red[entry(decltype(qc)::value, kg - (kg > o ? 1 : 0))] = tile_acc(qc);
  });
  __syncthreads();

  // acc[m][j]: outputs 16 (nh kMT + m) + 4 grp + e of patch 16 tile + col, tile
  // = nh kOwn + j for j < kOwn, else (1 - nh) kOwn + j - kOwn
  float* dst = part + ((int64_t)split * n_total + row0 + p_base) * kFc1Out;
  static_for<kSlots>([&](auto qc) {
    constexpr int q = decltype(qc)::value, o = q / kPer, m = q / kTiles, j = q % kTiles;
    if (kg == o) {
      floatx4 v[kGroups];
#pragma unroll
      for (int g = 0; g < kGroups; ++g)
        v[g] = (g == o) ? tile_acc(qc) : red[entry(q, g - (g > o ? 1 : 0))];
      const floatx4 sum = (v[0] + v[2]) + (v[1] + v[3]);
      const int tile = j < kOwn ? nh * kOwn + j : (1 - nh) * kOwn + (j - kOwn);
      const int64_t p = (int64_t)tile * 16 + col;
      if (p_base + p < n)
        __builtin_nontemporal_store(sum, reinterpret_cast<floatx4*>(
                                             dst + p * kFc1Out + 16 * (nh * kMT + m) + 4 * grp));
    }
  });
}

// Tiles t < n_big hold kBigTile patches; the ones after them kSmallTile.  A
// patch's sums do not depend on the size of the tile it is in: every MFMA
// column and every reduction step is per patch.
__global__ __launch_bounds__(kThreads, 1) void conv_fc1_f32_kernel(
    const float* __restrict__ patches, int64_t n, int64_t n_big, const float* __restrict__ conv_w,
    const float* __restrict__ conv_b, const float* __restrict__ w1t, float* __restrict__ part,
    int64_t row0, int64_t n_total) {
  __shared__ __attribute__((aligned(16))) float lds[Tile<kBigTile>::kLds];
  const int split = blockIdx.x % kSplits;
  const int64_t t = blockIdx.x / kSplits;
  if (t < n_big)
    conv_fc1_f32_block<kBigTile>(lds, split, t * kBigTile, patches, n, conv_w, conv_b, w1t, part,
                                 row0, n_total);
  else
    conv_fc1_f32_block<kSmallTile>(lds, split, n_big * kBigTile + (t - n_big) * kSmallTile,
                                   patches, n, conv_w, conv_b, w1t, part, row0, n_total);
}

// W1t[o][k] = W1[k][o], once at create: 32 x 32 tiles through LDS, both sides
// coalesced.
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

int conv_fc1_f32_splits() { return kSplits; }

// As for the 16-bit kernel: big tiles fill whole rounds of the CUs (one block
// per CU), and the rest is cut into small tiles when they fit in one round.
void conv_fc1_f32_tiles(int64_t n, int cus, int64_t* n_big, int64_t* n_small) {
  const int64_t per_round = cus >= kSplits ? cus / kSplits : 1;     // tiles per round
  int64_t big = n / (kBigTile * per_round) * per_round;
  const int64_t rest = n - big * kBigTile;
  int64_t small = (rest + kSmallTile - 1) / kSmallTile;
  if (small > per_round) {                   // more than one round of small tiles
    big += (rest + kBigTile - 1) / kBigTile;
    small = 0;
  }
  *n_big = big;
  *n_small = small;
}

hipError_t launch_transpose_w1(const float* w1, float* w1t, hipStream_t stream) {
  static_assert(kFc1In % 32 == 0 && kFc1Out % 32 == 0, "whole 32 x 32 tiles");
  return launch_kernel(transpose_w1_kernel, dim3(kFc1In / 32, kFc1Out / 32), dim3(256), 0, stream,
                       w1, w1t);
}

hipError_t launch_conv_fc1_f32(const float* patches, int64_t n, int64_t row0, int64_t n_total,
                               const float* conv_w, const float* conv_b, const float* w1t,
                               float* part, hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  int dev = 0, cus = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return e;
  int64_t n_big = 0, n_small = 0;
  conv_fc1_f32_tiles(n, cus, &n_big, &n_small);
  const dim3 grid((unsigned)((n_big + n_small) * kSplits));
  return launch_kernel(conv_fc1_f32_kernel, grid, dim3(kThreads), 0, stream, patches, n, n_big,
                       conv_w, conv_b, w1t, part, row0, n_total);
}

}  // namespace pointid
