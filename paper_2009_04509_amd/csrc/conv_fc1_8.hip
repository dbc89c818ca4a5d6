// Fused conv 5x5 (1->48) + ReLU + FC1 (92928->128) with FC1 on 8-bit float
// operands: the 8-bit operation of the paper's outlook (§4) applied to the
// network of §2.2.
//
// The conv runs on fp16 MFMAs exactly as in conv_fc1_16.hip (fp16 patch rows
// in an LDS ring, a pair of map positions per 5x6 window, the bias in window
// slots 30-31).  Its ReLU output is clamped to 448 and rounded to OCP e4m3
// (v_med3 + v_cvt_pk_fp8, nearest even), and FC1 runs on
// v_mfma_scale_f32_16x16x128_f8f6f4 with unit scales and fp32 accumulation.
// FC1 column n is stored multiplied by 2^k_n (the largest power of two that
// keeps the column within 448) and rounded to e4m3 at create time; the tail
// kernel multiplies the column's sums by 2^-k_n, which is exact.
//
// Work split as in the fp16 kernel: a block owns 64 patches (32 in the blocks
// that finish a batch) and one of 8 ranges of map positions (blockIdx % 8, so
// each XCD's L2 holds one eighth of the 11.9 MB of fp8 weights); 8 waves = 4
// position groups x 2 output halves; the two waves of a group take the same
// pairs, each computes the conv of half of the block's 16-patch tiles, and the
// two exchange their quantized fragments through LDS.  (96-patch blocks, as
// in the fp16 kernel, need more than the 256 registers two waves per SIMD
// allow: the 8-register operand tuples and the conv filters held in registers.)
//
// One K step is one pair of map positions (P = y * 22 + x / 2, positions x
// and x + 1 of map row y): its 2 x 48 FC1 inputs fill 24 of the 32 operand
// bytes of a lane.  Lane (col, g) of the B operand (and lane (row, g) of A)
// holds, in dword d < 6, the conv tile (shift d / 3, channel tile d % 3):
// byte e is channel 16 (d % 3) + 4g + e at position x + d / 3.  Dwords 6-7
// are zero in both operands.  Per K step a wave issues 16 FC1 MFMAs (4 output
// tiles x 4 patch tiles) and 6 conv MFMAs per own patch tile, and the block
// passes one barrier.  The FC1 weights of the wave's 4 output tiles sit in
// one register set; each fragment is reloaded for the next pair right after
// its last use, most of a K step before it is needed.
//
// The partial sums are reduced over the position groups in LDS in a fixed
// order and written as fp32 partials [split][patch][128], as in the fp16 kernel.
#include "internal.h"
#include "op16.h"

namespace pointid {
namespace {

typedef int v8i __attribute__((ext_vector_type(8)));

constexpr int kKGroups = 4;                   // position groups (interleaved pairs)
constexpr int kNHalves = 2;                   // output halves
constexpr int kWaves = kKGroups * kNHalves;   // 8
constexpr int kThreads = kWaves * 64;         // 512
constexpr int kMT = 8 / kNHalves;             // 16-output tiles per wave
constexpr int kPairsPerRow = kFm / 2;         // 22
constexpr int kRing = 8;                      // patch-row ring slots
constexpr int kPrologueRows = 2 + 5 - 1;      // rows of the first two steps
constexpr int kRP = 26;                       // LDS row pitch, dwords (24 used)
constexpr int kBigTile = 64;                  // patches per block (most blocks)
constexpr int kSmallTile = 32;                // patches per block (the last ones)
constexpr int kFrag8 = 1536;                  // bytes per (pair, output tile) fragment
constexpr int kSwapTile = 64 * 6;             // dwords per swapped patch tile

// LDS of a block of kBt patches (dwords): ring | conv filter fragments | swap
// buffers; the final reduction reuses it from the start.
template <int kBt>
struct Tile8 {
  static constexpr int kTiles = kBt / 16;
  static constexpr int kOwn = kTiles / kNHalves;
  static constexpr int kSlot = kBt * kRP;
  static constexpr int kConvOff = kRing * kSlot;
  static constexpr int kSwapOff = kConvOff + 6 * 64 * 4;
  static constexpr int kSwapWave = kOwn * kSwapTile;
  static constexpr int kSwapBuf = kWaves * kSwapWave;
  // the reduction: per output half, 3 tiles from the other groups per accumulator tile
  static constexpr int kRed = kNHalves * kMT * kTiles * (kKGroups - 1) * 4 * 64;
  static constexpr int kMain = kSwapOff + 2 * kSwapBuf;
  static constexpr int kLdsDwords = (kMain > kRed) ? kMain : kRed;
  static constexpr int kRowChunks = kBt * 6;
  static constexpr int kRowMain = kRowChunks < kThreads ? kRowChunks : kThreads;
  static constexpr int kRowExtra = kRowChunks - kRowMain;
  static_assert(kTiles % kNHalves == 0 && kOwn <= 3, "whole tiles per output half");
  static_assert(kRowMain % 64 == 0 && kRowExtra % 64 == 0 && kRowExtra <= kThreads,
                "row chunking in whole waves");
  static_assert(kLdsDwords * 4 <= 160 * 1024, "LDS of one block");
};
static_assert(Tile8<kBigTile>::kLdsDwords >= Tile8<kSmallTile>::kLdsDwords, "LDS sized by the big tile");

// Patch rows: 16 B chunks of fp16 patches; patches past the end of the batch
// read the last patch (their results are never stored).
__device__ __forceinline__ uint4 row_chunk_load(const uint16_t* __restrict__ patches, int64_t n,
                                                int64_t p_base, int r, int c) {
  typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
  const int p = c / 6, h = c - (c / 6) * 6;
  int64_t gp = p_base + p;
  gp = gp < n ? gp : n - 1;
  const uint16_t* src = patches + gp * kPatchPix + r * kPatch + h * 8;
  return __builtin_bit_cast(uint4, __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(src)));
}

template <int kBt>
__device__ __forceinline__ void row_chunk_store(uint32_t* lds, int r, int c, const uint4& v) {
  const int p = c / 6, h = c - (c / 6) * 6;
  uint32_t* d = lds + (r & (kRing - 1)) * Tile8<kBt>::kSlot + p * kRP + h * 4;
  *reinterpret_cast<uint2*>(d) = make_uint2(v.x, v.y);
  *reinterpret_cast<uint2*>(d + 2) = make_uint2(v.z, v.w);
}

template <int kBt>
__device__ __forceinline__ void row_load(const uint16_t* __restrict__ patches, int64_t n,
                                         int64_t p_base, int r, bool main, bool extra,
                                         uint4 (&v)[2]) {
  if (main) v[0] = row_chunk_load(patches, n, p_base, r, threadIdx.x);
  if (extra) v[1] = row_chunk_load(patches, n, p_base, r, threadIdx.x + kThreads);
}

template <int kBt>
__device__ __forceinline__ void row_store(uint32_t* lds, int r, bool main, bool extra,
                                          const uint4 (&v)[2]) {
  if (main) row_chunk_store<kBt>(lds, r, threadIdx.x, v[0]);
  if (extra) row_chunk_store<kBt>(lds, r, threadIdx.x + kThreads, v[1]);
}

// ReLU, clamp to the largest e4m3 value and round four fp32 values to e4m3
// (nearest even); value e in byte e.  `old` is the register's previous value:
// the two conversions overwrite its low and its high half.
__device__ __forceinline__ int to_e4m3x4(const floatx4& c, int old) {
  const float a0 = __builtin_amdgcn_fmed3f(c[0], 0.f, 448.f);
  const float a1 = __builtin_amdgcn_fmed3f(c[1], 0.f, 448.f);
  const float a2 = __builtin_amdgcn_fmed3f(c[2], 0.f, 448.f);
  const float a3 = __builtin_amdgcn_fmed3f(c[3], 0.f, 448.f);
  const int lo = __builtin_amdgcn_cvt_pk_fp8_f32(a0, a1, old, false);
  return __builtin_amdgcn_cvt_pk_fp8_f32(a2, a3, lo, true);
}

__device__ __forceinline__ floatx4 mfma8(const v8i& a, const v8i& b, const floatx4& c) {
  // operand formats 0 (e4m3) for A and B; scale exponents 127 = 2^0
  return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, b, c, 0, 0, 0, 127, 0, 127);
}

typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef int i32x2 __attribute__((ext_vector_type(2)));

// One block: patches p_base .. p_base + kBt - 1 (clamped to the batch) and
// position range `split`.
template <int kSplits, int kBt>
__device__ __forceinline__ void conv_fc1_8_block(
    uint32_t* lds, int split, int64_t p_base, const uint16_t* __restrict__ patches, int64_t n,
    const uint8_t* __restrict__ w1p, const uint4* __restrict__ convp, float* __restrict__ part,
    int64_t row0, int64_t n_total) {
  using T = Tile8<kBt>;
  constexpr int kTiles = T::kTiles, kOwn = T::kOwn, kSlot = T::kSlot;
  using Op = Op16<true>;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int kg = wave % kKGroups;
  const int nh = wave / kKGroups;
  const int partner = kg + kKGroups * (1 - nh);
  const bool rmain = wave < T::kRowMain / 64;
  const bool extra = wave < T::kRowExtra / 64;
  const int col = lane & 15;
  const int grp = lane >> 4;
  constexpr int kGroups = kPos / 2 / kKGroups;          // 242
  const int G0 = (kGroups * split) / kSplits;
  const int steps = (kGroups * (split + 1)) / kSplits - G0;
  const int P0 = kKGroups * G0;

  uint4* cwl = reinterpret_cast<uint4*>(lds + T::kConvOff);
  static_assert(6 * 64 <= kThreads, "one filter chunk per thread");
  uint32_t* swp = lds + T::kSwapOff;

  // this lane's 4 window dwords: slot pair f = 8*grp + 2d -> pixel (u, c)
  int woff[4], wrow[4];
#pragma unroll
  for (int d = 0; d < 4; ++d) {
    int f = 8 * grp + 2 * d;
    if (f > 28) f = 28;
    wrow[d] = f / 6;
    woff[d] = (f % 6) / 2 + col * kRP + nh * kOwn * 16 * kRP;
  }
  const bool const_slot = (grp == 3);

  floatx4 acc_own[kMT][kOwn], acc_oth[kMT][kOwn];
#pragma unroll
  for (int m = 0; m < kMT; ++m)
#pragma unroll
    for (int i = 0; i < kOwn; ++i) {
      acc_own[m][i] = (floatx4){0.f, 0.f, 0.f, 0.f};
      acc_oth[m][i] = (floatx4){0.f, 0.f, 0.f, 0.f};
    }

  auto top_row = [&](int step) {             // highest input row a step needs
    int pl = P0 + kKGroups * step + kKGroups - 1;
    if (pl > kPos / 2 - 1) pl = kPos / 2 - 1;
    return pl / kPairsPerRow + kK - 1;
  };
  int loaded_hi = top_row(1);
  {
    const int r0 = P0 / kPairsPerRow;
    uint4 v[kPrologueRows][2], fv;
    if (tid < 6 * 64) fv = convp[tid];
#pragma unroll
    for (int j = 0; j < kPrologueRows; ++j)
      if (r0 + j <= loaded_hi) row_load<kBt>(patches, n, p_base, r0 + j, rmain, extra, v[j]);
    if (tid < 6 * 64) cwl[tid] = fv;
#pragma unroll
    for (int j = 0; j < kPrologueRows; ++j)
      if (r0 + j <= loaded_hi) row_store<kBt>(lds, r0 + j, rmain, extra, v[j]);
  }

  // FC1 fragments of this wave's output tiles through a buffer resource:
  // reads past the end of the weights return 0
  const __amdgpu_buffer_rsrc_t w1r = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(w1p), (short)0, (int)((int64_t)(kPos / 2) * 8 * kFrag8), 0x00020000);
  // Operand tuples (weights w, the wave's own conv fragments, the partner's)
  // live across the whole loop and are updated in place in dwords 0-5, so
  // their zero dwords 6-7 are set once.
  auto load_w = [&](int P, int m, v8i& a) {
    const int base = (P * 8 + nh * kMT + m) * kFrag8;
    a.s0123 = __builtin_bit_cast(i32x4, __builtin_amdgcn_raw_buffer_load_b128(w1r, lane * 16, base, 0));
    a.s45 = __builtin_bit_cast(i32x2, __builtin_amdgcn_raw_buffer_load_b64(w1r, 1024 + lane * 8, base, 0));
  };
  const v8i zero8 = {0, 0, 0, 0, 0, 0, 0, 0};
  v8i w[kMT];
#pragma unroll
  for (int m = 0; m < kMT; ++m) {
    w[m] = zero8;
    load_w(P0 + kg, m, w[m]);
  }
  __syncthreads();

  // window of pair P (the constant slots set by fix_win)
  auto read_win_raw = [&](int P, uint4 (&win)[kOwn]) {
    const int y = P / kPairsPerRow;
    const int xh = P - y * kPairsPerRow;
    int base[4];
#pragma unroll
    for (int d = 0; d < 4; ++d) base[d] = ((y + wrow[d]) & (kRing - 1)) * kSlot + woff[d] + xh;
#pragma unroll
    for (int i = 0; i < kOwn; ++i) {
      const int o = i * 16 * kRP;
      win[i].x = lds[base[0] + o];
      win[i].y = lds[base[1] + o];
      win[i].z = lds[base[2] + o];
      win[i].w = lds[base[3] + o];
    }
  };
  auto fix_win = [&](uint4 (&win)[kOwn]) {
#pragma unroll
    for (int i = 0; i < kOwn; ++i) win[i].w = const_slot ? Op::kOnes : win[i].w;
  };
  // the conv of channel tile t (both shifts) for every own tile, rounded to
  // e4m3: dwords t and 3 + t (the prologue's conv of the first pair)
  // (the six filter fragments stay in registers for the whole block)
  uint4 filt[6];
  auto conv_t = [&](int t, const uint4 (&win)[kOwn], v8i (&nd)[kOwn]) {
    const uint4 f0 = filt[t];
    const uint4 f1 = filt[3 + t];
    const floatx4 z = {0.f, 0.f, 0.f, 0.f};
    floatx4 c0[kOwn], c1[kOwn];
#pragma unroll
    for (int i = 0; i < kOwn; ++i) {
      c0[i] = Op::mfma(f0, win[i], z);
      c1[i] = Op::mfma(f1, win[i], z);
    }
#pragma unroll
    for (int i = 0; i < kOwn; ++i) {
      nd[i][t] = to_e4m3x4(c0[i], nd[i][t]);
      nd[i][3 + t] = to_e4m3x4(c1[i], nd[i][3 + t]);
    }
  };
  // swap buffers: [buffer][wave][own tile] x (64 lanes x 16 B, then 64 lanes x 8 B)
  auto put = [&](int buf, const v8i (&nd)[kOwn]) {
#pragma unroll
    for (int i = 0; i < kOwn; ++i) {
      uint32_t* d = swp + (buf * kWaves + wave) * T::kSwapWave + i * kSwapTile;
      *reinterpret_cast<i32x4*>(d + lane * 4) = nd[i].s0123;
      *reinterpret_cast<i32x2*>(d + 256 + lane * 2) = nd[i].s45;
    }
  };
  auto get = [&](int buf, v8i (&oth)[kOwn]) {
#pragma unroll
    for (int i = 0; i < kOwn; ++i) {
      const uint32_t* s = swp + (buf * kWaves + partner) * T::kSwapWave + i * kSwapTile;
      oth[i].s0123 = *reinterpret_cast<const i32x4*>(s + lane * 4);
      oth[i].s45 = *reinterpret_cast<const i32x2*>(s + 256 + lane * 2);
    }
  };

  // prologue: the conv of the wave's first pair, published in swap buffer 0
  v8i own_a[kOwn], own_b[kOwn], oth[kOwn];
#pragma unroll
  for (int i = 0; i < kOwn; ++i) {
    own_a[i] = zero8;
    own_b[i] = zero8;
    oth[i] = zero8;
  }
#pragma unroll
  for (int j = 0; j < 6; ++j) filt[j] = cwl[j * 64 + lane];
  {
    uint4 win[kOwn];
    read_win_raw(P0 + kg, win);
    fix_win(win);
#pragma unroll
    for (int t = 0; t < 3; ++t) conv_t(t, win, own_a);
    put(0, own_a);
  }
  int buf = 0;
  __syncthreads();

  // One K step: pair P of this wave with its own fragments in `cur`; the conv
  // of its next pair goes into `nxt` and the swap buffer the partner reads in
  // the next step.
  auto step_fn = [&](int step, v8i (&cur)[kOwn], v8i (&nxt)[kOwn]) {
    uint4 rv[2];
    const int want_hi = top_row(step + 2);
    const bool new_row = want_hi > loaded_hi;
    if (new_row) row_load<kBt>(patches, n, p_base, want_hi, rmain, extra, rv);

    const int Pn = P0 + kKGroups * (step + 1) + kg;   // the wave's next pair
    uint4 win[kOwn];
    // LDS reads in the order they are needed: the partner's fragments, then
    // the next pair's window
    get(buf, oth);
    read_win_raw(Pn, win);
    // output tile m: own tiles, partner's tiles, then the fragment is reloaded
    // for the next pair; the conv of the next pair's channel tiles in between
    // (the empty asm statements keep each group of MFMAs at its place in the
    // step: their results are next used one step later, and the compiler would
    // otherwise move them all past the step's barrier, away from the conv)
    auto own_m = [&](int m) {
#pragma unroll
      for (int i = 0; i < kOwn; ++i) acc_own[m][i] = mfma8(w[m], cur[i], acc_own[m][i]);
#pragma unroll
      for (int i = 0; i < kOwn; ++i) asm volatile("" : "+v"(acc_own[m][i]));
    };
    auto oth_m = [&](int m) {
#pragma unroll
      for (int i = 0; i < kOwn; ++i) acc_oth[m][i] = mfma8(w[m], oth[i], acc_oth[m][i]);
#pragma unroll
      for (int i = 0; i < kOwn; ++i) asm volatile("" : "+v"(acc_oth[m][i]));
      load_w(Pn, m, w[m]);
    };
    // own tiles first (their operands are in registers), the partner's once
    // its fragments are back from LDS
    // the conv of the next pair in three channel tiles: each tile's MFMAs are
    // issued one FC1 group before their results are rounded, so the rounding
    // does not wait on them
    floatx4 cA[kOwn], cB[kOwn];
    const floatx4 z = {0.f, 0.f, 0.f, 0.f};
    auto conv_issue = [&](int t) {
#pragma unroll
      for (int i = 0; i < kOwn; ++i) {
        cA[i] = Op::mfma(filt[t], win[i], z);
        cB[i] = Op::mfma(filt[3 + t], win[i], z);
      }
    };
    auto conv_quant = [&](int t) {
#pragma unroll
      for (int i = 0; i < kOwn; ++i) {
        nxt[i][t] = to_e4m3x4(cA[i], nxt[i][t]);
        nxt[i][3 + t] = to_e4m3x4(cB[i], nxt[i][3 + t]);
      }
    };
    // Wave priorities stepped down through the step: the two waves of a SIMD
    // run the same sequence, and the arbiter favours the older one, so without
    // this the younger one finished each step about a quarter of a step later
    // (alone on the SIMD, its conversions no longer hidden behind MFMAs);
    // a wave past a checkpoint yields to one that has not reached it.
    __builtin_amdgcn_s_setprio(3);
    own_m(0);
    __builtin_amdgcn_sched_barrier(0);
    fix_win(win);
    conv_issue(0);
    __builtin_amdgcn_sched_barrier(0);
    own_m(1);
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_setprio(2);
    conv_quant(0);
    conv_issue(1);
    __builtin_amdgcn_sched_barrier(0);
    oth_m(0);
    __builtin_amdgcn_sched_barrier(0);
    own_m(2);
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_setprio(1);
    conv_quant(1);
    conv_issue(2);
    __builtin_amdgcn_sched_barrier(0);
    oth_m(1);
    __builtin_amdgcn_sched_barrier(0);
    own_m(3);
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_setprio(0);
    conv_quant(2);
    __builtin_amdgcn_sched_barrier(0);
    oth_m(2);
    __builtin_amdgcn_sched_barrier(0);
    oth_m(3);
    __builtin_amdgcn_sched_barrier(0);
    put(buf ^ 1, nxt);
    // the slot a new row overwrites held a row below every row any wave still
    // reads; the barrier publishes it before the step that first needs it
    if (new_row) {
      row_store<kBt>(lds, want_hi, rmain, extra, rv);
      loaded_hi = want_hi;
    }
    buf ^= 1;
    __syncthreads();
  };
  // two steps per iteration, so the own fragments alternate between two sets
  // of registers instead of being copied
  int step = 0;
#pragma unroll 1
  for (; step + 1 < steps; step += 2) {
    step_fn(step, own_a, own_b);
    step_fn(step + 1, own_b, own_a);
  }
  if (step < steps) step_fn(step, own_a, own_b);

  // ---- fixed-order reduction over position groups, per output half:
  //      (g0 + g2) + (g1 + g3), finished by one wave per accumulator tile.
  // The four waves of an output half hold the same tiles; position group g
  // finishes the g-th quarter of them, so after one barrier every wave adds
  // and stores its own quarter.
  constexpr int kSlots = kMT * kTiles;
  constexpr int kPer = kSlots / kKGroups;
  static_assert(kSlots % kKGroups == 0, "whole quarters");
  floatx4* red = reinterpret_cast<floatx4*>(lds);
  auto entry = [&](int q, int src) { return ((nh * kSlots + q) * (kKGroups - 1) + src) * 64 + lane; };
  auto tile = [&](auto qc) -> floatx4& {
    constexpr int q = decltype(qc)::value, m = q / kTiles, j = q % kTiles;
    if constexpr (j < kOwn) return acc_own[m][j];
    else return acc_oth[m][j - kOwn];
  };
  static_for<kSlots>([&](auto qc) {
    constexpr int o = decltype(qc)::value / kPer;
    if (kg != o) red[entry(decltype(qc)::value, kg - (kg > o ? 1 : 0))] = tile(qc);
  });
  __syncthreads();

  // tile q = m * kTiles + j: outputs 16(nh*kMT + m) + 4*grp + e for patch
  // 16*(block tile) + col, the block tile nh*kOwn + j (own) or
  // (1-nh)*kOwn + j - kOwn (partner's)
  float* dst = part + ((int64_t)split * n_total + row0 + p_base) * kFc1Out;
  static_for<kSlots>([&](auto qc) {
    constexpr int q = decltype(qc)::value, o = q / kPer, m = q / kTiles, j = q % kTiles;
    if (kg == o) {
      floatx4 v[kKGroups];
#pragma unroll
      for (int g = 0; g < kKGroups; ++g)
        v[g] = (g == o) ? tile(qc) : red[entry(q, g - (g > o ? 1 : 0))];
      const floatx4 sum = (v[0] + v[2]) + (v[1] + v[3]);
      const int64_t pt = (int64_t)((j < kOwn) ? nh * kOwn + j : (1 - nh) * kOwn + (j - kOwn)) * 16 + col;
      const int out = 16 * (nh * kMT + m) + 4 * grp;
      if (p_base + pt < n) __builtin_nontemporal_store(sum, reinterpret_cast<floatx4*>(dst + pt * kFc1Out + out));
    }
  });
}

// Tiles t < n_big hold kBigTile patches; the ones after them kSmallTile.  A
// patch's sums do not depend on the size of the tile it is in.
template <int kSplits>
__global__ __launch_bounds__(kThreads, 1) void conv_fc1_8_kernel(
    const uint16_t* __restrict__ patches, int64_t n, int64_t n_big, const uint8_t* __restrict__ w1p,
    const uint4* __restrict__ convp, float* __restrict__ part, int64_t row0, int64_t n_total) {
  __shared__ __attribute__((aligned(16))) uint32_t lds[Tile8<kBigTile>::kLdsDwords];
  const int split = blockIdx.x % kSplits;
  const int64_t t = blockIdx.x / kSplits;
  if (t < n_big)
    conv_fc1_8_block<kSplits, kBigTile>(lds, split, t * kBigTile, patches, n, w1p, convp, part,
                                        row0, n_total);
  else
    conv_fc1_8_block<kSplits, kSmallTile>(lds, split, n_big * kBigTile + (t - n_big) * kSmallTile,
                                          patches, n, w1p, convp, part, row0, n_total);
}

constexpr int kSplits8 = 8;

}  // namespace

int conv_fc1_8_splits() { return kSplits8; }

// As for the fp16 kernel: big tiles fill whole rounds of the CUs; the rest is
// cut into small tiles when they fit in one round.
void conv_fc1_8_tiles(int64_t n, int cus, int64_t* n_big, int64_t* n_small) {
  const int64_t per_round = cus >= kSplits8 ? cus / kSplits8 : 1;
  int64_t big = n / (kBigTile * per_round) * per_round;
  const int64_t rest = n - big * kBigTile;
  int64_t small = (rest + kSmallTile - 1) / kSmallTile;
  if (small > per_round) {
    big += (rest + kBigTile - 1) / kBigTile;
    small = 0;
  }
  *n_big = big;
  *n_small = small;
}

hipError_t launch_conv_fc1_8(const uint16_t* patches, int64_t n, int64_t row0, int64_t n_total,
                             const uint8_t* w1p, const uint4* convp, float* part, hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  int dev = 0, cus = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return e;
  int64_t n_big = 0, n_small = 0;
  conv_fc1_8_tiles(n, cus, &n_big, &n_small);
  const dim3 grid((unsigned)((n_big + n_small) * kSplits8));
  return launch_kernel(conv_fc1_8_kernel<kSplits8>, grid, dim3(kThreads), 0, stream, patches, n,
                       n_big, w1p, convp, part, row0, n_total);
}

}  // namespace pointid
