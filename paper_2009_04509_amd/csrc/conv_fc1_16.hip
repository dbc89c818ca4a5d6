// Fused conv 5x5 (1->48) + ReLU + FC1 (92928->128) on 16-bit MFMA (paper §2.2),
// with bf16 or fp16 operands and fp32 accumulation.
//
// FC1 is a skinny, very deep GEMM (M = patches, N = 128, K = 92,928) whose A
// operand — the conv maps, 185,856 B per patch in 16 bits — would cost twice its
// size in HBM traffic if written out and read back.  Here the conv is FC1's
// operand producer: the maps exist only in registers.
//
// Work split.  A block owns 96 patches (64 in the blocks of the last rounds of
// some batches: see conv_fc1_16_tiles; small batches run the thin tiles
// further below, with the same sums) and one of kSplits contiguous ranges of
// map positions (split-K); blockIdx % 8 selects the range, so every block on one
// XCD reads the same 1/8 of the FC1 weights and that slice (2.97 MB) stays in
// the XCD's 4 MB L2.  Positions are taken in pairs (x, x+1) with x even: the
// 5x6 pixel window of a pair (30 values) fits one K=32 MFMA operand, shared by
// both positions.  The block's 8 waves (2 per SIMD, so one wave's conversions
// overlap the other's MFMAs) form 4 position groups x 2 output halves.  The two
// waves of a group take the same interleaved pairs; each computes the conv of
// half of the 96 patches, and the pair swaps the converted 16-bit fragments
// through LDS (double-buffered, one block barrier per K-step), so the conv is
// computed once and each wave streams only the FC1 weights of its 64 outputs:
// every weight fragment fetched through L1 feeds 6 MFMAs.  LDS also holds a
// ring of 8 patch rows (the 5 rows a map row needs, plus those prefetched two
// steps ahead) for the block's 96 patches, and the conv filter fragments.
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
constexpr int kPairsPerRow = kFm / 2;         // 22
constexpr int kRing = 8;                      // patch-row ring slots
// rows the first two steps of a split need: pairs P0 .. P0 + 2 kKGroups - 1 span
// at most two map rows, plus the filter height
constexpr int kPrologueRows = 2 + 5 - 1;
constexpr int kRP = 26;                       // LDS row pitch, dwords (24 used)
constexpr int kBigTile = 96;                  // patches per block (most blocks)
constexpr int kMidTile = 64;                  // patches per block (the last rounds, some batches)

// Layout of a block of kBt patches.  LDS (dwords): ring | conv filter
// fragments | swap buffers; the final reduction reuses it from the start.
// A patch row (96 B) of each of the block's patches is kBt x 6 chunks of 16 B:
// chunk c = tid for the first kRowMain threads, plus c = kThreads + tid for
// the first kRowExtra threads (whole waves, so no lane diverges).
template <int kBt>
struct Tile {
  static constexpr int kTiles = kBt / 16;                 // 16-patch MFMA tiles
  static constexpr int kOwn = kTiles / kNHalves;          // tiles whose conv a wave computes
  static constexpr int kSlot = kBt * kRP;                 // dwords per ring slot
  static constexpr int kConvOff = kRing * kSlot;
  static constexpr int kSwapOff = kConvOff + 6 * 64 * 4;
  static constexpr int kSwapWave = kOwn * 64 * 4;         // one wave's fragments
  static constexpr int kSwapBuf = kWaves * kSwapWave;     // one buffer
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
};
static_assert(Tile<kBigTile>::kLdsDwords >= Tile<kMidTile>::kLdsDwords, "LDS sized by the big tile");

// Patches past the end of the batch are read from the last patch instead:
// their results are never stored.  `In` is the patches' element type: 16-bit
// bit patterns (from the gather or the cast), or fp32 pre-cut patches rounded
// here, on the way into LDS, with the same round-to-nearest-even as the cast.
template <int kBt, bool kFp16, class In>
__device__ __forceinline__ uint4 row_chunk_load(const In* __restrict__ patches, int64_t n,
                                                int64_t p_base, int r, int c) {
  typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
  const int p = c / 6, h = c - (c / 6) * 6;
  int64_t gp = p_base + p;
  gp = gp < n ? gp : n - 1;
  // streamed once per block: non-temporal, so it does not push the block's FC1
  // weight slice out of L2
  const In* src = patches + gp * kPatchPix + r * kPatch + h * 8;
  if constexpr (sizeof(In) == 2) {
    return __builtin_bit_cast(uint4, __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(src)));
  } else {
    typedef float f32x4 __attribute__((ext_vector_type(4)));
    const f32x4 a = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(src));
    const f32x4 b = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(src) + 1);
    using Op = Op16<kFp16>;
    return make_uint4(Op::pack(a[0], a[1]), Op::pack(a[2], a[3]), Op::pack(b[0], b[1]),
                      Op::pack(b[2], b[3]));
  }
}

template <int kBt>
__device__ __forceinline__ void row_chunk_store(uint32_t* lds, int r, int c, const uint4& v) {
  const int p = c / 6, h = c - (c / 6) * 6;
  uint32_t* d = lds + (r & (kRing - 1)) * Tile<kBt>::kSlot + p * kRP + h * 4;
  *reinterpret_cast<uint2*>(d) = make_uint2(v.x, v.y);
  *reinterpret_cast<uint2*>(d + 2) = make_uint2(v.z, v.w);
}

// `main` and `extra`: wave-uniform, whether this thread has a first / second chunk
template <int kBt, bool kFp16, class In>
__device__ __forceinline__ void row_load(const In* __restrict__ patches, int64_t n,
                                         int64_t p_base, int r, bool main, bool extra,
                                         uint4 (&v)[2]) {
  if (main) v[0] = row_chunk_load<kBt, kFp16, In>(patches, n, p_base, r, threadIdx.x);
  if (extra) v[1] = row_chunk_load<kBt, kFp16, In>(patches, n, p_base, r, threadIdx.x + kThreads);
}

template <int kBt>
__device__ __forceinline__ void row_store(uint32_t* lds, int r, bool main, bool extra,
                                          const uint4 (&v)[2]) {
  if (main) row_chunk_store<kBt>(lds, r, threadIdx.x, v[0]);
  if (extra) row_chunk_store<kBt>(lds, r, threadIdx.x + kThreads, v[1]);
}

// One block: patches p_base .. p_base + kBt - 1 (clamped to the batch) and
// position range `split`.
template <bool kFp16, int kSplits, int kBt, class In>
__device__ __forceinline__ void conv_fc1_block(
    uint32_t* lds, int split, int64_t p_base,
    const In* __restrict__ patches, int64_t n, const uint4* __restrict__ w1p,
    const uint4* __restrict__ convp, float* __restrict__ part, int64_t row0, int64_t n_total) {
  using T = Tile<kBt>;
  constexpr int kTiles = T::kTiles, kOwn = T::kOwn, kSlot = T::kSlot;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int kg = wave % kKGroups;            // position group
  const int nh = wave / kKGroups;            // output half; also the half of the tiles it convolves
  const int partner = kg + kKGroups * (1 - nh);
  const bool rmain = wave < T::kRowMain / 64;   // wave-uniform
  const bool extra = wave < T::kRowExtra / 64;
  const int col = lane & 15;                 // MFMA column (patch within tile) / row
  const int grp = lane >> 4;                 // MFMA K-slot group
  // split boundaries on whole steps of kKGroups pairs: every wave runs `steps` pairs
  constexpr int kGroups = kPos / 2 / kKGroups;          // 242
  const int G0 = (kGroups * split) / kSplits;
  const int steps = (kGroups * (split + 1)) / kSplits - G0;
  const int P0 = kKGroups * G0;
  using Op = Op16<kFp16>;

  // conv filter fragments [shift][channel tile] in LDS; a K-step reads two
  // (copied below, with the first patch rows, so both loads are in flight together)
  uint4* cwl = reinterpret_cast<uint4*>(lds + T::kConvOff);
  static_assert(6 * 64 <= kThreads, "one filter chunk per thread");
  // swap buffers: [buffer][wave][own tile][lane] x 16 B
  uint4* swp = reinterpret_cast<uint4*>(lds + T::kSwapOff);

  // this lane's 4 window dwords: slot pair f = 8*grp + 2d -> pixel (u, c)
  int woff[4], wrow[4];
#pragma unroll
  for (int d = 0; d < 4; ++d) {
    int f = 8 * grp + 2 * d;
    if (f > 28) f = 28;                      // slots 30-31 are constants (masked below)
    wrow[d] = f / 6;
    woff[d] = (f % 6) / 2 + col * kRP + nh * kOwn * 16 * kRP;
  }
  const bool const_slot = (grp == 3);

  // accumulators for the wave's own conv tiles (block tiles nh*kOwn + i) and
  // for the partner's (tiles (1-nh)*kOwn + i); indexed statically only, so
  // they stay in registers
  floatx4 acc_own[kMT][kOwn], acc_oth[kMT][kOwn];
#pragma unroll
  for (int m = 0; m < kMT; ++m)
#pragma unroll
    for (int i = 0; i < kOwn; ++i) {
      acc_own[m][i] = (floatx4){0.f, 0.f, 0.f, 0.f};
      acc_oth[m][i] = (floatx4){0.f, 0.f, 0.f, 0.f};
    }

  // ---- patch rows.  The ring is filled two steps ahead of the step being
  // computed, so the window of step s+1 can be read during step s.
  auto top_row = [&](int step) {             // highest input row a step needs
    int pl = P0 + kKGroups * step + kKGroups - 1;
    if (pl > kPos / 2 - 1) pl = kPos / 2 - 1;
    return pl / kPairsPerRow + kK - 1;
  };
  // all rows in flight at once (at most kPrologueRows), then into the ring
  int loaded_hi = top_row(1);
  {
    const int r0 = P0 / kPairsPerRow;
    uint4 v[kPrologueRows][2], fv;
    if (tid < 6 * 64) fv = convp[tid];
#pragma unroll
    for (int j = 0; j < kPrologueRows; ++j)
      if (r0 + j <= loaded_hi)
        row_load<kBt, kFp16, In>(patches, n, p_base, r0 + j, rmain, extra, v[j]);
    if (tid < 6 * 64) cwl[tid] = fv;
#pragma unroll
    for (int j = 0; j < kPrologueRows; ++j)
      if (r0 + j <= loaded_hi) row_store<kBt>(lds, r0 + j, rmain, extra, v[j]);
  }
  __syncthreads();

  // window of pair P; the constant slots are set by fix_win, which the main
  // loop issues a few MFMAs later so that no VALU op waits on the LDS reads
  auto read_win_raw = [&](int P, uint4 (&win)[kOwn]) {
    const int y = P / kPairsPerRow;
    const int xh = P - y * kPairsPerRow;     // x / 2
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
  // filter fragments of K-step q: conv tiles (shift, channel tile) feeding it
  auto read_filters = [&](int q, uint4& fa, uint4& fb) {
    const int sa = (q == 2) ? 1 : 0, ta = (q == 0) ? 0 : (q == 1 ? 2 : 1);
    const int sb = (q == 0) ? 0 : 1, tb = (q == 0) ? 1 : (q == 1 ? 0 : 2);
    fa = cwl[(sa * 3 + ta) * 64 + lane];
    fb = cwl[(sb * 3 + tb) * 64 + lane];
  };
  // ReLU + round to 16 bits: a conv tile pair becomes an FC1 B operand
  auto convert1 = [&](const floatx4& ca, const floatx4& cb) {
    return make_uint4(relu2(Op::pack(ca[0], ca[1])), relu2(Op::pack(ca[2], ca[3])),
                      relu2(Op::pack(cb[0], cb[1])), relu2(Op::pack(cb[2], cb[3])));
  };
  auto put1 = [&](int buf, int i, const uint4& bf) {
    swp[((buf * kWaves + wave) * kOwn + i) * 64 + lane] = bf;
  };
  auto get_swap = [&](int buf, uint4 (&bf)[kOwn]) {
#pragma unroll
    for (int i = 0; i < kOwn; ++i) bf[i] = swp[((buf * kWaves + partner) * kOwn + i) * 64 + lane];
  };

  // FC1 fragments of this wave's outputs through a buffer resource: the
  // fragment base is a scalar offset and the output tiles are immediate
  // offsets, so the loads need no per-lane address arithmetic; reads past the
  // end return 0.
  const __amdgpu_buffer_rsrc_t w1r = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint4*>(w1p), (short)0, (int)(kFc1Frags * 16), 0x00020000);
  const int voff = lane * 16 + nh * kMT * 1024;
  auto load_one = [&](int P, int q, int m) {
    return __builtin_bit_cast(
        uint4, __builtin_amdgcn_raw_buffer_load_b128(w1r, voff + m * 1024, (P * 3 + q) * 8 * 1024, 0));
  };

  // ---- software pipeline.  Entering a K-step, this wave's own conv fragments
  // are in registers and the partner's are in swap buffer `buf` (published by
  // the last barrier).  While the FC1 MFMAs run, the conv of the next K-step is
  // issued, converted and published in the other buffer.  The FC1 weights sit
  // in a ring of 3 register sets, one per K-step of a pair (set q for K-step
  // q), each loaded two K-steps before it is used.
  uint4 w[3][kMT], win[kOwn], own[kOwn];
#pragma unroll
  for (int m = 0; m < kMT; ++m) {
    w[0][m] = load_one(P0 + kg, 0, m);
    w[1][m] = load_one(P0 + kg, 1, m);
  }
  read_win_raw(P0 + kg, win);
  fix_win(win);
  {
    uint4 fa, fb;
    read_filters(0, fa, fb);
    const floatx4 z = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int i = 0; i < kOwn; ++i) own[i] = convert1(Op::mfma(fa, win[i], z), Op::mfma(fb, win[i], z));
  }
  int buf = 0;
#pragma unroll
  for (int i = 0; i < kOwn; ++i) put1(buf, i, own[i]);
  __syncthreads();

#pragma unroll 1
  for (int step = 0; step < steps; ++step) {
    // the patch row two steps ahead (at most one per step; block-uniform)
    uint4 rv[2];
    const int want_hi = top_row(step + 2);
    const bool new_row = want_hi > loaded_hi;
    if (new_row) row_load<kBt, kFp16, In>(patches, n, p_base, want_hi, rmain, extra, rv);

    const int P = P0 + kKGroups * step + kg;
    uint4 win_next[kOwn];
#pragma unroll
    for (int q = 0; q < 3; ++q) {
      const int nq = (q + 1) % 3;            // the next K-step
      const int fq = (q + 2) % 3;            // the K-step after it
      const int fP = (q < 1) ? P : P + kKGroups;
      uint4 oth[kOwn], nxt[kOwn], fa, fb;
      floatx4 ca[kOwn], cb[kOwn];
      const floatx4 z = {0.f, 0.f, 0.f, 0.f};
      // One K-step in ten groups of 3 MFMAs, the other work spread between
      // them: the two waves sharing a SIMD run the same sequence at about the
      // same time, so neither may bunch its VALU or LDS work.  The weight
      // register set q is used by groups 0-1, 4-5 (own tiles) and 6-9
      // (partner's tiles); set fq, last used in the previous K-step, is
      // reloaded for two K-steps ahead (past the end of the weights this reads 0).
      auto own_group = [&](int m) {
#pragma unroll
        for (int i = 0; i < kOwn; ++i) acc_own[m][i] = Op::mfma(w[q][m], own[i], acc_own[m][i]);
      };
      auto oth_group = [&](int m) {
#pragma unroll
        for (int i = 0; i < kOwn; ++i) acc_oth[m][i] = Op::mfma(w[q][m], oth[i], acc_oth[m][i]);
      };
      // g0: next filters, then the partner's fragments, from LDS (LDS returns
      // in order, and the filters are needed first)
      read_filters(nq, fa, fb);
      get_swap(buf, oth);
      own_group(0);
      w[fq][0] = load_one(fP, fq, 0);
      __builtin_amdgcn_sched_barrier(0);
      own_group(1);
      w[fq][1] = load_one(fP, fq, 1);
      __builtin_amdgcn_sched_barrier(0);
      // g2, g3: conv of the next K-step
#pragma unroll
      for (int i = 0; i < kOwn; ++i) ca[i] = Op::mfma(fa, (q == 2) ? win_next[i] : win[i], z);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int i = 0; i < kOwn; ++i) cb[i] = Op::mfma(fb, (q == 2) ? win_next[i] : win[i], z);
      __builtin_amdgcn_sched_barrier(0);
      own_group(2);
      w[fq][2] = load_one(fP, fq, 2);
      if (q == 1) read_win_raw(P + kKGroups, win_next);
      __builtin_amdgcn_sched_barrier(0);
      own_group(3);
      w[fq][3] = load_one(fP, fq, 3);
      nxt[0] = convert1(ca[0], cb[0]);
      __builtin_amdgcn_sched_barrier(0);
      oth_group(0);
      if constexpr (kOwn > 1) nxt[1] = convert1(ca[1], cb[1]);
      put1(buf ^ 1, 0, nxt[0]);
      __builtin_amdgcn_sched_barrier(0);
      oth_group(1);
      if constexpr (kOwn > 2) nxt[2] = convert1(ca[2], cb[2]);
      if constexpr (kOwn > 1) put1(buf ^ 1, 1, nxt[1]);
      if (q == 1) fix_win(win_next);
      __builtin_amdgcn_sched_barrier(0);
      oth_group(2);
      if constexpr (kOwn > 2) put1(buf ^ 1, 2, nxt[2]);
      __builtin_amdgcn_sched_barrier(0);
      oth_group(3);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int i = 0; i < kOwn; ++i) own[i] = nxt[i];
      if (q == 2) {
#pragma unroll
        for (int i = 0; i < kOwn; ++i) win[i] = win_next[i];
        // The slot a new row overwrites held a row below every row that any
        // wave still reads; the barrier below publishes it before the step
        // that first needs it (two steps later).
        if (new_row) {
          row_store<kBt>(lds, want_hi, rmain, extra, rv);
          loaded_hi = want_hi;
        }
      }
      buf ^= 1;
      // publishes the next K-step's swap fragments (and a new row); the
      // buffer written next was last read before this barrier
      __syncthreads();
    }
  }

  // ---- fixed-order reduction over position groups, per output half:
  //      (g0 + g2) + (g1 + g3), finished by one wave per accumulator tile.
  // The four waves of an output half hold the same tiles (they share the
  // own/partner tile order); position group g finishes the g-th quarter of
  // them, so after one barrier every wave adds and stores its own quarter.
  // One 16 B accumulator tile per lane and access (conflict-free b128).
  constexpr int kSlots = kMT * kTiles;         // accumulator tiles of a wave
  constexpr int kPer = kSlots / kKGroups;      // tiles a wave finishes
  static_assert(kSlots % kKGroups == 0, "whole quarters");
  floatx4* red = reinterpret_cast<floatx4*>(lds);
  // slot q of output half nh, written by the src-th of the other three groups
  auto entry = [&](int q, int src) { return ((nh * kSlots + q) * (kKGroups - 1) + src) * 64 + lane; };
  auto tile = [&](auto qc) -> floatx4& {
    constexpr int q = decltype(qc)::value, m = q / kTiles, j = q % kTiles;
    if constexpr (j < kOwn) return acc_own[m][j];
    else return acc_oth[m][j - kOwn];
  };
  static_for<kSlots>([&](auto qc) {
    constexpr int o = decltype(qc)::value / kPer;     // the group that finishes it
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
      // the partials are read once, by the tail kernel: non-temporal stores keep
      // them from evicting the FC1 weight slices from L2
      if (p_base + pt < n) __builtin_nontemporal_store(sum, reinterpret_cast<floatx4*>(dst + pt * kFc1Out + out));
    }
  });
}

// Tiles t < n_big hold kBigTile patches, the ones after them kMidTile.  A
// patch's sums do not depend on the size of the tile it is in: every MFMA
// column and every reduction step is per patch.
template <bool kFp16, int kSplits, class In>
__global__ __launch_bounds__(kThreads, 1) void conv_fc1_16_kernel(
    const In* __restrict__ patches, int64_t n, int64_t n_big, const uint4* __restrict__ w1p,
    const uint4* __restrict__ convp, float* __restrict__ part, int64_t row0, int64_t n_total) {
  __shared__ __attribute__((aligned(16))) uint32_t lds[Tile<kBigTile>::kLdsDwords];
  const int split = blockIdx.x % kSplits;
  const int64_t t = blockIdx.x / kSplits;
  if (t < n_big)
    conv_fc1_block<kFp16, kSplits, kBigTile, In>(lds, split, t * kBigTile, patches, n, w1p, convp,
                                                 part, row0, n_total);
  else
    conv_fc1_block<kFp16, kSplits, kMidTile, In>(lds, split,
                                                 n_big * kBigTile + (t - n_big) * kMidTile,
                                                 patches, n, w1p, convp, part, row0, n_total);
}


// ---- Thin tiles: batches that leave most of the chip idle.  Then one block's
// K-loop is the whole call, and the barrier per K-step and the swap through
// LDS are latency, not throughput.  A thin block holds 16 or 32 patches (1 or
// 2 MFMA patch tiles) with the same 8 waves (position group x output half);
// each wave computes the conv of every tile of the block (the two output
// halves of a position group both compute it: twice the conv MFMAs, on a chip
// that is mostly idle) and feeds it to its own FC1 MFMAs, so no fragment
// crosses waves.  All input rows of the block's position range (at most 11)
// are staged in LDS once, so the loop has no barrier.  Every FC1 accumulator
// sees the same operands in the same order as in the tiles above, and the
// reduction over position groups is the same: a patch's sums are bit for bit
// those of the other tile shapes.
// With kParts = 2 or 4 the 128 FC1 outputs are shared by that many blocks
// (each wave takes 4 / kParts of the 16-output tiles): more blocks, each
// streaming a part of the position range's weights, for batches that would
// leave CUs idle; every block computes the conv.
constexpr int kThinRows = 11;                 // input rows of one position range, at most
template <int kBt, int kParts>
struct Thin {
  static constexpr int kTiles = kBt / 16;
  static constexpr int kMTw = kMT / kParts;                // 16-output tiles per wave
  static constexpr int kSlot = kBt * kRP;                  // dwords per staged row
  // the reduction: per output half, 3 tiles from the other groups per accumulator tile
  static constexpr int kRed = kNHalves * kMTw * kTiles * (kKGroups - 1) * 4 * 64;
  // one row slot more than a range needs: the loop reads the window of the
  // pair after its last one (the result is never used), which may lie one row lower
  static constexpr int kRowsDw = (kThinRows + 1) * kSlot;
  static constexpr int kLdsDwords = kRowsDw > kRed ? kRowsDw : kRed;
  static constexpr int kRowChunks = kBt * 6;               // 16 B chunks per staged row
  static constexpr int kPer = (kThinRows * kRowChunks + kThreads - 1) / kThreads;
  static_assert(kTiles >= 1 && kTiles <= 2, "1 or 2 patch tiles");
  static_assert(kParts == 1 || kParts == 2 || kParts == 4, "whole, half or quarter of the outputs");
};

// input rows a position range spans, at most, over the ranges of `splits`
constexpr int thin_rows_needed(int splits) {
  int most = 0;
  for (int s = 0; s < splits; ++s) {
    const int g0 = (kPos / 2 / kKGroups) * s / splits;
    const int g1 = (kPos / 2 / kKGroups) * (s + 1) / splits;
    const int rows = (kKGroups * g1 - 1) / kPairsPerRow + kK - (kKGroups * g0) / kPairsPerRow;
    most = rows > most ? rows : most;
  }
  return most;
}

template <bool kFp16, int kSplits, int kBt, int kParts, class In>
__device__ __forceinline__ void thin_block(
    uint32_t* lds, int split, int opart, int64_t p_base, const In* __restrict__ patches,
    int64_t n, const uint4* __restrict__ w1p, const uint4* __restrict__ convp,
    float* __restrict__ part, int64_t row0, int64_t n_total) {
  using T = Thin<kBt, kParts>;
  constexpr int kTiles = T::kTiles, kSlot = T::kSlot, kMTw = T::kMTw;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int kg = wave % kKGroups;
  const int nh = wave / kKGroups;
  const int col = lane & 15;
  const int grp = lane >> 4;
  constexpr int kGroups = kPos / 2 / kKGroups;
  const int G0 = (kGroups * split) / kSplits;
  const int steps = (kGroups * (split + 1)) / kSplits - G0;
  const int P0 = kKGroups * G0;
  const int r0 = P0 / kPairsPerRow;                        // first input row of the range
  const int nrows = (P0 + kKGroups * steps - 1) / kPairsPerRow + kK - r0;
  using Op = Op16<kFp16>;

  // ---- every input row of the range, all loads in flight together
  {
    const int total = nrows * T::kRowChunks;
    uint4 v[T::kPer];
#pragma unroll
    for (int k = 0; k < T::kPer; ++k) {
      const int c = tid + k * kThreads;
      if (c < total) {
        const int j = c / T::kRowChunks;
        v[k] = row_chunk_load<kBt, kFp16, In>(patches, n, p_base, r0 + j, c - j * T::kRowChunks);
      }
    }
#pragma unroll
    for (int k = 0; k < T::kPer; ++k) {
      const int c = tid + k * kThreads;
      if (c < total) {
        const int j = c / T::kRowChunks, cc = c - j * T::kRowChunks;
        const int p = cc / 6, h = cc - (cc / 6) * 6;
        uint32_t* d = lds + j * kSlot + p * kRP + h * 4;
        *reinterpret_cast<uint2*>(d) = make_uint2(v[k].x, v[k].y);
        *reinterpret_cast<uint2*>(d + 2) = make_uint2(v[k].z, v[k].w);
      }
    }
  }
  // the six conv filter fragments [shift][channel tile], kept in registers:
  // K-step q uses fragments 2q and 2q + 1
  uint4 filt[6];
#pragma unroll
  for (int k = 0; k < 6; ++k) filt[k] = convp[k * 64 + lane];

  int woff[4], wrow[4];
#pragma unroll
  for (int d = 0; d < 4; ++d) {
    int f = 8 * grp + 2 * d;
    if (f > 28) f = 28;                      // slots 30-31 are constants (set below)
    wrow[d] = f / 6 - r0;
    woff[d] = (f % 6) / 2 + col * kRP;
  }
  const bool const_slot = (grp == 3);
  auto read_win = [&](int P, uint4 (&win)[kTiles]) {
    const int y = P / kPairsPerRow;
    const int xh = P - y * kPairsPerRow;
    int base[4];
#pragma unroll
    for (int d = 0; d < 4; ++d) base[d] = (y + wrow[d]) * kSlot + woff[d] + xh;
#pragma unroll
    for (int i = 0; i < kTiles; ++i) {
      const int o = i * 16 * kRP;
      win[i].x = lds[base[0] + o];
      win[i].y = lds[base[1] + o];
      win[i].z = lds[base[2] + o];
      win[i].w = const_slot ? Op::kOnes : lds[base[3] + o];
    }
  };
  auto convert1 = [&](const floatx4& ca, const floatx4& cb) {
    return make_uint4(relu2(Op::pack(ca[0], ca[1])), relu2(Op::pack(ca[2], ca[3])),
                      relu2(Op::pack(cb[0], cb[1])), relu2(Op::pack(cb[2], cb[3])));
  };
  const __amdgpu_buffer_rsrc_t w1r = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint4*>(w1p), (short)0, (int)(kFc1Frags * 16), 0x00020000);
  const int ot0 = (opart * kNHalves + nh) * kMTw;           // the wave's first output tile
  const int voff = lane * 16 + ot0 * 1024;
  auto load_one = [&](int P, int q, int m) {
    return __builtin_bit_cast(
        uint4, __builtin_amdgcn_raw_buffer_load_b128(w1r, voff + m * 1024, (P * 3 + q) * 8 * 1024, 0));
  };

  floatx4 acc[kMTw][kTiles];
#pragma unroll
  for (int m = 0; m < kMTw; ++m)
#pragma unroll
    for (int i = 0; i < kTiles; ++i) acc[m][i] = (floatx4){0.f, 0.f, 0.f, 0.f};
  // FC1 weights: 3 register sets, set q for K-step q of a pair, each reloaded
  // for the next pair as soon as its MFMAs have issued (three K-steps ahead:
  // with one or two patch tiles a K-step is short)
  uint4 w[3][kMTw], win[kTiles], own[kTiles];
#pragma unroll
  for (int m = 0; m < kMTw; ++m) {
    w[0][m] = load_one(P0 + kg, 0, m);
    w[1][m] = load_one(P0 + kg, 1, m);
    w[2][m] = load_one(P0 + kg, 2, m);
  }
  __syncthreads();                           // the staged rows
  const floatx4 z = {0.f, 0.f, 0.f, 0.f};
  read_win(P0 + kg, win);
#pragma unroll
  for (int i = 0; i < kTiles; ++i) own[i] = convert1(Op::mfma(filt[0], win[i], z), Op::mfma(filt[1], win[i], z));

#pragma unroll 1
  for (int step = 0; step < steps; ++step) {
    const int P = P0 + kKGroups * step + kg;
    uint4 win_next[kTiles];
#pragma unroll
    for (int q = 0; q < 3; ++q) {
      const int nq = (q + 1) % 3;            // the next K-step
      // FC1 of K-step q (past the end of the weights the reload reads 0)
#pragma unroll
      for (int m = 0; m < kMTw; ++m) {
#pragma unroll
        for (int i = 0; i < kTiles; ++i) acc[m][i] = Op::mfma(w[q][m], own[i], acc[m][i]);
        w[q][m] = load_one(P + kKGroups, q, m);
      }
      // conv of the next K-step (its window: this pair's, or the next pair's
      // after the last K-step)
      if (q == 1) read_win(P + kKGroups, win_next);
#pragma unroll
      for (int i = 0; i < kTiles; ++i) {
        const uint4& wi = (q == 2) ? win_next[i] : win[i];
        own[i] = convert1(Op::mfma(filt[2 * nq], wi, z), Op::mfma(filt[2 * nq + 1], wi, z));
      }
      if (q == 2) {
#pragma unroll
        for (int i = 0; i < kTiles; ++i) win[i] = win_next[i];
      }
    }
  }

  // ---- the fixed-order reduction of the tiles above: (g0 + g2) + (g1 + g3),
  // each position group finishing a quarter of its output half's tiles, as in
  // the tiles above (with 2 tiles per half groups 0 and 2 finish one each,
  // with 1 group 0 finishes it)
  __syncthreads();                           // every wave is done with the rows
  constexpr int kSlots = kMTw * kTiles;
  static_assert(kSlots % kKGroups == 0 || kKGroups % kSlots == 0, "tiles spread evenly");
  // the position group that finishes slot q
  constexpr auto owner = [](int q) {
    return kSlots >= kKGroups ? q / (kSlots / kKGroups) : q * (kKGroups / kSlots);
  };
  floatx4* red = reinterpret_cast<floatx4*>(lds);
  auto entry = [&](int q, int src) { return ((nh * kSlots + q) * (kKGroups - 1) + src) * 64 + lane; };
  auto tile = [&](auto qc) -> floatx4& {
    constexpr int q = decltype(qc)::value;
    return acc[q / kTiles][q % kTiles];
  };
  static_for<kSlots>([&](auto qc) {
    constexpr int o = owner(decltype(qc)::value);
    if (kg != o) red[entry(decltype(qc)::value, kg - (kg > o ? 1 : 0))] = tile(qc);
  });
  __syncthreads();

  float* dst = part + ((int64_t)split * n_total + row0 + p_base) * kFc1Out;
  static_for<kSlots>([&](auto qc) {
    constexpr int q = decltype(qc)::value, o = owner(q), m = q / kTiles, i = q % kTiles;
    if (kg == o) {
      floatx4 v[kKGroups];
#pragma unroll
      for (int g = 0; g < kKGroups; ++g)
        v[g] = (g == o) ? tile(qc) : red[entry(q, g - (g > o ? 1 : 0))];
      const floatx4 sum = (v[0] + v[2]) + (v[1] + v[3]);
      const int64_t po = (int64_t)i * 16 + col;
      const int out = 16 * (ot0 + m) + 4 * grp;
      if (p_base + po < n)
        __builtin_nontemporal_store(sum, reinterpret_cast<floatx4*>(dst + po * kFc1Out + out));
    }
  });
}

// Block b: split b % kSplits, then output part, then patch tile.
template <bool kFp16, int kSplits, int kBt, int kParts, class In>
__global__ __launch_bounds__(kThreads, 1) void conv_fc1_16_thin_kernel(
    const In* __restrict__ patches, int64_t n, const uint4* __restrict__ w1p,
    const uint4* __restrict__ convp, float* __restrict__ part, int64_t row0, int64_t n_total) {
  static_assert(thin_rows_needed(kSplits) <= kThinRows, "a position range's rows fit the stage");
  __shared__ __attribute__((aligned(16))) uint32_t lds[Thin<kBt, kParts>::kLdsDwords];
  const int split = blockIdx.x % kSplits;
  const int64_t r = blockIdx.x / kSplits;
  const int opart = (int)(r % kParts);
  const int64_t t = r / kParts;
  thin_block<kFp16, kSplits, kBt, kParts, In>(lds, split, opart, t * kBt, patches, n, w1p, convp,
                                              part, row0, n_total);
}

constexpr int kSplits16 = 8;

}  // namespace

int conv_fc1_16_splits() { return kSplits16; }

// One block per CU and (tile, split), so a round of the CUs holds `per_round`
// tiles.  Whole rounds of big tiles, then the rest as rounds of mid tiles or
// of big tiles, whichever ends first by the relative round time of mid
// tiles (a 64-patch block takes about 0.72 of a 96-patch block's time: its
// weight fragments feed 4 MFMAs instead of 6).  Giving up one or two rounds
// of big tiles for rounds of mid tiles often ends sooner than a last, partly
// filled round of big tiles (B = 16,384: 4 rounds of 96 and 2 of 64 = 5.44
// against 6 rounds of 96).  (A last round of 32-patch tiles, at about 0.55 of
// a big round, never beats two rounds of mid tiles after one big round fewer;
// batches of at most one round of 32-patch tiles run thin tiles.)
void conv_fc1_16_tiles(int64_t n, int cus, int64_t* n_big, int64_t* n_mid) {
  constexpr double kRoundMid = 0.72;
  const int64_t per_round = cus >= kSplits16 ? cus / kSplits16 : 1;   // tiles per round
  const int64_t full = n / (kBigTile * per_round);
  auto rounds = [&](int64_t tiles) { return (tiles + per_round - 1) / per_round; };
  double best = 0.0;
  bool have = false;
  for (int64_t r = full; r >= 0 && r >= full - 2; --r) {
    const int64_t big = r * per_round;
    const int64_t rest = n - big * kBigTile;
    const int64_t t_mid = (rest + kMidTile - 1) / kMidTile;
    const int64_t t_big = (rest + kBigTile - 1) / kBigTile;
    auto consider = [&](double cost, int64_t b, int64_t m) {
      if (have && !(cost < best - 1e-9)) return;
      have = true;
      best = cost;
      *n_big = b;
      *n_mid = m;
    };
    consider(r + kRoundMid * (double)rounds(t_mid), big, t_mid);
    consider(r + (double)rounds(t_big), big + t_big, 0);
  }
}

// Thin tiles (16 or 32 patches) when the batch in them fills at most one
// round of the CUs: the call is then one block's K-loop long.  0: the tiles above.
int conv_fc1_16_thin_tile(int64_t n, int cus) {
  const int64_t per_round = cus >= kSplits16 ? cus / kSplits16 : 1;   // tiles per round
  if (n <= 16 * per_round) return 16;
  if (n <= 32 * per_round) return 32;
  return 0;
}

// Output parts of a 16-patch thin tile: the most (4, 2 or 1) whose blocks
// still fit one round of the CUs.  (Two blocks per CU were slower than one
// block with all the outputs: 512 patches 54.5 against 51.5 us per call,
// 1,024 in 32-patch tiles 71.6 against 60.9 us.)
int conv_fc1_16_thin_parts(int64_t n, int cus, int thin) {
  if (thin != 16) return 1;
  const int64_t blocks = (n + thin - 1) / thin * kSplits16;
  if (4 * blocks <= cus) return 4;
  return 2 * blocks <= cus ? 2 : 1;
}

template <bool kFp16, class In>
hipError_t launch_typed(const In* patches, int64_t n, int64_t row0, int64_t n_total,
                        const uint4* w1p, const uint4* convp, float* part, hipStream_t stream) {
  int dev = 0, cus = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return e;
  const int thin = conv_fc1_16_thin_tile(n, cus);
  if (thin) {
    const int parts = conv_fc1_16_thin_parts(n, cus, thin);
    const dim3 grid((unsigned)((n + thin - 1) / thin * kSplits16 * parts));
    auto go = [&](auto kernel) {
      return launch_kernel(kernel, grid, dim3(kThreads), 0, stream, patches, n, w1p, convp, part,
                           row0, n_total);
    };
    if (thin == 32) return go(conv_fc1_16_thin_kernel<kFp16, kSplits16, 32, 1, In>);
    if (parts == 4) return go(conv_fc1_16_thin_kernel<kFp16, kSplits16, 16, 4, In>);
    return parts == 2 ? go(conv_fc1_16_thin_kernel<kFp16, kSplits16, 16, 2, In>)
                      : go(conv_fc1_16_thin_kernel<kFp16, kSplits16, 16, 1, In>);
  }
  int64_t n_big = 0, n_mid = 0;
  conv_fc1_16_tiles(n, cus, &n_big, &n_mid);
  const dim3 grid((unsigned)((n_big + n_mid) * kSplits16));
  return launch_kernel(conv_fc1_16_kernel<kFp16, kSplits16, In>, grid, dim3(kThreads), 0, stream,
                       patches, n, n_big, w1p, convp, part, row0, n_total);
}

hipError_t launch_conv_fc1_16(bool fp16, const void* patches, bool f32_in, int64_t n, int64_t row0,
                              int64_t n_total, const uint4* w1p, const uint4* convp,
                              float* part, hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  if (f32_in) {
    const float* p = static_cast<const float*>(patches);
    return fp16 ? launch_typed<true>(p, n, row0, n_total, w1p, convp, part, stream)
                : launch_typed<false>(p, n, row0, n_total, w1p, convp, part, stream);
  }
  const uint16_t* p = static_cast<const uint16_t*>(patches);
  return fp16 ? launch_typed<true>(p, n, row0, n_total, w1p, convp, part, stream)
              : launch_typed<false>(p, n, row0, n_total, w1p, convp, part, stream);
}

}  // namespace pointid
