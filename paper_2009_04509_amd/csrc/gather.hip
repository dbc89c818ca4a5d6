// Patch construction (paper §2.1): for hit (w, t) the 48x48 patch
// P[r][c] = image[w - 24 + r][t - 24 + c], zero outside the plane.
//
// One wavefront builds one patch; each lane writes whole 16-byte output chunks
// (4 fp32 or 8 bf16/fp16 pixels of one patch row), so a wavefront writes 1 KiB
// of contiguous output per store.  A chunk's pixels are read as the aligned
// 16-byte words that cover them (the run starts 0-3 floats into the first
// word) and shifted into place in registers: no LDS, no barrier.  A lane
// issues the loads of all its chunks before it shifts any (78 VGPRs, 6 waves
// per SIMD): with the loads of only two chunks in flight, as the compiler
// schedules them at 8 waves per SIMD, waves spent most of their time waiting.  The loads go through a buffer resource
// that starts at the image's 16-byte-aligned base and ends with the image, so
// a word outside it reads as 0; words partly outside a row hold pixels of the
// neighbouring row (or bytes just outside the image, in the same 16-byte
// block), and every pixel whose wire or tick is outside the plane is set to 0
// after the load.  Planes of 2 GiB or more take a per-pixel path instead.
// Values are copied, never computed (bf16 / fp16 output is the
// round-to-nearest-even of the fp32 pixel), so the result is bit-exact.
#include "pointid.h"
#include "internal.h"
#include "op16.h"

namespace pointid {
namespace {

constexpr int kWaves = 4;                 // patches per block (one per wave)

// Hit i of a hit array: (wire, tick) on plane 0 (stride 2) or (plane, wire,
// tick); with `div` ticks per image column the tick becomes its column,
// floor(tick / div).
struct HitArray {
  const int32_t* hits;
  int stride;
  int div;
  __device__ void get(int64_t i, int& plane, int& w, int& t) const {
    const int32_t* h = hits + i * stride;
    if (stride == 3) {
      plane = h[0];
      w = h[1];
      t = h[2];
    } else {
      plane = 0;
      w = h[0];
      t = h[1];
    }
    if (div > 1) {
      const int q = t / div;
      t = (q * div != t && t < 0) ? q - 1 : q;
    }
  }
};

// Hit i of a batch of requests: request r holds patches start[r] .. start[r+1]-1
// (i is wave-uniform, so the search runs on scalar registers).
struct RequestHits {
  RequestTable tab;
  __device__ void get(int64_t i, int& plane, int& w, int& t) const {
    int lo = 0, hi = tab.n - 1;              // the last request starting at or before i
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (tab.start[mid] <= i) lo = mid;
      else hi = mid - 1;
    }
    const int64_t j = i - tab.start[lo];
    if (tab.plane[lo] >= 0) {
      const int32_t* h = tab.hits[lo] + 2 * j;
      plane = tab.plane[lo];
      w = h[0];
      t = h[1];
    } else {
      const int32_t* h = tab.hits[lo] + 3 * j;
      plane = h[0];
      w = h[1];
      t = h[2];
    }
  }
};

// Blocks are dispatched round-robin over the 8 XCDs (block b to XCD b % 8).
// Logical block order: the blocks one XCD runs take consecutive patches, so
// hits that arrive in wire order share their windows' image lines in that
// XCD's L2.  A bijection of [0, nb).
__device__ __forceinline__ int64_t xcd_major_block(int64_t b, int64_t nb) {
  const int64_t x = b % 8, s = b / 8;
  const int64_t q = nb / 8, r = nb % 8;
  return x * q + (x < r ? x : r) + s;
}

template <int kOut, class Src>
__global__ __launch_bounds__(256) void gather_kernel(PlaneTable planes, Src src, int64_t n,
                                                     void* __restrict__ out) {
  constexpr int kPix = (kOut == POINTID_FP32) ? 4 : 8;   // pixels per 16-byte chunk
  constexpr int kPerRow = kPatch / kPix;                 // chunks per patch row
  constexpr int kChunks = kPatch * kPerRow;              // chunks per patch
  constexpr int kIter = (kChunks + 63) / 64;
  constexpr int kLoads = kPix / 4;                       // 16-byte loads of a chunk
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int64_t i = xcd_major_block(blockIdx.x, gridDim.x) * kWaves + wave;
  if (i >= n) return;                                    // wave-uniform

  int plane = 0, w = 0, t = 0;
  src.get(i, plane, w, t);
  // one patch per wave: the hit is wave-uniform, so plane lookups are scalar
  plane = __builtin_amdgcn_readfirstlane(plane);
  w = __builtin_amdgcn_readfirstlane(w);
  t = __builtin_amdgcn_readfirstlane(t);
  const bool plane_ok = plane >= 0 && plane < planes.n;
  const float* img = plane_ok ? planes.p[plane].image : nullptr;
  const int64_t W = plane_ok ? planes.p[plane].n_wires : 0;
  const int64_t T = plane_ok ? planes.p[plane].n_ticks : 1;
  const uint64_t base = reinterpret_cast<uint64_t>(img) & ~uint64_t(15);
  const uint64_t lead = reinterpret_cast<uint64_t>(img) - base;       // 0, 4, 8 or 12
  const uint64_t span = lead + 4 * (uint64_t)W * (uint64_t)T;         // bytes base .. image end
  const bool small = span < (uint64_t(1) << 31);                      // wave-uniform

  uint4* o = reinterpret_cast<uint4*>(static_cast<char*>(out) +
                                      i * kPatchPix * (kOut == POINTID_FP32 ? 4 : 2));
  auto emit = [&](int k, const float (&v)[kPix]) {
    if (k >= kChunks) return;
    if constexpr (kOut == POINTID_FP32) {
      o[k] = make_uint4(__float_as_uint(v[0]), __float_as_uint(v[1]), __float_as_uint(v[2]),
                        __float_as_uint(v[3]));
    } else {
      using Op = Op16<kOut == POINTID_FP16>;
      o[k] = make_uint4(Op::pack(v[0], v[1]), Op::pack(v[2], v[3]), Op::pack(v[4], v[5]),
                        Op::pack(v[6], v[7]));
    }
  };
  if (small) {
    const __amdgpu_buffer_rsrc_t rsrc = __builtin_amdgcn_make_buffer_rsrc(
        reinterpret_cast<void*>(base), (short)0, (int)span, 0x00020000);
    // every load of the wave first (all in flight together): a chunk's
    // pixels are kPix consecutive floats at a 4-byte aligned offset, read as
    // kPix / 4 16-byte loads at that offset when they lie inside the image
    floatx4 q[kIter][kLoads];
    bool inside[kIter];
#pragma unroll
    for (int it = 0; it < kIter; ++it) {
      const int k = lane + 64 * it;
      const int r = k / kPerRow, hc = k - (k / kPerRow) * kPerRow;
      const int64_t wire = (int64_t)w - kHalf + r;
      const int64_t tick0 = (int64_t)t - kHalf + kPix * hc;
      const bool row_ok = k < kChunks && wire >= 0 && wire < W;
      // byte offset of the chunk's first pixel from `base`
      const int64_t rel = (int64_t)lead + 4 * (wire * T + tick0);
      inside[it] = row_ok && rel >= 0 && rel + 4 * kPix <= (int64_t)span;
      // offsets are taken mod 2^32: every offset at or past 2^31 is out of range
      const uint32_t a0 = inside[it] ? (uint32_t)rel : 0x80000000u;
#pragma unroll
      for (int j = 0; j < kLoads; ++j)
        q[it][j] = __builtin_bit_cast(
            floatx4, __builtin_amdgcn_raw_buffer_load_b128(rsrc, a0 + 16u * j, 0, 0));
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int it = 0; it < kIter; ++it) {
      const int k = lane + 64 * it;
      const int r = k / kPerRow, hc = k - (k / kPerRow) * kPerRow;
      const int64_t wire = (int64_t)w - kHalf + r;
      const int64_t tick0 = (int64_t)t - kHalf + kPix * hc;
      const bool row_ok = k < kChunks && wire >= 0 && wire < W;
      // columns j_lo <= j < j_hi of the chunk are inside the row
      const int64_t lo64 = -tick0, hi64 = T - tick0;
      const int j_lo = row_ok ? (int)(lo64 < 0 ? 0 : (lo64 > kPix ? kPix : lo64)) : kPix;
      const int j_hi = (int)(hi64 < 0 ? 0 : (hi64 > kPix ? kPix : hi64));
      float v[kPix];
#pragma unroll
      for (int j = 0; j < kPix; ++j) v[j] = (j >= j_lo && j < j_hi) ? q[it][j / 4][j % 4] : 0.f;
      if (row_ok && !inside[it]) {
        // a chunk over the first or last bytes of the image: pixel by pixel
#pragma unroll
        for (int j = 0; j < kPix; ++j) v[j] = (j >= j_lo && j < j_hi) ? img[wire * T + tick0 + j] : 0.f;
      }
      emit(k, v);
    }
  } else {
#pragma unroll 1
    for (int it = 0; it < kIter; ++it) {
      const int k = lane + 64 * it;
      const int r = k / kPerRow, hc = k - (k / kPerRow) * kPerRow;
      const int64_t wire = (int64_t)w - kHalf + r;
      const int64_t tick0 = (int64_t)t - kHalf + kPix * hc;
      const bool row_ok = k < kChunks && wire >= 0 && wire < W;
      float v[kPix];
#pragma unroll
      for (int j = 0; j < kPix; ++j) {
        const int64_t tk = tick0 + j;
        v[j] = (row_ok && tk >= 0 && tk < T) ? img[wire * T + tk] : 0.f;
      }
      emit(k, v);
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

// Columns of D ticks (paper §2.1: a pixel holds the charge its wire collects in
// the time interval of its column): out[w][j] is the charge of the interval,
// the sum of in[w][jD + k] over the ticks k < D that exist (missing ticks
// count as 0), accumulated in fp64 in tick order and rounded to fp32 once.  blockIdx.z is the plane, blockIdx.y strides over wires, and the
// lanes of a block take consecutive columns, so a wave's loads of one k cover
// consecutive memory.
// kVec4: D is a multiple of 4 and every row starts 16-byte aligned, so a
// column is D / 4 whole 16-byte words and lanes read them as such.
template <bool kVec4>
__global__ __launch_bounds__(256) void bin_ticks_kernel(PlaneTable in, PlaneTable out, int D) {
  const int p = blockIdx.z;
  const int64_t T = in.p[p].n_ticks;
  const int64_t J = out.p[p].n_ticks;
  const int64_t W = in.p[p].n_wires;
  const int64_t j = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (j >= J) return;
  const int n = (int)(T - j * D < D ? T - j * D : D);
  float* o = const_cast<float*>(out.p[p].image);
  // kWires wires per pass, their loads in flight together (4 with float4
  // loads: 63 against 72 us on the event at D = 4; the scalar loads of other
  // D keep one wire per pass, where four measured slower); each column's sum
  // still runs in tick order from its first tick
  constexpr int kWires = kVec4 ? 4 : 1;
  const int64_t step = gridDim.y;
  for (int64_t w0 = blockIdx.y; w0 < W; w0 += kWires * step) {
    double s[kWires];
    for (int k0 = 0; k0 < n; k0 += 8) {
      float xs[kWires][8];
#pragma unroll
      for (int g = 0; g < kWires; ++g) {
        const int64_t w = w0 + g * step;
        const float* x = in.p[p].image + (w < W ? w : W - 1) * T + j * D;
        if constexpr (kVec4) {              // n is a multiple of 4 here (T % 4 == 0)
          const float4* x4 = reinterpret_cast<const float4*>(x + k0);
          const float4 a = x4[0];
          const float4 b = k0 + 4 < n ? x4[1] : make_float4(0.f, 0.f, 0.f, 0.f);
          xs[g][0] = a.x; xs[g][1] = a.y; xs[g][2] = a.z; xs[g][3] = a.w;
          xs[g][4] = b.x; xs[g][5] = b.y; xs[g][6] = b.z; xs[g][7] = b.w;
        } else {
#pragma unroll
          for (int k = 0; k < 8; ++k) xs[g][k] = k0 + k < n ? x[k0 + k] : 0.f;
        }
      }
#pragma unroll
      for (int g = 0; g < kWires; ++g)
#pragma unroll
        for (int k = 0; k < 8; ++k)
          if (k0 + k < n) s[g] = (k0 + k == 0) ? (double)xs[g][k] : s[g] + xs[g][k];
    }
#pragma unroll
    for (int g = 0; g < kWires; ++g) {
      const int64_t w = w0 + g * step;
      if (w < W) o[w * J + j] = (float)s[g];
    }
  }
}

}  // namespace

hipError_t launch_bin_ticks(const PlaneTable& in, const PlaneTable& out, int ticks_per_column,
                            hipStream_t stream) {
  int64_t jmax = 0, wmax = 0;
  for (int i = 0; i < in.n; ++i) {
    if (out.p[i].n_ticks > jmax) jmax = out.p[i].n_ticks;
    if (in.p[i].n_wires > wmax) wmax = in.p[i].n_wires;
  }
  if (jmax <= 0 || in.n <= 0) return hipSuccess;
  bool vec4 = ticks_per_column % 4 == 0;
  for (int i = 0; i < in.n; ++i)
    vec4 = vec4 && (reinterpret_cast<uintptr_t>(in.p[i].image) & 15) == 0 && in.p[i].n_ticks % 4 == 0;
  const int64_t wy = vec4 ? (wmax + 3) / 4 : wmax;   // wires per thread and pass: 4 or 1
  const dim3 grid((unsigned)((jmax + 255) / 256), (unsigned)(wy < 65535 ? wy : 65535),
                  (unsigned)in.n);
  if (vec4) return launch_kernel(bin_ticks_kernel<true>, grid, dim3(256), 0, stream, in, out, ticks_per_column);
  return launch_kernel(bin_ticks_kernel<false>, grid, dim3(256), 0, stream, in, out, ticks_per_column);
}

hipError_t launch_patches_to_16(bool fp16, const float* in, int64_t n, uint16_t* out,
                                hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  const int64_t n8 = n * kPatchPix / 8;
  const dim3 grid((unsigned)((n8 + 255) / 256));
  const float4* src = reinterpret_cast<const float4*>(in);
  uint4* dst = reinterpret_cast<uint4*>(out);
  if (fp16) return launch_kernel(to_16_kernel<true>, grid, dim3(256), 0, stream, src, n8, dst);
  return launch_kernel(to_16_kernel<false>, grid, dim3(256), 0, stream, src, n8, dst);
}

template <class Src>
hipError_t launch_gather_src(const PlaneTable& planes, const Src& src, int64_t n, void* out,
                             int out_dtype, hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  const dim3 grid((unsigned)((n + kWaves - 1) / kWaves));
  if (out_dtype == POINTID_BF16)
    return launch_kernel(gather_kernel<POINTID_BF16, Src>, grid, dim3(256), 0, stream, planes, src, n, out);
  if (out_dtype == POINTID_FP16)
    return launch_kernel(gather_kernel<POINTID_FP16, Src>, grid, dim3(256), 0, stream, planes, src, n, out);
  return launch_kernel(gather_kernel<POINTID_FP32, Src>, grid, dim3(256), 0, stream, planes, src, n, out);
}

hipError_t launch_gather(const PlaneTable& planes, const int32_t* hits,
                         int hit_stride, int64_t n, void* out, int out_dtype,
                         hipStream_t stream, int tick_div) {
  return launch_gather_src(planes, HitArray{hits, hit_stride, tick_div}, n, out, out_dtype,
                           stream);
}

hipError_t launch_gather_requests(const PlaneTable& planes, const RequestTable& reqs, void* out,
                                  int out_dtype, hipStream_t stream) {
  if (reqs.n < 1 || reqs.n > kMaxRequests) return hipErrorInvalidValue;
  return launch_gather_src(planes, RequestHits{reqs}, reqs.start[reqs.n], out, out_dtype, stream);
}

}  // namespace pointid
