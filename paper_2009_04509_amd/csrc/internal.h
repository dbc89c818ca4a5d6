// Internal interface between the C-ABI layer (api.hip) and the HIP kernels.
// Not installed; nothing here is part of the public ABI.
#pragma once

#include <string>
#include <tuple>
#include <utility>

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include "pointid.h"

#include <cstdint>

namespace pointid {

// f(std::integral_constant<int, I>) for I = 0 .. N-1, unrolled
template <class F, int... I>
__device__ __forceinline__ void static_for_seq(F&& f, std::integer_sequence<int, I...>) {
  (f(std::integral_constant<int, I>{}), ...);
}
template <int N, class F>
__device__ __forceinline__ void static_for(F&& f) {
  static_for_seq(f, std::make_integer_sequence<int, N>{});
}

// Events the next kernel launched by this thread through launch_kernel
// attaches to its own dispatch (start: when the kernel begins, stop: when it
// ends; the library sets only `stop`, a call's completion event, which then
// needs no packet of its own on the stream).  The next launch takes both (and
// clears them); a scope that launches nothing leaves them set.
struct LaunchEvents {
  hipEvent_t start = nullptr;
  hipEvent_t stop = nullptr;
};
LaunchEvents& launch_events();    // the calling thread's

// kernel<<<grid, block, shmem, stream>>>(args...), with the calling thread's
// launch events attached when it has any.  The arguments are converted to the
// kernel's parameter types before their addresses are taken.
template <class... KArgs, class... Args>
hipError_t launch_kernel(void (*kernel)(KArgs...), dim3 grid, dim3 block, size_t shmem,
                         hipStream_t stream, Args&&... args) {
  static_assert(sizeof...(KArgs) == sizeof...(Args), "argument count");
  std::tuple<KArgs...> vals(std::forward<Args>(args)...);
  void* ptrs[sizeof...(KArgs) > 0 ? sizeof...(KArgs) : 1];
  std::apply([&](auto&... v) {
    int i = 0;
    ((ptrs[i++] = static_cast<void*>(&v)), ...);
  }, vals);
  LaunchEvents& ev = launch_events();
  hipError_t e;
  if (ev.start || ev.stop) {
    e = hipExtLaunchKernel(reinterpret_cast<const void*>(kernel), grid, block, ptrs, shmem, stream,
                           ev.start, ev.stop, 0);
    ev = LaunchEvents();
  } else {
    e = hipLaunchKernel(reinterpret_cast<const void*>(kernel), grid, block, ptrs, shmem, stream);
  }
  return e;
}

constexpr int kPatch = 48;                  // patch side (paper §2.1)
constexpr int kHalf = 24;                   // hit sits at patch pixel (24, 24)
constexpr int kK = 5;                       // filter side (paper §2.2)
constexpr int kCh = 48;                     // filters
constexpr int kFm = 44;                     // map side = 48 - 5 + 1
constexpr int kPos = kFm * kFm;             // 1936 map positions
constexpr int kFc1In = kPos * kCh;          // 92928
constexpr int kFc1Out = 128;
constexpr int kFc2Out = 32;
constexpr int kNcls = 3;
constexpr int kPatchPix = kPatch * kPatch;  // 2304
constexpr int kMaxPlanes = 64;

struct PlaneDesc {
  const float* image;
  int32_t n_wires;
  int32_t n_ticks;
};

// Passed by value as a kernel argument (64 * 16 B + 4 B, inside the 4 KiB limit).
struct PlaneTable {
  PlaneDesc p[kMaxPlanes];
  int32_t n;
};

// Device-resident parameters of one handle.  fp32 tensors are in the ABI
// layouts; packed tensors are in the layouts the MFMA kernels read.
struct DeviceWeights {
  int precision;             // POINTID_FP32 / POINTID_BF16 / POINTID_FP16 / POINTID_FP8
  const float* conv_w;       // [48][25] fp32
  const float* conv_b;       // [48]
  const float* fc1_wt;       // [128][92928] fp32, FC1 transposed (fp32 handles)
  const float* fc1_b;        // [128]
  const float* fc2_w;        // [128][32]
  const float* fc2_b;        // [32]
  const float* cls_w;        // [32][3]
  const float* cls_b;        // [3]
  const float* mic_w;        // [32]
  const float* mic_b;        // [1]
  // 16-bit handles: MFMA operand fragments (see conv_fc1_16.hip)
  const uint4* conv_frag;    // [2 shifts][3 channel tiles][64 lanes] x 8 halves
  const uint4* fc1_frag;     // [968 pairs][3 K-steps][8 output tiles][64 lanes] x 8 halves
  // 8-bit handles (see conv_fc1_8.hip): e4m3 fragments [968 pairs][8 output
  // tiles] x (64 lanes x 16 B, then 64 lanes x 8 B), and the factor 2^-k_n
  // the tail multiplies FC1 output n's sums by (nullptr on other handles)
  const uint8_t* fc1_frag8;
  const float* fc1_scale;
};

// Bytes of the 8-bit packed FC1 weights.
constexpr int64_t kFc1Frag8Bytes = (int64_t)(kPos / 2) * 8 * 1536;

// Fragment counts of the 16-bit packed weights.
constexpr int64_t kConvFrags = 2 * 3 * 64;
constexpr int64_t kFc1Frags = (int64_t)(kPos / 2) * 3 * 8 * 64;

// Patch construction.  hits: int32 rows of `hit_stride` (2 = (wire, tick) on
// plane 0, 3 = (plane, wire, tick)).  out: [n][48][48] of `out_dtype`
// (POINTID_FP32, or POINTID_BF16 / POINTID_FP16 bit patterns, RNE).  With
// tick_div > 1 the planes hold columns of tick_div ticks and a hit's tick t
// selects column floor(t / tick_div).
hipError_t launch_gather(const PlaneTable& planes, const int32_t* hits,
                         int hit_stride, int64_t n, void* out, int out_dtype,
                         hipStream_t stream, int tick_div = 1);

// Planes binned into columns of D ticks: out.p[i] is [n_wires][ceil(n_ticks / D)]
// of in.p[i] (its n_ticks holds that column count).
hipError_t launch_bin_ticks(const PlaneTable& in, const PlaneTable& out, int ticks_per_column,
                            hipStream_t stream);

// Several requests classified by one launch sequence (kernel argument, by
// value): request r owns patches start[r] .. start[r + 1] - 1 of the launch;
// its hits are (wire, tick) on plane[r] when plane[r] >= 0, else
// (plane, wire, tick); its scores go to scores[r].
constexpr int kMaxRequests = 64;
struct RequestTable {
  int64_t start[kMaxRequests + 1];
  const int32_t* hits[kMaxRequests];
  float* scores[kMaxRequests];
  int32_t plane[kMaxRequests];
  int32_t n;
};

// Gather of the hits of the requests of `reqs` into patches [start[n]][48][48].
hipError_t launch_gather_requests(const PlaneTable& planes, const RequestTable& reqs, void* out,
                                  int out_dtype, hipStream_t stream);

// Round fp32 patches [n][2304] to bf16 or fp16 (RNE) bit patterns.
hipError_t launch_patches_to_16(bool fp16, const float* in, int64_t n, uint16_t* out,
                                hipStream_t stream);

// Repack fp32 conv/FC1 weights into 16-bit MFMA fragments.
hipError_t launch_pack_16(bool fp16, const float* conv_w, const float* conv_b,
                          const float* fc1_w, uint4* conv_frag, uint4* fc1_frag,
                          hipStream_t stream);

// The fp16 conv filter fragments alone (8-bit handles).
hipError_t launch_pack_conv_fp16(const float* conv_w, const float* conv_b, uint4* conv_frag,
                                 hipStream_t stream);
// Repack fp32 FC1 weights (on the device) into the e4m3 fragments of the
// 8-bit kernel: column n multiplied by 2^exp2[n] (exact) and rounded to e4m3.
hipError_t launch_pack_fc1_8(const float* fc1_w, const int* exp2, uint8_t* fc1_frag8,
                             hipStream_t stream);

// Error text for pointid_last_error (this thread); returns `code`.
int set_error(int code, const std::string& msg);
// Device ordinal of a handle.
int handle_device(pointid_handle h);

// Fused conv + ReLU + FC1 on 16-bit MFMA: patches [n][2304] (bf16 or fp16
// bits, or fp32 when f32_in: rounded in the kernel) -> part[s][row0 + i][128]
// for s < conv_fc1_16_splits().
int conv_fc1_16_splits();
// Tiles of the launch over n patches on `cus` CUs: n_big tiles of 96 patches,
// then n_mid of 64 (a batch that fits one round of thin tiles of 16 or 32
// patches, conv_fc1_16_thin_tile, runs those instead).
void conv_fc1_16_tiles(int64_t n, int cus, int64_t* n_big, int64_t* n_mid);
int conv_fc1_16_thin_tile(int64_t n, int cus);
int conv_fc1_16_thin_parts(int64_t n, int cus, int thin);
hipError_t launch_conv_fc1_16(bool fp16, const void* patches, bool f32_in, int64_t n, int64_t row0,
                              int64_t n_total, const uint4* w1p, const uint4* convp,
                              float* part, hipStream_t stream);

// Fused conv (fp16 MFMA) + ReLU + FC1 on e4m3 MFMA operands: fp16 patches
// [n][2304] -> part[s][row0 + i][128] for s < conv_fc1_8_splits(), the sums
// of FC1 column n still multiplied by 2^k_n.
int conv_fc1_8_splits();
// Tiles of the 8-bit launch for n patches on `cus` CUs (64 and 32 patches).
void conv_fc1_8_tiles(int64_t n, int cus, int64_t* n_big, int64_t* n_small);
hipError_t launch_conv_fc1_8(const uint16_t* patches, int64_t n, int64_t row0, int64_t n_total,
                             const uint8_t* w1p, const uint4* convp, float* part, hipStream_t stream);

// Fused fp32 conv + ReLU + FC1 on fp32 MFMA: patches [n][2304] fp32 ->
// part[s][row0 + i][128] for s < conv_fc1_f32_splits(), from the conv filters
// and biases and the transposed FC1 weights w1t[o][k].
int conv_fc1_f32_splits();
// Tiles of the fused fp32 launch for n patches on `cus` CUs (64 and 32 patches).
void conv_fc1_f32_tiles(int64_t n, int cus, int64_t* n_big, int64_t* n_small);
hipError_t launch_conv_fc1_f32(const float* patches, int64_t n, int64_t row0, int64_t n_total,
                               const float* conv_w, const float* conv_b, const float* w1t,
                               float* part, hipStream_t stream);

// w1t[o][k] = w1[k][o] for the FC1 weights.
hipError_t launch_transpose_w1(const float* w1, float* w1t, hipStream_t stream);

// Reduce the split-K partials in fixed order, then bias+ReLU, FC2+ReLU, the
// softmax and sigmoid heads: scores [n][4].
hipError_t launch_tail(const float* part, int splits, int64_t n,
                       const DeviceWeights& w, float* scores,
                       hipStream_t stream);
// The same, with patch p's scores written to its request's output.
hipError_t launch_tail_requests(const float* part, int splits, const DeviceWeights& w,
                                const RequestTable& reqs, hipStream_t stream);

// Hit finding (hits.hip).  The waveforms of all planes are cut into steps of
// 256 ticks, numbered plane by plane, wire by wire, then along the wire; step
// g covers ticks 256*s .. 256*s + 255 of one wire.  Each of `workers` waves
// takes the steps [w * per, min((w + 1) * per, total)).
constexpr int kHitStep = 256;
constexpr int kHitMaxWorkers = 8192;
struct HitSteps {
  int64_t step0[kMaxPlanes + 1];    // first step of plane p; step0[n] = total
  int32_t per_row[kMaxPlanes];      // steps per wire of plane p
  int64_t per;                      // steps per worker
  int32_t workers;
  int32_t n;
};
void hit_steps(const PlaneTable& planes, HitSteps* st);
// Every step's hit bits (4 uint64 words: bit l of word j = tick 4l + j of the
// step) into mask[4g ...]; each worker's hit count into counts[w].  kVec
// (every image 16-byte aligned, every n_ticks a multiple of 4) allows 16-byte
// loads.
hipError_t launch_hits_mask(const PlaneTable& planes, const HitSteps& st, float threshold,
                            uint64_t* mask, int32_t* counts, hipStream_t stream);
// offsets[w] = sum of counts[0 .. w-1]; *total = sum of all counts.
hipError_t launch_hits_scan(const int32_t* counts, int32_t n, int64_t* offsets, int64_t* total,
                            hipStream_t stream);
// (plane, wire, tick) of every hit with output index below `capacity`.
hipError_t launch_hits_emit(const PlaneTable& planes, const HitSteps& st, const uint64_t* mask,
                            const int32_t* counts, const int64_t* offsets, int32_t* hits,
                            int64_t capacity, hipStream_t stream);

}  // namespace pointid
