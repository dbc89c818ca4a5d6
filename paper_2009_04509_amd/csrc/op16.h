// 16-bit MFMA operand helpers shared by the fused conv/FC1 kernel, the weight
// packing kernels and the patch gather: bf16 or fp16 per a compile-time flag.
// All conversions are the hardware round-to-nearest-even ones.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace pointid {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef _Float16 halfx8 __attribute__((ext_vector_type(8)));
typedef _Float16 halfx2 __attribute__((ext_vector_type(2)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef float floatx2 __attribute__((ext_vector_type(2)));
typedef short shortx2 __attribute__((ext_vector_type(2)));

template <bool kFp16>
struct Op16;

template <>
struct Op16<false> {                          // bf16
  static constexpr uint32_t kOnes = 0x3F803F80u;   // two 1.0
  static __device__ __forceinline__ floatx4 mfma(const uint4& a, const uint4& b, const floatx4& c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                   __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
  }
  // (a, b) rounded and packed, a in the low half
  static __device__ __forceinline__ uint32_t pack(float a, float b) {
    return __builtin_bit_cast(uint32_t, __builtin_convertvector((floatx2){a, b}, bf16x2));
  }
  static __device__ __forceinline__ float value(uint16_t h) {
    return __uint_as_float((uint32_t)h << 16);
  }
};

template <>
struct Op16<true> {                           // fp16
  static constexpr uint32_t kOnes = 0x3C003C00u;
  static __device__ __forceinline__ floatx4 mfma(const uint4& a, const uint4& b, const floatx4& c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(halfx8, a),
                                                  __builtin_bit_cast(halfx8, b), c, 0, 0, 0);
  }
  static __device__ __forceinline__ uint32_t pack(float a, float b) {
    return __builtin_bit_cast(uint32_t, __builtin_convertvector((floatx2){a, b}, halfx2));
  }
  static __device__ __forceinline__ float value(uint16_t h) {
    return (float)__builtin_bit_cast(_Float16, h);
  }
};

// ReLU on two packed 16-bit floats: a negative value has its sign bit set, so
// it is negative as an int16 and max(x, 0) over int16 lanes zeroes it (-0 too).
__device__ __forceinline__ uint32_t relu2(uint32_t v) {
  shortx2 s = __builtin_elementwise_max(__builtin_bit_cast(shortx2, v), (shortx2){0, 0});
  return __builtin_bit_cast(uint32_t, s);
}

}  // namespace pointid
