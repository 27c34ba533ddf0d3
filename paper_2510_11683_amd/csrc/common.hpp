// Device-side helpers shared by the BGPO ELBO-head kernels (gfx950).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace bgpo {

typedef uint16_t bf16_t;                                   // bfloat16 bit pattern
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));  // MFMA operand
typedef float f32x16 __attribute__((ext_vector_type(16)));  // 32x32 MFMA accumulator

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11): 10 rounds of two 32x32->64
// multiplies with key mixing; the key advances by the Weyl constants between
// rounds.
struct u32x4 {
  uint32_t x, y, z, w;
};

__device__ __forceinline__ u32x4 philox4x32_10(u32x4 c, uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r) {
      k0 += 0x9E3779B9u;
      k1 += 0xBB67AE85u;
    }
    const uint32_t hi0 = __umulhi(0xD2511F53u, c.x), lo0 = 0xD2511F53u * c.x;
    const uint32_t hi1 = __umulhi(0xCD9E8D57u, c.z), lo1 = 0xCD9E8D57u * c.z;
    c = u32x4{hi1 ^ c.y ^ k0, lo1, hi0 ^ c.w ^ k1, lo0};
  }
  return c;
}

__device__ __forceinline__ uint32_t pick_word(const u32x4& v, int i) {
  return i == 0 ? v.x : i == 1 ? v.y : i == 2 ? v.z : v.w;
}

// Integer timestep T24 in [1, 2^24): t = T24 * 2^-24 (exact in fp32 and fp64).
__device__ __forceinline__ uint32_t timestep_t24(uint32_t k0, uint32_t k1, uint32_t seq, int j,
                                                 int n_t, int t_mode) {
  if (t_mode == 0) {
    const u32x4 w = philox4x32_10(u32x4{0u, seq, (uint32_t)j, 1u}, k0, k1);
    const uint32_t T = w.x >> 8;
    return T ? T : 1u;
  }
  const u32x4 w = philox4x32_10(u32x4{0u, seq, 0u, 2u}, k0, k1);
  const uint64_t u24 = w.x >> 8;
  const uint64_t T = (((uint64_t)j << 24) + u24) / (uint64_t)n_t;
  return T ? (uint32_t)T : 1u;
}

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

// float -> bfloat16, round to nearest even (the hardware v_cvt_pk_bf16_f32).
__device__ __forceinline__ bf16_t f32_to_bf16(float f) {
  return __builtin_bit_cast(bf16_t, static_cast<__bf16>(f));
}

// two floats -> packed bfloat16 pair (lo = a, hi = b), one conversion instruction
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  const f32x2_t v = {a, b};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
}

__device__ __forceinline__ float bf16_to_f32(bf16_t h) { return __uint_as_float((uint32_t)h << 16); }

// Head inputs as bf16 bit patterns, 8 or 4 consecutive elements at a time:
// bf16 inputs as they are, fp32 inputs rounded to nearest even (so both
// element types give the same bits for the same rounded values).  p must be
// 16-byte (bf16 x8, fp32 x4) or 8-byte (bf16 x4) aligned.
template <typename T>
__device__ __forceinline__ uint4 load_bf16x8(const T* p);
template <>
__device__ __forceinline__ uint4 load_bf16x8<uint16_t>(const uint16_t* p) {
  return *reinterpret_cast<const uint4*>(p);
}
template <>
__device__ __forceinline__ uint4 load_bf16x8<float>(const float* p) {
  const float4 a = *reinterpret_cast<const float4*>(p);
  const float4 b = *reinterpret_cast<const float4*>(p + 4);
  return make_uint4(pack_bf16x2(a.x, a.y), pack_bf16x2(a.z, a.w), pack_bf16x2(b.x, b.y),
                    pack_bf16x2(b.z, b.w));
}
template <typename T>
__device__ __forceinline__ uint2 load_bf16x4(const T* p);
template <>
__device__ __forceinline__ uint2 load_bf16x4<uint16_t>(const uint16_t* p) {
  return *reinterpret_cast<const uint2*>(p);
}
template <>
__device__ __forceinline__ uint2 load_bf16x4<float>(const float* p) {
  const float4 a = *reinterpret_cast<const float4*>(p);
  return make_uint2(pack_bf16x2(a.x, a.y), pack_bf16x2(a.z, a.w));
}

}  // namespace bgpo
