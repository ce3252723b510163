// Device-side helpers shared by the fcngrad kernels (gfx950 / CDNA4).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fg {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kWave = 64;

// fp32 -> fp16 bits, round to nearest even, overflow to infinity.
__device__ __forceinline__ uint16_t f32_to_h(float v) {
  _Float16 h = (_Float16)v;
  return __builtin_bit_cast(uint16_t, h);
}

__device__ __forceinline__ float h_to_f32(uint16_t b) {
  return (float)__builtin_bit_cast(_Float16, b);
}

// fp64 -> fp16 bits, one nearest-even rounding (overflow to infinity).
// The value is first rounded in fp64 to a multiple of the fp16 spacing at its
// magnitude (rint rounds half to even); the result is an fp16 number, so the
// remaining conversions are exact.
__device__ __forceinline__ uint16_t f64_to_h(double d) {
  if (d != d) return 0x7E00;
  double ad = fabs(d);
  double r;
  if (ad >= 65520.0) {
    r = __builtin_inf();
  } else if (ad == 0.0) {
    r = 0.0;
  } else {
    int e = ilogb(ad);                 // ad in [2^e, 2^(e+1))
    int ue = (e < -14 ? -14 : e) - 10; // spacing 2^ue of fp16 at this size
    r = ldexp(rint(ldexp(ad, -ue)), ue);
  }
  r = copysign(r, d);
  _Float16 h = (_Float16)(float)r;
  return __builtin_bit_cast(uint16_t, h);
}

// 32x32x16 fp16 MFMA with fp32 accumulate. Operand lane layout: lane l holds
// row (A) / column (B) l % 32 and the 8 reduction elements 8*(l/32)..+7.
// Accumulator layout: lane l, register v holds C[8*(v/4) + 4*(l/32) + v%4]
// [l % 32].
__device__ __forceinline__ f32x16 mfma32(const u32x4 &a, const u32x4 &b,
                                         const f32x16 &c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(half8, a),
                                                __builtin_bit_cast(half8, b),
                                                c, 0, 0, 0);
}

// Select the low (sel=0) or high (sel=1) 16-bit half of each of two words
// and pack them as (lo_word_part, hi_word_part).
__device__ __forceinline__ uint32_t pack_lo(uint32_t a, uint32_t b) {
  return (a & 0xFFFFu) | (b << 16);
}
__device__ __forceinline__ uint32_t pack_hi(uint32_t a, uint32_t b) {
  return (a >> 16) | (b & 0xFFFF0000u);
}

// True if either fp16 value packed in w is +-inf or NaN (exponent all ones).
__device__ __forceinline__ bool nonfinite_h2(uint32_t w) {
  return ((w & 0x7C00u) == 0x7C00u) | ((w & 0x7C000000u) == 0x7C000000u);
}

// *flag = 1 from one lane of each wave in which some lane has `bad` (a plain
// store of the same value: no atomics needed). One-dimensional workgroups.
__device__ __forceinline__ void flag_nonfinite(int32_t *flag, bool bad) {
  const unsigned long long b = __ballot(bad);
  if (b != 0 && (threadIdx.x & 63) == (unsigned)__builtin_ctzll(b)) *flag = 1;
}

}  // namespace fg
