// Sustained fp16 MFMA rate of the GPU: the on-chip ceiling the convolution
// rates are read against. Register-only chains of v_mfma_f32_32x32x16_f16,
// no memory traffic in the loop, so the rate is that of the matrix pipes at
// the clock the chip holds under this load.
//
// Operands come from a hash of (thread, operand slot, element): about half
// of them zero; the rest random fp16 values in (-1, 1) (mode 0, whose
// toggling bits draw the power of real data) or integers in -2..2 (mode 1,
// whose sums stay exact in fp32, so a test can check the result in closed
// form).
#include "common.h"
#include "internal.h"

namespace fg {
namespace {

__device__ __forceinline__ uint32_t operand_hash(uint32_t t, uint32_t slot, uint32_t e) {
  uint32_t h = t * 0x9E3779B1u + slot * 0x85EBCA77u + e * 0xC2B2AE3Du;
  h ^= h >> 15;
  h *= 0x2C1B3C6Du;
  h ^= h >> 12;
  return h;
}

// The 8 fp16 values of this lane's operand in a slot (A: slots 0-3, B: 4-7).
__device__ __forceinline__ u32x4 operand(uint32_t t, uint32_t slot, int mode) {
  half8 v;
#pragma unroll
  for (uint32_t e = 0; e < 8; ++e) {
    const uint32_t h = operand_hash(t, slot, e);
    float f = 0.f;
    if (!(h & 1u))
      f = mode ? (float)((int)((h >> 1) % 5u) - 2)
               : ((h >> 31) ? -1.f : 1.f) * (float)((h >> 2) & 0x3FFFu) * (1.f / 16384.f);
    v[e] = (_Float16)f;
  }
  return __builtin_bit_cast(u32x4, v);
}

// Four accumulator chains per wave; each iteration issues 8 MFMAs that
// rotate through the operands: c0 += A0 B0 + A1 B2, c1 += A1 B1 + A2 B3,
// c2 += A2 B2 + A3 B0, c3 += A3 B3 + A0 B1. Each thread then writes the sum
// of its 64 accumulator values.
__global__ __launch_bounds__(256) void mfma_loop_kernel(float *out, int iters, int mode) {
  const uint32_t t = blockIdx.x * 256u + threadIdx.x;
  const u32x4 a0 = operand(t, 0, mode), a1 = operand(t, 1, mode);
  const u32x4 a2 = operand(t, 2, mode), a3 = operand(t, 3, mode);
  const u32x4 b0 = operand(t, 4, mode), b1 = operand(t, 5, mode);
  const u32x4 b2 = operand(t, 6, mode), b3 = operand(t, 7, mode);
  f32x16 c0 = {}, c1 = {}, c2 = {}, c3 = {};
  for (int i = 0; i < iters; ++i) {
    c0 = mfma32(a0, b0, c0);
    c1 = mfma32(a1, b1, c1);
    c2 = mfma32(a2, b2, c2);
    c3 = mfma32(a3, b3, c3);
    c0 = mfma32(a1, b2, c0);
    c1 = mfma32(a2, b3, c1);
    c2 = mfma32(a3, b0, c2);
    c3 = mfma32(a0, b1, c3);
  }
  float s = 0.f;
#pragma unroll
  for (int v = 0; v < 16; ++v) s += (c0[v] + c1[v]) + (c2[v] + c3[v]);
  out[t] = s;
}

}  // namespace

hipError_t launch_mfma_loop(float *out, int32_t blocks, int32_t iters, int32_t mode,
                            hipStream_t st) {
  hipLaunchKernelGGL(mfma_loop_kernel, dim3(blocks), dim3(256), 0, st, out, iters, mode);
  return hipGetLastError();
}

}  // namespace fg
