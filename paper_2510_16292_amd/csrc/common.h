// Device-side helpers shared by the QSVD kernels (gfx950 only).
#pragma once
#include <hip/hip_runtime.h>
#include <hip/hip_fp16.h>
#include <stdint.h>

#include "qsvd.h"

namespace qsvd {

typedef int32_t  i32x4  __attribute__((ext_vector_type(4)));
typedef int32_t  i32x16 __attribute__((ext_vector_type(16)));
typedef float    f32x4  __attribute__((ext_vector_type(4)));
typedef float    f32x16 __attribute__((ext_vector_type(16)));
typedef _Float16 f16x8  __attribute__((ext_vector_type(8)));
typedef _Float16 f16x4  __attribute__((ext_vector_type(4)));
typedef _Float16 f16x2  __attribute__((ext_vector_type(2)));

constexpr int kWave = 64;

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
  return v;
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}

// IEEE fp32 operations with no contraction into FMA: the stored results of the
// quantizers and epilogues depend on each rounding step.
__device__ __forceinline__ float mul_rn(float a, float b) { return __fmul_rn(a, b); }
__device__ __forceinline__ float add_rn(float a, float b) { return __fadd_rn(a, b); }
__device__ __forceinline__ float div_rn(float a, float b) { return __fdiv_rn(a, b); }

// fp32 -> fp16 with round-to-nearest-even, applied to an fp32 value that has
// already been rounded: the empty asm keeps the backend from folding a
// preceding multiply into v_fma_mix (a single rounding straight to fp16).
__device__ __forceinline__ _Float16 to_f16(float v) {
  __asm__("" : "+v"(v));
  return (_Float16)v;
}

// Symmetric code: clamp(rint(v), -qm, qm), rint ties to even.
__device__ __forceinline__ int quant_code(float v, float qm) {
  float t = __builtin_rintf(v);
  t = fminf(fmaxf(t, -qm), qm);
  return (int)t;
}

// Signed int4 from a nibble.
__device__ __forceinline__ int nib_lo(uint32_t b) { return ((int)(b << 28)) >> 28; }
__device__ __forceinline__ int nib_hi(uint32_t b) { return ((int)(b << 24)) >> 28; }

}  // namespace qsvd
