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

// Symmetric code clamp(rint(x * inv), -qm, qm) (rint ties to even) in four VALU
// operations: y = fl(x * inv) (an FMA with a -0 addend rounds the exact product
// once, as the product alone does, and keeps its sign), clamped to [-qm, qm],
// then rounded half to even to an integer by adding 1.5 * 2^23 (for |y| <= 2^22
// the sum holds that integer in its low mantissa bits).  The low byte (nibble)
// of the returned word is the two's-complement code; inv == 0 (an all-zero
// row) gives code 0.
__device__ __forceinline__ uint32_t code_bits(float x, float inv, float qm) {
  const float y = __builtin_amdgcn_fmed3f(__builtin_fmaf(x, inv, -0.0f), -qm, qm);
  return __float_as_uint(add_rn(y, 12582912.0f));
}

// Low bytes of four code words -> one word, element e in byte e.
__device__ __forceinline__ uint32_t pack4_codes8(uint32_t b0, uint32_t b1, uint32_t b2, uint32_t b3) {
  const uint32_t p01 = __builtin_amdgcn_perm(b1, b0, 0x0c0c0400u);
  const uint32_t p23 = __builtin_amdgcn_perm(b3, b2, 0x0c0c0400u);
  return __builtin_amdgcn_perm(p23, p01, 0x05040100u);
}

// Low nibbles of eight code words -> one word, element e in bits 4e .. 4e+3.
__device__ __forceinline__ uint32_t pack8_codes4(const uint32_t* b) {
  const uint32_t lo = pack4_codes8(b[0], b[1], b[2], b[3]) & 0x0f0f0f0fu;
  const uint32_t hi = pack4_codes8(b[4], b[5], b[6], b[7]) & 0x0f0f0f0fu;
  const uint32_t l2 = lo | (lo >> 4), h2 = hi | (hi >> 4);   // bytes 0 and 2 hold nibble pairs
  return __builtin_amdgcn_perm(h2, l2, 0x06040200u);
}

// Running max of |x| over fp16 values as bit patterns, two halves per lane
// word: for non-NaN fp16 values |x| orders like the bits of |x|.
typedef uint16_t u16x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ u16x2 absmax_f16x8(u16x2 m, f16x8 v) {
  const i32x4 w = __builtin_bit_cast(i32x4, v);
#pragma unroll
  for (int k = 0; k < 4; ++k) m = __builtin_elementwise_max(m, __builtin_bit_cast(u16x2, (uint32_t)w[k] & 0x7fff7fffu));
  return m;
}
__device__ __forceinline__ float absmax_value(u16x2 m) {
  const uint16_t b = m.x > m.y ? m.x : m.y;
  return (float)__builtin_bit_cast(_Float16, b);
}

// Output-tile order of the GEMM grids.  The chip dispatches workgroup i to
// XCD i % 8, and each XCD has its own L2.  The ids one XCD receives are made
// consecutive, and consecutive ids walk a block of gm tile rows column by
// column, so the tiles that run together on one XCD form a compact
// gm x (tiles / 8 / gm) block and fetch each operand row block into that L2
// once.  (A bijection on [0, tiles); gm comes from xcd_group_rows.)
__device__ __forceinline__ void xcd_tile(int id, int tiles, int tiles_n, int gm, int* tm, int* tn) {
  if (tiles % 8 == 0) id = (id % 8) * (tiles / 8) + id / 8;
  const int tiles_m = tiles / tiles_n, per_group = gm * tiles_n, grp = id / per_group, first = grp * gm;
  const int rows = min(tiles_m - first, gm), in_g = id - grp * per_group;
  *tm = first + in_g % rows;
  *tn = in_g / rows;
}

// Tile rows per group: the block height that minimizes the operand row
// blocks one XCD touches, gm + (tiles / 8) / gm.  When an XCD's share is
// many rounds of the `conc` tiles it runs at once, the L2 only ever holds the
// operands of the tiles in flight, so the block height that keeps those
// fewest, about sqrt(conc) (a column-first walk of gm rows has gm row blocks
// and conc / gm column blocks in flight), is taken instead.
inline int xcd_group_rows(int64_t tiles_m, int64_t tiles_n, int conc = 0) {
  const double per_xcd = (double)(tiles_m * tiles_n) / 8;
  if (conc > 0 && per_xcd > 4.0 * conc && tiles_n * tiles_n >= conc) {
    int g = 1;
    while ((g + 1) * (g + 1) <= conc) ++g;
    if ((int64_t)g < tiles_m) return g;
  }
  int best = (int)tiles_m;
  double best_cost = 1e300;
  for (int c = 1; c <= tiles_m; ++c) {
    const double cost = c + per_xcd / c;
    if (cost < best_cost) { best_cost = cost; best = c; }
  }
  return best;
}

// Signed int4 from a nibble.
__device__ __forceinline__ int nib_lo(uint32_t b) { return ((int)(b << 28)) >> 28; }
__device__ __forceinline__ int nib_hi(uint32_t b) { return ((int)(b << 24)) >> 28; }

}  // namespace qsvd
