// Per-token symmetric quantization of fp16 rows (activations X, and the latent C).
#include "common.h"
#include "launch.h"

namespace qsvd {

// One wavefront per row.  Lane l holds the 8-element (16-byte) chunks
// l, l + 64, ... of the row in registers (up to MAXC per lane), so the row is
// read once; longer rows take a second pass over memory (MAXC == 0).
template <int BITS, int MAXC>
__global__ void __launch_bounds__(64)
quantize_rows_kernel(const _Float16* __restrict__ x, int64_t M, int32_t K, int64_t ldx, float clip,
                     uint8_t* __restrict__ xq, float* __restrict__ sx) {
  const int lane = threadIdx.x;
  const int64_t m = blockIdx.x;
  const _Float16* row = x + m * ldx;
  const int nch = K >> 3;
  constexpr int REG = MAXC > 0 ? MAXC : 1;
  f16x8 v[REG];
  float amax = 0.f;
  if (MAXC > 0) {
#pragma unroll
    for (int i = 0; i < REG; ++i) {
      const int c = lane + 64 * i;
      v[i] = c < nch ? *reinterpret_cast<const f16x8*>(row + c * 8) : f16x8{};
    }
#pragma unroll
    for (int i = 0; i < REG; ++i)
#pragma unroll
      for (int e = 0; e < 8; ++e) amax = fmaxf(amax, fabsf((float)v[i][e]));
  } else {
    for (int c = lane; c < nch; c += 64) {
      const f16x8 t = *reinterpret_cast<const f16x8*>(row + c * 8);
#pragma unroll
      for (int e = 0; e < 8; ++e) amax = fmaxf(amax, fabsf((float)t[e]));
    }
  }
  amax = wave_max(amax);
  const float qm = (float)((1 << (BITS - 1)) - 1);
  const float a = mul_rn(clip, amax);
  float inv = 0.f, s = 1.f;
  if (a != 0.f) {
    inv = div_rn(qm, a);
    s = div_rn(a, qm);
  }
  if (lane == 0) sx[m] = s;
  auto emit = [&](int c, const f16x8& t) {
    int q[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) q[e] = (a != 0.f) ? quant_code(mul_rn((float)t[e], inv), qm) : 0;
    if (BITS == 8) {
      uint32_t lo = (q[0] & 0xff) | ((q[1] & 0xff) << 8) | ((q[2] & 0xff) << 16) | ((uint32_t)(q[3] & 0xff) << 24);
      uint32_t hi = (q[4] & 0xff) | ((q[5] & 0xff) << 8) | ((q[6] & 0xff) << 16) | ((uint32_t)(q[7] & 0xff) << 24);
      *reinterpret_cast<uint2*>(xq + m * (int64_t)K + c * 8) = make_uint2(lo, hi);
    } else {
      uint32_t p = 0;
#pragma unroll
      for (int e = 0; e < 8; ++e) p |= (uint32_t)(q[e] & 0xf) << (4 * e);
      *reinterpret_cast<uint32_t*>(xq + m * (int64_t)(K / 2) + c * 4) = p;
    }
  };
  if (MAXC > 0) {
#pragma unroll
    for (int i = 0; i < REG; ++i) {
      const int c = lane + 64 * i;
      if (c < nch) emit(c, v[i]);
    }
  } else {
    for (int c = lane; c < nch; c += 64) emit(c, *reinterpret_cast<const f16x8*>(row + c * 8));
  }
}

hipError_t launch_quantize_rows(const void* x, int64_t M, int32_t K, int64_t ldx, int32_t bits,
                                float clip, void* xq, float* sx, hipStream_t s) {
  if (M == 0) return hipSuccess;
  dim3 grid((unsigned)M), block(64);
  const bool regs = K <= 64 * 8 * 16;
  KernelScope ks("quantize_rows", s);
  const _Float16* xp = (const _Float16*)x;
  uint8_t* q = (uint8_t*)xq;
  if (bits == 8) {
    if (regs) QSVD_LAUNCH(ks, (quantize_rows_kernel<8, 16>), grid, block, 0, s, xp, M, K, ldx, clip, q, sx);
    else QSVD_LAUNCH(ks, (quantize_rows_kernel<8, 0>), grid, block, 0, s, xp, M, K, ldx, clip, q, sx);
  } else {
    if (regs) QSVD_LAUNCH(ks, (quantize_rows_kernel<4, 16>), grid, block, 0, s, xp, M, K, ldx, clip, q, sx);
    else QSVD_LAUNCH(ks, (quantize_rows_kernel<4, 0>), grid, block, 0, s, xp, M, K, ldx, clip, q, sx);
  }
  return hipGetLastError();
}

}  // namespace qsvd
