// Per-token symmetric quantization of fp16 rows (activations X, and the latent C).
#include "common.h"
#include "launch.h"

namespace qsvd {

// One wavefront per row; lanes stride over 8-element (16-byte) chunks.
template <int BITS>
__global__ void __launch_bounds__(256)
quantize_rows_kernel(const _Float16* __restrict__ x, int64_t M, int32_t K, int64_t ldx, float clip,
                     uint8_t* __restrict__ xq, float* __restrict__ sx) {
  const int lane = threadIdx.x & 63;
  const int64_t m = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (m >= M) return;
  const _Float16* row = x + m * ldx;
  const int nch = K >> 3;
  float amax = 0.f;
  for (int c = lane; c < nch; c += 64) {
    f16x8 v = *reinterpret_cast<const f16x8*>(row + c * 8);
#pragma unroll
    for (int i = 0; i < 8; ++i) amax = fmaxf(amax, fabsf((float)v[i]));
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
  for (int c = lane; c < nch; c += 64) {
    f16x8 v = *reinterpret_cast<const f16x8*>(row + c * 8);
    int q[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) q[i] = (a != 0.f) ? quant_code(mul_rn((float)v[i], inv), qm) : 0;
    if (BITS == 8) {
      uint32_t lo = (q[0] & 0xff) | ((q[1] & 0xff) << 8) | ((q[2] & 0xff) << 16) | ((uint32_t)(q[3] & 0xff) << 24);
      uint32_t hi = (q[4] & 0xff) | ((q[5] & 0xff) << 8) | ((q[6] & 0xff) << 16) | ((uint32_t)(q[7] & 0xff) << 24);
      *reinterpret_cast<uint2*>(xq + m * (int64_t)K + c * 8) = make_uint2(lo, hi);
    } else {
      uint32_t p = 0;
#pragma unroll
      for (int i = 0; i < 8; ++i) p |= (uint32_t)(q[i] & 0xf) << (4 * i);
      *reinterpret_cast<uint32_t*>(xq + m * (int64_t)(K / 2) + c * 4) = p;
    }
  }
}

hipError_t launch_quantize_rows(const void* x, int64_t M, int32_t K, int64_t ldx, int32_t bits,
                                float clip, void* xq, float* sx, hipStream_t s) {
  if (M == 0) return hipSuccess;
  dim3 grid((unsigned)((M + 3) / 4)), block(256);
  KernelScope ks("quantize_rows", s);
  if (bits == 8)
    hipLaunchKernelGGL(quantize_rows_kernel<8>, grid, block, 0, s, (const _Float16*)x, M, K, ldx,
                       clip, (uint8_t*)xq, sx);
  else
    hipLaunchKernelGGL(quantize_rows_kernel<4>, grid, block, 0, s, (const _Float16*)x, M, K, ldx,
                       clip, (uint8_t*)xq, sx);
  return hipGetLastError();
}

}  // namespace qsvd
