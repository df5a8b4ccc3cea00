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
  u16x2 mb = u16x2{0, 0};
  if (MAXC > 0) {
#pragma unroll
    for (int i = 0; i < REG; ++i) {
      const int c = lane + 64 * i;
      v[i] = c < nch ? *reinterpret_cast<const f16x8*>(row + c * 8) : f16x8{};
    }
#pragma unroll
    for (int i = 0; i < REG; ++i) mb = absmax_f16x8(mb, v[i]);
  } else {
    for (int c = lane; c < nch; c += 64) mb = absmax_f16x8(mb, *reinterpret_cast<const f16x8*>(row + c * 8));
  }
  const float amax = wave_max(absmax_value(mb));
  const float qm = (float)((1 << (BITS - 1)) - 1);
  const float a = mul_rn(clip, amax);
  float inv = 0.f, s = 1.f;
  if (a != 0.f) {
    inv = div_rn(qm, a);
    s = div_rn(a, qm);
  }
  if (lane == 0) sx[m] = s;
  auto emit = [&](int c, const f16x8& t) {
    uint32_t q[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) q[e] = code_bits((float)t[e], inv, qm);
    if (BITS == 8)
      *reinterpret_cast<uint2*>(xq + m * (int64_t)K + c * 8) =
          make_uint2(pack4_codes8(q[0], q[1], q[2], q[3]), pack4_codes8(q[4], q[5], q[6], q[7]));
    else
      *reinterpret_cast<uint32_t*>(xq + m * (int64_t)(K / 2) + c * 4) = pack8_codes4(q);
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

// ---------------------------------------------------------------------------
// Quantization of rotated rows, Q(X H1^T) with H1 = blockdiag(H_B) diag(s) /
// sqrt(B) (Eq. 11-12; an online H1 for inputs whose rotation is not folded
// into the previous layer).  One workgroup of 256 threads per row; the row
// lives in LDS as fp32.  In fp32: x_i * s_i, the Walsh-Hadamard stages
// h = 1, 2, ..., B/2 ((v_i, v_{i+h}) -> (v_i + v_{i+h}, v_i - v_{i+h})), then
// one product by c = fp32(1/sqrt(B)); the quantizer of quantize_rows_kernel
// follows.  Stages 1, 2, 4 run in registers on 8-element chunks; the rest in
// radix-8 (then radix-4 / radix-2) passes through LDS.  Which thread does a
// butterfly does not change its operands, so the result is that of the
// stage-by-stage definition.
// ---------------------------------------------------------------------------
constexpr int kRotThreads = 256;
constexpr int kRotMaxChunks = 8;       // 8-element chunks per thread: K <= 8 * 8 * 256

// LDS word of row element i: 8 pad words after every 64 elements, so that the
// strided groups of every pass (stride 8 included) fall on distinct banks.
__device__ __forceinline__ int rot_addr(int i) { return i + ((i >> 6) << 3); }

template <int R>
__device__ __forceinline__ void rot_pass(float* buf, int K, int lh) {
  // groups of R elements i + k h (h = 2^lh, k = 0..R-1), i with bits h .. (R/2) h clear
  constexpr int LR = R == 8 ? 3 : R == 4 ? 2 : 1;
  const int ngroups = K / R, h = 1 << lh;
  for (int g = threadIdx.x; g < ngroups; g += kRotThreads) {
    const int i = ((g >> lh) << (lh + LR)) | (g & (h - 1));
    float v[R];
#pragma unroll
    for (int k = 0; k < R; ++k) v[k] = buf[rot_addr(i + k * h)];
#pragma unroll
    for (int st = 1; st < R; st <<= 1)
#pragma unroll
      for (int k = 0; k < R; ++k)
        if (!(k & st)) {
          const float a = v[k], b = v[k + st];
          v[k] = add_rn(a, b);
          v[k + st] = add_rn(a, -b);
        }
#pragma unroll
    for (int k = 0; k < R; ++k) buf[rot_addr(i + k * h)] = v[k];
  }
}

template <int BITS>
__global__ void __launch_bounds__(kRotThreads)
quantize_rotated_kernel(const _Float16* __restrict__ x, int64_t M, int32_t K, int64_t ldx, float clip,
                        const int8_t* __restrict__ signs, int32_t block, float c, uint8_t* __restrict__ xq,
                        float* __restrict__ sx) {
  extern __shared__ __attribute__((aligned(16))) float rbuf[];
  __shared__ float wmax[kRotThreads / 64];
  const int tid = threadIdx.x;
  const int64_t m = blockIdx.x;
  const _Float16* row = x + m * ldx;
  const int nch = K >> 3;
  // signs, stages 1, 2, 4 on 8-element chunks (B >= 8, so a chunk lies in one block)
  for (int ch = tid; ch < nch; ch += kRotThreads) {
    const f16x8 t = *reinterpret_cast<const f16x8*>(row + ch * 8);
    float v[8];
    if (signs) {
      const uint2 sb = *reinterpret_cast<const uint2*>(signs + ch * 8);
      const uint32_t sw[2] = {sb.x, sb.y};
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float f = (float)t[e];
        v[e] = (int8_t)(sw[e >> 2] >> (8 * (e & 3))) < 0 ? -f : f;
      }
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = (float)t[e];
    }
#pragma unroll
    for (int st = 1; st < 8; st <<= 1)
#pragma unroll
      for (int k = 0; k < 8; ++k)
        if (!(k & st)) {
          const float a = v[k], b = v[k + st];
          v[k] = add_rn(a, b);
          v[k + st] = add_rn(a, -b);
        }
    float* dst = rbuf + rot_addr(ch * 8);
    *reinterpret_cast<f32x4*>(dst) = f32x4{v[0], v[1], v[2], v[3]};
    *reinterpret_cast<f32x4*>(dst + 4) = f32x4{v[4], v[5], v[6], v[7]};
  }
  __syncthreads();
  int lh = 3;
  while ((1 << lh) < block) {
    const int h = 1 << lh;
    if (h * 8 <= block) rot_pass<8>(rbuf, K, lh), lh += 3;
    else if (h * 4 <= block) rot_pass<4>(rbuf, K, lh), lh += 2;
    else rot_pass<2>(rbuf, K, lh), lh += 1;
    __syncthreads();
  }
  // y = v * c kept in registers, row absmax, then the per-token quantizer
  float y[kRotMaxChunks][8];
  float amax = 0.f;
#pragma unroll
  for (int j = 0; j < kRotMaxChunks; ++j) {
    const int ch = tid + j * kRotThreads;
    if (ch < nch) {
      const float* srcp = rbuf + rot_addr(ch * 8);
      const f32x4 lo = *reinterpret_cast<const f32x4*>(srcp), hi = *reinterpret_cast<const f32x4*>(srcp + 4);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        y[j][e] = mul_rn(lo[e], c);
        y[j][4 + e] = mul_rn(hi[e], c);
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) amax = fmaxf(amax, fabsf(y[j][e]));
    }
  }
  amax = wave_max(amax);
  if ((tid & 63) == 0) wmax[tid >> 6] = amax;
  __syncthreads();
  amax = fmaxf(fmaxf(wmax[0], wmax[1]), fmaxf(wmax[2], wmax[3]));
  const float qm = (float)((1 << (BITS - 1)) - 1);
  const float a = mul_rn(clip, amax);
  float inv = 0.f, s = 1.f;
  if (a != 0.f) {
    inv = div_rn(qm, a);
    s = div_rn(a, qm);
  }
  if (tid == 0) sx[m] = s;
#pragma unroll
  for (int j = 0; j < kRotMaxChunks; ++j) {
    const int ch = tid + j * kRotThreads;
    if (ch >= nch) continue;
    uint32_t q[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) q[e] = code_bits(y[j][e], inv, qm);
    if (BITS == 8)
      *reinterpret_cast<uint2*>(xq + m * (int64_t)K + ch * 8) =
          make_uint2(pack4_codes8(q[0], q[1], q[2], q[3]), pack4_codes8(q[4], q[5], q[6], q[7]));
    else
      *reinterpret_cast<uint32_t*>(xq + m * (int64_t)(K / 2) + ch * 4) = pack8_codes4(q);
  }
}

// The same for K = B = 4096 with one wavefront per row and no workgroup
// barrier: lane l holds elements 64 l .. 64 l + 63, stages h = 1 .. 32 run in
// its registers; one transpose through LDS (16.6 KB) gives lane l the
// elements 64 k + l, k = 0 .. 63, so stages h = 64 .. 2048 run in
// registers too; then the product by c, the row max (a wave reduction), a
// transpose back, and the codes of 64 consecutive elements per lane.  Each
// element sees the same fp32 operations in the same order as above.
constexpr int kRw = 64;          // elements per lane
constexpr int kRwLd = kRw + 1;   // LDS words per lane row (odd: no bank conflicts either way)

__device__ __forceinline__ void rw_butterflies(float* v, int hmin, int hmax) {
#pragma unroll
  for (int h = 1; h < kRw; h <<= 1) {
    if (h < hmin || h > hmax) continue;
#pragma unroll
    for (int k = 0; k < kRw; ++k)
      if (!(k & h)) {
        const float a = v[k], b = v[k + h];
        v[k] = add_rn(a, b);
        v[k + h] = add_rn(a, -b);
      }
  }
}

template <int BITS>
__global__ void __launch_bounds__(64)
quantize_rotated_w64_kernel(const _Float16* __restrict__ x, int64_t M, int64_t ldx, float clip,
                            const int8_t* __restrict__ signs, float c, uint8_t* __restrict__ xq,
                            float* __restrict__ sx) {
  constexpr int K = kRw * 64;
  __shared__ float tb[64 * kRwLd];   // [lane][element] of one wave
  const int lane = threadIdx.x;
  const int64_t m = blockIdx.x;
  const _Float16* row = x + m * ldx + kRw * lane;
  float v[kRw];
#pragma unroll
  for (int i = 0; i < kRw / 8; ++i) {
    const f16x8 t = *reinterpret_cast<const f16x8*>(row + 8 * i);
#pragma unroll
    for (int e = 0; e < 8; ++e) v[8 * i + e] = (float)t[e];
  }
  if (signs) {
#pragma unroll
    for (int i = 0; i < kRw / 16; ++i) {
      const uint4 sb = *reinterpret_cast<const uint4*>(signs + kRw * lane + 16 * i);
      const uint32_t sw[4] = {sb.x, sb.y, sb.z, sb.w};
#pragma unroll
      for (int e = 0; e < 16; ++e)
        if ((int8_t)(sw[e >> 2] >> (8 * (e & 3))) < 0) v[16 * i + e] = -v[16 * i + e];
    }
  }
  rw_butterflies(v, 1, kRw / 2);                  // h = 1 .. 32
  // transpose: element 64 l + k of lane l -> lane k, register l (one wave:
  // its LDS accesses execute in order; the empty asm keeps the compiler's)
#pragma unroll
  for (int k = 0; k < kRw; ++k) tb[lane * kRwLd + k] = v[k];
  asm volatile("" ::: "memory");
#pragma unroll
  for (int k = 0; k < kRw; ++k) v[k] = tb[k * kRwLd + lane];
  asm volatile("" ::: "memory");
  rw_butterflies(v, 1, kRw / 2);                  // h = 64 .. 2048 (register index bits)
  float amax = 0.f;
#pragma unroll
  for (int k = 0; k < kRw; ++k) {
    v[k] = mul_rn(v[k], c);
    amax = fmaxf(amax, fabsf(v[k]));
  }
  amax = wave_max(amax);
  // transpose back: lane l (register k = element 64 k + l) -> lane k, register l
#pragma unroll
  for (int k = 0; k < kRw; ++k) tb[k * kRwLd + lane] = v[k];
  asm volatile("" ::: "memory");
  float z[kRw];
#pragma unroll
  for (int k = 0; k < kRw; ++k) z[k] = tb[lane * kRwLd + k];
  const float qm = (float)((1 << (BITS - 1)) - 1);
  const float a = mul_rn(clip, amax);
  float inv = 0.f, sc = 1.f;
  if (a != 0.f) {
    inv = div_rn(qm, a);
    sc = div_rn(a, qm);
  }
  if (lane == 0) sx[m] = sc;
#pragma unroll
  for (int i = 0; i < kRw / 16; ++i) {
    uint32_t q[16];
#pragma unroll
    for (int e = 0; e < 16; ++e) q[e] = code_bits(z[16 * i + e], inv, qm);
    if (BITS == 8)
      *reinterpret_cast<uint4*>(xq + m * (int64_t)K + kRw * lane + 16 * i) =
          make_uint4(pack4_codes8(q[0], q[1], q[2], q[3]), pack4_codes8(q[4], q[5], q[6], q[7]),
                     pack4_codes8(q[8], q[9], q[10], q[11]), pack4_codes8(q[12], q[13], q[14], q[15]));
    else
      *reinterpret_cast<uint2*>(xq + m * (int64_t)(K / 2) + (kRw * lane + 16 * i) / 2) =
          make_uint2(pack8_codes4(q), pack8_codes4(q + 8));
  }
}

hipError_t launch_quantize_rotated(const void* x, int64_t M, int32_t K, int64_t ldx, int32_t bits, float clip,
                                   const int8_t* signs, int32_t block, float c, void* xq, float* sx,
                                   hipStream_t s) {
  if (M == 0) return hipSuccess;
  // (the one-wave kernel moves 16-byte runs of signs and 8-bit codes)
  if (K == kRw * 64 && block == K && ldx % 8 == 0 && ((uintptr_t)signs & 15) == 0 &&
      (bits == 4 || ((uintptr_t)xq & 15) == 0)) {
    KernelScope ks("quantize_rotated", s);
    if (bits == 8)
      QSVD_LAUNCH(ks, quantize_rotated_w64_kernel<8>, dim3((unsigned)M), dim3(64), 0, s, (const _Float16*)x, M, ldx,
                  clip, signs, c, (uint8_t*)xq, sx);
    else
      QSVD_LAUNCH(ks, quantize_rotated_w64_kernel<4>, dim3((unsigned)M), dim3(64), 0, s, (const _Float16*)x, M, ldx,
                  clip, signs, c, (uint8_t*)xq, sx);
    return hipGetLastError();
  }
  const size_t lds = (size_t)(K + K / 8) * sizeof(float);     // with the pad words
  auto kern = bits == 8 ? quantize_rotated_kernel<8> : quantize_rotated_kernel<4>;
  if (lds + 1024 > 64 * 1024) {     // (plus the kernel's static LDS)
    hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  KernelScope ks("quantize_rotated", s);
  QSVD_LAUNCH(ks, kern, dim3((unsigned)M), dim3(kRotThreads), lds, s, (const _Float16*)x, M, K, ldx, clip, signs,
              block, c, (uint8_t*)xq, sx);
  return hipGetLastError();
}

hipError_t launch_quantize_rows(const void* x, int64_t M, int32_t K, int64_t ldx, int32_t bits,
                                float clip, void* xq, float* sx, hipStream_t s, const char* name) {
  if (M == 0) return hipSuccess;
  dim3 grid((unsigned)M), block(64);
  const bool regs = K <= 64 * 8 * 16;
  KernelScope ks(name, s);
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
