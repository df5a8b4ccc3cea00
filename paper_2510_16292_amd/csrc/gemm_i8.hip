// int8 x int8 -> int32 products on the gfx950 matrix cores (v_mfma_i32_32x32x32_i8)
// with the per-row / per-column dequantization epilogue of the quantized
// projections Q(X) Q(W^d) and Q(C) Q(W^u) (Eq. 11-12).
//
// Operand layout of one 32x32x32 MFMA: lane l supplies row (l % 32) of A and
// column (l % 32) of B, 16 bytes each along the contraction.  Which 16 bytes a
// lane supplies only has to agree between A and B: integer sums are exact in
// any order, so each kernel assigns contraction bytes to lanes in whatever
// order its loads are cheapest.  Output: lane l holds column (l % 32) and rows
// 8*(v/4) + 4*(l/32) + (v%4) for accumulator registers v = 0..15.
#include "common.h"
#include "launch.h"

namespace qsvd {

struct DevSegs {
  _Float16* ptr[3];
  int64_t ld[3];
  int32_t n0[3];
  int32_t n[3];
  int32_t n_seg;
};

__device__ __forceinline__ void store_out(const DevSegs& sg, int64_t m, int32_t n, float y) {
#pragma unroll
  for (int s = 0; s < 3; ++s) {
    if (s < sg.n_seg && n >= sg.n0[s] && n < sg.n0[s] + sg.n[s]) {
      if (sg.ptr[s]) sg.ptr[s][m * sg.ld[s] + (n - sg.n0[s])] = to_f16(y);
      return;
    }
  }
}

// Dequantize one integer accumulator: (f32(acc) * row_scale) * col_scale, each
// product rounded to fp32 on its own.
__device__ __forceinline__ float dequant(int32_t acc, float rs, float cs) {
  return mul_rn(mul_rn((float)acc, rs), cs);
}

// ---------------------------------------------------------------------------
// Tiled kernel: 128 x 128 output tile per workgroup, 4 waves of 64 x 64,
// K staged through LDS 64 bytes at a time with a register double buffer.
// ---------------------------------------------------------------------------
constexpr int TBM = 128, TBN = 128, TBK = 64, TPAD = 16, TLD = TBK + TPAD;

__global__ void __launch_bounds__(256)
gemm_i8_tiled_kernel(const int8_t* __restrict__ A, const int8_t* __restrict__ B,
                     const float* __restrict__ rs, const float* __restrict__ cs,
                     int64_t M, int32_t N, int32_t K, DevSegs sg, int32_t* __restrict__ dbg) {
  __shared__ __attribute__((aligned(16))) int8_t As[2][TBM * TLD];
  __shared__ __attribute__((aligned(16))) int8_t Bs[2][TBN * TLD];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int wm = w >> 1, wn = w & 1;
  const int64_t m0 = (int64_t)blockIdx.y * TBM;
  const int32_t n0 = blockIdx.x * TBN;

  // global -> register loader: chunk c in [0, 512) of 16 bytes; row c/4, col 16*(c%4)
  i32x4 ra[2], rb[2];
  auto gload = [&](int kt) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int c = tid + 256 * h, row = c >> 2, col = (c & 3) * 16;
      const int64_t gm = m0 + row;
      const int32_t gn = n0 + row;
      const int64_t k = (int64_t)kt * TBK + col;
      ra[h] = (gm < M) ? *reinterpret_cast<const i32x4*>(A + gm * K + k) : i32x4{0, 0, 0, 0};
      rb[h] = (gn < N) ? *reinterpret_cast<const i32x4*>(B + (int64_t)gn * K + k) : i32x4{0, 0, 0, 0};
    }
  };
  auto sstore = [&](int buf) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int c = tid + 256 * h, row = c >> 2, col = (c & 3) * 16;
      *reinterpret_cast<i32x4*>(&As[buf][row * TLD + col]) = ra[h];
      *reinterpret_cast<i32x4*>(&Bs[buf][row * TLD + col]) = rb[h];
    }
  };

  i32x16 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = i32x16{};

  const int nk = K / TBK;
  gload(0);
  sstore(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) gload(kt + 1);
#pragma unroll
    for (int kk = 0; kk < TBK; kk += 32) {
      i32x4 af[2], bf[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const int row = wm * 64 + i * 32 + (lane & 31);
        af[i] = *reinterpret_cast<const i32x4*>(&As[cur][row * TLD + kk + 16 * (lane >> 5)]);
      }
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int row = wn * 64 + j * 32 + (lane & 31);
        bf[j] = *reinterpret_cast<const i32x4*>(&Bs[cur][row * TLD + kk + 16 * (lane >> 5)]);
      }
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(af[i], bf[j], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < nk) sstore(cur ^ 1);
    __syncthreads();
  }

#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int32_t n = n0 + wn * 64 + j * 32 + (lane & 31);
      if (n >= N) continue;
      const float csn = cs[n];
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int64_t m = m0 + wm * 64 + i * 32 + 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
        if (m >= M) continue;
        const int32_t a = acc[i][j][v];
        if (dbg) dbg[m * N + n] = a;
        store_out(sg, m, n, dequant(a, rs[m], csn));
      }
    }
}

// ---------------------------------------------------------------------------
// Skinny kernel for M <= 32 (decode): the weight is streamed once by many
// workgroups, each owning 128 columns and one slice of the contraction, and
// writing its int32 partial tile to part[slice][m][n].  The epilogue adds the
// slices in a fixed order (integer sums are exact in any order anyway).
// ---------------------------------------------------------------------------
constexpr int SBN = 128;

__global__ void __launch_bounds__(256)
gemm_i8_splitk_kernel(const int8_t* __restrict__ A, const int8_t* __restrict__ B, int64_t M,
                      int32_t N, int32_t K, int32_t kchunk, int32_t* __restrict__ part) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int32_t ncol = blockIdx.x * SBN + w * 32 + (lane & 31);
  const int64_t mrow = lane & 31;
  const int32_t kbeg = blockIdx.y * kchunk;
  const int half = lane >> 5;
  const bool arow = mrow < M, brow = ncol < N;
  const int8_t* pa = A + mrow * K + kbeg + 32 * half;
  const int8_t* pb = B + (int64_t)ncol * K + kbeg + 32 * half;
  i32x16 acc = i32x16{};
  // 64 contraction bytes per step: lane half h supplies bytes [32h, 32h + 32).
#pragma unroll 4
  for (int32_t k = 0; k < kchunk; k += 64) {
    i32x4 a0 = arow ? *reinterpret_cast<const i32x4*>(pa + k) : i32x4{0, 0, 0, 0};
    i32x4 a1 = arow ? *reinterpret_cast<const i32x4*>(pa + k + 16) : i32x4{0, 0, 0, 0};
    i32x4 b0 = brow ? *reinterpret_cast<const i32x4*>(pb + k) : i32x4{0, 0, 0, 0};
    i32x4 b1 = brow ? *reinterpret_cast<const i32x4*>(pb + k + 16) : i32x4{0, 0, 0, 0};
    acc = __builtin_amdgcn_mfma_i32_32x32x32_i8(a0, b0, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_i32_32x32x32_i8(a1, b1, acc, 0, 0, 0);
  }
  if (!brow) return;
  int32_t* pp = part + (int64_t)blockIdx.y * M * N;
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    const int64_t m = 8 * (v >> 2) + 4 * half + (v & 3);
    if (m < M) pp[m * N + ncol] = acc[v];
  }
}

// Sum the slices of 4 consecutive columns, dequantize, store fp16.
__global__ void __launch_bounds__(256)
splitk_epilogue_kernel(const int32_t* __restrict__ part, int32_t split, const float* __restrict__ rs,
                       const float* __restrict__ cs, int64_t M, int32_t N, DevSegs sg,
                       int32_t* __restrict__ dbg) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int32_t n4 = N / 4;
  if (i >= M * n4) return;
  const int64_t m = i / n4;
  const int32_t n = 4 * (int32_t)(i - m * n4);
  i32x4 acc = i32x4{0, 0, 0, 0};
#pragma unroll 8
  for (int sl = 0; sl < split; ++sl) acc += *reinterpret_cast<const i32x4*>(part + ((int64_t)sl * M + m) * N + n);
  if (dbg) *reinterpret_cast<i32x4*>(dbg + m * N + n) = acc;
  const float r_s = rs[m];
  for (int e = 0; e < 4; ++e) store_out(sg, m, n + e, dequant(acc[e], r_s, cs[n + e]));
}

// Down-projection epilogue for M <= 32 fused with the latent quantization:
// one workgroup per token row.  Each thread owns 8 consecutive latent
// columns per pass (two passes cover r <= 4096): sum the slices, dequantize
// to fp16 C, keep it in registers, reduce max |C| over the row, then quantize
// the row exactly as the stand-alone quantizer does (clip 1).
template <int ABITS>
__global__ void __launch_bounds__(256)
splitk_latent_epilogue_kernel(const int32_t* __restrict__ part, int32_t split, const float* __restrict__ sx,
                              const float* __restrict__ sa, int64_t M, int32_t r, _Float16* __restrict__ c_h,
                              uint8_t* __restrict__ cq, float* __restrict__ sc, int32_t* __restrict__ dbg) {
  __shared__ float red[4];
  const int64_t m = blockIdx.x;
  const int tid = threadIdx.x;
  const float rs = sx[m];
  f16x8 hv[2];
  float amax = 0.f;
#pragma unroll
  for (int pass = 0; pass < 2; ++pass) {
    const int32_t n = 8 * (tid + 256 * pass);
    hv[pass] = f16x8{};
    if (n < r) {
      i32x4 a0 = i32x4{0, 0, 0, 0}, a1 = i32x4{0, 0, 0, 0};
#pragma unroll 8
      for (int sl = 0; sl < split; ++sl) {
        const int32_t* src = part + ((int64_t)sl * M + m) * r + n;
        a0 += *reinterpret_cast<const i32x4*>(src);
        a1 += *reinterpret_cast<const i32x4*>(src + 4);
      }
      if (dbg) {
        *reinterpret_cast<i32x4*>(dbg + m * r + n) = a0;
        *reinterpret_cast<i32x4*>(dbg + m * r + n + 4) = a1;
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const _Float16 hval = to_f16(dequant(e < 4 ? a0[e] : a1[e - 4], rs, sa[n + e]));
        hv[pass][e] = hval;
        amax = fmaxf(amax, fabsf((float)hval));
      }
      *reinterpret_cast<f16x8*>(c_h + m * r + n) = hv[pass];
    }
  }
  amax = wave_max(amax);
  if ((tid & 63) == 0) red[tid >> 6] = amax;
  __syncthreads();
  amax = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  const float qm = (float)((1 << (ABITS - 1)) - 1);
  const float a = mul_rn(1.f, amax);
  float inv = 0.f, s = 1.f;
  if (a != 0.f) {
    inv = div_rn(qm, a);
    s = div_rn(a, qm);
  }
  if (tid == 0) sc[m] = s;
#pragma unroll
  for (int pass = 0; pass < 2; ++pass) {
    const int32_t n = 8 * (tid + 256 * pass);
    if (n >= r) continue;
    int q[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) q[e] = (a != 0.f) ? quant_code(mul_rn((float)hv[pass][e], inv), qm) : 0;
    if (ABITS == 8) {
      uint32_t lo = (q[0] & 0xff) | ((q[1] & 0xff) << 8) | ((q[2] & 0xff) << 16) | ((uint32_t)(q[3] & 0xff) << 24);
      uint32_t hi = (q[4] & 0xff) | ((q[5] & 0xff) << 8) | ((q[6] & 0xff) << 16) | ((uint32_t)(q[7] & 0xff) << 24);
      *reinterpret_cast<uint2*>(cq + m * r + n) = make_uint2(lo, hi);
    } else {
      uint32_t p = 0;
#pragma unroll
      for (int e = 0; e < 8; ++e) p |= (uint32_t)(q[e] & 0xf) << (4 * e);
      *reinterpret_cast<uint32_t*>(cq + m * (r / 2) + n / 2) = p;
    }
  }
}

static DevSegs to_dev(const GemmArgs& g) {
  DevSegs d{};
  d.n_seg = g.n_seg;
  for (int s = 0; s < 3; ++s) {
    d.ptr[s] = s < g.n_seg ? g.seg[s].ptr : nullptr;
    d.ld[s] = s < g.n_seg ? g.seg[s].ld : 0;
    d.n0[s] = s < g.n_seg ? g.seg[s].n0 : 0;
    d.n[s] = s < g.n_seg ? g.seg[s].n : 0;
  }
  return d;
}

static bool use_splitk(int64_t M) { return M <= 32; }

// Number of contraction slices: about 256 workgroups stream the weight, at
// most 16 slices for the epilogue to add.
static int splitk_slices(int32_t N, int32_t K) {
  const int nblk = (N + SBN - 1) / SBN;
  const int steps = K / 64;
  int split = 256 / nblk;
  if (split < 1) split = 1;
  if (split > 16) split = 16;
  if (split > steps) split = steps;
  while (steps % split) --split;
  return split;
}

size_t gemm_i8_workspace(int64_t M, int32_t N, int32_t K) {
  return use_splitk(M) ? (size_t)splitk_slices(N, K) * M * N * sizeof(int32_t) : 0;
}

hipError_t launch_gemm_i8(const GemmArgs& g, void* ws, size_t ws_bytes, hipStream_t s) {
  if (g.M == 0 || g.N == 0) return hipSuccess;
  const size_t need = gemm_i8_workspace(g.M, g.N, g.K);
  if (need > 0 && (!ws || ws_bytes < need)) return hipErrorInvalidValue;
  const DevSegs sg = to_dev(g);
  const bool latent = g.cq != nullptr;
  if (!use_splitk(g.M)) {
    dim3 grid((g.N + TBN - 1) / TBN, (unsigned)((g.M + TBM - 1) / TBM));
    {
      KernelScope ks("gemm_i8_tiled", s);
      hipLaunchKernelGGL(gemm_i8_tiled_kernel, grid, dim3(256), 0, s, g.a, g.b, g.row_scale, g.col_scale, g.M,
                         g.N, g.K, sg, g.dbg);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || !latent) return e;
    return launch_quantize_rows(g.seg[0].ptr, g.M, g.N, g.seg[0].ld, g.abits, 1.f, g.cq, g.sc, s);
  }
  int32_t* part = (int32_t*)ws;
  const int split = splitk_slices(g.N, g.K);
  const int32_t kchunk = (g.K / 64 / split) * 64;
  {
    KernelScope ks("gemm_i8_splitk", s);
    hipLaunchKernelGGL(gemm_i8_splitk_kernel, dim3((g.N + SBN - 1) / SBN, split), dim3(256), 0, s, g.a, g.b, g.M,
                       g.N, g.K, kchunk, part);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (latent) {
    KernelScope ks("splitk_latent_epilogue", s);
    if (g.abits == 8)
      hipLaunchKernelGGL(splitk_latent_epilogue_kernel<8>, dim3((unsigned)g.M), dim3(256), 0, s, part, split,
                         g.row_scale, g.col_scale, g.M, g.N, g.seg[0].ptr, (uint8_t*)g.cq, g.sc, g.dbg);
    else
      hipLaunchKernelGGL(splitk_latent_epilogue_kernel<4>, dim3((unsigned)g.M), dim3(256), 0, s, part, split,
                         g.row_scale, g.col_scale, g.M, g.N, g.seg[0].ptr, (uint8_t*)g.cq, g.sc, g.dbg);
  } else {
    const int64_t total = g.M * (g.N / 4);
    KernelScope ks("splitk_epilogue", s);
    hipLaunchKernelGGL(splitk_epilogue_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, s, part, split,
                       g.row_scale, g.col_scale, g.M, g.N, sg, g.dbg);
  }
  return hipGetLastError();
}

}  // namespace qsvd
