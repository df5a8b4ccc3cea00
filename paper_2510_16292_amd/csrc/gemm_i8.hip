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

hipError_t launch_gemm_i8(const GemmArgs& g, hipStream_t s) {
  if (g.M == 0 || g.N == 0) return hipSuccess;
  const DevSegs sg = to_dev(g);
  dim3 grid((g.N + TBN - 1) / TBN, (unsigned)((g.M + TBM - 1) / TBM));
  {
    KernelScope ks("gemm_i8_tiled", s);
    hipLaunchKernelGGL(gemm_i8_tiled_kernel, grid, dim3(256), 0, s, g.a, g.b, g.row_scale, g.col_scale, g.M, g.N,
                       g.K, sg, g.dbg);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || !g.cq) return e;
  return launch_quantize_rows(g.seg[0].ptr, g.M, g.N, g.seg[0].ld, g.abits, 1.f, g.cq, g.sc, s);
}

}  // namespace qsvd
