// Decode-size projections (M <= 32 token rows) on v_mfma_i32_16x16x64_i8.
//
// The weight is the large operand here (M is the decode batch), so each
// workgroup owns 16 output columns over the whole contraction: up to 16 waves
// split the contraction, each streaming its slice of the 16 weight rows once
// with all of its loads in flight together, and leave exact int32 partial sums
// in LDS.  No partial sums go through HBM and no second kernel is needed.
//
// 16x16x64 operand layout: lane l supplies row (l % 16) of A and column
// (l % 16) of B, 16 contraction bytes each (which bytes only has to agree
// between A and B: integer sums are exact in any order).  Output: lane l holds
// column l % 16 and rows 4 * (l / 16) + v, v = 0..3.
//
// Per-channel weights: the waves' int32 sums are added (exact) and dequantized
// as (f32(acc) * s_row) * s_col.  Per-group weights (int4, groups of G along the
// contraction): every group's int32 sum is kept in LDS and one thread per
// output adds f32(acc_g) * s[g][n] over the groups in order, then * s_row --
// the same sequence of fp32 roundings as the stand-alone definition.
//
// Up-projection (A = the fp16 latent C): every workgroup first takes each row's
// max |C|, quantizes the rows into LDS (Q(C), Section 4's per-token symmetric
// rule) and uses them as the A operand; workgroup (m mod grid) also stores row
// m's codes and scale.  The first batch of weight loads is issued before this
// so that its HBM latency overlaps the row pass.
#include <algorithm>

#include "common.h"
#include "launch.h"
#include "rowpass.h"

namespace qsvd {

constexpr int kSkCols = 16;        // output columns of one 16x16x64 product
constexpr int kSkMinGrid = 256;    // workgroups wanted: one per CU
constexpr int kSkMaxWaves = 16;
constexpr int kSkBatch = 4;        // 64-byte contraction steps loaded per batch
constexpr int kSkMaxGroups = 64;   // scale groups along the contraction
constexpr size_t kSkLdsLimit = 160 * 1024 - 5 * 1024;   // dynamic LDS beside the static scale arrays

struct SkinnyOut {
  _Float16* ptr[3];
  int64_t ld[3];
  int32_t n0[3];
  int32_t n[3];
  int32_t n_seg;
};

// Selects rather than indexes the segment arrays, so that the argument struct
// is only ever read at constant offsets (an indexed copy would go to scratch).
__device__ __forceinline__ void sk_store(const SkinnyOut& so, int64_t m, int32_t n, float y) {
  const bool in0 = so.n_seg > 0 && n >= so.n0[0] && n < so.n0[0] + so.n[0];
  const bool in1 = !in0 && so.n_seg > 1 && n >= so.n0[1] && n < so.n0[1] + so.n[1];
  const bool in2 = !in0 && !in1 && so.n_seg > 2 && n >= so.n0[2] && n < so.n0[2] + so.n[2];
  _Float16* base = in0 ? so.ptr[0] : in1 ? so.ptr[1] : in2 ? so.ptr[2] : nullptr;
  if (!base) return;
  const int64_t ld = in0 ? so.ld[0] : in1 ? so.ld[1] : so.ld[2];
  const int32_t n0 = in0 ? so.n0[0] : in1 ? so.n0[1] : so.n0[2];
  base[m * ld + (n - n0)] = to_f16(y);
}

// 16 int4 codes (8 bytes, element 2i in the low nibble of byte i) -> 16 int8.
__device__ __forceinline__ i32x4 unpack16_i4(uint2 p) {
  i32x4 o;
  const uint32_t w[2] = {p.x, p.y};
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    uint32_t lo = 0, hi = 0;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      lo |= (uint32_t)((((int)(w[h] << (28 - 4 * e))) >> 28) & 0xff) << (8 * e);
      hi |= (uint32_t)((((int)(w[h] << (12 - 4 * e))) >> 28) & 0xff) << (8 * e);
    }
    o[2 * h] = (int32_t)lo;
    o[2 * h + 1] = (int32_t)hi;
  }
  return o;
}

// A operand source: int8 or packed int4 codes (down-projection: the quantized
// activations), or fp16 rows quantized per row by the workgroup itself (the
// latent C in the up-projection, clip 1; or the activations X in the fused
// decode down-projection, with the caller's clip), 8- or 4-bit codes.
enum { SK_A_I8 = 0, SK_A_F16Q = 1 };

// Contraction steps [s0, s1) of wave w: contiguous ranges, whole groups when the
// weights carry per-group scales.
__device__ __forceinline__ void sk_span(int w, int nw, int32_t K, int32_t group, int& s0, int& s1) {
  if (group) {
    const int ng = K / group, gs = group / 64;
    s0 = (w * ng / nw) * gs;
    s1 = ((w + 1) * ng / nw) * gs;
  } else {
    const int steps = K / 64;
    s0 = w * steps / nw;
    s1 = (w + 1) * steps / nw;
  }
}

template <int ASRC, int WBITS, bool WIDE = false>
__global__ void __launch_bounds__(64 * kSkMaxWaves)
skinny_gemm_kernel(const void* __restrict__ a_src, int64_t lda, float clip, const float* __restrict__ row_scale_in,
                   const uint8_t* __restrict__ bt, const float* __restrict__ col_scale, int32_t sstride,
                   int32_t M, int32_t N, int32_t K, int32_t group, int32_t nw, int32_t abits, int32_t qa_off,
                   SkinnyOut so, int32_t* __restrict__ dbg, uint8_t* __restrict__ cq_out, float* __restrict__ sc_out,
                   SkinnyAppend ap, int32_t cols) {
  // [0, qa_off): int32 tiles, [slot][row block][lane] (slot = wave for
  // per-channel weights, group for per-group ones); [qa_off, ...): Q(C) rows.
  extern __shared__ __attribute__((aligned(16))) uint8_t sk_lds[];
  i32x4* red = reinterpret_cast<i32x4*>(sk_lds);
  int8_t* qa = reinterpret_cast<int8_t*>(sk_lds + qa_off);
  __shared__ float rsc[32];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int l16 = lane & 15, quad = lane >> 4;
  // the workgroup's first `cols` (16, 8 or 4) product columns are output
  // columns, the rest of the product stays zero
  const int32_t n = blockIdx.x * cols + l16;           // this lane's weight row (output column)
  const bool ncol = l16 < cols && n < N;
  const int rbl = (M + 15) / 16;
  const int qa_ld = K + 16;

  int s0, s1;
  sk_span(w, nw, K, group, s0, s1);

  // Epilogue scales are fetched first, so that their latency hides behind
  // the weight stream: this thread's first output (row, column) scales in
  // registers, per-group column scales of the tile in LDS.
  __shared__ float s_gscale[kSkMaxGroups * kSkCols];
  const int ng = group ? K / group : 0;
  float pre_rs = 1.f, pre_cs = 0.f;
  if (tid < M * cols) {
    const int32_t nn = blockIdx.x * cols + tid % cols;
    if (nn < N) {
      if (ASRC == SK_A_I8) pre_rs = row_scale_in[tid / cols];
      if (!group) pre_cs = col_scale[nn];
    }
  }
  for (int i = tid; i < ng * kSkCols; i += 64 * nw) {
    const int32_t nn = blockIdx.x * cols + i % kSkCols;
    s_gscale[i] = i % kSkCols < cols && nn < N ? col_scale[(int64_t)(i / kSkCols) * sstride + nn] : 0.f;
  }

  i32x4 bw[kSkBatch];
  auto load_b = [&](int st0) {
#pragma unroll
    for (int s = 0; s < kSkBatch; ++s) {
      const int st = st0 + s;
      const int32_t k = 64 * st + 16 * quad;
      if (st < s1 && ncol) {
        if (WBITS == 8)
          bw[s] = *reinterpret_cast<const i32x4*>(bt + (int64_t)n * K + k);
        else
          bw[s] = unpack16_i4(*reinterpret_cast<const uint2*>(bt + ((int64_t)n * K + k) / 2));
      } else {
        bw[s] = i32x4{0, 0, 0, 0};
      }
    }
  };
  load_b(s0);

  if (ASRC == SK_A_F16Q) {
    sk_row_pass<WIDE>(reinterpret_cast<const _Float16*>(a_src), lda, clip, M, K, abits, w, nw, lane, qa, qa_ld,
                      rsc, cq_out, sc_out, ap);
    __syncthreads();
    sk_advance(ap, M, tid);
  }

  // --- contraction over this wave's steps ------------------------------------
  const int gsteps = group ? group / 64 : 0;
  i32x4 acc[2] = {i32x4{0, 0, 0, 0}, i32x4{0, 0, 0, 0}};
  int step_in_group = 0;
  for (int st0 = s0; st0 < s1; st0 += kSkBatch) {
    if (st0 != s0) load_b(st0);
    i32x4 aw[kSkBatch][2];
#pragma unroll
    for (int s = 0; s < kSkBatch; ++s) {
      const int32_t k = 64 * (st0 + s) + 16 * quad;
#pragma unroll
      for (int rb = 0; rb < 2; ++rb) {
        const int m = 16 * rb + l16;
        if (st0 + s < s1 && rb < rbl && m < M) {
          if (ASRC == SK_A_I8 && abits == 8)
            aw[s][rb] = *reinterpret_cast<const i32x4*>(reinterpret_cast<const int8_t*>(a_src) + (int64_t)m * K + k);
          else if (ASRC == SK_A_I8)     // 4-bit codes, two per byte
            aw[s][rb] = unpack16_i4(*reinterpret_cast<const uint2*>(reinterpret_cast<const uint8_t*>(a_src) +
                                                                   ((int64_t)m * K + k) / 2));
          else
            aw[s][rb] = *reinterpret_cast<const i32x4*>(qa + m * qa_ld + k);
        } else {
          aw[s][rb] = i32x4{0, 0, 0, 0};
        }
      }
    }
#pragma unroll
    for (int s = 0; s < kSkBatch; ++s) {
      if (st0 + s >= s1) continue;     // (not break: keeps the register arrays statically indexed)
#pragma unroll
      for (int rb = 0; rb < 2; ++rb)
        if (rb < rbl) acc[rb] = __builtin_amdgcn_mfma_i32_16x16x64_i8(aw[s][rb], bw[s], acc[rb], 0, 0, 0);
      if (gsteps && ++step_in_group == gsteps) {
        const int g = (st0 + s) / gsteps;
#pragma unroll
        for (int rb = 0; rb < 2; ++rb) {
          if (rb < rbl) red[(g * rbl + rb) * 64 + lane] = acc[rb];
          acc[rb] = i32x4{0, 0, 0, 0};
        }
        step_in_group = 0;
      }
    }
  }
  if (!gsteps)
#pragma unroll
    for (int rb = 0; rb < 2; ++rb)
      if (rb < rbl) red[(w * rbl + rb) * 64 + lane] = acc[rb];
  __syncthreads();

  // --- epilogue: one thread per output (row m, column n) ------------------------
  for (int t = tid; t < M * cols; t += 64 * nw) {
    const int m = t / cols, nl = t % cols;
    const int32_t nn = blockIdx.x * cols + nl;
    if (nn >= N) continue;
    const int rb = m >> 4, mm = m & 15, src = 16 * (mm >> 2) + nl, v = mm & 3;
    const bool first = t == tid;
    const float rs = ASRC == SK_A_I8 ? (first ? pre_rs : row_scale_in[m]) : rsc[m];
    float y;
    if (!group) {
      int32_t tot = 0;
      for (int ww = 0; ww < nw; ++ww) tot += red[(ww * rbl + rb) * 64 + src][v];
      if (dbg) dbg[(int64_t)m * N + nn] = tot;
      y = mul_rn(mul_rn((float)tot, rs), first ? pre_cs : col_scale[nn]);
    } else {
      float S = 0.f;
      for (int g = 0; g < ng; ++g)
        S = add_rn(S, mul_rn((float)red[(g * rbl + rb) * 64 + src][v], s_gscale[g * kSkCols + nl]));
      y = mul_rn(S, rs);
    }
    sk_store(so, m, nn, y);
    if (ap.mode == SK_APPEND_F16_ROW) {
      const int32_t pos = ap.seq_len[m];
      if (pos >= 0 && pos < ap.capacity)
        reinterpret_cast<_Float16*>(ap.data)[((int64_t)m * ap.capacity + pos) * N + nn] = to_f16(y);
    }
  }
}

struct SkinnyPlan {
  int nw;            // waves per workgroup
  int32_t qa_off;    // LDS bytes of the int32 tiles
  size_t lds;        // dynamic LDS bytes
  int32_t cols;      // output columns per workgroup
};

// Narrower column strips (8 or 4 of the product's 16 columns) while the grid
// still fits one workgroup per CU: the weight stream then spreads over more
// CUs, at the price of a repeated A operand (and row pass) per workgroup and
// idle product columns.  (A second round of workgroups would double the time.)
static SkinnyPlan skinny_plan(int64_t M, int32_t K, int32_t N, int32_t group, bool f16q) {
  SkinnyPlan p{};
  p.cols = kSkCols;
  while (p.cols > 4 && (N + p.cols / 2 - 1) / (p.cols / 2) <= kSkMinGrid) p.cols /= 2;
  const int steps = K / 64, ng = group ? K / group : 0;
  p.nw = std::min(kSkMaxWaves, group ? ng : steps);
  // more column blocks than CUs: workgroups of at most half the waves, so
  // that two share a CU and the grid still takes one round
  if ((N + p.cols - 1) / p.cols > kSkMinGrid) p.nw = std::min(p.nw, kSkMaxWaves / 2);
  const int rbl = (int)((M + 15) / 16);
  const size_t tiles = (size_t)(group ? ng : p.nw) * rbl * 64 * sizeof(i32x4);
  p.qa_off = (int32_t)tiles;
  p.lds = tiles + (f16q ? (size_t)M * (K + 16) : 0);
  return p;
}

bool skinny_supported(int64_t M, int32_t K, int32_t group, bool f16q) {
  if (M < 1 || M > 32 || K < 64 || K % 64) return false;
  if (group && (group % 64 || K % group || K / group > kSkMaxGroups)) return false;
  if (f16q && K > kSkMaxRowK) return false;
  return skinny_plan(M, K, kSkCols, group, f16q).lds <= kSkLdsLimit;
}

hipError_t launch_skinny(const GemmArgs& g, bool a_is_f16_latent, int32_t wbits, int32_t group, int32_t sstride,
                         hipStream_t s) {
  return launch_skinny_fused(g, a_is_f16_latent ? SKA_F16_LATENT : SKA_CODES, 1.f, g.K, wbits, group, sstride,
                             SkinnyAppendArgs{}, s);
}

hipError_t launch_skinny_fused(const GemmArgs& g, int32_t asrc, float clip, int64_t lda, int32_t wbits, int32_t group,
                               int32_t sstride, const SkinnyAppendArgs& aa, hipStream_t s) {
  const bool a_is_f16_latent = asrc != SKA_CODES;
  if (g.M == 0 || g.N == 0) return hipSuccess;
  if (!skinny_supported(g.M, g.K, group, a_is_f16_latent)) return hipErrorInvalidValue;
  SkinnyOut so{};
  so.n_seg = g.n_seg;
  for (int i = 0; i < 3; ++i) {
    so.ptr[i] = i < g.n_seg ? g.seg[i].ptr : nullptr;
    so.ld[i] = i < g.n_seg ? g.seg[i].ld : 0;
    so.n0[i] = i < g.n_seg ? g.seg[i].n0 : 0;
    so.n[i] = i < g.n_seg ? g.seg[i].n : 0;
  }
  const SkinnyPlan p = skinny_plan(g.M, g.K, g.N, group, a_is_f16_latent);
  dim3 grid((g.N + p.cols - 1) / p.cols), block(64 * p.nw);
  const int32_t M = (int32_t)g.M;
  const uint8_t* bt = (const uint8_t*)g.b;
  // more than 64 KB of dynamic LDS has to be allowed per kernel before the launch
  auto allow = [&](const void* fn) -> hipError_t {
    return p.lds > 65536 ? hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)p.lds)
                         : hipSuccess;
  };
  SkinnyAppend ap{(uint8_t*)aa.data, aa.scale, aa.seq_len, aa.overflow, aa.capacity, aa.mode};
  KernelScope ks(asrc == SKA_F16_ACT ? "skinny_down_q" : a_is_f16_latent ? "skinny_up" : "skinny_down", s);
  if (!a_is_f16_latent) {
    auto k = wbits == 8 ? skinny_gemm_kernel<SK_A_I8, 8> : skinny_gemm_kernel<SK_A_I8, 4>;
    if (hipError_t e = allow((const void*)k); e != hipSuccess) return e;
    QSVD_LAUNCH(ks, k, grid, block, p.lds, s, (const void*)g.a, (int64_t)g.K, 1.f, g.row_scale, bt, g.col_scale,
                       sstride, M, g.N, g.K, group, p.nw, g.abits, p.qa_off, so, g.dbg, (uint8_t*)nullptr,
                       (float*)nullptr, ap, p.cols);
  } else {
    // rows wider than the row pass holds at once take the two-read variant
    const bool wide = g.K > 64 * 8 * kSkMaxRowChunks;
    auto k = wbits == 8 ? (wide ? skinny_gemm_kernel<SK_A_F16Q, 8, true> : skinny_gemm_kernel<SK_A_F16Q, 8>)
                        : (wide ? skinny_gemm_kernel<SK_A_F16Q, 4, true> : skinny_gemm_kernel<SK_A_F16Q, 4>);
    if (hipError_t e = allow((const void*)k); e != hipSuccess) return e;
    QSVD_LAUNCH(ks, k, grid, block, p.lds, s, (const void*)g.a, lda, clip, (const float*)nullptr, bt, g.col_scale,
                       sstride, M, g.N, g.K, group, p.nw, g.abits, p.qa_off, so, g.dbg, (uint8_t*)g.cq, g.sc, ap, p.cols);
  }
  return hipGetLastError();
}

}  // namespace qsvd
