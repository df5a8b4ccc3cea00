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
#include <type_traits>

namespace qsvd {

// Output segments (columns [n0, n0 + n) of the product go to ptr with row
// stride ld); fields are spelled out per segment so that a store only ever
// reads kernel arguments at constant offsets.
struct DevSegs {
  _Float16* p0; _Float16* p1; _Float16* p2;
  int64_t ld0, ld1, ld2;
  int32_t a0, a1, a2;      // first column of each segment
  int32_t e0, e1, e2;      // one past the last column
};

// Where column n of the product goes: its first element's address and the row
// stride (NULL if the column is not stored).  Selects rather than branches, so
// the three segment pointers stay in registers.
struct ColOut {
  _Float16* p;
  int64_t ld;
};

__device__ __forceinline__ ColOut col_out(const DevSegs& sg, int32_t n) {
  const bool in0 = n >= sg.a0 && n < sg.e0;
  const bool in1 = n >= sg.a1 && n < sg.e1;
  const bool in2 = n >= sg.a2 && n < sg.e2;
  _Float16* p = in0 ? sg.p0 + (n - sg.a0) : in1 ? sg.p1 + (n - sg.a1) : in2 ? sg.p2 + (n - sg.a2) : nullptr;
  if (!(in0 ? sg.p0 : in1 ? sg.p1 : in2 ? sg.p2 : nullptr)) p = nullptr;
  const int64_t ld = in0 ? sg.ld0 : in1 ? sg.ld1 : sg.ld2;
  return ColOut{p, ld};
}

// Dequantize one integer accumulator: (f32(acc) * row_scale) * col_scale, each
// product rounded to fp32 on its own.
__device__ __forceinline__ float dequant(int32_t acc, float rs, float cs) {
  return mul_rn(mul_rn((float)acc, rs), cs);
}
__device__ __forceinline__ float dequant(float acc, float rs, float cs) { return mul_rn(mul_rn(acc, rs), cs); }

// ---------------------------------------------------------------------------
// Pipelined kernel: BM x BN output tile per workgroup of 4 or 8 waves (each
// WM x WN), the contraction in stages of 64 bytes.  With F16 the operands are
// fp16 (a stage is 32 contraction elements, v_mfma_f32_32x32x16_f16, fp32
// accumulators; a 16-byte slot is 8 elements, so the slot layout, the loads
// and the fragment reads are the same) and K counts bytes per row.  Operands go from global
// memory straight into LDS (global_load_lds_dwordx4: lane i of a wave writes
// 16 bytes at base + 16 i), NS stages deep, so NS - 1 stages are in flight
// while one is multiplied; one barrier per stage.
//
// LDS layout of a stage: blocks of 16 rows x 64 bytes (1 KB); in a block,
// 16-byte slot 4 * (row % 16) + (chunk ^ ((row / 4) % 4)) holds contraction
// chunk `chunk` of that row.  A fragment read (16 consecutive rows, one chunk)
// then touches every bank once.
// ---------------------------------------------------------------------------
typedef __attribute__((address_space(3))) void lds_void_t;
typedef __attribute__((address_space(1))) void glb_void_t;

constexpr int PBK = 64;

// Wait until at most N direct loads of this wave are outstanding (and its LDS
// reads are done), then meet the other waves.  Written as one asm statement
// so that the compiler neither adds a full wait nor moves LDS accesses across.
template <int N>
__device__ __forceinline__ void vm_wait_barrier() {
  asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(N) : "memory");
}

// The stage being consumed was issued `rem` stages before the newest one.
template <int LPW, int R>
__device__ __forceinline__ void vm_wait_stage(int rem) {
  if constexpr (R == 0) {
    vm_wait_barrier<0>();
  } else {
    if (rem >= R) vm_wait_barrier<R * LPW>();
    else vm_wait_stage<LPW, R - 1>(rem);
  }
}

__device__ __forceinline__ int pipe_slot(int row, int chunk) {
  return (row >> 4) * 1024 + (4 * (row & 15) + (chunk ^ ((row >> 2) & 3))) * 16;
}

template <int BM, int BN, int WM, int WN, int NS>
struct PipeCfg {
  static constexpr int kWaves = (BM / WM) * (BN / WN);
  static_assert(kWaves == 4 || kWaves == 8, "four or eight waves");
  static constexpr int kThreads = 64 * kWaves;
  static constexpr int kABlocks = BM / 16, kBBlocks = BN / 16;
  static_assert((kABlocks + kBBlocks) % kWaves == 0, "whole 1 KB loads per wave");
  static constexpr int kLPW = (kABlocks + kBBlocks) / kWaves;   // direct loads per wave per stage
  static constexpr int kStage = (kABlocks + kBBlocks) * 1024;
  static constexpr size_t kStages = (size_t)NS * kStage;
  static constexpr size_t kOut = (size_t)kWaves * WM * (WN + 8) * 2;   // fp16 output staging
  static constexpr size_t kLds = kStages > kOut ? kStages : kOut;
};

template <int BM, int BN, int WM, int WN, int NS, bool DBG, bool F16, bool RS = false>
__global__ void __launch_bounds__((PipeCfg<BM, BN, WM, WN, NS>::kThreads))
gemm_i8_pipe_kernel(const int8_t* __restrict__ A, const int8_t* __restrict__ B,
                    const float* __restrict__ rs, const float* __restrict__ cs,
                    int64_t M, int32_t N, int32_t K, int32_t n_tiles_n, int32_t gm, DevSegs sg,
                    int32_t* __restrict__ dbg, RopeEpi re) {
  using C = PipeCfg<BM, BN, WM, WN, NS>;
  using Acc = std::conditional_t<F16, f32x16, i32x16>;
  static_assert(!(DBG && F16), "accumulator dumps are for the integer products");
  constexpr int TI = WM / 32, TJ = WN / 32;
  extern __shared__ __attribute__((aligned(1024))) uint8_t pipe_smem[];
  __shared__ __attribute__((aligned(16))) float s_rs[BM];
  __shared__ __attribute__((aligned(16))) float s_cs[BN];
  const int tid = threadIdx.x, lane = tid & 63, w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = w / (BN / WN), wn = w % (BN / WN);
  const int l32 = lane & 31, hl = lane >> 5;
  int tm, tn;
  xcd_tile(blockIdx.x, gridDim.x, n_tiles_n, gm, &tm, &tn);
  const int64_t m0 = (int64_t)tm * BM;
  const int32_t n0 = tn * BN;
  const int nk = K / PBK;

  // Each direct load of this wave covers one 16-row block of A or B; its
  // per-lane source offset from the tile's first row is fixed, so a stage
  // only advances the (scalar) tile base by 64 bytes.
  const int8_t* a_tile = A + m0 * K;
  const int8_t* b_tile = B + (int64_t)n0 * K;
  uint32_t voff[C::kLPW];
#pragma unroll
  for (int j = 0; j < C::kLPW; ++j) {
    const int blk = w * C::kLPW + j;                         // wave-uniform
    const bool is_a = blk < C::kABlocks;
    const int row = 16 * (is_a ? blk : blk - C::kABlocks) + (lane >> 2);
    const int chunk = (lane & 3) ^ ((row >> 2) & 3);
    const int64_t last = is_a ? M - 1 - m0 : (int64_t)N - 1 - n0;   // clamp ragged tiles to the last row
    voff[j] = (uint32_t)(min((int64_t)row, last) * K + 16 * chunk);
  }
  auto issue = [&](int st) {
    uint8_t* base = pipe_smem + (st % NS) * C::kStage;
    const int64_t k0 = (int64_t)st * PBK;
#pragma unroll
    for (int j = 0; j < C::kLPW; ++j) {
      const int blk = w * C::kLPW + j;
      const int8_t* src = (blk < C::kABlocks ? a_tile : b_tile) + k0 + voff[j];
      __builtin_amdgcn_global_load_lds((glb_void_t*)src, (lds_void_t*)(base + blk * 1024), 16, 0, 0);
    }
  };

  // scales first: their wait then leaves the stage loads in flight
  // (fp16 operands: a NULL scale vector means no scale)
  for (int i = tid; i < BM; i += C::kThreads) s_rs[i] = (!F16 || rs) ? rs[min(m0 + i, M - 1)] : 1.f;
  for (int i = tid; i < BN; i += C::kThreads) s_cs[i] = (!F16 || cs) ? cs[min(n0 + i, N - 1)] : 1.f;
#pragma unroll
  for (int st = 0; st < NS - 1; ++st)
    if (st < nk) issue(st);

  Acc acc[TI][TJ];
#pragma unroll
  for (int i = 0; i < TI; ++i)
#pragma unroll
    for (int j = 0; j < TJ; ++j) acc[i][j] = Acc{};

  // Fragments of one stage, by contraction half kk: af[kk][i], bf[kk][j].
  // Half 1 of a stage is read while half 0's products run, and half 0 of the
  // next stage while half 1's products run.
  i32x4 af[2][TI], bf[2][TJ];
  auto read_half = [&](int kt, int kk) {
    const uint8_t* sa = pipe_smem + (kt % NS) * C::kStage;
    const uint8_t* sb = sa + C::kABlocks * 1024;
#pragma unroll
    for (int i = 0; i < TI; ++i)
      af[kk][i] = *reinterpret_cast<const i32x4*>(sa + pipe_slot(wm * WM + 32 * i + l32, 2 * kk + hl));
#pragma unroll
    for (int j = 0; j < TJ; ++j)
      bf[kk][j] = *reinterpret_cast<const i32x4*>(sb + pipe_slot(wn * WN + 32 * j + l32, 2 * kk + hl));
  };
  auto products = [&](int kk) {
#pragma unroll
    for (int i = 0; i < TI; ++i)
#pragma unroll
      for (int j = 0; j < TJ; ++j)
        if constexpr (F16)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, bf[kk][j]),
                                                             __builtin_bit_cast(f16x8, af[kk][i]), acc[i][j], 0, 0, 0);
        else
          acc[i][j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(bf[kk][j], af[kk][i], acc[i][j], 0, 0, 0);
  };

  // One MFMA goes out before each LDS read of the other half, so the reads
  // run under the products and every wait the compiler places before a
  // product only covers reads issued before it.
  auto interleave = [&]() {
    if constexpr (C::kWaves == 8) return;     // two waves per SIMD interleave by themselves
#pragma unroll
    for (int r = 0; r < TI + TJ; ++r) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // one MFMA
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);   // one LDS read
    }
    __builtin_amdgcn_sched_group_barrier(0x008, TI * TJ - (TI + TJ), 0);
  };
  static_assert(TI * TJ >= TI + TJ, "at least as many products as reads per half");

  // Waiting for stage s (its loads landed; every wave has finished reading
  // stage s - 1) frees slot (s - 1) % NS for stage s + NS - 1.
  vm_wait_stage<C::kLPW, NS - 2>(nk - 1);
  if (NS - 1 < nk) issue(NS - 1);
  read_half(0, 0);
  for (int kt = 0; kt < nk; ++kt) {
    __builtin_amdgcn_sched_barrier(0);
    products(0);
    read_half(kt, 1);
    interleave();
    __builtin_amdgcn_sched_barrier(0);
    // (on the last stage: a full wait and barrier, nothing left to issue)
    vm_wait_stage<C::kLPW, NS - 2>(nk - 2 - kt);
    if (kt + NS < nk) issue(kt + NS);
    __builtin_amdgcn_sched_barrier(0);
    // the next stage's first half (after the last stage: an unused read of a
    // stage slot, which keeps this loop free of branches around products)
    products(1);
    read_half(kt + 1, 0);
    interleave();
    __builtin_amdgcn_sched_barrier(0);
  }

  // Epilogue.  The integer accumulators are dumped as they are (debug only);
  // the dequantized fp16 tile of each wave is staged in LDS (the stages are
  // free once every wave is past its last product) and written back as
  // 16-byte runs of one row.  The products take B's fragment as their first
  // operand, so lane holds row wm*WM + 32i + l32 and the four consecutive
  // columns wn*WN + 32j + 8(v/4) + 4hl + 0..3: one 8-byte LDS write per
  // four outputs.
  if constexpr (DBG) {
#pragma unroll
    for (int j = 0; j < TJ; ++j) {
#pragma unroll
      for (int i = 0; i < TI; ++i)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int64_t m = m0 + wm * WM + 32 * i + l32;
          const int32_t n = n0 + wn * WN + 32 * j + 8 * (v >> 2) + 4 * hl + (v & 3);
          if (m < M && n < N) dbg[m * N + n] = acc[i][j][v];
        }
    }
  }
  vm_wait_barrier<0>();
  constexpr int OST = WN + 8;                   // staged row stride in halves
  _Float16* ost = reinterpret_cast<_Float16*>(pipe_smem) + w * WM * OST;
#pragma unroll
  for (int i = 0; i < TI; ++i) {
    const int rl = 32 * i + l32;                 // this lane's row
    const float rsm = s_rs[wm * WM + rl];
#pragma unroll
    for (int j = 0; j < TJ; ++j)
#pragma unroll
      for (int vq = 0; vq < 4; ++vq) {
        const int cl = 32 * j + 8 * vq + 4 * hl;  // its 4 consecutive columns
        const f32x4 c4 = *reinterpret_cast<const f32x4*>(&s_cs[wn * WN + cl]);
        f16x4 o4;
#pragma unroll
        for (int e = 0; e < 4; ++e) o4[e] = to_f16(dequant(acc[i][j][4 * vq + e], rsm, c4[e]));
        *reinterpret_cast<f16x4*>(ost + rl * OST + cl) = o4;
        // one accumulator block at a time: keeps the live registers few
        __builtin_amdgcn_sched_barrier(0);
      }
  }
  if constexpr (RS) {
    // Rotary scores of the tile's rows: item (row, head of the tile), the
    // threads of a wave on consecutive rows of one head.  The staged element
    // (row, col) sits in the LDS rows of wave (row / WM, col / WN).
    __syncthreads();
    const int dh = re.dh, half = dh >> 1, hpt = BN / dh;
    auto staged = [&](int row, int col) {
      const int wv = (row / WM) * (BN / WN) + col / WN;
      return *reinterpret_cast<const f16x8*>(reinterpret_cast<const _Float16*>(pipe_smem) +
                                             (size_t)wv * WM * OST + (row % WM) * OST + col % WN);
    };
    for (int it = tid; it < BM * hpt; it += C::kThreads) {
      const int row = it % BM, hl = it / BM;
      const int64_t m = m0 + row;
      const int32_t col0 = hl * dh, gkv = (n0 + col0) / dh;
      if (m >= M || n0 + col0 >= N) continue;
      const int64_t bt = re.row0 + m;
      const int b = (int)(bt / re.capacity), t = (int)(bt - (int64_t)b * re.capacity);
      if (t >= min(re.seq_len[b], re.capacity)) continue;
      float* prow = re.pre + bt * 32;
      const float4* cst = reinterpret_cast<const float4*>(re.rope + (int64_t)t * half);
      for (int g = 0; g < re.G; ++g) {
        const float4* qh = reinterpret_cast<const float4*>(re.qrot + ((int64_t)b * re.Hq + gkv * re.G + g) * dh);
        // rot(k) . q over the pairs (j, j + half):
        //   cos * (k_j q_j + k'_j q'_j) + sin * (k_j q'_j - k'_j q_j)
        float acc = 0.f;
        for (int j0 = 0; j0 < half; j0 += 8) {
          const f16x8 ka = staged(row, col0 + j0), kb = staged(row, col0 + half + j0);
          float4 c4[4], qa[2], qb[2];
#pragma unroll
          for (int u = 0; u < 4; ++u) c4[u] = cst[j0 / 2 + u];
#pragma unroll
          for (int u = 0; u < 2; ++u) {
            qa[u] = qh[j0 / 4 + u];
            qb[u] = qh[(half + j0) / 4 + u];
          }
#pragma unroll
          for (int i = 0; i < 8; ++i) {
            const float a = (float)ka[i], bb = (float)kb[i];
            const float qj = qa[i / 4][i % 4], qk = qb[i / 4][i % 4];
            const float cs_c = (i & 1) ? c4[i / 2].z : c4[i / 2].x, cs_s = (i & 1) ? c4[i / 2].w : c4[i / 2].y;
            const float uu = fmaf(bb, qk, a * qj), vv = fmaf(-bb, qj, a * qk);
            acc = fmaf(cs_c, uu, acc);
            acc = fmaf(cs_s, vv, acc);
          }
        }
        prow[gkv * re.G + g] = acc;
      }
      if (n0 + col0 == 0)
        for (int h = re.Hq; h < 32; ++h) prow[h] = 0.f;
    }
    return;
  }
  // Output rows leave non-temporally: the tile is written once and read by
  // a later kernel, so it need not displace the operands in L2.
  constexpr int CPR = WN / 8;                   // 16-byte chunks per staged row
  for (int e = lane; e < WM * CPR; e += 64) {
    const int row = e / CPR, c8 = e % CPR;
    const int64_t m = m0 + wm * WM + row;
    const int32_t n = n0 + wn * WN + 8 * c8;
    if (m >= M || n >= N) continue;
    const ColOut co = col_out(sg, n);
    if (co.p) __builtin_nontemporal_store(*reinterpret_cast<const f16x8*>(ost + row * OST + 8 * c8), reinterpret_cast<f16x8*>(co.p + m * co.ld));
  }
}

// Segments are consecutive and ascending in the column range; missing ones
// become empty ranges past the last column.
static DevSegs to_dev(const GemmArgs& g) {
  DevSegs d{};
  _Float16** ps[3] = {&d.p0, &d.p1, &d.p2};
  int64_t* lds[3] = {&d.ld0, &d.ld1, &d.ld2};
  int32_t* as[3] = {&d.a0, &d.a1, &d.a2};
  int32_t* es[3] = {&d.e0, &d.e1, &d.e2};
  for (int s = 0; s < 3; ++s) {
    if (s < g.n_seg) {
      *ps[s] = g.seg[s].ptr;
      *lds[s] = g.seg[s].ld;
      *as[s] = g.seg[s].n0;
      *es[s] = g.seg[s].n0 + g.seg[s].n;
    } else {
      *ps[s] = nullptr;
      *lds[s] = 0;
      *as[s] = *es[s] = s > 0 ? *es[s - 1] : 0;
    }
  }
  return d;
}

// Tiles one XCD runs at once: its 32 CUs, one workgroup each.
constexpr int kGemmTilesPerXcd = 32;

template <int BM, int BN, int WM, int WN, int NS, bool DBG, bool F16 = false, bool RS = false>
static hipError_t launch_pipe(const GemmArgs& g, const DevSegs& sg, hipStream_t s, const RopeEpi& re = RopeEpi{}) {
  using C = PipeCfg<BM, BN, WM, WN, NS>;
  auto kern = gemm_i8_pipe_kernel<BM, BN, WM, WN, NS, DBG, F16, RS>;
  hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)C::kLds);
  if (e != hipSuccess) return e;
  const int tn = (g.N + BN - 1) / BN;
  const int64_t tm = (g.M + BM - 1) / BM;
  const int32_t kbytes = F16 ? 2 * g.K : g.K;
  KernelScope ks(RS ? "rope_rebuild_scores" : F16 ? "gemm_f16_pipe" : "gemm_i8_pipe", s);
  QSVD_LAUNCH(ks, kern, dim3((unsigned)(tm * tn)), dim3(C::kThreads), C::kLds, s, g.a, g.b, g.row_scale, g.col_scale,
                     g.M, g.N, kbytes, tn, xcd_group_rows(tm, tn, kGemmTilesPerXcd), sg, g.dbg, re);
  return hipGetLastError();
}

hipError_t launch_gemm_i8(const GemmArgs& g, hipStream_t s) {
  if (g.M == 0 || g.N == 0) return hipSuccess;
  if (g.K % PBK) return hipErrorInvalidValue;
  // outputs are written in 16-byte runs of 8 columns
  for (int i = 0; i < g.n_seg; ++i)
    if (g.seg[i].n0 % 8 || g.seg[i].n % 8 || g.seg[i].ld % 8 || ((uintptr_t)g.seg[i].ptr & 15))
      return hipErrorInvalidValue;
  const DevSegs sg = to_dev(g);
  // 256 x 256 tiles once they fill the chip, 128 x 128 otherwise (and for
  // the accumulator dumps)
  const int64_t big_tiles = ((g.M + 255) / 256) * ((g.N + 255) / 256);
  hipError_t e = g.dbg ? launch_pipe<128, 128, 64, 64, 6, true>(g, sg, s)
                 : big_tiles >= 256 ? launch_pipe<256, 256, 128, 64, 4, false>(g, sg, s)
                                    : launch_pipe<128, 128, 64, 64, 6, false>(g, sg, s);
  if (e != hipSuccess || !g.cq) return e;
  return launch_quantize_rows(g.seg[0].ptr, g.M, g.N, g.seg[0].ld, g.abits, 1.f, g.cq, g.sc, s, "latent_quant");
}

hipError_t launch_gemm_f16(const GemmArgs& g, hipStream_t s) {
  if (g.M == 0 || g.N == 0) return hipSuccess;
  if (g.K % (PBK / 2) || g.dbg || g.cq) return hipErrorInvalidValue;
  for (int i = 0; i < g.n_seg; ++i)
    if (g.seg[i].n0 % 8 || g.seg[i].n % 8 || g.seg[i].ld % 8 || ((uintptr_t)g.seg[i].ptr & 15))
      return hipErrorInvalidValue;
  const DevSegs sg = to_dev(g);
  const int64_t big_tiles = ((g.M + 255) / 256) * ((g.N + 255) / 256);
  return big_tiles >= 256 ? launch_pipe<256, 256, 128, 64, 4, false, true>(g, sg, s)
                          : launch_pipe<128, 128, 64, 64, 6, false, true>(g, sg, s);
}

hipError_t launch_gemm_rope_scores(const GemmArgs& g, const RopeEpi& re, bool f16, hipStream_t s) {
  if (g.M == 0 || g.N == 0) return hipSuccess;
  if ((f16 ? g.K % (PBK / 2) : g.K % PBK) || g.dbg || g.cq) return hipErrorInvalidValue;
  if (re.dh < 32 || 128 % re.dh || g.N % re.dh || re.Hq > 32 || re.G < 1) return hipErrorInvalidValue;
  const DevSegs sg{};
  const int64_t big_tiles = ((g.M + 255) / 256) * ((g.N + 255) / 256);
  if (f16)
    return big_tiles >= 256 ? launch_pipe<256, 256, 128, 64, 4, false, true, true>(g, sg, s, re)
                            : launch_pipe<128, 128, 64, 64, 6, false, true, true>(g, sg, s, re);
  return big_tiles >= 256 ? launch_pipe<256, 256, 128, 64, 4, false, false, true>(g, sg, s, re)
                          : launch_pipe<128, 128, 64, 64, 6, false, false, true>(g, sg, s, re);
}

}  // namespace qsvd
