// Prefill-size products (M > 32) with 4-bit operands and per-group weight
// scales: Q(X) Q(W^d) and Q(C) Q(W^u) for W4A8 / W4A4 / W8A4 layers (Eq. 11-12,
// Section 4's per-group int4 weights).
//
// Same pipeline as the int8 kernel (operands global -> LDS with
// global_load_lds_dwordx4, NS stages of 64 contraction elements, one barrier
// per stage) on 128 x 128 tiles of four 64 x 64 waves.  A stage row holds 64
// codes: 64 bytes (int8) or 32 bytes (int4, element 2i in the low nibble of
// byte i); int4 fragments are read 8 bytes at a time and widened in registers
// to int8 bytes holding 16 * code before v_mfma_i32_32x32x32_i8, so every
// product is exact and the int32 sums are exact multiples of 16 or 256.
//
// Per-group scales (groups of G contraction elements, G a multiple of 64):
// at the end of each group the int32 tile is folded into an fp32 tile as
// S = S + f32(acc_g) * s[g][n] (each product and sum rounded to fp32, groups
// in order) and the int32 tile restarts from zero; the output is S * s_row.
// Per-channel scales: (f32(acc) * s_row) * s_col.  Both are the definition's
// rounding sequence.
#include "common.h"
#include "launch.h"

namespace qsvd {

typedef __attribute__((address_space(3))) void q4_lds_void_t;
typedef __attribute__((address_space(1))) void q4_glb_void_t;

constexpr int QBM = 128, QBN = 128, QWM = 64, QWN = 64, QNS = 6, QBK = 64;

template <int N>
__device__ __forceinline__ void q4_wait_barrier() {
  asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(N) : "memory");
}

template <int LPW, int R>
__device__ __forceinline__ void q4_wait_stage(int rem) {
  if constexpr (R == 0) {
    q4_wait_barrier<0>();
  } else {
    if (rem >= R) q4_wait_barrier<R * LPW>();
    else q4_wait_stage<LPW, R - 1>(rem);
  }
}

// LDS slot of (row, 16-byte chunk) in an operand tile whose rows are RB bytes
// (64: four chunks, 32: two).  The XOR keeps the rows of one fragment read
// (16 consecutive rows, same chunk) on distinct banks.
template <int RB>
__device__ __forceinline__ int q4_slot(int row, int chunk) {
  if constexpr (RB == 64) return row * 64 + 16 * (chunk ^ ((row >> 2) & 3));
  else return row * 32 + 16 * (chunk ^ ((row >> 3) & 1));
}

// 16 int4 codes (8 bytes, element 2i in the low nibble of byte i) -> 16 int8
// holding 16 * code, in the element order 0,2,4,6, 1,3,5,7, 8,10,12,14,
// 9,11,13,15: (w << 4) & 0xF0F0F0F0 moves every even element into the high
// half of its byte and w & 0xF0F0F0F0 keeps every odd one there, so each
// code's sign bit lands on bit 7 (three operations per eight codes).
__device__ __forceinline__ i32x4 q4_widen(uint2 p) {
  return i32x4{(int32_t)((p.x << 4) & 0xF0F0F0F0u), (int32_t)(p.x & 0xF0F0F0F0u),
               (int32_t)((p.y << 4) & 0xF0F0F0F0u), (int32_t)(p.y & 0xF0F0F0F0u)};
}

// 16 int8 codes in element order -> the element order of q4_widen (one byte
// permute per four codes), for an int8 operand multiplied with an int4 one.
__device__ __forceinline__ i32x4 q4_interleave(i32x4 v) {
  return i32x4{(int32_t)__builtin_amdgcn_perm((uint32_t)v[1], (uint32_t)v[0], 0x06040200u),
               (int32_t)__builtin_amdgcn_perm((uint32_t)v[1], (uint32_t)v[0], 0x07050301u),
               (int32_t)__builtin_amdgcn_perm((uint32_t)v[3], (uint32_t)v[2], 0x06040200u),
               (int32_t)__builtin_amdgcn_perm((uint32_t)v[3], (uint32_t)v[2], 0x07050301u)};
}

// Fragment for sub-step kk (32 contraction elements) of a 32x32x32 MFMA: lane
// (row, hl) supplies elements 32*kk + 16*hl .. +15 of its row, in natural
// order when both operands are int8, else in q4_widen's order (the same
// order in both operands, so the sum runs over the same products).
template <int BITS, int OTHER>
__device__ __forceinline__ i32x4 q4_frag(const uint8_t* base, int row, int kk, int hl) {
  if constexpr (BITS == 8) {
    const i32x4 v = *reinterpret_cast<const i32x4*>(base + q4_slot<64>(row, 2 * kk + hl));
    if constexpr (OTHER == 8) return v;
    else return q4_interleave(v);
  } else {
    return q4_widen(*reinterpret_cast<const uint2*>(base + q4_slot<32>(row, kk) + 8 * hl));
  }
}

struct Q4Segs {
  _Float16* p0; _Float16* p1; _Float16* p2;
  int64_t ld0, ld1, ld2;
  int32_t a0, a1, a2, e0, e1, e2;
};

__device__ __forceinline__ _Float16* q4_col(const Q4Segs& sg, int32_t n, int64_t* ld) {
  const bool in0 = n >= sg.a0 && n < sg.e0, in1 = n >= sg.a1 && n < sg.e1, in2 = n >= sg.a2 && n < sg.e2;
  _Float16* base = in0 ? sg.p0 : in1 ? sg.p1 : in2 ? sg.p2 : nullptr;
  *ld = in0 ? sg.ld0 : in1 ? sg.ld1 : sg.ld2;
  return base ? base + (n - (in0 ? sg.a0 : in1 ? sg.a1 : sg.a2)) : nullptr;
}

template <int ABITS, int BBITS, bool GROUPED>
__global__ void __launch_bounds__(256)
gemm_q4_pipe_kernel(const uint8_t* __restrict__ A, const uint8_t* __restrict__ B,
                    const float* __restrict__ rs, const float* __restrict__ cs, int32_t sstride,
                    int64_t M, int32_t N, int32_t K, int32_t group, int32_t n_tiles_n, int32_t gm, Q4Segs sg) {
  constexpr int RBA = QBK * ABITS / 8, RBB = QBK * BBITS / 8;        // stage row bytes
  constexpr int SA = QBM * RBA, SB = QBN * RBB, STAGE = SA + SB;
  constexpr int LPW = STAGE / 1024 / 4;                               // direct loads per wave per stage
  static_assert(STAGE % 4096 == 0, "whole 1 KB loads per wave");
  constexpr int TI = QWM / 32, TJ = QWN / 32;
  extern __shared__ __attribute__((aligned(1024))) uint8_t q4_smem[];
  __shared__ __attribute__((aligned(16))) float s_rs[QBM];
  // int4 operands enter the products as 16 * code: the int32 sums are exact
  // multiples of 16 (or 256) and are shifted back exactly before use
  constexpr int SH = (ABITS == 4 ? 4 : 0) + (BBITS == 4 ? 4 : 0);
  const int tid = threadIdx.x, lane = tid & 63, w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = w >> 1, wn = w & 1;
  const int l32 = lane & 31, hl = lane >> 5;
  int tm, tn;
  xcd_tile(blockIdx.x, gridDim.x, n_tiles_n, gm, &tm, &tn);
  const int64_t m0 = (int64_t)tm * QBM;
  const int32_t n0 = tn * QBN;
  const int nk = K / QBK;
  const int64_t KA = (int64_t)K * ABITS / 8, KB = (int64_t)K * BBITS / 8;   // row bytes in memory

  // byte o of a stage: A tile rows first, then B tile rows; lane p of load j
  // of wave w covers bytes 1024*(w*LPW + j) + 16p
  // Per-lane source offsets of this wave's direct loads from the tile's first
  // row (fixed over the contraction; a stage advances the base by a row's
  // stage bytes): byte o of a stage holds A tile rows first, then B tile
  // rows; lane p of load j of wave w covers bytes 1024*(w*LPW + j) + 16p.
  const uint8_t* a_tile = A + m0 * KA;
  const uint8_t* b_tile = B + (int64_t)n0 * KB;
  uint32_t voff[LPW];
#pragma unroll
  for (int j = 0; j < LPW; ++j) {
    const int blk = w * LPW + j;                                     // wave-uniform
    const int o = blk * 1024 + 16 * lane;
    if (blk * 1024 < SA) {
      const int row = o / RBA, phys = (o % RBA) / 16;
      const int chunk = RBA == 64 ? (phys ^ ((row >> 2) & 3)) : (phys ^ ((row >> 3) & 1));
      voff[j] = (uint32_t)(min((int64_t)row, M - 1 - m0) * KA + 16 * chunk);
    } else {
      const int ob = o - SA;
      const int row = ob / RBB, phys = (ob % RBB) / 16;
      const int chunk = RBB == 64 ? (phys ^ ((row >> 2) & 3)) : (phys ^ ((row >> 3) & 1));
      voff[j] = (uint32_t)(min((int64_t)row, (int64_t)N - 1 - n0) * KB + 16 * chunk);
    }
  }
  auto issue = [&](int st) {
    uint8_t* base = q4_smem + (st % QNS) * STAGE;
#pragma unroll
    for (int j = 0; j < LPW; ++j) {
      const int blk = w * LPW + j;
      const uint8_t* src = blk * 1024 < SA ? a_tile + (int64_t)st * RBA + voff[j] : b_tile + (int64_t)st * RBB + voff[j];
      __builtin_amdgcn_global_load_lds((q4_glb_void_t*)src, (q4_lds_void_t*)(base + blk * 1024), 16, 0, 0);
    }
  };

  // row scales and this lane's column scales first (their waits leave the
  // stage loads in flight)
  for (int i = tid; i < QBM; i += 256) s_rs[i] = rs[min(m0 + i, M - 1)];
  int32_t ncol[TJ];
  float csn[TJ];
#pragma unroll
  for (int j = 0; j < TJ; ++j) {
    ncol[j] = n0 + wn * QWN + 32 * j + l32;
    csn[j] = GROUPED ? 0.f : cs[min(ncol[j], N - 1)];
  }
  const int gsteps = GROUPED ? group / QBK : 0;
  float gsc[TJ];               // scales of the group being accumulated
  if constexpr (GROUPED) {
#pragma unroll
    for (int j = 0; j < TJ; ++j) gsc[j] = cs[min(ncol[j], N - 1)];
  }
#pragma unroll
  for (int st = 0; st < QNS - 1; ++st)
    if (st < nk) issue(st);

  i32x16 acc[TI][TJ];
  f32x16 S[GROUPED ? TI : 1][GROUPED ? TJ : 1];
#pragma unroll
  for (int i = 0; i < TI; ++i)
#pragma unroll
    for (int j = 0; j < TJ; ++j) acc[i][j] = i32x16{};
  if constexpr (GROUPED) {
#pragma unroll
    for (int i = 0; i < TI; ++i)
#pragma unroll
      for (int j = 0; j < TJ; ++j) S[i][j] = f32x16{};
  }

  // Fragments by contraction half kk (32 elements): half 1 of a stage is read
  // while half 0's products run, half 0 of the next stage while half 1's run;
  // one MFMA goes out before each read so that the reads run under them.
  i32x4 af[2][TI], bf[2][TJ];
  auto read_half = [&](int kt, int kk) {
    const uint8_t* sa = q4_smem + (kt % QNS) * STAGE;
    const uint8_t* sb = sa + SA;
#pragma unroll
    for (int i = 0; i < TI; ++i) af[kk][i] = q4_frag<ABITS, BBITS>(sa, wm * QWM + 32 * i + l32, kk, hl);
#pragma unroll
    for (int j = 0; j < TJ; ++j) bf[kk][j] = q4_frag<BBITS, ABITS>(sb, wn * QWN + 32 * j + l32, kk, hl);
  };
  auto products = [&](int kk) {
#pragma unroll
    for (int i = 0; i < TI; ++i)
#pragma unroll
      for (int j = 0; j < TJ; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(af[kk][i], bf[kk][j], acc[i][j], 0, 0, 0);
  };
  auto interleave = [&]() {
#pragma unroll
    for (int r = 0; r < TI + TJ; ++r) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // one MFMA
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);   // one LDS read
    }
  };
  static_assert(TI * TJ == TI + TJ, "as many products as reads per half");

  // Waiting for stage s (its loads landed; every wave has finished reading
  // stage s - 1) frees slot (s - 1) % QNS for stage s + QNS - 1.
  q4_wait_stage<LPW, QNS - 2>(nk - 1);
  if (QNS - 1 < nk) issue(QNS - 1);
  read_half(0, 0);
  for (int kt = 0; kt < nk; ++kt) {
    __builtin_amdgcn_sched_barrier(0);
    products(0);
    read_half(kt, 1);
    interleave();
    __builtin_amdgcn_sched_barrier(0);
    // (on the last stage: a full wait and barrier, nothing left to issue)
    q4_wait_stage<LPW, QNS - 2>(nk - 2 - kt);
    if (kt + QNS < nk) issue(kt + QNS);
    __builtin_amdgcn_sched_barrier(0);
    // after the last stage this reads a stage slot whose values go unused
    products(1);
    read_half(kt + 1, 0);
    interleave();
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (GROUPED) {
      if ((kt + 1) % gsteps == 0) {
        // group g = (kt + 1) / gsteps - 1 ends here: fold it, fetch the next group's scales
        const int gn = (kt + 1) / gsteps;
        // (float)acc * (s_g 2^-SH) is the same real number as
        // (float)(acc >> SH) * s_g (acc is an exact multiple of 2^SH below
        // 2^24, and scaling s_g by a power of two is exact), so it rounds the
        // same; the shift is saved on every element
        float gss[TJ];
#pragma unroll
        for (int j = 0; j < TJ; ++j) gss[j] = mul_rn(gsc[j], 1.f / (float)(1 << SH));
#pragma unroll
        for (int i = 0; i < TI; ++i)
#pragma unroll
          for (int j = 0; j < TJ; ++j) {
#pragma unroll
            for (int v = 0; v < 16; ++v) S[i][j][v] = add_rn(S[i][j][v], mul_rn((float)acc[i][j][v], gss[j]));
            acc[i][j] = i32x16{};
          }
        if (gn * gsteps < nk) {
#pragma unroll
          for (int j = 0; j < TJ; ++j) gsc[j] = cs[(int64_t)gn * sstride + min(ncol[j], N - 1)];
        }
      }
    }
  }

  // Epilogue: the dequantized fp16 tile of each wave is staged in LDS and
  // written back as 16-byte runs of one row.  Lane holds column
  // wn*64 + 32j + l32 and rows wm*64 + 32i + 8(v/4) + 4hl + v%4.
  q4_wait_barrier<0>();
  constexpr int OST = QWN + 8;
  _Float16* ost = reinterpret_cast<_Float16*>(q4_smem) + w * QWM * OST;
#pragma unroll
  for (int j = 0; j < TJ; ++j)
#pragma unroll
    for (int i = 0; i < TI; ++i)
#pragma unroll
      for (int vq = 0; vq < 4; ++vq) {
        const int rl = 32 * i + 8 * vq + 4 * hl;
        const f32x4 r4 = *reinterpret_cast<const f32x4*>(&s_rs[wm * QWM + rl]);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int v = 4 * vq + e;
          const float y = GROUPED ? mul_rn(S[i][j][v], r4[e]) : mul_rn(mul_rn((float)(acc[i][j][v] >> SH), r4[e]), csn[j]);
          ost[(rl + e) * OST + 32 * j + l32] = to_f16(y);
        }
      }
  constexpr int CPR = QWN / 8;
  for (int e = lane; e < QWM * CPR; e += 64) {
    const int row = e / CPR, c8 = e % CPR;
    const int64_t m = m0 + wm * QWM + row;
    const int32_t n = n0 + wn * QWN + 8 * c8;
    if (m >= M || n >= N) continue;
    int64_t ld;
    _Float16* p = q4_col(sg, n, &ld);
    if (p) __builtin_nontemporal_store(*reinterpret_cast<const f16x8*>(ost + row * OST + 8 * c8), reinterpret_cast<f16x8*>(p + m * ld));
  }
}

template <int ABITS, int BBITS, bool GROUPED>
static hipError_t launch_q4(const GemmArgs& g, const Q4Segs& sg, int32_t group, int32_t sstride, hipStream_t s) {
  constexpr int STAGE = QBM * QBK * ABITS / 8 + QBN * QBK * BBITS / 8;
  constexpr size_t lds = (size_t)QNS * STAGE > (size_t)4 * QWM * (QWN + 8) * 2 ? (size_t)QNS * STAGE
                                                                             : (size_t)4 * QWM * (QWN + 8) * 2;
  auto kern = gemm_q4_pipe_kernel<ABITS, BBITS, GROUPED>;
  hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  const int tn = (g.N + QBN - 1) / QBN;
  const int64_t tm = (g.M + QBM - 1) / QBM;
  KernelScope ks("gemm_q4_pipe", s);
  QSVD_LAUNCH(ks, kern, dim3((unsigned)(tm * tn)), dim3(256), lds, s, (const uint8_t*)g.a, (const uint8_t*)g.b,
              g.row_scale, g.col_scale, sstride, g.M, g.N, g.K, group, tn, xcd_group_rows(tm, tn), sg);
  return hipGetLastError();
}

hipError_t launch_gemm_q4(const GemmArgs& g, int32_t abits, int32_t wbits, int32_t group, int32_t sstride,
                          hipStream_t s) {
  if (g.M == 0 || g.N == 0) return hipSuccess;
  if (g.K % QBK || (group && (group % QBK || g.K % group))) return hipErrorInvalidValue;
  if ((abits != 8 && abits != 4) || (wbits != 8 && wbits != 4) || (wbits == 4 && !group)) return hipErrorInvalidValue;
  for (int i = 0; i < g.n_seg; ++i)
    if (g.seg[i].n0 % 8 || g.seg[i].n % 8 || g.seg[i].ld % 8 || ((uintptr_t)g.seg[i].ptr & 15))
      return hipErrorInvalidValue;
  Q4Segs sg{};
  _Float16** ps[3] = {&sg.p0, &sg.p1, &sg.p2};
  int64_t* lds[3] = {&sg.ld0, &sg.ld1, &sg.ld2};
  int32_t* as[3] = {&sg.a0, &sg.a1, &sg.a2};
  int32_t* es[3] = {&sg.e0, &sg.e1, &sg.e2};
  for (int i = 0; i < 3; ++i) {
    if (i < g.n_seg) {
      *ps[i] = g.seg[i].ptr; *lds[i] = g.seg[i].ld; *as[i] = g.seg[i].n0; *es[i] = g.seg[i].n0 + g.seg[i].n;
    } else {
      *ps[i] = nullptr; *lds[i] = 0; *as[i] = *es[i] = i > 0 ? *es[i - 1] : 0;
    }
  }
  hipError_t e;
  if (abits == 8 && wbits == 4) e = launch_q4<8, 4, true>(g, sg, group, sstride, s);
  else if (abits == 4 && wbits == 4) e = launch_q4<4, 4, true>(g, sg, group, sstride, s);
  else if (abits == 4 && group) e = launch_q4<4, 8, true>(g, sg, group, sstride, s);
  else if (abits == 4) e = launch_q4<4, 8, false>(g, sg, 0, sstride, s);
  else e = launch_q4<8, 8, true>(g, sg, group, sstride, s);     // 8-bit codes, per-group scales
  if (e != hipSuccess || !g.cq) return e;
  return launch_quantize_rows(g.seg[0].ptr, g.M, g.N, g.seg[0].ld, g.abits, 1.f, g.cq, g.sc, s, "latent_quant");
}

}  // namespace qsvd
