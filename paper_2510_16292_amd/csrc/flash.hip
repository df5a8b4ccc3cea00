// Causal self-attention of a prefill block over its own projections.
//
// In prefill every prompt token's keys and values are at hand: the
// up-projection Y' = Q(C) Q(W^u) (Eq. 11) produces Q, K and V of all tokens at
// once (K = C W^u_k, V = C W^u_v, Eq. 5), so the prompt attends over those
// rows directly: 4 Hq dh flop per (query, key) pair, against 4 Hq r for the
// latent form, which the decode path uses because there only one query row
// per sequence meets the whole cache.
//
// One workgroup of eight waves takes 128 consecutive queries of one
// (sequence, query head); wave w owns the 16-query block q0 + 16w .. +15 (the
// code also takes several blocks per wave, which then share every key and
// value fragment read from LDS; one block per wave with eight waves measured
// fastest).  Key/value tiles of 64 tokens are staged in LDS (shared by the
// waves; the next tile's rows are already in registers while the current one
// is used).  Per tile, wave and query block, on the 16x16x32 fp16 matrix cores:
//   S^T (64 keys x 16 queries) = K_tile Q_b^T        (contraction over dh)
//   online softmax per query in fp32 (a query is one lane column; its 64
//   scores sit in that lane and the three lanes l ^ 16, l ^ 32, l ^ 48)
//   O^T (dh x 16 queries) += V_tile^T P^T            (contraction over keys)
// (16x16 products keep the accumulators small enough for two waves per SIMD.)
// The query rows stay in registers for the whole kernel.  Keys past a query's
// position, or past the sequence end, are masked.
//
// Rotary layers (ROPE): a query row is turned once, in registers, at its
// position within the sequence; a key row is turned while its tile moves from
// registers into LDS, at its own position (rotate-half pairs j, j + dh/2 by
// the angle pos * theta^(-2j/dh)).  The angle is formed in revolutions in
// fp64 and reduced to [0, 1) there, then sine and cosine come from the
// hardware's revolution-based instructions in fp32; the turned rows are
// rounded to fp16 for the matrix cores, like the unturned ones.
#include <math.h>

#include "common.h"
#include "launch.h"

namespace qsvd {

constexpr int kFaQ = 128;       // queries per workgroup
constexpr int kFaK = 64;        // keys per tile
constexpr int kFaWaves = 8;
constexpr int kFaQW = kFaQ / kFaWaves;   // queries per wave
constexpr int kFaQB = kFaQW / 16;        // 16-query blocks per wave
constexpr float kFaLog2e = 1.4426950408889634f;

template <int DH>
struct FaCfg {
  static constexpr int KST = DH + 8;       // K tile row stride (halves): 16-byte row reads hit every bank once
  static constexpr int VST = DH + 16;      // V tile row stride: the transposing reads hit distinct banks
  static constexpr int OST = DH + 8;       // output staging row stride
  static constexpr size_t kK = (size_t)kFaK * KST * 2, kV = (size_t)kFaK * VST * 2;
  static constexpr size_t kOut = (size_t)kFaWaves * kFaQW * OST * 2;
  static constexpr size_t kLds = kK + kV > kOut ? kK + kV : kOut;
  static constexpr size_t kLdsRope = kLds + (size_t)(DH / 2) * sizeof(double);   // + revolutions per position of each pair
  static constexpr int kChunks = kFaK * DH / 8;               // 16-byte runs per K (or V) tile
  static constexpr int kPerThread = kChunks / (kFaWaves * 64);
  static_assert(kChunks % (kFaWaves * 64) == 0, "whole runs per thread");
};

// Max and sum over the four 16-lane rows of a wave (lanes l, l ^ 16, l ^ 32,
// l ^ 48), every lane receiving the result: gfx950's v_permlane32_swap and
// v_permlane16_swap with both registers holding the value give each lane its
// partner's value at vector-ALU latency (issued as asm with both registers
// read-write; the s_nop covers the hazard of a vector write just before).
__device__ __forceinline__ void fa_swap32(uint32_t& a, uint32_t& b) {
  asm volatile("s_nop 1\n\tv_permlane32_swap_b32 %0, %1" : "+v"(a), "+v"(b));
}
__device__ __forceinline__ void fa_swap16(uint32_t& a, uint32_t& b) {
  asm volatile("s_nop 1\n\tv_permlane16_swap_b32 %0, %1" : "+v"(a), "+v"(b));
}
__device__ __forceinline__ float fa_rows4_max(float x) {
  uint32_t a = __builtin_bit_cast(uint32_t, x), b = a;
  fa_swap32(a, b);
  uint32_t c = __builtin_bit_cast(uint32_t, fmaxf(__builtin_bit_cast(float, a), __builtin_bit_cast(float, b))), e = c;
  fa_swap16(c, e);
  return fmaxf(__builtin_bit_cast(float, c), __builtin_bit_cast(float, e));
}
__device__ __forceinline__ float fa_rows4_sum(float x) {
  uint32_t a = __builtin_bit_cast(uint32_t, x), b = a;
  fa_swap32(a, b);
  uint32_t c = __builtin_bit_cast(uint32_t, __builtin_bit_cast(float, a) + __builtin_bit_cast(float, b)), e = c;
  fa_swap16(c, e);
  return __builtin_bit_cast(float, c) + __builtin_bit_cast(float, e);
}

// Rotary staging of a key tile: thread tid turns the 8 pairs of run pc
// (channels 8 pc .. +7 with their partners dh/2 further) of row tid / PR.
template <int DH>
struct FaRope {
  static constexpr int PR = DH / 16;                     // pair runs per row
  static constexpr int kActive = kFaK * PR;              // threads with a key row to turn
  static_assert(kActive <= kFaWaves * 64, "one pair run per thread");
  static constexpr int KR = FaCfg<DH>::kPerThread > 2 ? FaCfg<DH>::kPerThread : 2;   // key registers per thread
};

// Key/value tile t of the rows this thread stages (rows past the sequence end
// re-read its last row; they are masked).  With ROPE the key registers hold
// the two halves of one pair run instead.
template <int DH, bool ROPE>
__device__ __forceinline__ void fa_load_tile(const _Float16* __restrict__ k, const _Float16* __restrict__ v, int tok0,
                                             int n, int ldkv, int g, int t, int tid,
                                             i32x4 (&kr)[FaRope<DH>::KR], i32x4 (&vr)[FaCfg<DH>::kPerThread]) {
  constexpr int RUNS = DH / 8;
#pragma unroll
  for (int i = 0; i < FaCfg<DH>::kPerThread; ++i) {
    const int e = tid + kFaWaves * 64 * i, row = e / RUNS, c8 = e - row * RUNS;
    const int key = min(t * kFaK + row, n - 1);
    const int64_t off = (int64_t)(tok0 + key) * ldkv + g * DH + 8 * c8;
    if (!ROPE) kr[i] = *reinterpret_cast<const i32x4*>(k + off);
    vr[i] = *reinterpret_cast<const i32x4*>(v + off);
  }
  if (ROPE && tid < FaRope<DH>::kActive) {
    constexpr int PR = FaRope<DH>::PR;
    const int row = tid / PR, pc = tid - row * PR;
    const int key = min(t * kFaK + row, n - 1);
    const _Float16* src = k + (int64_t)(tok0 + key) * ldkv + g * DH + 8 * pc;
    kr[0] = *reinterpret_cast<const i32x4*>(src);
    kr[1] = *reinterpret_cast<const i32x4*>(src + DH / 2);
  }
}

// Turn the rotate-half pairs (a[e], b[e]) of channels j0 + e by the angle
// pos * theta^(-2j/dh): freq[j] holds theta^(-2j/dh) / (2 pi), so the angle
// in revolutions is formed and reduced to [0, 1) in fp64 before the fp32
// sine and cosine.
__device__ __forceinline__ void fa_rope8(f16x8& a, f16x8& b, int pos, const double* freq) {
  f16x8 ra, rb;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    double rev = (double)pos * freq[e];
    rev -= floor(rev);
    const float x = (float)rev;
    const float c = __builtin_amdgcn_cosf(x), sn = __builtin_amdgcn_sinf(x);
    const float fa = (float)a[e], fb = (float)b[e];
    ra[e] = (_Float16)(fa * c - fb * sn);
    rb[e] = (_Float16)(fb * c + fa * sn);
  }
  a = ra;
  b = rb;
}

// ... and its copy into the LDS tiles (turning the keys of a rotary layer at
// positions t * 64 + row).
template <int DH, bool ROPE>
__device__ __forceinline__ void fa_store_tile(_Float16* ks, _Float16* vs, int tid, int t, const double* freq,
                                              const i32x4 (&kr)[FaRope<DH>::KR],
                                              const i32x4 (&vr)[FaCfg<DH>::kPerThread]) {
  constexpr int RUNS = DH / 8;
#pragma unroll
  for (int i = 0; i < FaCfg<DH>::kPerThread; ++i) {
    const int e = tid + kFaWaves * 64 * i, row = e / RUNS, c8 = e - row * RUNS;
    if (!ROPE) *reinterpret_cast<i32x4*>(ks + row * FaCfg<DH>::KST + 8 * c8) = kr[i];
    *reinterpret_cast<i32x4*>(vs + row * FaCfg<DH>::VST + 8 * c8) = vr[i];
  }
  if (ROPE && tid < FaRope<DH>::kActive) {
    constexpr int PR = FaRope<DH>::PR;
    const int row = tid / PR, pc = tid - row * PR;
    f16x8 a = __builtin_bit_cast(f16x8, kr[0]), b = __builtin_bit_cast(f16x8, kr[1]);
    fa_rope8(a, b, t * kFaK + row, freq + 8 * pc);
    *reinterpret_cast<f16x8*>(ks + row * FaCfg<DH>::KST + 8 * pc) = a;
    *reinterpret_cast<f16x8*>(ks + row * FaCfg<DH>::KST + 8 * pc + DH / 2) = b;
  }
}

// Cache mode: the queries are the last q_len positions of each sequence of a
// cache and the keys and values its rebuilt rows (row b * capacity + t,
// position t < seq_len[b], row stride ldkv).
struct FaCacheArgs {
  const int32_t* seq_len;
  int32_t capacity, q_len, ldkv;
};

template <int DH, bool ROPE, bool CACHE>
__global__ void __launch_bounds__(kFaWaves * 64, 2)
prefill_flash_kernel(const _Float16* __restrict__ q, const _Float16* __restrict__ k, const _Float16* __restrict__ v,
                     const int32_t* __restrict__ cu, int32_t n_seq, int32_t Hq, int32_t Hkv, int32_t n_qt,
                     float scale_log2, double log2_theta, FaCacheArgs ca, _Float16* __restrict__ out) {
  using C = FaCfg<DH>;
  constexpr int KS = DH / 32;      // contraction steps of the score product
  constexpr int OB = DH / 16;      // 16-channel blocks of the output
  constexpr int RUNS = DH / 8;     // 16-byte runs per row
  extern __shared__ __attribute__((aligned(16))) uint8_t fa_smem[];
  _Float16* ks = reinterpret_cast<_Float16*>(fa_smem);
  _Float16* vs = reinterpret_cast<_Float16*>(fa_smem + C::kK);
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int l16 = lane & 15, g = lane >> 4;

  // Workgroup -> (sequence, head, query tile).  The query tiles of one
  // (sequence, head) read the same key/value rows, so they get ids that one
  // XCD receives (the chip hands workgroup i to XCD i % 8) and share its L2;
  // within a group the longest tiles (most keys) go first.
  const int groups = n_seq * Hq, total = groups * n_qt;
  int lin = blockIdx.x;
  if (total % 8 == 0) lin = (lin % 8) * (total / 8) + lin / 8;
  const int grp = lin / n_qt, qt = n_qt - 1 - (lin - grp * n_qt);
  const int b = grp / Hq, h = grp - b * Hq;
  // this sequence's rows: query i (i < nq) is row q_row0 + i at position
  // q_off + i, key t (t < nk) is row k_row0 + t at position t; query i sees
  // the keys at positions <= q_off + i
  int q_row0, nq, k_row0, nk, q_off;
  if (CACHE) {
    nk = min(ca.seq_len[b], ca.capacity);
    nq = ca.q_len;
    q_row0 = b * nq;
    k_row0 = b * ca.capacity;
    q_off = nk - nq;
  } else {
    q_row0 = k_row0 = cu[b];
    nq = nk = cu[b + 1] - q_row0;
    q_off = 0;
  }
  const int q0 = qt * kFaQ;
  if (q0 >= nq) return;
  double* freq = reinterpret_cast<double*>(fa_smem + C::kLds);
  if (ROPE) {
    if (tid < DH / 2) freq[tid] = exp2(-2.0 * tid / DH * log2_theta) * 0.15915494309189533576888376337251;
    __syncthreads();
  }
  const int g_kv = (h * Hkv) / Hq;
  const int ldq = Hq * DH, ldkv = CACHE ? ca.ldkv : Hkv * DH;
  const int kend = min(nk, q_off + min(nq, q0 + kFaQ));   // keys this tile of queries can see
  if (CACHE && kend <= 0) {
    // no query of the tile sees a position (a cache shorter than the query
    // block): zeros, as for every query without a visible position
#pragma unroll
    for (int i = 0; i < kFaQ * RUNS / (kFaWaves * 64); ++i) {
      const int e = tid + kFaWaves * 64 * i, row = e / RUNS, c8 = e - row * RUNS;
      if (q0 + row < nq) *reinterpret_cast<f16x8*>(out + (int64_t)(q_row0 + q0 + row) * ldq + h * DH + 8 * c8) = f16x8{};
    }
    return;
  }
  const int n_tiles = (kend + kFaK - 1) / kFaK;
  const int qw0 = q0 + kFaQW * w;                   // this wave's first query
  int my_q[kFaQB];                                  // this lane's query in each block
#pragma unroll
  for (int qb = 0; qb < kFaQB; ++qb) my_q[qb] = qw0 + 16 * qb + l16;

  // query slots of the score product: step s, lane group g -> channels 32 s + 8 g .. +7
  f16x8 qf[kFaQB][KS];
#pragma unroll
  for (int qb = 0; qb < kFaQB; ++qb) {
    const _Float16* qrow = q + (int64_t)(q_row0 + min(my_q[qb], nq - 1)) * ldq + h * DH + 8 * g;
#pragma unroll
    for (int s = 0; s < KS; ++s) qf[qb][s] = *reinterpret_cast<const f16x8*>(qrow + 32 * s);
    if (ROPE) {                                     // slot s pairs with slot s + KS/2 (channels dh/2 further)
#pragma unroll
      for (int s = 0; s < KS / 2; ++s)
        fa_rope8(qf[qb][s], qf[qb][s + KS / 2], q_off + min(my_q[qb], nq - 1), freq + 32 * s + 8 * g);
    }
  }

  i32x4 kr[FaRope<DH>::KR], vr[C::kPerThread];
  f32x4 o[kFaQB][OB];
  float m_run[kFaQB], l_run[kFaQB];
#pragma unroll
  for (int qb = 0; qb < kFaQB; ++qb) {
#pragma unroll
    for (int ob = 0; ob < OB; ++ob) o[qb][ob] = f32x4{};
    m_run[qb] = -INFINITY;
    l_run[qb] = 0.f;
  }
  typedef short s16x4 __attribute__((ext_vector_type(4)));
  typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

  fa_load_tile<DH, ROPE>(k, v, k_row0, nk, ldkv, g_kv, 0, tid, kr, vr);
  for (int t = 0; t < n_tiles; ++t) {
    __syncthreads();                                // every wave is done with the previous tile
    fa_store_tile<DH, ROPE>(ks, vs, tid, t, freq, kr, vr);
    __syncthreads();
    if (t + 1 < n_tiles) fa_load_tile<DH, ROPE>(k, v, k_row0, nk, ldkv, g_kv, t + 1, tid, kr, vr);
    const int kt0 = t * kFaK;
    if (kt0 > q_off + qw0 + kFaQW - 1) continue;    // every key of the tile is after this wave's queries
    // S^T: key block kb, lane (query l16 of block qb, group g) holds keys kt0 + 16 kb + 4 g + v
    f32x4 sacc[kFaQB][4];
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
#pragma unroll
      for (int qb = 0; qb < kFaQB; ++qb) sacc[qb][kb] = f32x4{};
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        const f16x8 kf = *reinterpret_cast<const f16x8*>(ks + (16 * kb + l16) * C::KST + 32 * s + 8 * g);
#pragma unroll
        for (int qb = 0; qb < kFaQB; ++qb)
          sacc[qb][kb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(kf, qf[qb][s], sacc[qb][kb], 0, 0, 0);
      }
    }
    // softmax per query block; the scores become the probabilities in place
    // (tiles wholly before this wave's first query and inside the sequence
    // need no mask)
    const bool full = kt0 + kFaK - 1 <= q_off + qw0 && kt0 + kFaK <= nk;
    float p[kFaQB][4][4];
#pragma unroll
    for (int qb = 0; qb < kFaQB; ++qb) {
      float mx = -INFINITY;
      if (full) {
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
#pragma unroll
          for (int vv = 0; vv < 4; ++vv) {
            p[qb][kb][vv] = sacc[qb][kb][vv] * scale_log2;
            mx = fmaxf(mx, p[qb][kb][vv]);
          }
      } else {
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
#pragma unroll
          for (int vv = 0; vv < 4; ++vv) {
            const int key = kt0 + 16 * kb + 4 * g + vv;
            p[qb][kb][vv] = (key <= q_off + my_q[qb] && key < nk) ? sacc[qb][kb][vv] * scale_log2 : -INFINITY;
            mx = fmaxf(mx, p[qb][kb][vv]);
          }
      }
      const float m_new = fmaxf(m_run[qb], fa_rows4_max(mx));
      float alpha = 1.f, ps = 0.f;
      if (m_new == -INFINITY) {
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
#pragma unroll
          for (int vv = 0; vv < 4; ++vv) p[qb][kb][vv] = 0.f;
      } else {
        alpha = __builtin_amdgcn_exp2f(m_run[qb] - m_new);
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
#pragma unroll
          for (int vv = 0; vv < 4; ++vv) {
            p[qb][kb][vv] = __builtin_amdgcn_exp2f(p[qb][kb][vv] - m_new);
            ps += p[qb][kb][vv];
          }
      }
      l_run[qb] = l_run[qb] * alpha + fa_rows4_sum(ps);
      m_run[qb] = m_new;
      if (__any(alpha != 1.f)) {
#pragma unroll
        for (int ob = 0; ob < OB; ++ob) o[qb][ob] *= alpha;
      }
    }
    // O^T += V^T P^T in two 32-key steps st: k-slot e of lane group g is key
    // 32 st + 16 (e / 4) + 4 g + e % 4, i.e. score p[2 st + e / 4][e % 4].
    // The A operand comes from transposing reads: lane a of group g addresses
    // key 4g + a/4 of the 16-key block, channels 16 ob + 4 (a % 4) .. +3, and
    // lane i receives element i % 4 of the chunks of lanes i/4, 4 + i/4,
    // 8 + i/4, 12 + i/4: channel 16 ob + i at keys 4g .. 4g+3 of the block.
#pragma unroll
    for (int st = 0; st < 2; ++st) {
      f16x8 pf[kFaQB];
#pragma unroll
      for (int qb = 0; qb < kFaQB; ++qb)
#pragma unroll
        for (int e = 0; e < 8; ++e) pf[qb][e] = (_Float16)p[qb][2 * st + (e >> 2)][e & 3];
      const int key = 32 * st + 4 * g + (l16 >> 2);
#pragma unroll
      for (int ob = 0; ob < OB; ++ob) {
        const _Float16* a0 = vs + key * C::VST + 16 * ob + 4 * (l16 & 3);
        const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)a0);
        const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(a0 + 16 * C::VST));
        const f16x4 flo = __builtin_bit_cast(f16x4, lo), fhi = __builtin_bit_cast(f16x4, hi);
        const f16x8 a = {flo[0], flo[1], flo[2], flo[3], fhi[0], fhi[1], fhi[2], fhi[3]};
#pragma unroll
        for (int qb = 0; qb < kFaQB; ++qb) o[qb][ob] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, pf[qb], o[qb][ob], 0, 0, 0);
      }
    }
  }

  // O / l through LDS, so that each query row leaves as 16-byte runs: lane
  // (l16, g) holds query qw0 + 16 qb + l16 at channels 16 ob + 4 g .. +3.
  __syncthreads();
  _Float16* ost = reinterpret_cast<_Float16*>(fa_smem) + w * kFaQW * C::OST;
#pragma unroll
  for (int qb = 0; qb < kFaQB; ++qb) {
    const float inv_l = l_run[qb] > 0.f ? 1.f / l_run[qb] : 0.f;
#pragma unroll
    for (int ob = 0; ob < OB; ++ob) {
      const f16x4 v4 = {(_Float16)(o[qb][ob][0] * inv_l), (_Float16)(o[qb][ob][1] * inv_l),
                        (_Float16)(o[qb][ob][2] * inv_l), (_Float16)(o[qb][ob][3] * inv_l)};
      *reinterpret_cast<f16x4*>(ost + (16 * qb + l16) * C::OST + 16 * ob + 4 * g) = v4;
    }
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < kFaQW * RUNS / 64; ++i) {
    const int e = lane + 64 * i, row = e / RUNS, c8 = e - row * RUNS;
    const int qq = qw0 + row;
    if (qq < nq)
      *reinterpret_cast<f16x8*>(out + (int64_t)(q_row0 + qq) * ldq + h * DH + 8 * c8) =
          *reinterpret_cast<const f16x8*>(ost + row * C::OST + 8 * c8);
  }
}

template <int DH, bool ROPE, bool CACHE>
static hipError_t launch_flash(const PrefillAttnArgs& a, const FaCacheArgs& ca, hipStream_t s) {
  using C = FaCfg<DH>;
  auto kern = prefill_flash_kernel<DH, ROPE, CACHE>;
  const size_t lds = ROPE ? C::kLdsRope : C::kLds;
  hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  const int n_qt = ((CACHE ? ca.q_len : a.max_seqlen) + kFaQ - 1) / kFaQ;
  const int64_t blocks = (int64_t)a.batch * a.n_q_heads * n_qt;
  KernelScope ks(CACHE ? "cache_flash" : ROPE ? "prefill_flash_rope" : "prefill_flash", s);
  QSVD_LAUNCH(ks, kern, dim3((unsigned)blocks), dim3(kFaWaves * 64), lds, s, a.q, a.k, a.v, a.cu_seqlens, a.batch,
              a.n_q_heads, a.n_kv_heads, n_qt, a.sm_scale * kFaLog2e, ROPE ? log2((double)a.rope_theta) : 0.0, ca,
              a.out);
  return hipGetLastError();
}

bool prefill_attention_supported(int32_t head_dim) { return head_dim == 64 || head_dim == 128; }

hipError_t launch_prefill_attention(const PrefillAttnArgs& a, hipStream_t s) {
  if (a.batch == 0 || a.max_seqlen == 0) return hipSuccess;
  const FaCacheArgs none{};
  if (a.rope_theta > 0.f)
    return a.head_dim == 128 ? launch_flash<128, true, false>(a, none, s) : launch_flash<64, true, false>(a, none, s);
  return a.head_dim == 128 ? launch_flash<128, false, false>(a, none, s) : launch_flash<64, false, false>(a, none, s);
}

// Queries of several positions per sequence over a cache's rebuilt K^ | V^
// rows (the reconstruct form with q_len > 1).
hipError_t launch_cache_attention(const CacheAttnArgs& c, hipStream_t s) {
  if (c.batch == 0 || c.q_len == 0) return hipSuccess;
  const int nkv = c.n_kv_heads * c.head_dim;
  PrefillAttnArgs a{c.q, c.kv, c.kv + nkv, nullptr, c.batch, c.q_len, c.n_q_heads, c.n_kv_heads, c.head_dim,
                    c.sm_scale, c.out, c.rope_theta};
  const FaCacheArgs ca{c.seq_len, c.capacity, c.q_len, 2 * nkv};
  if (c.rope_theta > 0.f)
    return c.head_dim == 128 ? launch_flash<128, true, true>(a, ca, s) : launch_flash<64, true, true>(a, ca, s);
  return c.head_dim == 128 ? launch_flash<128, false, true>(a, ca, s) : launch_flash<64, false, true>(a, ca, s);
}

}  // namespace qsvd
