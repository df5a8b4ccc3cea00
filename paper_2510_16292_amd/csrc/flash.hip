// Causal self-attention of a prefill block over its own projections.
//
// In prefill every prompt token's keys and values are at hand: the
// up-projection Y' = Q(C) Q(W^u) (Eq. 11) produces Q, K and V of all tokens at
// once (K = C W^u_k, V = C W^u_v, Eq. 5), so the prompt attends over those
// rows directly: 4 Hq dh flop per (query, key) pair, against 4 Hq r for the
// latent form, which the decode path uses because there only one query row
// per sequence meets the whole cache.
//
// One workgroup of four waves takes 128 consecutive queries of one
// (sequence, query head); wave w owns queries q0 + 32w .. +31.  Key/value
// tiles of 64 tokens are staged in LDS (shared by the four waves; the next
// tile's rows are already in registers while the current one is used).  Per
// tile and wave, on the 32x32x16 fp16 matrix cores:
//   S^T (64 keys x 32 queries) = K_tile Q_w^T        (contraction over dh)
//   online softmax per query in fp32 (a query is one lane column; its 64
//   scores sit in that lane and its partner lane l ^ 32)
//   O^T (dh x 32 queries) += V_tile^T P^T            (contraction over keys)
// The query rows stay in registers for the whole kernel.  Keys past a query's
// position, or past the sequence end, are masked.
#include <math.h>

#include "common.h"
#include "launch.h"

namespace qsvd {

constexpr int kFaQ = 128;       // queries per workgroup
constexpr int kFaK = 64;        // keys per tile
constexpr int kFaWaves = 4;
constexpr float kFaLog2e = 1.4426950408889634f;

template <int DH>
struct FaCfg {
  static constexpr int KST = DH + 8;       // K tile row stride (halves): 16-byte row reads hit every bank once
  static constexpr int VST = DH + 16;      // V tile row stride: the transposing reads hit distinct banks
  static constexpr int OST = DH + 8;       // output staging row stride
  static constexpr size_t kK = (size_t)kFaK * KST * 2, kV = (size_t)kFaK * VST * 2;
  static constexpr size_t kOut = (size_t)kFaWaves * 32 * OST * 2;
  static constexpr size_t kLds = kK + kV > kOut ? kK + kV : kOut;
  static constexpr int kChunks = kFaK * DH / 8;               // 16-byte runs per K (or V) tile
  static constexpr int kPerThread = kChunks / (kFaWaves * 64);
  static_assert(kChunks % (kFaWaves * 64) == 0, "whole runs per thread");
};

// Key/value tile t of the rows this thread stages (rows past the sequence end
// re-read its last row; they are masked).
template <int DH>
__device__ __forceinline__ void fa_load_tile(const _Float16* __restrict__ k, const _Float16* __restrict__ v, int tok0,
                                             int n, int ldkv, int g, int t, int tid,
                                             i32x4 (&kr)[FaCfg<DH>::kPerThread], i32x4 (&vr)[FaCfg<DH>::kPerThread]) {
  constexpr int RUNS = DH / 8;
#pragma unroll
  for (int i = 0; i < FaCfg<DH>::kPerThread; ++i) {
    const int e = tid + kFaWaves * 64 * i, row = e / RUNS, c8 = e - row * RUNS;
    const int key = min(t * kFaK + row, n - 1);
    const int64_t off = (int64_t)(tok0 + key) * ldkv + g * DH + 8 * c8;
    kr[i] = *reinterpret_cast<const i32x4*>(k + off);
    vr[i] = *reinterpret_cast<const i32x4*>(v + off);
  }
}

// ... and its copy into the LDS tiles.
template <int DH>
__device__ __forceinline__ void fa_store_tile(_Float16* ks, _Float16* vs, int tid,
                                              const i32x4 (&kr)[FaCfg<DH>::kPerThread],
                                              const i32x4 (&vr)[FaCfg<DH>::kPerThread]) {
  constexpr int RUNS = DH / 8;
#pragma unroll
  for (int i = 0; i < FaCfg<DH>::kPerThread; ++i) {
    const int e = tid + kFaWaves * 64 * i, row = e / RUNS, c8 = e - row * RUNS;
    *reinterpret_cast<i32x4*>(ks + row * FaCfg<DH>::KST + 8 * c8) = kr[i];
    *reinterpret_cast<i32x4*>(vs + row * FaCfg<DH>::VST + 8 * c8) = vr[i];
  }
}

template <int DH>
__global__ void __launch_bounds__(kFaWaves * 64)
prefill_flash_kernel(const _Float16* __restrict__ q, const _Float16* __restrict__ k, const _Float16* __restrict__ v,
                     const int32_t* __restrict__ cu, int32_t n_seq, int32_t Hq, int32_t Hkv, int32_t n_qt,
                     float scale_log2, _Float16* __restrict__ out) {
  using C = FaCfg<DH>;
  constexpr int KS = DH / 16;      // contraction steps of the score product
  constexpr int OB = DH / 32;      // 32-channel blocks of the output
  constexpr int RUNS = DH / 8;     // 16-byte runs per row
  extern __shared__ __attribute__((aligned(16))) uint8_t fa_smem[];
  _Float16* ks = reinterpret_cast<_Float16*>(fa_smem);
  _Float16* vs = reinterpret_cast<_Float16*>(fa_smem + C::kK);
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int l32 = lane & 31, half = lane >> 5, s16 = lane & 15, q16 = (lane >> 4) & 1;

  // Workgroup -> (sequence, head, query tile).  The query tiles of one
  // (sequence, head) read the same key/value rows, so they get ids that one
  // XCD receives (the chip hands workgroup i to XCD i % 8) and share its L2;
  // within a group the longest tiles (most keys) go first.
  const int groups = n_seq * Hq, total = groups * n_qt;
  int lin = blockIdx.x;
  if (total % 8 == 0) lin = (lin % 8) * (total / 8) + lin / 8;
  const int grp = lin / n_qt, qt = n_qt - 1 - (lin - grp * n_qt);
  const int b = grp / Hq, h = grp - b * Hq;
  const int tok0 = cu[b], n = cu[b + 1] - tok0;
  const int q0 = qt * kFaQ;
  if (q0 >= n) return;
  const int g = (h * Hkv) / Hq;
  const int ldq = Hq * DH, ldkv = Hkv * DH;
  const int kend = min(n, q0 + kFaQ);              // keys this tile of queries can see
  const int n_tiles = (kend + kFaK - 1) / kFaK;
  const int qw0 = q0 + 32 * w;                      // this wave's first query
  const int my_q = qw0 + l32;

  // query slots of the score product: step s, lane half -> channels 16 s + 8 half .. +7
  f16x8 qf[KS];
  {
    const _Float16* qrow = q + (int64_t)(tok0 + min(my_q, n - 1)) * ldq + h * DH + 8 * half;
#pragma unroll
    for (int s = 0; s < KS; ++s) qf[s] = *reinterpret_cast<const f16x8*>(qrow + 16 * s);
  }

  // this thread's 16-byte runs of a K (and V) tile: run e = tid + 256 i is
  // row e / RUNS, columns 8 (e % RUNS) .. +7
  i32x4 kr[C::kPerThread], vr[C::kPerThread];

  f32x16 o[OB];
#pragma unroll
  for (int ob = 0; ob < OB; ++ob) o[ob] = f32x16{};
  float m_run = -INFINITY, l_run = 0.f;
  typedef short s16x4 __attribute__((ext_vector_type(4)));
  typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

  fa_load_tile<DH>(k, v, tok0, n, ldkv, g, 0, tid, kr, vr);
  for (int t = 0; t < n_tiles; ++t) {
    __syncthreads();                                // every wave is done with the previous tile
    fa_store_tile<DH>(ks, vs, tid, kr, vr);
    __syncthreads();
    if (t + 1 < n_tiles) fa_load_tile<DH>(k, v, tok0, n, ldkv, g, t + 1, tid, kr, vr);
    const int kt0 = t * kFaK;
    if (kt0 > qw0 + 31) continue;                   // every key of the tile is after this wave's queries
    // S^T: block kb holds keys kt0 + 32 kb + 8 (v / 4) + 4 half + v % 4 of query my_q
    f32x16 sacc[2] = {f32x16{}, f32x16{}};
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        const f16x8 kf = *reinterpret_cast<const f16x8*>(ks + (32 * kb + l32) * C::KST + 16 * s + 8 * half);
        sacc[kb] = __builtin_amdgcn_mfma_f32_32x32x16_f16(kf, qf[s], sacc[kb], 0, 0, 0);
      }
    float sv[32];
    float mx = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int vv = 0; vv < 16; ++vv) {
        const int key = kt0 + 32 * kb + 8 * (vv >> 2) + 4 * half + (vv & 3);
        const float x = sacc[kb][vv] * scale_log2;
        sv[16 * kb + vv] = (key <= my_q && key < n) ? x : -INFINITY;
        mx = fmaxf(mx, sv[16 * kb + vv]);
      }
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    const float m_new = fmaxf(m_run, mx);
    float alpha = 1.f, ps = 0.f;
    float p[32];
    if (m_new == -INFINITY) {
#pragma unroll
      for (int i = 0; i < 32; ++i) p[i] = 0.f;
    } else {
      alpha = __builtin_amdgcn_exp2f(m_run - m_new);
#pragma unroll
      for (int i = 0; i < 32; ++i) {
        p[i] = __builtin_amdgcn_exp2f(sv[i] - m_new);
        ps += p[i];
      }
    }
    ps += __shfl_xor(ps, 32, 64);
    l_run = l_run * alpha + ps;
    m_run = m_new;
    if (__any(alpha != 1.f)) {
#pragma unroll
      for (int ob = 0; ob < OB; ++ob) o[ob] *= alpha;
    }
    // O^T += V^T P^T over the four 16-key steps (kb, mf): k-slot e of this lane
    // is key 32 kb + 16 mf + 8 (e / 4) + 4 half + e % 4, i.e. score p[16 kb + 8 mf + e].
    // The A operand comes from transposing reads: lane s of the 16-lane group
    // (half, q16) addresses key 32 kb + 16 mf + 4 half + s / 4 (and + 8),
    // channels 32 ob + 16 q16 + 4 (s % 4) .. +3, and receives its 4 keys of
    // one channel.
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int mf = 0; mf < 2; ++mf) {
        f16x8 pf;
#pragma unroll
        for (int e = 0; e < 8; ++e) pf[e] = (_Float16)p[16 * kb + 8 * mf + e];
        const int key = 32 * kb + 16 * mf + 4 * half + (s16 >> 2);
#pragma unroll
        for (int ob = 0; ob < OB; ++ob) {
          const int col = 32 * ob + 16 * q16 + 4 * (s16 & 3);
          const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(vs + key * C::VST + col));
          const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(vs + (key + 8) * C::VST + col));
          const f16x4 flo = __builtin_bit_cast(f16x4, lo), fhi = __builtin_bit_cast(f16x4, hi);
          const f16x8 a = {flo[0], flo[1], flo[2], flo[3], fhi[0], fhi[1], fhi[2], fhi[3]};
          o[ob] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, pf, o[ob], 0, 0, 0);
        }
      }
  }

  // O / l through LDS, so that each query row leaves as 16-byte runs: lane
  // (l32, half) holds query qw0 + l32 at channels 32 ob + 8 vq + 4 half .. +3.
  __syncthreads();
  const float inv_l = l_run > 0.f ? 1.f / l_run : 0.f;
  _Float16* ost = reinterpret_cast<_Float16*>(fa_smem) + w * 32 * C::OST;
#pragma unroll
  for (int ob = 0; ob < OB; ++ob)
#pragma unroll
    for (int vq = 0; vq < 4; ++vq) {
      const f16x4 v4 = {(_Float16)(o[ob][4 * vq] * inv_l), (_Float16)(o[ob][4 * vq + 1] * inv_l),
                        (_Float16)(o[ob][4 * vq + 2] * inv_l), (_Float16)(o[ob][4 * vq + 3] * inv_l)};
      *reinterpret_cast<f16x4*>(ost + l32 * C::OST + 32 * ob + 8 * vq + 4 * half) = v4;
    }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < 32 * RUNS / 64; ++i) {
    const int e = lane + 64 * i, row = e / RUNS, c8 = e - row * RUNS;
    const int qq = qw0 + row;
    if (qq < n)
      *reinterpret_cast<f16x8*>(out + (int64_t)(tok0 + qq) * ldq + h * DH + 8 * c8) =
          *reinterpret_cast<const f16x8*>(ost + row * C::OST + 8 * c8);
  }
}

template <int DH>
static hipError_t launch_flash(const PrefillAttnArgs& a, hipStream_t s) {
  using C = FaCfg<DH>;
  auto kern = prefill_flash_kernel<DH>;
  hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)C::kLds);
  if (e != hipSuccess) return e;
  const int n_qt = (a.max_seqlen + kFaQ - 1) / kFaQ;
  const int64_t blocks = (int64_t)a.batch * a.n_q_heads * n_qt;
  KernelScope ks("prefill_flash", s);
  QSVD_LAUNCH(ks, kern, dim3((unsigned)blocks), dim3(kFaWaves * 64), C::kLds, s, a.q, a.k, a.v, a.cu_seqlens, a.batch,
              a.n_q_heads, a.n_kv_heads, n_qt, a.sm_scale * kFaLog2e, a.out);
  return hipGetLastError();
}

bool prefill_attention_supported(int32_t head_dim) { return head_dim == 64 || head_dim == 128; }

hipError_t launch_prefill_attention(const PrefillAttnArgs& a, hipStream_t s) {
  if (a.batch == 0 || a.max_seqlen == 0) return hipSuccess;
  return a.head_dim == 128 ? launch_flash<128>(a, s) : launch_flash<64>(a, s);
}

}  // namespace qsvd
