// Row pass of the decode-size kernels: per-token symmetric quantization
// (Section 4) of up to 32 fp16 rows by every workgroup that needs them as an
// integer A operand, with the latent cache append folded in.
#pragma once
#include "common.h"

namespace qsvd {

constexpr int kSkMaxRowChunks = 8;  // 8-element chunks per lane held at once: 8 * 64 * 8 = 4096 columns
constexpr int kSkMaxRowK = 16384;   // wider rows are read twice (max pass, then codes)

// The latent cache append fused into the decode-size projections (one new
// row per sequence, row m of the product being sequence m's):
//   SK_APPEND_F16_ROW  down-projection: the fp16 C row also goes to the cache
//                      row seq_len[m] (the epilogue stores each element twice)
//   SK_APPEND_CODES    up-projection: the row's Q(C) codes and scale also go to
//                      the cache row seq_len[m], then seq_len[m] advances
//   SK_APPEND_ADVANCE  up-projection over an fp16 cache: seq_len[m] advances
// A row at or past capacity is not written; seq_len stops at capacity and the
// overflow flag (when given) is set.
enum { SK_APPEND_NONE = 0, SK_APPEND_F16_ROW = 1, SK_APPEND_CODES = 2, SK_APPEND_ADVANCE = 3 };
struct SkinnyAppend {
  uint8_t* data;       // cache rows
  float* scale;        // integer caches: per-row scales
  int32_t* seq_len;
  int32_t* overflow;   // optional
  int32_t capacity;
  int32_t mode;
};

// Quantize rows m = w, w + nw, ... < M of the fp16 rows `ch` (row stride lda,
// K <= 4096 columns): wave w holds a row in registers (8-element chunks lane,
// lane + 64, ...), takes its max |x| round the wave, and writes its codes to
// LDS (qa, row stride qa_ld, one byte per code) and its scale to rsc[m].  The
// owning workgroup of row m (blockIdx.x == m mod gridDim.x) also stores the
// codes and scale to cq_out / sc_out (when given) and, for SK_APPEND_CODES,
// to the cache row seq_len[m].  MAXCH bounds the chunks per lane (K <= 512 MAXCH).
template <int MAXCH = kSkMaxRowChunks>
__device__ __forceinline__ void sk_row_pass_narrow(const _Float16* __restrict__ ch, int64_t lda, float clip, int32_t M,
                                            int32_t K, int32_t abits, int w, int nw, int lane, int8_t* qa,
                                            int qa_ld, float* rsc, uint8_t* __restrict__ cq_out,
                                            float* __restrict__ sc_out, const SkinnyAppend& ap) {
  const float qm = (float)((1 << (abits - 1)) - 1);
  const int nch = K / 8;
  for (int m = w; m < M; m += nw) {
    f16x8 v[MAXCH];
#pragma unroll
    for (int i = 0; i < MAXCH; ++i) {
      const int c = lane + 64 * i;
      v[i] = c < nch ? *reinterpret_cast<const f16x8*>(ch + (int64_t)m * lda + 8 * c) : f16x8{};
    }
    u16x2 mb = u16x2{0, 0};
#pragma unroll
    for (int i = 0; i < MAXCH; ++i) mb = absmax_f16x8(mb, v[i]);
    const float a = mul_rn(clip, wave_max(absmax_value(mb)));
    const float inv = a != 0.f ? div_rn(qm, a) : 0.f;
    const float sc = a != 0.f ? div_rn(a, qm) : 1.f;
    const bool own = (m % (int)gridDim.x) == (int)blockIdx.x;
    // the cache row this sequence's codes also go to (integer caches)
    const bool app = own && ap.mode == SK_APPEND_CODES;
    const int32_t pos = app ? ap.seq_len[m] : 0;
    const bool app_row = app && pos >= 0 && pos < ap.capacity;
    uint8_t* crow = ap.data + ((int64_t)m * ap.capacity + (app_row ? pos : 0)) * (abits == 8 ? K : K / 2);
    if (lane == 0) {
      rsc[m] = sc;
      if (own && sc_out) sc_out[m] = sc;
      if (app_row) ap.scale[(int64_t)m * ap.capacity + pos] = sc;
    }
#pragma unroll
    for (int i = 0; i < MAXCH; ++i) {
      const int c = lane + 64 * i;
      if (c >= nch) continue;
      uint32_t q[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) q[e] = code_bits((float)v[i][e], inv, qm);
      const uint32_t lo = pack4_codes8(q[0], q[1], q[2], q[3]), hi = pack4_codes8(q[4], q[5], q[6], q[7]);
      *reinterpret_cast<uint2*>(qa + m * qa_ld + 8 * c) = make_uint2(lo, hi);
      if (own && (cq_out || app_row)) {
        if (abits == 8) {
          if (cq_out) *reinterpret_cast<uint2*>(cq_out + (int64_t)m * K + 8 * c) = make_uint2(lo, hi);
          if (app_row) *reinterpret_cast<uint2*>(crow + 8 * c) = make_uint2(lo, hi);
        } else {
          const uint32_t p = pack8_codes4(q);
          if (cq_out) *reinterpret_cast<uint32_t*>(cq_out + (int64_t)m * (K / 2) + 4 * c) = p;
          if (app_row) *reinterpret_cast<uint32_t*>(crow + 4 * c) = p;
        }
      }
    }
  }
}

// The same for rows of more than 512 MAXCH columns.  A row is split into S
// parts (S = nw / M, at most 4, when the workgroup has at least two waves per
// row; else 1), one wave per part: every part's max |x| goes to LDS, and
// after a barrier each wave forms its row's max from the parts and writes
// its part's codes.  A part that fits the registers (512 MAXCH columns, one
// part per wave) is read once; otherwise it is read again for the codes.
// Every wave reaches the one barrier.
template <int MAXCH = kSkMaxRowChunks>
__device__ __forceinline__ void sk_row_pass_wide(const _Float16* __restrict__ ch, int64_t lda, float clip, int32_t M,
                                            int32_t K, int32_t abits, int w, int nw, int lane, int8_t* qa,
                                            int qa_ld, float* rsc, uint8_t* __restrict__ cq_out,
                                            float* __restrict__ sc_out, const SkinnyAppend& ap) {
  __shared__ float part_max[32];     // M * S <= 32: M <= 32, and M * S <= nw <= 16 for S > 1
  const float qm = (float)((1 << (abits - 1)) - 1);
  const int nch = K / 8;
  const int S = nw >= 2 * M ? min(nw / M, 4) : 1;
  const int per = (nch + S - 1) / S;                  // chunks per part
  const bool keep = M * S <= nw && per <= 64 * MAXCH;  // each wave's one part stays in registers
  f16x8 v[MAXCH];
  auto load = [&](int m, int c0, int c_end) {
#pragma unroll
    for (int i = 0; i < MAXCH; ++i) {
      const int c = c0 + lane + 64 * i;
      v[i] = c < c_end ? *reinterpret_cast<const f16x8*>(ch + (int64_t)m * lda + 8 * c) : f16x8{};
    }
  };
  for (int it = w; it < M * S; it += nw) {
    const int m = it / S, pt = it - m * S, cb = pt * per, ce = min(nch, cb + per);
    u16x2 mb = u16x2{0, 0};
    for (int c0 = cb; c0 < ce; c0 += 64 * MAXCH) {
      load(m, c0, ce);
#pragma unroll
      for (int i = 0; i < MAXCH; ++i) mb = absmax_f16x8(mb, v[i]);
    }
    const float pm = wave_max(absmax_value(mb));
    if (lane == 0) part_max[it] = pm;
  }
  __syncthreads();
  for (int it = w; it < M * S; it += nw) {
    const int m = it / S, pt = it - m * S, cb = pt * per, ce = min(nch, cb + per);
    float mx = part_max[m * S];
    for (int q2 = 1; q2 < S; ++q2) mx = fmaxf(mx, part_max[m * S + q2]);
    const float a = mul_rn(clip, mx);
    const float inv = a != 0.f ? div_rn(qm, a) : 0.f;
    const float sc = a != 0.f ? div_rn(a, qm) : 1.f;
    const bool own = (m % (int)gridDim.x) == (int)blockIdx.x;
    // the cache row this sequence's codes also go to (integer caches)
    const bool app = own && ap.mode == SK_APPEND_CODES;
    const int32_t pos = app ? ap.seq_len[m] : 0;
    const bool app_row = app && pos >= 0 && pos < ap.capacity;
    uint8_t* crow = ap.data + ((int64_t)m * ap.capacity + (app_row ? pos : 0)) * (abits == 8 ? K : K / 2);
    if (lane == 0 && pt == 0) {
      rsc[m] = sc;
      if (own && sc_out) sc_out[m] = sc;
      if (app_row) ap.scale[(int64_t)m * ap.capacity + pos] = sc;
    }
    for (int c0 = cb; c0 < ce; c0 += 64 * MAXCH) {
      if (!keep) load(m, c0, ce);
#pragma unroll
      for (int i = 0; i < MAXCH; ++i) {
        const int c = c0 + lane + 64 * i;
        if (c >= ce) continue;
        uint32_t q[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) q[e] = code_bits((float)v[i][e], inv, qm);
        const uint32_t lo = pack4_codes8(q[0], q[1], q[2], q[3]), hi = pack4_codes8(q[4], q[5], q[6], q[7]);
        *reinterpret_cast<uint2*>(qa + m * qa_ld + 8 * c) = make_uint2(lo, hi);
        if (own && (cq_out || app_row)) {
          if (abits == 8) {
            if (cq_out) *reinterpret_cast<uint2*>(cq_out + (int64_t)m * K + 8 * c) = make_uint2(lo, hi);
            if (app_row) *reinterpret_cast<uint2*>(crow + 8 * c) = make_uint2(lo, hi);
          } else {
            const uint32_t p = pack8_codes4(q);
            if (cq_out) *reinterpret_cast<uint32_t*>(cq_out + (int64_t)m * (K / 2) + 4 * c) = p;
            if (app_row) *reinterpret_cast<uint32_t*>(crow + 4 * c) = p;
          }
        }
      }
    }
  }
}

// The row pass of a kernel built for rows up to 512 MAXCH columns (WIDE
// false) or wider ones.
template <bool WIDE, int MAXCH = kSkMaxRowChunks>
__device__ __forceinline__ void sk_row_pass(const _Float16* __restrict__ ch, int64_t lda, float clip, int32_t M,
                                            int32_t K, int32_t abits, int w, int nw, int lane, int8_t* qa,
                                            int qa_ld, float* rsc, uint8_t* __restrict__ cq_out,
                                            float* __restrict__ sc_out, const SkinnyAppend& ap) {
  if constexpr (WIDE)
    sk_row_pass_wide<MAXCH>(ch, lda, clip, M, K, abits, w, nw, lane, qa, qa_ld, rsc, cq_out, sc_out, ap);
  else
    sk_row_pass_narrow<MAXCH>(ch, lda, clip, M, K, abits, w, nw, lane, qa, qa_ld, rsc, cq_out, sc_out, ap);
}

// After the row pass (and a barrier): the cache row of each sequence this
// workgroup owns is complete, so its length advances (only the owning
// workgroup reads or writes seq_len[m] here).
__device__ __forceinline__ void sk_advance(const SkinnyAppend& ap, int32_t M, int tid) {
  if ((ap.mode == SK_APPEND_CODES || ap.mode == SK_APPEND_ADVANCE) && tid < M &&
      (tid % (int)gridDim.x) == (int)blockIdx.x) {
    const int32_t base = ap.seq_len[tid];
    if (base >= ap.capacity && ap.overflow) *ap.overflow = 1;
    ap.seq_len[tid] = base >= ap.capacity ? ap.capacity : base + 1;
  }
}

}  // namespace qsvd
