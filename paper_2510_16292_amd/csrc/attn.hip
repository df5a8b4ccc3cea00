// Decode attention over the latent cache (Section 3.1: only C is cached and
// K = C W^u_k, V = C W^u_v are recomputed from it, Eq. 5).
//
// Absorbed form (default): since q . (C_t W^u_k)^T = (q W^u_k^T) . C_t and
// sum_t p_t C_t W^u_v = (sum_t p_t C_t) W^u_v, the query is first mapped into
// the rank-r latent space once per step, every head then attends directly over
// the cached latent rows, and W^u_v is applied once to the latent-space result.
//
//   absorb_kernel       q~[b][h][:] = (sm_scale * log2 e) * q[b][h] W^u_k,g(h)^T     (fp16)
//   latent_attn_kernel  per (sequence, context chunk): S = q~ C^T, online softmax,
//                       O = P C over the chunk -> split partials (m, l, O)
//   merge_latent_kernel merge the chunk partials of each sequence
//   vproj_kernel        o[b][h] = O[b][h] W^u_v,g(h)                               (fp16)
//
// Reconstruct form (for comparison): K^, V^ are rebuilt for every cached token
// with an fp16 matrix-core GEMM and a plain split-context attention follows.
#include <math.h>

#include <algorithm>
#include <type_traits>

#include "common.h"
#include "launch.h"

namespace qsvd {

constexpr float kLog2e = 1.4426950408889634f;
constexpr int kHeadBlk = 32;   // query heads are padded to one 32-wide MFMA block
constexpr int kMaxChunks = 256;  // context chunks per sequence the merge supports
constexpr int kMaxAbsorbedHeads = 64;   // query heads per sequence in the absorbed form

// ---------------------------------------------------------------------------
// Exact integer code -> fp16 conversion by exponent bias: a code made unsigned
// (offset binary, by flipping its sign bit) is placed in the low mantissa bits
// of 1024.0 (0x6400), where every integer below 1024 is exact, and the bias is
// removed with one packed fp16 operation per two codes.
// ---------------------------------------------------------------------------
__device__ inline f16x2 bias_sub(uint32_t d, f16x2 mul, f16x2 add) {
  return __builtin_elementwise_fma(__builtin_bit_cast(f16x2, d), mul, add);
}

// 8 int8 codes (bytes of w0 then w1, lowest first) -> fp16, in order.
__device__ inline f16x8 cvt_i8x8(uint32_t w0, uint32_t w1) {
  const uint32_t u0 = w0 ^ 0x80808080u, u1 = w1 ^ 0x80808080u;
  const f16x2 one = {(_Float16)1.f, (_Float16)1.f}, off = {(_Float16)-1152.f, (_Float16)-1152.f};
  // perm: byte k of the result is byte sel_k of (0x64646464 : u), 4 = a 0x64 byte
  const f16x2 a = bias_sub(__builtin_amdgcn_perm(0x64646464u, u0, 0x04010400u), one, off);
  const f16x2 b = bias_sub(__builtin_amdgcn_perm(0x64646464u, u0, 0x04030402u), one, off);
  const f16x2 c = bias_sub(__builtin_amdgcn_perm(0x64646464u, u1, 0x04010400u), one, off);
  const f16x2 d = bias_sub(__builtin_amdgcn_perm(0x64646464u, u1, 0x04030402u), one, off);
  return f16x8{a[0], a[1], b[0], b[1], c[0], c[1], d[0], d[1]};
}

// 8 int4 codes (nibbles of w, lowest first) -> fp16, in order.  Byte i holds
// codes 2i (low nibble) and 2i + 1 (high nibble): the low one lands in
// 1024 + n, the high one in 1024 + 16 n, undone by (x * 1/16 - 72).
__device__ inline f16x8 cvt_i4x8(uint32_t w) {
  const uint32_t u = w ^ 0x88888888u;
  const f16x2 mul = {(_Float16)1.f, (_Float16)0.0625f}, off = {(_Float16)-1032.f, (_Float16)-72.f};
  f16x8 r;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint32_t sel = 0x04000400u | ((uint32_t)i << 16) | (uint32_t)i;
    const f16x2 h = bias_sub(__builtin_amdgcn_perm(0x64646464u, u, sel) & 0xFFF0FF0Fu, mul, off);
    r[2 * i] = h[0];
    r[2 * i + 1] = h[1];
  }
  return r;
}

// Max and sum of a value over the four 16-lane rows of a wave (lanes l, l ^ 16,
// l ^ 32, l ^ 48), every lane receiving the result, at vector-ALU latency
// with gfx950's lane swaps: v_permlane32_swap a, b exchanges rows 2-3 of a
// with rows 0-1 of b (a row is 16 lanes) and v_permlane16_swap a, b rows 1, 3
// of a with rows 0, 2 of b, so with a = b = x the pair (a, b) holds each
// lane's value and its partner's.  (Issued as asm with both registers
// read-write: the compiler builtin's second result is not usable here; the
// s_nop covers the hazard of a vector write just before the swap.)  The sum
// adds in the same order in every lane.
__device__ __forceinline__ void swap32(uint32_t& a, uint32_t& b) {
  asm volatile("s_nop 1\n\tv_permlane32_swap_b32 %0, %1" : "+v"(a), "+v"(b));
}
__device__ __forceinline__ void swap16(uint32_t& a, uint32_t& b) {
  asm volatile("s_nop 1\n\tv_permlane16_swap_b32 %0, %1" : "+v"(a), "+v"(b));
}

__device__ __forceinline__ float rows4_max(float x) {
  uint32_t a = __builtin_bit_cast(uint32_t, x), b = a;
  swap32(a, b);
  uint32_t c = __builtin_bit_cast(uint32_t, fmaxf(__builtin_bit_cast(float, a), __builtin_bit_cast(float, b))), e = c;
  swap16(c, e);
  return fmaxf(__builtin_bit_cast(float, c), __builtin_bit_cast(float, e));
}

__device__ __forceinline__ float rows4_sum(float x) {
  uint32_t a = __builtin_bit_cast(uint32_t, x), b = a;
  swap32(a, b);
  uint32_t c = __builtin_bit_cast(uint32_t, __builtin_bit_cast(float, a) + __builtin_bit_cast(float, b)), e = c;
  swap16(c, e);
  return __builtin_bit_cast(float, c) + __builtin_bit_cast(float, e);
}

// ---------------------------------------------------------------------------
// q~ = scale * q W^u_k^T on the 16x16x32 fp16 matrix cores.  One wave per
// (head h, 64 latent columns j): the dh x 64 block of W^u_k codes (rows
// c = key channel, contiguous in j) is staged in LDS as exact fp16 codes, and
// the channel scales multiply the query, which enters as an fp16 hi/lo pair
// (two MFMAs, about fp32 accuracy); the MFMA needs 8 consecutive c of one column j per lane, which
// two LDS transpose reads deliver (lane s of each 16-lane group addresses row
// base + s/4 at columns 4*(s%4)..+3 and receives 4 rows of one column).  Rows
// of the product are 16 sequences (query rows loaded straight from memory),
// columns 16 latent indices, the contraction the dh key channels.
// ---------------------------------------------------------------------------
constexpr int kAbsorbJ = 64;
constexpr int kAbsorbLd = kAbsorbJ + 16;   // stride 40 dwords = 8 (mod 32): conflict-free transpose reads

// NT 16 x 16 tiles of q~ (16 query rows x 16 latent columns, at columns
// col0 + 16 jj of the staged codes wk: row c = key channel, stride ld halves,
// ld = 8 mod 32 dwords).  a[k]: this lane's query channels 32 k + 8 quad + e
// of row l16; sc4[k][hh]: the weight scales of those channels.  For every
// 32-channel step the scaled query q_c * s_c enters as an fp16 pair hi + lo
// (the product of two fp16 MFMAs then carries it to about fp32 accuracy); the
// MFMA needs 8 consecutive c of one column per lane, which two LDS transpose
// reads deliver (lane s of each 16-lane group addresses row base + s/4 at
// columns 4*(s%4)..+3 and receives 4 rows of one column).
template <int NT>
__device__ __forceinline__ void absorb_tiles(const f16x8* a, const f32x4 (*sc4)[2], int dh, const _Float16* wk,
                                             int ld, int col0, int lane, f32x4* acc) {
  typedef short s16x4 __attribute__((ext_vector_type(4)));
  typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
  const int s16 = lane & 15, quad = lane >> 4;
#pragma unroll
  for (int jj = 0; jj < NT; ++jj) acc[jj] = f32x4{};
#pragma unroll
  for (int k = 0; k < 128 / 32; ++k) {
    const int c0 = 32 * k;
    if (c0 >= dh) break;
    f16x8 ahi, alo;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float x = (float)a[k][e] * sc4[k][e >> 2][e & 3];
      ahi[e] = to_f16(x);        // x rounded to fp32 first (no fused single rounding)
      alo[e] = to_f16(x - (float)ahi[e]);
    }
#pragma unroll
    for (int jj = 0; jj < NT; ++jj) {
      const int row = c0 + 8 * quad + (s16 >> 2);
      const int col = col0 + jj * 16 + 4 * (s16 & 3);
      const s16x4 x0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)&wk[row * ld + col]);
      const s16x4 x1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)&wk[(row + 4) * ld + col]);
      const f16x4 f0 = __builtin_bit_cast(f16x4, x0), f1 = __builtin_bit_cast(f16x4, x1);
      const f16x8 bw = {f0[0], f0[1], f0[2], f0[3], f1[0], f1[1], f1[2], f1[3]};
      acc[jj] = __builtin_amdgcn_mfma_f32_16x16x32_f16(ahi, bw, acc[jj], 0, 0, 0);
      acc[jj] = __builtin_amdgcn_mfma_f32_16x16x32_f16(alo, bw, acc[jj], 0, 0, 0);
    }
  }
}

// int8 codes (16 per i32x4, element e in byte e) -> two fp16 x 8 (exact)
__device__ __forceinline__ void codes16_to_f16(const uint32_t* wv, f16x8& lo, f16x8& hi) {
  lo = cvt_i8x8(wv[0], wv[1]);
  hi = cvt_i8x8(wv[2], wv[3]);
}

__global__ void __launch_bounds__(64)
absorb_kernel(const _Float16* __restrict__ q, const uint8_t* __restrict__ bt, const float* __restrict__ sb,
              int32_t B, int32_t r, int32_t Hq, int32_t Hkv, int32_t dh, int32_t N, int32_t bits,
              int32_t group, float scale, int32_t hp, _Float16* __restrict__ qt) {
  __shared__ __attribute__((aligned(16))) _Float16 wk[128 * kAbsorbLd];
  __shared__ __attribute__((aligned(16))) _Float16 ot[16 * (kAbsorbJ + 8)];   // output tile, 16 sequences
  const int h = blockIdx.x, lane = threadIdx.x;
  const int32_t jb = blockIdx.y * kAbsorbJ;
  if (h >= Hq) {
    for (int e = lane; e < B * (kAbsorbJ / 8); e += 64) {
      const int b = e / (kAbsorbJ / 8), j8 = e - b * (kAbsorbJ / 8);
      *reinterpret_cast<f16x8*>(qt + ((int64_t)b * hp + h) * r + jb + 8 * j8) = f16x8{};
    }
    return;
  }
  const int g = (h * Hkv) / Hq;
  const int32_t nk0 = Hq * dh + g * dh;
  // The weight scale of key channel c (per channel, or of this block's group:
  // a 64-column block never straddles a group) multiplies the query, not the
  // staged codes, which stay exact in fp16.
  const float* srow = sb + (group ? (int64_t)(jb / group) * N : 0) + nk0;
  // stage: chunk e -> row c = e / 4, 16 codes at columns 16 * (e % 4); every
  // lane's loads (dh <= 128: at most 8 chunks) go out before any is used
  constexpr int kStageIt = 128 * 4 / 64;
  uint4 raw[kStageIt];
#pragma unroll
  for (int it = 0; it < kStageIt; ++it) {
    const int e = lane + 64 * it;
    if (e >= dh * 4) break;
    const int c = e >> 2, j16 = (e & 3) * 16;
    const int32_t n = nk0 + c;
    if (bits == 8) {
      raw[it] = *reinterpret_cast<const uint4*>(bt + (int64_t)n * r + jb + j16);
    } else {
      const uint2 r2 = *reinterpret_cast<const uint2*>(bt + ((int64_t)n * r + jb + j16) / 2);
      raw[it] = make_uint4(r2.x, r2.y, 0u, 0u);
    }
  }
  const int l16 = lane & 15, quad = lane >> 4;
  // this lane's contraction channels c = 32k + 8*quad + e: their scales, and
  // the query rows of the first 16 sequences, loaded while the weights arrive
  constexpr int KC = 128 / 32;
  f32x4 sc4[KC][2];
#pragma unroll
  for (int k = 0; k < KC; ++k)
#pragma unroll
    for (int hh = 0; hh < 2; ++hh)
      sc4[k][hh] = 32 * k < dh ? *reinterpret_cast<const f32x4*>(srow + 32 * k + 8 * quad + 4 * hh) : f32x4{};
  f16x8 qa[KC];
  {
    const int bA = l16;
    const _Float16* qrow = q + (int64_t)min(bA, B - 1) * Hq * dh + h * dh + 8 * quad;
#pragma unroll
    for (int k = 0; k < KC; ++k) qa[k] = (32 * k < dh && bA < B) ? *reinterpret_cast<const f16x8*>(qrow + 32 * k) : f16x8{};
  }
#pragma unroll
  for (int it = 0; it < kStageIt; ++it) {
    const int e = lane + 64 * it;
    if (e >= dh * 4) break;
    const int c = e >> 2, j16 = (e & 3) * 16;
    f16x8 lo, hi;
    if (bits == 8) {
      const uint32_t wv[4] = {raw[it].x, raw[it].y, raw[it].z, raw[it].w};
      codes16_to_f16(wv, lo, hi);
    } else {
      lo = cvt_i4x8(raw[it].x);
      hi = cvt_i4x8(raw[it].y);
    }
    *reinterpret_cast<f16x8*>(&wk[c * kAbsorbLd + j16]) = lo;
    *reinterpret_cast<f16x8*>(&wk[c * kAbsorbLd + j16 + 8]) = hi;
  }
  __syncthreads();
  for (int b0 = 0; b0 < B; b0 += 16) {
    const int bA = b0 + l16;
    const _Float16* qrow = q + (int64_t)min(bA, B - 1) * Hq * dh + h * dh + 8 * quad;
    f16x8 a[KC];
#pragma unroll
    for (int k = 0; k < KC; ++k) {
      a[k] = 32 * k >= dh ? f16x8{} : b0 == 0 ? qa[k] : *reinterpret_cast<const f16x8*>(qrow + 32 * k);
      if (bA >= B) a[k] = f16x8{};
    }
    f32x4 acc[kAbsorbJ / 16];
    absorb_tiles<kAbsorbJ / 16>(a, sc4, dh, wk, kAbsorbLd, 0, lane, acc);
    // lane holds column jb + 16*jj + l16 and sequences b0 + 4*quad + v; the
    // tile goes through LDS so that each sequence row leaves as 16-byte runs
#pragma unroll
    for (int jj = 0; jj < kAbsorbJ / 16; ++jj)
#pragma unroll
      for (int v = 0; v < 4; ++v)
        ot[(4 * quad + v) * (kAbsorbJ + 8) + 16 * jj + l16] = to_f16(acc[jj][v] * scale);
    __syncthreads();
#pragma unroll
    for (int i = 0; i < 16 * kAbsorbJ / 8 / 64; ++i) {
      const int e = lane + 64 * i, bl = e / (kAbsorbJ / 8), j8 = 8 * (e % (kAbsorbJ / 8));
      if (b0 + bl < B)
        *reinterpret_cast<f16x8*>(qt + ((int64_t)(b0 + bl) * hp + h) * r + jb + j8) =
            *reinterpret_cast<const f16x8*>(ot + bl * (kAbsorbJ + 8) + j8);
    }
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// Latent attention over one context chunk of one sequence.
//
// The workgroup has NW waves; wave w owns latent columns [w*RW, (w+1)*RW).
// Per 32-token tile:
//   S^T (tokens x heads) = C_tile[:, slice] q~[:, slice]^T   (fp16 MFMA, K = RW)
//   partial S^T of all waves are summed through LDS in a fixed order
//   online softmax per head in fp32 (lane l tracks head l % 32)
//   O^T[slice] (r x heads) += C_tile[:, slice]^T P^T          (fp16 MFMA, K = 32 tokens)
// Each wave copies its slice of the C tile (as exact fp16) into a private
// LDS area as soon as it arrives, reissues the next tile's loads into the
// same registers, and reads the copy back for both MFMAs (row reads for the
// scores, transposing reads for P C).
//
// PRE (rotary layers, decode): the scores come precomputed from the rotated
// keys, pre[b][t][32 heads] in fp32 (already scaled by sm_scale log2 e), and
// only the value side runs in latent space; every wave reads the scores of
// its tile itself, so the tile loop has no barrier.
// ---------------------------------------------------------------------------
template <int RW, int NW, int FMT, bool PRE>
__global__ void __launch_bounds__(NW * 64)
latent_attn_kernel(const _Float16* __restrict__ qt, const uint8_t* __restrict__ cdata,
                   const float* __restrict__ cscale, const int32_t* __restrict__ seq_len,
                   int32_t capacity, int32_t r, int32_t chunk, int32_t n_chunks, int32_t q_len,
                   const float* __restrict__ pre, _Float16* __restrict__ o_part, float* __restrict__ ml_part) {
  constexpr int KS = RW / 16;    // 16-wide contraction steps of the score MFMA
  constexpr int RB = RW / 32;    // 32-row blocks of the output MFMA
  // Staged row stride in halves: RW + 40 makes it an odd multiple of 4 dwords
  // (mod 64), so the 16-byte row accesses of 16 consecutive rows fall on
  // distinct groups of gfx950's 64 LDS banks (RW + 16, a multiple of 8, left
  // them two-way conflicted: 1.39 conflict cycles per active LDS cycle, now 0.35).
  constexpr int CST = RW + 40;
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int half = lane >> 5, l32 = lane & 31;
  _Float16* cst = reinterpret_cast<_Float16*>(smem) + w * 32 * CST;
  // Score exchange: wave w stores its 32x32 partial as f32x4 [w][v/4][lane],
  // 256 threads add the NW partials in wave order into ssum4 [v/4][lane].
  f32x4* spart4 = reinterpret_cast<f32x4*>(smem + NW * 32 * CST * 2);
  f32x4* ssum4 = spart4 + NW * 256;
  // Integer rows: the per-token scales of the wave's tile, staged with it
  // (each lane loads the scale of its own row, and reads back the 16 of the
  // tokens whose scores it holds).
  float* scl = reinterpret_cast<float*>(smem + NW * 32 * CST * 2 + (PRE ? 0 : (size_t)(NW + 1) * 1024 * 4)) + w * 32;

  // Workgroup row blockIdx.y is query i of sequence b (q_len queries per
  // sequence, the last q_len cached positions): it sees positions
  // [0, L - q_len + i], causally.  Decode has q_len = 1.
  const int vb = blockIdx.y, ch = blockIdx.x;
  const int b = vb / q_len, qi = vb - b * q_len;
  const int L = min(seq_len[b], capacity) - (q_len - 1 - qi);
  const int t_begin = ch * chunk;
  if (t_begin >= L) return;
  const int t_end = min(L, t_begin + chunk);
  const int slice0 = w * RW;

  // Contraction slots of the score MFMA: in step ks, lane (l32, half) feeds
  // token t0 + l32 at latent columns slice0 + kcol(ks, half) .. +7.  fp16 rows
  // come 8 columns (16 bytes) per load; int8 rows 16 columns per load, which
  // serve steps 2k and 2k + 1.  The query slots follow the same map.
  constexpr bool F16C = FMT == QSVD_CACHE_F16;
  auto kcol = [](int ks, int hf) { return F16C ? 16 * ks + 8 * hf : 32 * (ks >> 1) + 16 * hf + 8 * (ks & 1); };
  f16x8 qf[KS];
  f32x16 o[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) o[rb] = f32x16{};
  float m_run = -INFINITY, l_run = 0.f;

  // Raw tile registers: fp16 rows as they are, int8 rows as 16-byte chunks,
  // int4 rows as 8-byte chunks (16 codes, element 2i in the low nibble of
  // byte i); for the integer formats also the per-token scales of the 16
  // tokens whose scores and probabilities this lane holds
  // (t0 + 8*(v/4) + 4*half + v%4).
  constexpr bool I4C = FMT == QSVD_CACHE_I4;
  constexpr int NLD = F16C ? KS : KS / 2;
  // Staging the tile before the score product (and reissuing the loads
  // first) measured faster for fp16 rows and keeps the widest integer
  // slices from spilling; narrower integer slices convert in registers
  // and feed the score product directly.
  constexpr bool kStageFirst = F16C || RW >= 192;
  // Tiles in flight per wave: narrow integer slices keep two (a 32-token
  // tile of them is only 4 KB per wave, so one in flight leaves each tile
  // waiting most of a memory round trip); the loop then takes the tiles in
  // pairs, slot sl holding the tile 32 * sl tokens in, with every load
  // unconditional (clamped) so the loads in flight can be counted.
  constexpr int KD = (!kStageFirst && !PRE) ? 2 : 1;
  using RawT = typename std::conditional<F16C, f16x8, typename std::conditional<I4C, uint2, uint4>::type>::type;
  RawT raw[KD][NLD];
  float scr[KD], sc_cur[F16C ? 1 : 16];
  // Where load i of a lane goes in the wave's 32 x RW tile.  A tile that is
  // staged in LDS before any use is read row-major: consecutive lanes take
  // consecutive 16-byte (fp16, int8) or 8-byte (int4) chunks of a row slice
  // (24 lanes per 192-column fp16 slice), so one load instruction covers
  // whole cache lines (8 of them for fp16) instead of a 32-byte piece of 32
  // rows.  A tile that feeds the score product from registers keeps the
  // product's operand layout: row l32, the columns of contraction step i.
  constexpr bool kRowMajor = kStageFirst || PRE;
  constexpr int CPR = F16C ? RW / 8 : RW / 16;     // load chunks per row slice
  // the lane pattern repeats every P loads (64 P chunks = RPP whole rows),
  // so a lane holds only P distinct (row, column) pairs
  static_assert(CPR <= 64, "a row slice of at most 64 load chunks");
  constexpr int P = CPR / (CPR & -CPR);     // CPR / gcd(64, CPR)
  constexpr int RPP = 64 * P / CPR;
  auto trow = [&](int i) { return kRowMajor ? (i / P) * RPP + (64 * (i % P) + lane) / CPR : l32; };
  auto tcol = [&](int i) {
    return kRowMajor ? (F16C ? 8 : 16) * ((64 * (i % P) + lane) % CPR) : kcol(F16C ? i : 2 * i, half);
  };
  // this sequence's rows: element (t, x) at byte (t * r + x) * elem
  const int64_t seq_elems = (int64_t)b * capacity * r;
  const uint8_t* cseq = cdata + (F16C ? 2 * seq_elems : I4C ? seq_elems / 2 : seq_elems);
  // Row-major tiles come through range-checked buffer loads: one buffer per
  // group of RPP rows, ending at the chunk end, so rows past it read as zeros
  // (and are masked) without a memory access; a lane's offset into the group
  // is one of P constants.
  const int row_bytes = F16C ? 2 * r : I4C ? r / 2 : r;
  constexpr int CB = I4C ? 8 : 16;                  // bytes per load chunk
  int voff[P];
#pragma unroll
  for (int j = 0; j < P; ++j)
    voff[j] = trow(j) * row_bytes + CB * ((64 * j + lane) % CPR) + (F16C ? 2 * slice0 : I4C ? slice0 / 2 : slice0);
  auto load_tile = [&](int sl, int t0) {
    if constexpr (!F16C) scr[sl] = cscale[(int64_t)b * capacity + min(t0 + l32, L - 1)];
    if constexpr (kRowMajor) {
#pragma unroll
      for (int q = 0; q < NLD / P; ++q) {
        const int t = t0 + RPP * q;
        // (uniform; readfirstlane keeps the resource in scalar registers)
        const int nrows = __builtin_amdgcn_readfirstlane(max(0, min(RPP, t_end - t)));
        const auto rs = __builtin_amdgcn_make_buffer_rsrc((void*)(cseq + (int64_t)t * row_bytes), (short)0,
                                                          nrows * row_bytes, 0x00020000);
#pragma unroll
        for (int j = 0; j < P; ++j) {
          if constexpr (I4C)
            raw[sl][P * q + j] = __builtin_bit_cast(RawT, __builtin_amdgcn_raw_buffer_load_b64(rs, voff[j], 0, 0));
          else
            raw[sl][P * q + j] = __builtin_bit_cast(RawT, __builtin_amdgcn_raw_buffer_load_b128(rs, voff[j], 0, 0));
        }
      }
    } else {
      // rows past the chunk end are masked; re-read the last row instead of
      // fetching the next chunk's rows
      const int64_t off = ((int64_t)b * capacity + min(t0 + l32, t_end - 1)) * r + slice0;
#pragma unroll
      for (int i = 0; i < NLD; ++i) {
        if constexpr (I4C)
          raw[sl][i] = *reinterpret_cast<const RawT*>(cdata + (off + kcol(2 * i, half)) / 2);
        else
          raw[sl][i] = *reinterpret_cast<const RawT*>(reinterpret_cast<const int8_t*>(cdata) + off + kcol(2 * i, half));
      }
    }
  };
  // the scales of tokens t0 + 8*(v/4) + 4*half + v%4, from the wave's staged copy
  auto read_scales = [&]() {
    if constexpr (!F16C) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const f32x4 q4 = *reinterpret_cast<const f32x4*>(scl + 8 * j + 4 * half);
#pragma unroll
        for (int e = 0; e < 4; ++e) sc_cur[4 * j + e] = q4[e];
      }
    }
  };
  // With one tile in flight the query slice is read after the first tile's
  // loads are out (it is an L2 hit, the tile comes from HBM).  With two, the
  // loads go out in the order the loop consumes them (query, slot 0, slot 1),
  // so that the wait before each use can leave the later ones in flight.
  // The slice (32 heads x RW) is read row-major like a staged tile, whole
  // cache lines per load instruction, then passed through the wave's LDS
  // copy (free until the first tile is staged) into the score product's
  // operand layout.
  constexpr int CPQ = RW / 8;     // 16-byte chunks per head row of the slice
  auto load_query = [&]() {
    if constexpr (!PRE) {
      const _Float16* qb = qt + (int64_t)vb * kHeadBlk * r + slice0;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const int c = 64 * ks + lane;
        qf[ks] = *reinterpret_cast<const f16x8*>(qb + (int64_t)(c / CPQ) * r + 8 * (c % CPQ));
      }
    }
  };
  auto query_operands = [&]() {
    if constexpr (!PRE) {
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const int c = 64 * ks + lane;
        *reinterpret_cast<f16x8*>(cst + (c / CPQ) * CST + 8 * (c % CPQ)) = qf[ks];
      }
      asm volatile("" ::: "memory");
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) qf[ks] = *reinterpret_cast<const f16x8*>(cst + l32 * CST + kcol(ks, half));
      asm volatile("" ::: "memory");
    }
  };
  if constexpr (KD > 1) {
    load_query();
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int sl = 0; sl < KD; ++sl) {
      load_tile(sl, t_begin + 32 * sl);
      __builtin_amdgcn_sched_barrier(0);
    }
  } else {
    load_tile(0, t_begin);
    load_query();
  }
  query_operands();
  for (int tb = t_begin; tb < t_end; tb += 32 * KD) {
#pragma unroll
  for (int sl = 0; sl < KD; ++sl) {
    const int t0 = tb + 32 * sl;
    f32x16 sacc = f32x16{};
    float s[16];
    if constexpr (PRE) {
      // this lane's scores: head l32, tokens t0 + 8*(v/4) + 4*half + v%4
      const float* prow = pre + (int64_t)b * capacity * kHeadBlk + l32;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int t = t0 + 8 * (v >> 2) + 4 * half + (v & 3);
        s[v] = prow[(int64_t)min(t, t_end - 1) * kHeadBlk];
      }
      asm volatile("" ::: "memory");    // the previous tile's transposing reads stay before these stores
      if constexpr (F16C) {
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
          *reinterpret_cast<f16x8*>(cst + trow(ks) * CST + tcol(ks)) = raw[sl][ks];
      } else {
        scl[l32] = scr[sl];
#pragma unroll
        for (int i = 0; i < NLD; ++i) {
          f16x8 c0, c1;
          if constexpr (I4C) {
            c0 = cvt_i4x8(raw[sl][i].x);
            c1 = cvt_i4x8(raw[sl][i].y);
          } else {
            c0 = cvt_i8x8(raw[sl][i].x, raw[sl][i].y);
            c1 = cvt_i8x8(raw[sl][i].z, raw[sl][i].w);
          }
          *reinterpret_cast<f16x8*>(cst + trow(i) * CST + tcol(i)) = c0;
          *reinterpret_cast<f16x8*>(cst + trow(i) * CST + tcol(i) + 8) = c1;
        }
      }
      if (KD > 1 || t0 + 32 < t_end) load_tile(sl, t0 + 32 * KD);
      asm volatile("" ::: "memory");
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int t = t0 + 8 * (v >> 2) + 4 * half + (v & 3);
        if (t >= t_end) s[v] = -INFINITY;
      }
      read_scales();
    } else {
    if constexpr (kStageFirst) {
    // The tile (as exact fp16) goes to this wave's LDS copy first, so that
    // its registers take the next tile's loads before any product runs; the
    // score product reads its A operand back from the copy, one fragment per
    // MFMA.
    if constexpr (F16C) {
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
        *reinterpret_cast<f16x8*>(cst + trow(ks) * CST + tcol(ks)) = raw[sl][ks];
    } else {
      scl[l32] = scr[sl];
#pragma unroll
      for (int i = 0; i < NLD; ++i) {
        f16x8 c0, c1;
        if constexpr (I4C) {
          c0 = cvt_i4x8(raw[sl][i].x);
          c1 = cvt_i4x8(raw[sl][i].y);
        } else {
          c0 = cvt_i8x8(raw[sl][i].x, raw[sl][i].y);
          c1 = cvt_i8x8(raw[sl][i].z, raw[sl][i].w);
        }
        *reinterpret_cast<f16x8*>(cst + trow(i) * CST + tcol(i)) = c0;
        *reinterpret_cast<f16x8*>(cst + trow(i) * CST + tcol(i) + 8) = c1;
      }
    }
    if (KD > 1 || t0 + 32 < t_end) load_tile(sl, t0 + 32 * KD);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const f16x8 cf = *reinterpret_cast<const f16x8*>(cst + l32 * CST + kcol(ks, half));
      sacc = __builtin_amdgcn_mfma_f32_32x32x16_f16(cf, qf[ks], sacc, 0, 0, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);        // two fragment reads ahead
#pragma unroll
    for (int ks = 0; ks < KS - 2; ++ks) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);      // one MFMA
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);      // the next fragment read
    }
    __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
    __builtin_amdgcn_sched_barrier(0);
    } else {
    f16x8 cf[KS];
    if constexpr (F16C) {
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) cf[ks] = raw[sl][ks];
    } else {
      scl[l32] = scr[sl];
#pragma unroll
      for (int i = 0; i < NLD; ++i) {
        if constexpr (I4C) {
          cf[2 * i] = cvt_i4x8(raw[sl][i].x);
          cf[2 * i + 1] = cvt_i4x8(raw[sl][i].y);
        } else {
          cf[2 * i] = cvt_i8x8(raw[sl][i].x, raw[sl][i].y);
          cf[2 * i + 1] = cvt_i8x8(raw[sl][i].z, raw[sl][i].w);
        }
      }
    }
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      sacc = __builtin_amdgcn_mfma_f32_32x32x16_f16(cf[ks], qf[ks], sacc, 0, 0, 0);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      *reinterpret_cast<f16x8*>(cst + l32 * CST + kcol(ks, half)) = cf[ks];
    // The next tile streams in while this one is reduced, normalized and
    // multiplied into the output.
    if (KD > 1 || t0 + 32 < t_end) load_tile(sl, t0 + 32 * KD);
    }
#pragma unroll
    for (int vb = 0; vb < 4; ++vb)
      spart4[(w * 4 + vb) * 64 + lane] = f32x4{sacc[4 * vb], sacc[4 * vb + 1], sacc[4 * vb + 2], sacc[4 * vb + 3]};
    __syncthreads();
    if (tid < 256) {
      f32x4 acc = spart4[tid];
#pragma unroll
      for (int w2 = 1; w2 < NW; ++w2) acc += spart4[w2 * 256 + tid];
      ssum4[tid] = acc;
    }
    __syncthreads();
    // Lane l holds head l32 and tokens t0 + 8*(v/4) + 4*half + v%4.
    read_scales();
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int t = t0 + 8 * (v >> 2) + 4 * half + (v & 3);
      float x = ssum4[(v >> 2) * 64 + lane][v & 3];
      if constexpr (!F16C) x *= sc_cur[v];
      s[v] = (t < t_end) ? x : -INFINITY;
    }
    }
    float mx = s[0];
#pragma unroll
    for (int v = 1; v < 16; ++v) mx = fmaxf(mx, s[v]);
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    const float m_new = fmaxf(m_run, mx);
    float alpha = 1.f, ps = 0.f;
    float p[16];
    if (m_new == -INFINITY) {
#pragma unroll
      for (int v = 0; v < 16; ++v) p[v] = 0.f;
    } else {
      alpha = __builtin_amdgcn_exp2f(m_run - m_new);
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        p[v] = __builtin_amdgcn_exp2f(s[v] - m_new);
        ps += p[v];
      }
    }
    ps += __shfl_xor(ps, 32, 64);
    l_run = l_run * alpha + ps;
    m_run = m_new;
    // Once the running maxima settle, alpha is 1 for every head of the wave.
    if (__any(alpha != 1.f)) {
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)
#pragma unroll
        for (int v = 0; v < 16; ++v) o[rb][v] *= alpha;
    }
    // P^T as the B operand: k-slot (half, e) of MFMA mf is token 16*mf + 8*(e/4) + 4*half + e%4,
    // exactly the tokens this lane already holds in p[8*mf + e].
    f16x8 pf[2];
#pragma unroll
    for (int mf = 0; mf < 2; ++mf)
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        float pv = p[8 * mf + e];
        // token 16*mf + 8*(e/4) + 4*half + e%4 is score slot v = 8*mf + e
        if constexpr (!F16C) pv *= sc_cur[8 * mf + e];
        pf[mf][e] = (_Float16)pv;
      }
    // A operand of the output MFMA: lane l needs column rb*32 + l32 of the
    // staged tile at tokens 16*mf + 8*(e/4) + 4*half + e%4.  The LDS transpose
    // read returns, to lane i of each 16-lane group, element i%4 of the 4-half
    // chunk addressed by lane 4*e + i/4 of that group; so lane s of group
    // (half, q) addresses token 4*half + s/4 (+8 for the second read), columns
    // rb*32 + 16*q + 4*(s%4) .. +3, and receives its 4 tokens of one column.
    const int s16 = lane & 15, q16 = (lane >> 4) & 1;
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
      for (int mf = 0; mf < 2; ++mf) {
        const int tok = 16 * mf + 4 * half + (s16 >> 2);
        const int col = rb * 32 + 16 * q16 + 4 * (s16 & 3);
        typedef short s16x4 __attribute__((ext_vector_type(4)));
        typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
        const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (lds_s16x4*)(cst + tok * CST + col));
        const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (lds_s16x4*)(cst + (tok + 8) * CST + col));
        const f16x4 flo = __builtin_bit_cast(f16x4, lo), fhi = __builtin_bit_cast(f16x4, hi);
        const f16x8 a = {flo[0], flo[1], flo[2], flo[3], fhi[0], fhi[1], fhi[2], fhi[3]};
        o[rb] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, pf[mf], o[rb], 0, 0, 0);
      }
  }
  }

  const int64_t part = (int64_t)vb * n_chunks + ch;
  if (w == 0 && lane < 32) {
    ml_part[part * 64 + l32] = m_run;
    ml_part[part * 64 + 32 + l32] = l_run;
  }
  // O^T / l as fp16 (a weighted mean of latent rows, so it stays in range),
  // stored non-temporally (the merge reads it once, in another kernel),
  // stored in accumulator order [x/4][head][4]: lane (head l32, half) holds
  // latent columns slice0 + 32*rb + 8*vq + 4*half .. +3 in o[rb][4*vq ..],
  // so each store instruction writes 512 contiguous bytes.
  const float inv_l = l_run > 0.f ? 1.f / l_run : 0.f;
  _Float16* op = o_part + part * (int64_t)r * kHeadBlk;
#pragma unroll
  for (int rb = 0; rb < RB; ++rb)
#pragma unroll
    for (int vq = 0; vq < 4; ++vq) {
      const int x4 = (slice0 + 32 * rb + 8 * vq + 4 * half) >> 2;
      const f16x4 v4 = {(_Float16)(o[rb][4 * vq] * inv_l), (_Float16)(o[rb][4 * vq + 1] * inv_l),
                        (_Float16)(o[rb][4 * vq + 2] * inv_l), (_Float16)(o[rb][4 * vq + 3] * inv_l)};
      __builtin_nontemporal_store(v4, reinterpret_cast<f16x4*>(op + ((int64_t)x4 * kHeadBlk + l32) * 4));
    }
}

// ---------------------------------------------------------------------------
// Latent attention for wide layers: 16 query heads per workgroup (grid row =
// (sequence-query row, head block)), 16-token tiles, the latent columns split
// over 8 waves in units of 128.  Used where a 32-head block's output state
// (32 x r fp32) would not fit one CU's registers (r > 1536) or a sequence has
// more than 32 query heads.  Per tile:
//   S^T (16 tokens x 16 heads) = C_tile[:, slice] q~[:, slice]^T  (16x16x32 fp16 MFMA)
//   partial S^T of all waves summed through LDS in wave order
//   online softmax per head in fp32 (lane l: head l % 16, tokens 4(l/16) + v)
//   O^T[slice] (r x 16 heads) += C_tile[:, slice]^T P^T           (16x16x16 fp16 MFMA)
// The C tile reaches the first product straight from HBM (one 16-byte load
// per lane serves 1, 2 or 4 contraction steps for fp16, int8, int4 rows) and
// the second through a wave-private LDS copy read with transposing loads.
//
// Each wave keeps the next D tiles of its slice in flight in a ring of
// registers (D = 2, 3, 4 for fp16, int8, int4 rows: a 16-token tile of a
// narrow integer slice is only 0.5-1 KB per wave, so one tile in flight leaves
// every tile waiting a full memory round trip).  The loads are unconditional
// (rows past the chunk end re-read its last row and are masked), so the
// compiler can count them and wait only for the tile it is about to use; the
// unit count of a wave is a template parameter, so no product or fragment read
// sits behind a per-wave branch.
// ---------------------------------------------------------------------------
constexpr int kH16Waves = 8;

// Tokens per tile: 32 (two 16-token blocks per barrier pair) while a
// workgroup's fp16 staging of them fits LDS (two 128-column units per wave),
// else 16.
template <int UMAX>
struct H16Blocks {
  static constexpr int value = UMAX <= 2 ? 2 : 1;
};

// Ring depth: two tiles where the registers allow, one for fp16 rows, int8
// rows in 32-token tiles and three units per wave (whose accumulators take 96
// registers).  (Deeper rings measured slower: the tile body is unrolled once
// per slot.)
template <int UMAX, int U, int FMT>
struct H16Depth {
  static constexpr int value =
      (FMT == QSVD_CACHE_F16 || U >= 3 || (FMT == QSVD_CACHE_I8 && H16Blocks<UMAX>::value == 2)) ? 1 : 2;
};

template <int UMAX>
constexpr size_t h16_lds_bytes() {
  constexpr int NB = H16Blocks<UMAX>::value;
  return (size_t)kH16Waves * 16 * NB * (128 * UMAX + 24) * 2 + (size_t)(kH16Waves + 1) * NB * 64 * 16;
}

// One wave's pass over the chunk [t_begin, t_end) for a wave owning U units
// of 128 latent columns starting at slice0 (U may be 0: the wave then only
// takes part in the exchange and the softmax).  Tiles of T = 16 NB tokens,
// token block bb of a tile being tokens t0 + 16 bb .. +15.
template <int UMAX, int U, int FMT>
__device__ __forceinline__ void h16_wave(const _Float16* __restrict__ qrow, const uint8_t* __restrict__ cdata,
                                         const float* __restrict__ cscale, int64_t seq_row0, int r, int L,
                                         int t_begin, int t_end, int slice0, _Float16* cst, f32x4* spart,
                                         f32x4* ssum, int w, int lane, _Float16* __restrict__ op,
                                         float* __restrict__ mlp) {
  constexpr int NW = kH16Waves, NB = H16Blocks<UMAX>::value, T = 16 * NB;
  constexpr int D = H16Depth<UMAX, U, FMT>::value;
  constexpr bool F16C = FMT == QSVD_CACHE_F16, I4C = FMT == QSVD_CACHE_I4;
  constexpr int KS = 4 * U;                              // 32-wide contraction steps of the score product
  constexpr int RB = 8 * U;                              // 16-row blocks of the output product
  constexpr int NLD = F16C ? KS : (I4C ? U : KS / 2);    // 16-byte loads per token block
  constexpr int NLDA = NLD > 0 ? NLD : 1, KSA = KS > 0 ? KS : 1, RBA = RB > 0 ? RB : 1;
  // staged row stride in halves: 12 (mod 64) dwords, so the 16-byte row
  // writes of 16 consecutive rows and the transposing reads (4 rows x 8
  // dwords) fall on distinct banks of the 64
  constexpr int CST = 128 * UMAX + 24;
  const int l16 = lane & 15, g = lane >> 4;
  // contraction slots of the score product: in step ks, lane group g feeds
  // latent columns slice0 + kcol(ks, g) .. +7 of token t0 + 16 bb + l16
  auto kcol = [](int ks, int gg) {
    return F16C ? 32 * ks + 8 * gg : (I4C ? 128 * (ks >> 2) + 32 * gg + 8 * (ks & 3) : 64 * (ks >> 1) + 16 * gg + 8 * (ks & 1));
  };
  // The query slice (16 heads x 128 U columns) is read row-major, whole
  // cache lines per load instruction, and turned into the score product's
  // operand layout through the wave's LDS copy once the first tiles' loads
  // are out.
  constexpr int CPQ = 16 * U;      // 16-byte chunks per head row of the slice
  f16x8 qf[KSA];
  {
    const _Float16* qb = qrow - (int64_t)l16 * r;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const int c = 64 * ks + lane;
      qf[ks] = *reinterpret_cast<const f16x8*>(qb + (int64_t)(c / CPQ) * r + 8 * (c % CPQ));
    }
  }
  f32x4 o[RBA];
#pragma unroll
  for (int rb = 0; rb < RBA; ++rb) o[rb] = f32x4{};
  float m_run = -INFINITY, l_run = 0.f;

  i32x4 raw[D][NB][NLDA];
  float scr[D][NB];      // integer rows: the scale of token t0 + 16 bb + l16
  // tile starting at t0 into ring slot d (every load unconditional)
  auto load = [&](int d, int t0) {
#pragma unroll
    for (int bb = 0; bb < NB; ++bb) {
      const int t = t0 + 16 * bb + l16;
      if constexpr (!F16C) scr[d][bb] = cscale[seq_row0 + min(t, L - 1)];
      const int64_t off = (seq_row0 + min(t, t_end - 1)) * r + slice0;    // element index of the row slice
#pragma unroll
      for (int i = 0; i < NLD; ++i) {
        if constexpr (F16C)
          raw[d][bb][i] = *reinterpret_cast<const i32x4*>(reinterpret_cast<const _Float16*>(cdata) + off + kcol(i, g));
        else if constexpr (I4C)
          raw[d][bb][i] = *reinterpret_cast<const i32x4*>(cdata + (off + 128 * i + 32 * g) / 2);
        else
          raw[d][bb][i] = *reinterpret_cast<const i32x4*>(cdata + off + 64 * i + 16 * g);
      }
    }
  };
  typedef short s16x4 __attribute__((ext_vector_type(4)));
  typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

#pragma unroll
  for (int d = 0; d < D; ++d) load(d, t_begin + T * d);
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    const int c = 64 * ks + lane;
    *reinterpret_cast<f16x8*>(cst + (c / CPQ) * CST + 8 * (c % CPQ)) = qf[ks];
  }
  asm volatile("" ::: "memory");
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) qf[ks] = *reinterpret_cast<const f16x8*>(cst + l16 * CST + kcol(ks, g));
  asm volatile("" ::: "memory");
  for (int base = t_begin; base < t_end; base += T * D) {
#pragma unroll
    for (int d = 0; d < D; ++d) {
      const int t0 = base + T * d;
      // scales of the tokens t0 + 16 bb + 4g + v this lane's scores belong to
      float sc_cur[NB][4];
#pragma unroll
      for (int bb = 0; bb < NB; ++bb)
#pragma unroll
        for (int v = 0; v < 4; ++v) sc_cur[bb][v] = F16C ? 1.f : __shfl(scr[d][bb], 4 * g + v, 64);
      f32x4 sacc[NB];
#pragma unroll
      for (int bb = 0; bb < NB; ++bb) {
        sacc[bb] = f32x4{};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          f16x8 cf;
          if constexpr (F16C) {
            cf = __builtin_bit_cast(f16x8, raw[d][bb][ks]);
          } else if constexpr (I4C) {
            const i32x4 q4 = raw[d][bb][ks >> 2];
            cf = cvt_i4x8((uint32_t)q4[ks & 3]);
          } else {
            const i32x4 q8 = raw[d][bb][ks >> 1];
            cf = (ks & 1) ? cvt_i8x8((uint32_t)q8[2], (uint32_t)q8[3]) : cvt_i8x8((uint32_t)q8[0], (uint32_t)q8[1]);
          }
          sacc[bb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(cf, qf[ks], sacc[bb], 0, 0, 0);
          *reinterpret_cast<f16x8*>(cst + (16 * bb + l16) * CST + kcol(ks, g)) = cf;
        }
      }
      // the slot is refilled D tiles ahead while this tile is reduced and multiplied
      load(d, t0 + T * D);
#pragma unroll
      for (int bb = 0; bb < NB; ++bb) spart[(bb * NW + w) * 64 + lane] = sacc[bb];
      __syncthreads();
      // every wave adds, in wave order, the partials of 8 of the 64 lanes of each token block
      if (lane < 8 * NB) {
        const int bb = lane >> 3, ln = 8 * w + (lane & 7);
        f32x4 parts[NW];
#pragma unroll
        for (int w2 = 0; w2 < NW; ++w2) parts[w2] = spart[(bb * NW + w2) * 64 + ln];
        f32x4 acc = parts[0];
#pragma unroll
        for (int w2 = 1; w2 < NW; ++w2) acc += parts[w2];
        ssum[bb * 64 + ln] = acc;
      }
      __syncthreads();
      // lane holds head l16 at tokens t0 + 16 bb + 4g + v
      float s[NB][4];
      float mx = -INFINITY;
#pragma unroll
      for (int bb = 0; bb < NB; ++bb) {
        const f32x4 sv = ssum[bb * 64 + lane];
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          float x = sv[v];
          if constexpr (!F16C) x *= sc_cur[bb][v];
          s[bb][v] = (t0 + 16 * bb + 4 * g + v < t_end) ? x : -INFINITY;
          mx = fmaxf(mx, s[bb][v]);
        }
      }
      const float m_new = fmaxf(m_run, rows4_max(mx));
      float alpha = 1.f, ps = 0.f;
      float p[NB][4];
      if (m_new == -INFINITY) {
#pragma unroll
        for (int bb = 0; bb < NB; ++bb)
#pragma unroll
          for (int v = 0; v < 4; ++v) p[bb][v] = 0.f;
      } else {
        alpha = __builtin_amdgcn_exp2f(m_run - m_new);
#pragma unroll
        for (int bb = 0; bb < NB; ++bb)
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            p[bb][v] = __builtin_amdgcn_exp2f(s[bb][v] - m_new);
            ps += p[bb][v];
          }
      }
      l_run = l_run * alpha + rows4_sum(ps);
      m_run = m_new;
      if (__any(alpha != 1.f)) {
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) o[rb] *= alpha;
      }
      // P^T as the B operand, scaled per token: k-slot e of lane group g is
      // token 16 (e / 4) + 4g + e % 4 (one 16-token block: token 4g + e).
      // A operand: lane (l16, g) needs latent column 16rb + l16 at the same
      // tokens.  In a transposing read, lane a of group g addresses token
      // 4g + a/4 (of the block), columns 16rb + 4(a%4) .. +3, and lane i
      // receives element i%4 of the chunks of lanes i/4, 4 + i/4, 8 + i/4,
      // 12 + i/4: column 16rb + i at tokens 4g .. 4g+3 of the block.
      if constexpr (NB == 1) {
        f16x4 pf;
#pragma unroll
        for (int e = 0; e < 4; ++e) pf[e] = (_Float16)(F16C ? p[0][e] : p[0][e] * sc_cur[0][e]);
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) {
          const s16x4 x = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
              (lds_s16x4*)(cst + (4 * g + (l16 >> 2)) * CST + 16 * rb + 4 * (l16 & 3)));
          o[rb] = __builtin_amdgcn_mfma_f32_16x16x16f16(__builtin_bit_cast(f16x4, x), pf, o[rb], 0, 0, 0);
        }
      } else {
        f16x8 pf;
#pragma unroll
        for (int e = 0; e < 8; ++e) pf[e] = (_Float16)(F16C ? p[e >> 2][e & 3] : p[e >> 2][e & 3] * sc_cur[e >> 2][e & 3]);
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) {
          const _Float16* a0 = cst + (4 * g + (l16 >> 2)) * CST + 16 * rb + 4 * (l16 & 3);
          const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)a0);
          const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(a0 + 16 * CST));
          const f16x4 flo = __builtin_bit_cast(f16x4, lo), fhi = __builtin_bit_cast(f16x4, hi);
          const f16x8 a = {flo[0], flo[1], flo[2], flo[3], fhi[0], fhi[1], fhi[2], fhi[3]};
          o[rb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, pf, o[rb], 0, 0, 0);
        }
      }
    }
  }

  if (w == 0 && lane < 16) {
    mlp[l16] = m_run;
    mlp[16 + l16] = l_run;
  }
  // O^T / l as fp16 in [x/4][16 heads][4] order: lane (head l16, g) holds
  // latent columns slice0 + 16rb + 4g .. +3, so each store writes 512
  // contiguous bytes; non-temporal, as in the 32-head kernel.
  const float inv_l = l_run > 0.f ? 1.f / l_run : 0.f;
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    const int x4 = (slice0 + 16 * rb + 4 * g) >> 2;
    const f16x4 v4 = {(_Float16)(o[rb][0] * inv_l), (_Float16)(o[rb][1] * inv_l), (_Float16)(o[rb][2] * inv_l),
                      (_Float16)(o[rb][3] * inv_l)};
    __builtin_nontemporal_store(v4, reinterpret_cast<f16x4*>(op + ((int64_t)x4 * 16 + l16) * 4));
  }
}

template <int UMAX, int FMT>
__global__ void __launch_bounds__(kH16Waves * 64)
latent_attn_h16_kernel(const _Float16* __restrict__ qt, const uint8_t* __restrict__ cdata,
                       const float* __restrict__ cscale, const int32_t* __restrict__ seq_len,
                       int32_t capacity, int32_t r, int32_t hp, int32_t chunk, int32_t n_chunks,
                       int32_t q_len, _Float16* __restrict__ o_part, float* __restrict__ ml_part) {
  constexpr int NW = kH16Waves, NB = H16Blocks<UMAX>::value;
  constexpr int CST = 128 * UMAX + 24;
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int wu = __builtin_amdgcn_readfirstlane(w);     // wave-uniform copy: scalar branches below
  _Float16* cst = reinterpret_cast<_Float16*>(smem) + w * 16 * NB * CST;
  f32x4* spart = reinterpret_cast<f32x4*>(smem + (size_t)NW * 16 * NB * CST * 2);
  f32x4* ssum = spart + NB * NW * 64;

  const int n_hb = hp >> 4;
  // Workgroup -> (sequence-query row vb, head block hb, chunk ch).  The n_hb
  // head blocks of one (vb, ch) read the same cache rows, so they get ids
  // that one XCD receives together (the chip dispatches the i-th workgroup,
  // x fastest, to XCD i % 8) and share its L2 instead of each XCD fetching
  // the rows again.  A bijection on the grid.
  const int n_launch = gridDim.x, pairs = gridDim.x * gridDim.y / n_hb;
  const int lin = blockIdx.y * gridDim.x + blockIdx.x;
  int pair, hb;
  if (pairs % 8 == 0) {
    const int j = lin >> 3;
    pair = (lin & 7) * (pairs >> 3) + j / n_hb;
    hb = j % n_hb;
  } else {
    pair = lin / n_hb;
    hb = lin % n_hb;
  }
  const int vb = pair / n_launch, ch = pair % n_launch, row = vb * n_hb + hb;
  const int b = vb / q_len, qi = vb - b * q_len;
  const int L = min(seq_len[b], capacity) - (q_len - 1 - qi);
  const int t_begin = ch * chunk;
  if (t_begin >= L) return;
  const int t_end = min(L, t_begin + chunk);
  // this wave's latent units [u0, u0 + nu) of 128 columns: nu is UMAX or UMAX - 1
  const int m_units = r >> 7;
  const int u0 = (wu * m_units) / NW, nu = ((wu + 1) * m_units) / NW - u0;
  const int slice0 = 128 * u0;
  const int l16 = lane & 15;
  const _Float16* qrow = qt + ((int64_t)vb * hp + hb * 16 + l16) * r + slice0;
  const int64_t part = (int64_t)row * n_chunks + ch;
  _Float16* op = o_part + part * (int64_t)r * 16;
  float* mlp = ml_part + part * 32;
  const int64_t seq_row0 = (int64_t)b * capacity;
  if (nu == UMAX)
    h16_wave<UMAX, UMAX, FMT>(qrow, cdata, cscale, seq_row0, r, L, t_begin, t_end, slice0, cst, spart, ssum, w, lane,
                              op, mlp);
  else
    h16_wave<UMAX, UMAX - 1, FMT>(qrow, cdata, cscale, seq_row0, r, L, t_begin, t_end, slice0, cst, spart, ssum, w,
                                  lane, op, mlp);
}

// ---------------------------------------------------------------------------
// Merge the chunk partials of the latent form.  The attention grid row
// (sequence-query row vb, head block hb) of HB heads holds, per chunk c,
// m_c, l_c per head and the normalized O_c / l_c as fp16 in the [x/4][HB][4]
// order the attention kernels write.  With m = max m_c and
// w_c = 2^(m_c - m) l_c / sum, the result O[vb][h][x] = sum_c w_c (O_c / l_c)[h][x]
// is written head-major [vb][hp][r] at heads hb*HB ...
// A workgroup takes 2048 consecutive partial elements (2048 / (4 HB) latent
// quads x HB heads x 4); its threads first compute all the per-(chunk, head)
// weights into LDS (256 / HB lanes per head, chunks strided over them), then
// each thread streams 8 elements (two heads x 4 columns) of every chunk.
// ---------------------------------------------------------------------------
constexpr int kMergeElems = 2048;
constexpr int kMergeBatch = 16;   // chunk partials in flight per thread (one round trip for <= 16 chunks)

template <int HB>
__global__ void __launch_bounds__(256)
merge_latent_kernel(const _Float16* __restrict__ o_part, const float* __restrict__ ml_part,
                    const int32_t* __restrict__ seq_len, int32_t capacity, int32_t chunk, int32_t n_chunks,
                    int32_t n_launched, int32_t q_len, int32_t r, int32_t hp, _Float16* __restrict__ o_lat) {
  constexpr int LPH = 256 / HB;      // lanes per head in the weights phase
  __shared__ float wgt[kMaxChunks * HB];
  const int n_hb = hp / HB;
  const int row = blockIdx.y, vb = row / n_hb, hb = row - vb * n_hb, tid = threadIdx.x;
  const int L = min(seq_len[vb / q_len], capacity) - (q_len - 1 - vb % q_len);
  const int nv = L > 0 ? min(min((L + chunk - 1) / chunk, n_launched), kMaxChunks) : 0;
  const int64_t pb = (int64_t)row * n_chunks;
  // element e8 (8 halves): latent quad x4 = e8 / (HB / 2), heads 2*(e8 % (HB / 2)) and +1;
  // the first batch of partial loads goes out before the weights are known
  const int64_t e0 = (int64_t)blockIdx.x * kMergeElems + 8 * tid;
  const bool eok = e0 < (int64_t)r * HB;
  const _Float16* src = o_part + pb * (int64_t)r * HB + (eok ? e0 : 0);
  f16x8 v[kMergeBatch];
#pragma unroll
  for (int k = 0; k < kMergeBatch; ++k)
    v[k] = (eok && k < nv) ? *reinterpret_cast<const f16x8*>(src + (int64_t)k * r * HB) : f16x8{};
  {
    const int h = tid / LPH, sub = tid % LPH;
    float m = -INFINITY;
    for (int c = sub; c < nv; c += LPH) m = fmaxf(m, ml_part[(pb + c) * 2 * HB + h]);
#pragma unroll
    for (int o = 1; o < LPH; o <<= 1) m = fmaxf(m, __shfl_xor(m, o, 64));
    float tot = 0.f;
    for (int c = sub; c < nv; c += LPH) {
      const float wc = exp2f(ml_part[(pb + c) * 2 * HB + h] - m) * ml_part[(pb + c) * 2 * HB + HB + h];
      wgt[c * HB + h] = wc;
      tot += wc;
    }
#pragma unroll
    for (int o = 1; o < LPH; o <<= 1) tot += __shfl_xor(tot, o, 64);
    const float inv = tot > 0.f ? 1.f / tot : 0.f;
    for (int c = sub; c < nv; c += LPH) wgt[c * HB + h] *= inv;
  }
  __syncthreads();
  const int x4 = (int)(e0 / (4 * HB)), h0 = (int)((e0 / 4) % HB);
  float acc[8];
#pragma unroll
  for (int k = 0; k < 8; ++k) acc[k] = 0.f;
  for (int c0 = 0; eok && c0 < nv; c0 += kMergeBatch) {
    if (c0 > 0) {
#pragma unroll
      for (int k = 0; k < kMergeBatch; ++k)
        v[k] = (c0 + k < nv) ? *reinterpret_cast<const f16x8*>(src + (int64_t)(c0 + k) * r * HB) : f16x8{};
    }
#pragma unroll
    for (int k = 0; k < kMergeBatch; ++k) {
      if (c0 + k >= nv) continue;
      const float w0 = wgt[(c0 + k) * HB + h0], w1 = wgt[(c0 + k) * HB + h0 + 1];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        acc[q] = fmaf(w0, (float)v[k][q], acc[q]);
        acc[4 + q] = fmaf(w1, (float)v[k][4 + q], acc[4 + q]);
      }
    }
  }
  // The workgroup's kMergeElems / HB latent columns of its HB heads go
  // through LDS, so that each head row leaves as 16-byte runs.
  constexpr int COLS = kMergeElems / HB, OLD = COLS + 8;
  __shared__ __attribute__((aligned(16))) _Float16 ot[HB * OLD];
  const int xl = 4 * x4 - blockIdx.x * COLS;
#pragma unroll
  for (int hh = 0; hh < 2; ++hh) {
    const f16x4 o4 = {(_Float16)acc[4 * hh], (_Float16)acc[4 * hh + 1], (_Float16)acc[4 * hh + 2],
                      (_Float16)acc[4 * hh + 3]};
    *reinterpret_cast<f16x4*>(ot + (h0 + hh) * OLD + xl) = o4;
  }
  __syncthreads();
  static_assert(HB * COLS / 8 == 256, "one 16-byte run per thread");
  const int hr = tid / (COLS / 8), c8 = 8 * (tid % (COLS / 8));
  const int col = blockIdx.x * COLS + c8;
  if (col < r)
    *reinterpret_cast<f16x8*>(o_lat + ((int64_t)vb * hp + hb * HB + hr) * r + col) =
        *reinterpret_cast<const f16x8*>(ot + hr * OLD + c8);
}

// ---------------------------------------------------------------------------
// Merge the chunk partials of a sequence.  Chunk c holds m_c, l_c and the
// normalized O_c / l_c of a block of 32 heads as fp16 [x][32 heads]; with
// m = max m_c and w_c = 2^(m_c - m) l_c, the result is
// sum_c w_c (O_c / l_c) / sum_c w_c.  One workgroup per (64 rows x, sequence,
// head block): the per-head weights are computed once into LDS; each thread
// then streams 8 heads of one row x with 16-byte loads.  Output is the final
// fp16 [b][Hq*width], head-major.
// ---------------------------------------------------------------------------
__global__ void __launch_bounds__(256)
combine_kernel(const _Float16* __restrict__ o_part, const float* __restrict__ ml_part,
               const int32_t* __restrict__ seq_len, int32_t chunk, int32_t n_chunks, int32_t n_launched,
               int32_t width, int32_t Hq, int32_t n_hb, _Float16* __restrict__ out) {
  __shared__ float wgt[kMaxChunks * 32];
  __shared__ float tile[64][33];
  const int b = blockIdx.y / n_hb, hb = blockIdx.y - b * n_hb, x0 = blockIdx.x * 64, tid = threadIdx.x;
  const int L = seq_len[b];
  const int nv = L > 0 ? min(min((L + chunk - 1) / chunk, n_launched), kMaxChunks) : 0;
  const int64_t pb = ((int64_t)b * n_hb + hb) * n_chunks;
  if (tid < 32) {
    float m = -INFINITY;
    for (int c = 0; c < nv; ++c) m = fmaxf(m, ml_part[(pb + c) * 64 + tid]);
    float tot = 0.f;
    for (int c = 0; c < nv; ++c) {
      const float wc = exp2f(ml_part[(pb + c) * 64 + tid] - m) * ml_part[(pb + c) * 64 + 32 + tid];
      wgt[c * 32 + tid] = wc;
      tot += wc;
    }
    const float inv = tot > 0.f ? 1.f / tot : 0.f;
    for (int c = 0; c < nv; ++c) wgt[c * 32 + tid] *= inv;
  }
  __syncthreads();
  // thread -> row x0 + tid/4, heads 8*(tid%4) .. +8; chunk loads in batches of 8
  const int h0 = 8 * (tid & 3);
  const int xl = tid >> 2;
  const int x = x0 + xl;
  float acc[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) acc[e] = 0.f;
  if (x < width) {
    const _Float16* src = o_part + (pb * width + x) * kHeadBlk + h0;
    for (int c0 = 0; c0 < nv; c0 += 8) {
      f16x8 v[8];
#pragma unroll
      for (int k = 0; k < 8; ++k)
        v[k] = (c0 + k < nv) ? *reinterpret_cast<const f16x8*>(src + (int64_t)(c0 + k) * width * kHeadBlk) : f16x8{};
#pragma unroll
      for (int k = 0; k < 8; ++k)
        if (c0 + k < nv)
#pragma unroll
          for (int e = 0; e < 8; ++e) acc[e] = fmaf(wgt[(c0 + k) * 32 + h0 + e], (float)v[k][e], acc[e]);
    }
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) tile[xl][h0 + e] = acc[e];
  __syncthreads();
  // write head-major: pass i covers heads 4 i .. 4 i + 3 of the block, 64 rows each
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int e = tid + 256 * i, h = e >> 6, xl = e & 63, x = x0 + xl;
    const int hg = hb * kHeadBlk + h;
    if (x < width && hg < Hq) out[((int64_t)b * Hq + hg) * width + x] = (_Float16)tile[xl][h];
  }
}

// ---------------------------------------------------------------------------
// o[b][h*dh + c] = sum_j O[b][h][j] W^u_v[j][n], n = Hq*dh + Hkv*dh + g(h)*dh + c,
// on the 16x16x32 fp16 matrix cores: rows are 16 sequences, columns 16 output
// channels, the contraction runs over the latent index j.  One workgroup per
// (head, 16 columns); its 8 waves split the contraction into equal runs of
// 32-wide steps, load all fragments of a run at once, and add their partial
// results through LDS in a fixed order.  Both fragments come straight from
// memory (j-contiguous).  Integer codes convert to fp16 exactly; the
// per-channel scale multiplies the final sum, a per-group scale the product of
// each step (a step never straddles a group).
// ---------------------------------------------------------------------------
constexpr int kVprojWaves = 8;
constexpr int kVprojBatch = 8;

__global__ void __launch_bounds__(64 * kVprojWaves)
vproj_kernel(const _Float16* __restrict__ o_lat, const uint8_t* __restrict__ bt, const float* __restrict__ sb,
             int32_t B, int32_t r, int32_t Hq, int32_t Hkv, int32_t dh, int32_t N, int32_t bits,
             int32_t group, int32_t hp, _Float16* __restrict__ out) {
  __shared__ f32x4 red[kVprojWaves][64];
  const int h = blockIdx.x, c0 = blockIdx.y * 16, tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int l16 = lane & 15, quad = lane >> 4;
  const int g = (h * Hkv) / Hq;
  const int32_t n = Hq * dh + Hkv * dh + g * dh + c0 + l16;
  const int steps = r / 32;
  const int s_begin = (w * steps) / kVprojWaves, s_end = ((w + 1) * steps) / kVprojWaves;
  const float cs = group ? 1.f : sb[n];      // per-channel scale, fetched with the first loads
  for (int b0 = 0; b0 < B; b0 += 16) {
    const int bA = b0 + l16;
    const _Float16* arow = o_lat + ((int64_t)min(bA, B - 1) * hp + h) * r + 8 * quad;
    f32x4 res = f32x4{};
    for (int st0 = s_begin; st0 < s_end; st0 += kVprojBatch) {
      f16x8 a[kVprojBatch];
      uint2 raw[kVprojBatch];
      float gsc[kVprojBatch];      // per-group scales, loaded with the codes
#pragma unroll
      for (int k = 0; k < kVprojBatch; ++k) {
        const int j = (st0 + k) * 32;
        if (st0 + k < s_end) {
          a[k] = *reinterpret_cast<const f16x8*>(arow + j);
          if (bits == 8) {
            raw[k] = *reinterpret_cast<const uint2*>(bt + (int64_t)n * r + j + 8 * quad);
          } else {
            raw[k].x = *reinterpret_cast<const uint32_t*>(bt + ((int64_t)n * r + j + 8 * quad) / 2);
            raw[k].y = 0u;
          }
          gsc[k] = group ? sb[(int64_t)(j / group) * N + n] : 1.f;
        }
      }
#pragma unroll
      for (int k = 0; k < kVprojBatch; ++k) {
        if (st0 + k >= s_end) continue;
        const f16x8 bw = bits == 8 ? cvt_i8x8(raw[k].x, raw[k].y) : cvt_i4x8(raw[k].x);
        const f16x8 av = bA < B ? a[k] : f16x8{};
        const f32x4 acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(av, bw, f32x4{}, 0, 0, 0);
        if (group) {
          const float sc = gsc[k];
#pragma unroll
          for (int v = 0; v < 4; ++v) res[v] = fmaf(acc[v], sc, res[v]);
        } else {
          res += acc;
        }
      }
    }
    __syncthreads();
    red[w][lane] = res;
    __syncthreads();
    if (w == 0) {
      f32x4 tot = red[0][lane];
#pragma unroll
      for (int w2 = 1; w2 < kVprojWaves; ++w2) tot += red[w2][lane];
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int bb = b0 + 4 * quad + v;
        if (bb < B) out[(int64_t)bb * Hq * dh + h * dh + c0 + l16] = (_Float16)(tot[v] * cs);
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Host side of the absorbed form.
// ---------------------------------------------------------------------------
struct AbsorbPlan {
  int hb;            // heads per attention workgroup: 32 (latent_attn_kernel) or 16 (the wide variant)
  int n_hb, hp;      // head blocks per row and padded heads per row (n_hb * hb)
  int rw, nw;        // 32-head kernel: latent columns per wave, waves
  int umax;          // 16-head kernel: 128-column units per wave (at most)
  int chunk, n_chunks, n0;
  size_t qt_bytes, opart_bytes, ml_bytes, olat_bytes;
};

static int target_chunks(int rows) {
  const int n0 = (256 + rows - 1) / rows;
  return n0 < 1 ? 1 : n0;
}

static bool pick_slice(int r, int* rw, int* nw) {
  static const int opts[][2] = {{192, 8}, {128, 8}, {64, 8}, {32, 4}};
  for (auto& o : opts)
    if (r == o[0] * o[1]) { *rw = o[0]; *nw = o[1]; return true; }
  return false;
}

// The 16-head kernel takes r a multiple of 128 up to 3 * 128 columns per wave.
static bool h16_rank_ok(int r) { return r % 128 == 0 && r / 128 <= 3 * kH16Waves; }

static AbsorbPlan plan_absorbed(const qsvd_layer& w, const qsvd_cache& c, int32_t q_len) {
  AbsorbPlan p{};
  if (w.n_q_heads <= kHeadBlk && pick_slice(w.r, &p.rw, &p.nw)) {
    p.hb = kHeadBlk;
    p.n_hb = 1;
  } else {
    p.hb = 16;
    p.n_hb = (w.n_q_heads + 15) / 16;
    const int m_units = w.r / 128;
    p.umax = (m_units + kH16Waves - 1) / kH16Waves;
  }
  p.hp = p.hb * p.n_hb;
  const int64_t rows = (int64_t)c.batch * q_len;      // one query row per (sequence, query)
  const int64_t grows = rows * p.n_hb;                // attention grid rows
  // 32-head blocks: about one round of workgroups over the 256 CUs; 16-head
  // blocks (one workgroup per CU): at most one round
  p.n0 = p.hb == kHeadBlk ? target_chunks((int)grows) : (int)(grows >= 256 ? 1 : 256 / grows);
  const int len = c.max_len > 0 ? c.max_len : 1;
  int ch = (len + p.n0 - 1) / p.n0;
  const int gran = p.hb == kHeadBlk ? 16 : 64;      // 16-head plans: whole tiles and ring rounds
  ch = ((ch + gran - 1) / gran) * gran;
  p.chunk = ch;
  p.n_chunks = (len + ch - 1) / ch;
  p.qt_bytes = (size_t)rows * p.hp * w.r * sizeof(_Float16);
  p.opart_bytes = (size_t)grows * p.n0 * w.r * p.hb * sizeof(_Float16);
  p.ml_bytes = (size_t)grows * p.n0 * 2 * p.hb * sizeof(float);
  p.olat_bytes = (size_t)rows * p.hp * w.r * sizeof(_Float16);
  return p;
}

static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

bool absorbed_supported(const qsvd_layer& w, const qsvd_cache& c) {
  int rw, nw;
  if (w.n_q_heads <= kHeadBlk && pick_slice(w.r, &rw, &nw)) return true;
  return w.n_q_heads <= kMaxAbsorbedHeads && h16_rank_ok(w.r);
}

int64_t absorbed_grid_rows(const qsvd_layer& w, const qsvd_cache& c, int32_t q_len) {
  const AbsorbPlan p = plan_absorbed(w, c, 1);
  return (int64_t)c.batch * q_len * p.n_hb;
}

size_t attn_absorbed_workspace(const qsvd_layer& w, const qsvd_cache& c, int32_t q_len) {
  const AbsorbPlan p = plan_absorbed(w, c, q_len);
  return align256(p.qt_bytes) + align256(p.opart_bytes) + align256(p.ml_bytes) + align256(p.olat_bytes);
}

template <int RW, int NW, int FMT, bool PRE = false>
static hipError_t launch_latent(const AbsorbPlan& p, const qsvd_cache& c, int32_t q_len, const _Float16* qt,
                                _Float16* opart, float* ml, hipStream_t s, const float* pre = nullptr) {
  const size_t lds = (size_t)NW * 32 * (RW + 40) * 2 + (PRE ? 0 : (size_t)(NW + 1) * 1024 * 4) +
                     (FMT == QSVD_CACHE_F16 ? 0 : (size_t)NW * 32 * 4);
  auto kern = latent_attn_kernel<RW, NW, FMT, PRE>;
  hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  KernelScope ks("latent_attn", s);
  QSVD_LAUNCH(ks, kern, dim3(p.n_chunks, c.batch * q_len), dim3(NW * 64), lds, s, qt,
                     (const uint8_t*)c.data, c.scale, c.seq_len, c.capacity, c.r, p.chunk,
                     p.n0, q_len, pre, opart, ml);
  return hipGetLastError();
}

template <int UMAX, int FMT>
static hipError_t launch_latent_h16(const AbsorbPlan& p, const qsvd_cache& c, int32_t q_len, const _Float16* qt,
                                    _Float16* opart, float* ml, hipStream_t s) {
  const size_t lds = h16_lds_bytes<UMAX>();
  auto kern = latent_attn_h16_kernel<UMAX, FMT>;
  hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  KernelScope ks("latent_attn_h16", s);
  QSVD_LAUNCH(ks, kern, dim3(p.n_chunks, c.batch * q_len * p.n_hb), dim3(kH16Waves * 64), lds, s, qt,
              (const uint8_t*)c.data, c.scale, c.seq_len, c.capacity, c.r, p.hp, p.chunk, p.n0, q_len, opart, ml);
  return hipGetLastError();
}

template <int FMT>
static hipError_t dispatch_latent(const AbsorbPlan& p, const qsvd_cache& c, int32_t q_len, const _Float16* qt,
                                  _Float16* opart, float* ml, hipStream_t s) {
  if (p.hb == 16) {
    if (p.umax == 1) return launch_latent_h16<1, FMT>(p, c, q_len, qt, opart, ml, s);
    if (p.umax == 2) return launch_latent_h16<2, FMT>(p, c, q_len, qt, opart, ml, s);
    return launch_latent_h16<3, FMT>(p, c, q_len, qt, opart, ml, s);
  }
  if (p.rw == 192) return launch_latent<192, 8, FMT>(p, c, q_len, qt, opart, ml, s);
  if (p.rw == 128) return launch_latent<128, 8, FMT>(p, c, q_len, qt, opart, ml, s);
  if (p.rw == 64) return launch_latent<64, 8, FMT>(p, c, q_len, qt, opart, ml, s);
  return launch_latent<32, 4, FMT>(p, c, q_len, qt, opart, ml, s);
}

// Value side only, over precomputed scores (32-head plans, q_len 1).
template <int FMT>
static hipError_t dispatch_latent_pre(const AbsorbPlan& p, const qsvd_cache& c, const float* pre, _Float16* opart,
                                      float* ml, hipStream_t s) {
  if (p.rw == 192) return launch_latent<192, 8, FMT, true>(p, c, 1, nullptr, opart, ml, s, pre);
  if (p.rw == 128) return launch_latent<128, 8, FMT, true>(p, c, 1, nullptr, opart, ml, s, pre);
  if (p.rw == 64) return launch_latent<64, 8, FMT, true>(p, c, 1, nullptr, opart, ml, s, pre);
  return launch_latent<32, 4, FMT, true>(p, c, 1, nullptr, opart, ml, s, pre);
}

static hipError_t merge_and_project(const AttnArgs& a, const AbsorbPlan& p, const _Float16* opart, const float* ml,
                                    _Float16* olat, hipStream_t s);

// The absorbed form's workspace: q~, the chunk partials (O, then m and l), O_lat.
struct AbsorbWs {
  _Float16* qt;
  _Float16* opart;
  float* ml;
  _Float16* olat;
};
static AbsorbWs carve_absorbed(const AbsorbPlan& p, void* ws) {
  uint8_t* base = (uint8_t*)ws;
  AbsorbWs o;
  o.qt = (_Float16*)base;
  base += align256(p.qt_bytes);
  o.opart = (_Float16*)base;
  base += align256(p.opart_bytes);
  o.ml = (float*)base;
  base += align256(p.ml_bytes);
  o.olat = (_Float16*)base;
  return o;
}

// Everything after q~: the latent attention over the chunks, the merge and W^u_v.
static hipError_t absorbed_from_qt(const AttnArgs& a, const AbsorbPlan& p, const AbsorbWs& b, hipStream_t s) {
  const qsvd_cache& c = *a.c;
  hipError_t e = c.fmt == QSVD_CACHE_F16 ? dispatch_latent<QSVD_CACHE_F16>(p, c, a.q_len, b.qt, b.opart, b.ml, s)
                 : c.fmt == QSVD_CACHE_I8 ? dispatch_latent<QSVD_CACHE_I8>(p, c, a.q_len, b.qt, b.opart, b.ml, s)
                                          : dispatch_latent<QSVD_CACHE_I4>(p, c, a.q_len, b.qt, b.opart, b.ml, s);
  if (e != hipSuccess) return e;
  return merge_and_project(a, p, b.opart, b.ml, b.olat, s);
}

hipError_t launch_attn_absorbed(const AttnArgs& a, void* ws, hipStream_t s) {
  const qsvd_layer& w = *a.w;
  const qsvd_cache& c = *a.c;
  const AbsorbPlan p = plan_absorbed(w, c, a.q_len);
  const int32_t rows = c.batch * a.q_len;     // (sequence, query) rows, sequence-major
  const AbsorbWs b = carve_absorbed(p, ws);
  const int N = (w.n_q_heads + 2 * w.n_kv_heads) * w.head_dim;
  {
    KernelScope ks("absorb_q", s);
    QSVD_LAUNCH(ks, absorb_kernel, dim3(p.hp, w.r / kAbsorbJ), dim3(64), 0, s, a.q,
                       (const uint8_t*)w.b_t, w.s_b, rows, w.r, w.n_q_heads, w.n_kv_heads,
                       w.head_dim, N, w.w_bits, w.w_group, a.sm_scale * kLog2e, p.hp, b.qt);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return absorbed_from_qt(a, p, b, s);
}

// Merge the chunk partials into O_lat, then o = O_lat W^u_v.
static hipError_t merge_and_project(const AttnArgs& a, const AbsorbPlan& p, const _Float16* opart, const float* ml,
                                    _Float16* olat, hipStream_t s) {
  const qsvd_layer& w = *a.w;
  const qsvd_cache& c = *a.c;
  const int32_t rows = c.batch * a.q_len;
  const int N = (w.n_q_heads + 2 * w.n_kv_heads) * w.head_dim;
  {
    KernelScope ks("merge_latent", s);
    const dim3 grid((w.r * p.hb + kMergeElems - 1) / kMergeElems, rows * p.n_hb);
    if (p.hb == 16)
      QSVD_LAUNCH(ks, merge_latent_kernel<16>, grid, dim3(256), 0, s, opart, ml, c.seq_len, c.capacity, p.chunk,
                  p.n0, p.n_chunks, a.q_len, w.r, p.hp, olat);
    else
      QSVD_LAUNCH(ks, merge_latent_kernel<kHeadBlk>, grid, dim3(256), 0, s, opart, ml, c.seq_len, c.capacity,
                  p.chunk, p.n0, p.n_chunks, a.q_len, w.r, p.hp, olat);
  }
  {
    KernelScope ks("vproj", s);
    QSVD_LAUNCH(ks, vproj_kernel, dim3(w.n_q_heads, w.head_dim / 16), dim3(64 * kVprojWaves), 0, s, olat,
                       (const uint8_t*)w.b_t, w.s_b, rows, w.r, w.n_q_heads, w.n_kv_heads, w.head_dim, N,
                       w.w_bits, w.w_group, p.hp, a.out);
  }
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Reconstruct form: K^, V^ = C W^u_{k,v} rebuilt for every cached token
// (Eq. 5), then plain attention over them.
//
// The rebuild is one matrix-core product over all cache rows: int8 caches on
// the int8 products (exact integer sums, (acc * s_t) * s_n); fp16 caches on the
// fp16 products, with the weight columns first turned into fp16 in the
// workspace (the exact codes, per-channel scales in the epilogue; for per-group
// scales code * s_g rounded once to fp16, since a scale that varies along the
// contraction cannot leave the product).
// ---------------------------------------------------------------------------
__global__ void __launch_bounds__(256)
recon_weights_kernel(const uint8_t* __restrict__ bt, const float* __restrict__ sb, int32_t r, int32_t N, int32_t nq,
                     int32_t nkv2, int32_t bits, int32_t group, _Float16* __restrict__ w16) {
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;   // one 8-element run of a column
  const int per_col = r / 8;
  if (e >= (int64_t)nkv2 * per_col) return;
  const int np = (int)(e / per_col), k0 = 8 * (int)(e - (int64_t)np * per_col);
  const int n = nq + np;
  float v[8];
  if (bits == 8) {
    const int8_t* src = reinterpret_cast<const int8_t*>(bt) + (int64_t)n * r + k0;
    const uint2 u = *reinterpret_cast<const uint2*>(src);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      v[i] = (float)(int8_t)(u.x >> (8 * i));
      v[4 + i] = (float)(int8_t)(u.y >> (8 * i));
    }
  } else {
    const uint32_t u = *reinterpret_cast<const uint32_t*>(bt + (int64_t)n * (r / 2) + k0 / 2);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const uint32_t byte = (u >> (8 * i)) & 0xFFu;
      v[2 * i] = (float)nib_lo(byte);
      v[2 * i + 1] = (float)nib_hi(byte);
    }
  }
  if (group) {
    const float sg = sb[(int64_t)(k0 / group) * N + n];   // a run never crosses a group (group % 64 == 0)
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] = mul_rn(v[i], sg);
  }
  f16x8 o;
#pragma unroll
  for (int i = 0; i < 8; ++i) o[i] = to_f16(v[i]);
  *reinterpret_cast<f16x8*>(w16 + (int64_t)np * r + k0) = o;
}

// Rotary embedding table, once per call: cs[t][j] = (cos, sin) of the angle
// t * theta^(-2j/dh) of pair j at position t < len, formed and reduced modulo
// 2 pi in fp64, then evaluated in fp32 (so large positions keep their
// accuracy).  Every key/value head and sequence reads the same rows.
__global__ void __launch_bounds__(256)
rope_table_kernel(float2* __restrict__ cs, int32_t len, int32_t dh, double log2_theta) {
  const int half = dh >> 1;
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= (int64_t)len * half) return;
  const int t = (int)(e / half), j = (int)(e - (int64_t)t * half);
  const double two_pi = 6.283185307179586476925286766559;
  double ang = (double)t * exp2(-2.0 * (double)j / (double)dh * log2_theta);
  ang -= floor(ang * (1.0 / two_pi)) * two_pi;
  float c, sn;
  sincosf((float)ang, &sn, &c);
  cs[e] = make_float2(c, sn);
}

__device__ __forceinline__ void rope_pair(float a, float b, float c, float s, float* ra, float* rb) {
  *ra = add_rn(mul_rn(a, c), -mul_rn(b, s));
  *rb = add_rn(mul_rn(b, c), mul_rn(a, s));
}

// Split-context attention over the rebuilt rows kv[b][t][0 .. 2 Hkv dh)
// (K^ then V^): one workgroup per (chunk of RCH tokens, sequence, key/value
// head g) serves the G = Hq / Hkv query heads of g.  The chunk's K^ and V^
// rows are staged in LDS with 16-byte loads (with rotary embeddings, each K^
// pair (j, j + dh/2) is turned as it is staged, and the queries at position
// seq_len - 1); scores, the softmax (one wave per head, a lane per token) and
// P V^ read LDS.  Partials go out in the merge's layout: per block of 32
// heads, O/l as fp16 [chunk][x][32 heads] and (m, l) per head.
constexpr int RCH = 64;

__host__ __device__ constexpr int recon_kld(int dh) { return dh + 8; }   // staged row stride (halves)

static size_t recon_attn_lds(int dh, int G) {
  return 2 * (size_t)RCH * recon_kld(dh) * sizeof(_Float16) +
         (size_t)G * dh * sizeof(float) + (size_t)G * RCH * sizeof(float) + 2 * (size_t)G * sizeof(float);
}

__global__ void __launch_bounds__(256)
recon_attn_kernel(const _Float16* __restrict__ q, const _Float16* __restrict__ kv,
                  const int32_t* __restrict__ seq_len, int32_t capacity, int32_t Hq, int32_t Hkv,
                  int32_t dh, float scale, int32_t n_chunks, int32_t n_hb, const float2* __restrict__ rope,
                  _Float16* __restrict__ o_part, float* __restrict__ ml_part) {
  extern __shared__ __attribute__((aligned(16))) uint8_t recon_smem[];
  const int b = blockIdx.y, ch = blockIdx.x, g = blockIdx.z, tid = threadIdx.x;
  const int lane = tid & 63, wv = tid >> 6;
  const int L = min(seq_len[b], capacity);
  const int t0 = ch * RCH;
  if (t0 >= L) return;
  const int tn = min(RCH, L - t0);
  const int G = Hq / Hkv, h0 = g * G, half = dh >> 1, kld = recon_kld(dh);
  const int nkv = Hkv * dh, nkv2 = 2 * nkv;
  _Float16* Ks = reinterpret_cast<_Float16*>(recon_smem);
  _Float16* Vs = Ks + RCH * kld;
  float* qs = reinterpret_cast<float*>(Vs + RCH * kld);                // [G][dh], rotated and scaled
  float* ps = qs + G * dh;                                             // [G][RCH] scores, then weights
  float* red = ps + G * RCH;                                           // m[G], l[G]

  const _Float16* qb = q + (int64_t)b * Hq * dh + (int64_t)h0 * dh;
  for (int e = tid; e < G * dh; e += 256) {
    const int hg = e / dh, c = e - hg * dh;
    float y = (float)qb[e];
    if (rope) {
      const int j = c < half ? c : c - half;
      const float2 cs = rope[(int64_t)(L - 1) * half + j];
      float ra, rb;
      rope_pair((float)qb[hg * dh + j], (float)qb[hg * dh + j + half], cs.x, cs.y, &ra, &rb);
      y = c < half ? ra : rb;
    }
    qs[e] = y * scale;
  }
  // stage K^ (rotated) and V^ rows of the chunk; rows past the sequence are zero
  const _Float16* rows = kv + ((int64_t)b * capacity + t0) * nkv2 + (int64_t)g * dh;
  const int cpr = dh / 8;                                              // 16-byte runs per head row
  for (int e = tid; e < RCH * cpr; e += 256) {
    const int tl = e / cpr, x = e - tl * cpr;
    f16x8 v = f16x8{};
    if (tl < tn) v = *reinterpret_cast<const f16x8*>(rows + (int64_t)tl * nkv2 + nkv + 8 * x);
    *reinterpret_cast<f16x8*>(Vs + tl * kld + 8 * x) = v;
  }
  if (!rope) {
    for (int e = tid; e < RCH * cpr; e += 256) {
      const int tl = e / cpr, x = e - tl * cpr;
      f16x8 v = f16x8{};
      if (tl < tn) v = *reinterpret_cast<const f16x8*>(rows + (int64_t)tl * nkv2 + 8 * x);
      *reinterpret_cast<f16x8*>(Ks + tl * kld + 8 * x) = v;
    }
  } else {
    const int cph = half / 8;                                          // runs per half row
    for (int e = tid; e < RCH * cph; e += 256) {
      const int tl = e / cph, x = e - tl * cph;
      f16x8 lo = f16x8{}, hi = f16x8{};
      if (tl < tn) {
        lo = *reinterpret_cast<const f16x8*>(rows + (int64_t)tl * nkv2 + 8 * x);
        hi = *reinterpret_cast<const f16x8*>(rows + (int64_t)tl * nkv2 + half + 8 * x);
        const float4* cs4 = reinterpret_cast<const float4*>(rope + (int64_t)(t0 + tl) * half + 8 * x);
#pragma unroll
        for (int i2 = 0; i2 < 4; ++i2) {
          const float4 c2 = cs4[i2];       // pairs 2 i2 and 2 i2 + 1: (cos, sin, cos, sin)
          float ra, rb;
          rope_pair((float)lo[2 * i2], (float)hi[2 * i2], c2.x, c2.y, &ra, &rb);
          lo[2 * i2] = to_f16(ra);
          hi[2 * i2] = to_f16(rb);
          rope_pair((float)lo[2 * i2 + 1], (float)hi[2 * i2 + 1], c2.z, c2.w, &ra, &rb);
          lo[2 * i2 + 1] = to_f16(ra);
          hi[2 * i2 + 1] = to_f16(rb);
        }
      }
      *reinterpret_cast<f16x8*>(Ks + tl * kld + 8 * x) = lo;
      *reinterpret_cast<f16x8*>(Ks + tl * kld + half + 8 * x) = hi;
    }
  }
  __syncthreads();
  // scores (log2 domain): item (head hg, token tl)
  for (int e = tid; e < G * RCH; e += 256) {
    const int hg = e / RCH, tl = e - hg * RCH;
    float acc = -INFINITY;
    if (tl < tn) {
      acc = 0.f;
      const float* qh = qs + hg * dh;
      for (int c = 0; c < dh; c += 8) {
        const f16x8 k8 = *reinterpret_cast<const f16x8*>(Ks + tl * kld + c);
#pragma unroll
        for (int i = 0; i < 8; ++i) acc = fmaf(qh[c + i], (float)k8[i], acc);
      }
    }
    ps[e] = acc;
  }
  __syncthreads();
  // softmax per head: one wave, a lane per token (RCH == 64)
  for (int hg = wv; hg < G; hg += 4) {
    const float sv = ps[hg * RCH + lane];
    float m = sv;
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) m = fmaxf(m, __shfl_xor(m, o));
    const float pv = lane < tn ? exp2f(sv - m) : 0.f;
    float l = pv;
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) l += __shfl_xor(l, o);
    ps[hg * RCH + lane] = pv;
    if (lane == 0) {
      red[hg] = m;
      red[G + hg] = l;
    }
  }
  __syncthreads();
  // partial rows of head h: block h / 32, column h % 32
  auto part_of = [&](int h) { return ((int64_t)b * n_hb + h / kHeadBlk) * n_chunks + ch; };
  for (int hg = tid; hg < G; hg += 256) {
    const int h = h0 + hg;
    ml_part[part_of(h) * 64 + h % kHeadBlk] = red[hg];
    ml_part[part_of(h) * 64 + 32 + h % kHeadBlk] = red[G + hg];
  }
  if (g == 0) {
    // heads past Hq in the last block's partial rows: weight 0 in the merge
    const int pad = n_hb * kHeadBlk - Hq;
    for (int i = tid; i < pad; i += 256) {
      const int h = Hq + i;
      ml_part[part_of(h) * 64 + h % kHeadBlk] = 0.f;
      ml_part[part_of(h) * 64 + 32 + h % kHeadBlk] = 1.f;
    }
    for (int e = tid; e < dh * pad; e += 256) {
      const int c = e / pad, h = Hq + e - c * pad;
      o_part[(part_of(h) * dh + c) * kHeadBlk + h % kHeadBlk] = (_Float16)0.f;
    }
  }
  // O^T[c][h] / l = sum_t p[h][t] V^[t][c] / l[h]: item (head hg, column pair c2)
  for (int e = tid; e < G * half; e += 256) {
    const int hg = e / half, c = 2 * (e - hg * half);
    const int h = h0 + hg;
    const float* ph = ps + hg * RCH;
    float a0 = 0.f, a1 = 0.f;
    for (int tl = 0; tl < tn; ++tl) {
      const f16x2 v2 = *reinterpret_cast<const f16x2*>(Vs + tl * kld + c);
      a0 = fmaf(ph[tl], (float)v2[0], a0);
      a1 = fmaf(ph[tl], (float)v2[1], a1);
    }
    const float il = 1.f / red[G + hg];
    o_part[(part_of(h) * dh + c) * kHeadBlk + h % kHeadBlk] = (_Float16)(a0 * il);
    o_part[(part_of(h) * dh + c + 1) * kHeadBlk + h % kHeadBlk] = (_Float16)(a1 * il);
  }
}

// Scores of the rotary variant, pre[b][t][h] = (sm log2 e) q_rot(h) . K^_rot(t):
// one workgroup per (chunk of RCH tokens, sequence, run of up to HPB
// key/value heads).  A thread keeps the (cos, sin) of its staging slots in
// registers for every head of the run; per head, the rotated K^ rows go to
// LDS (the next head's rows are loaded meanwhile).  With G >= 4 query heads
// per key/value head the scores come from 16x16x16 fp16 MFMAs (wave w:
// tokens 16w .. 16w+15; the query enters as an fp16 hi/lo pair, about fp32
// accuracy); with fewer, four lanes share each (query head, token) product
// in fp32, a quarter of the head dimension each.  Heads past Hq (up to 32)
// get score 0 from the first run's workgroups.
constexpr int kRopeSlots = 2;     // staging slots per thread: RCH * dh / 16 <= 512 runs

__host__ __device__ constexpr int rope_gpad(int G) { return (G + 15) / 16 * 16; }
__host__ __device__ constexpr bool rope_mfma(int G) { return G >= 4; }

static size_t rope_scores_lds(int dh, int hpb, int G) {
  const size_t q = rope_mfma(G) ? 2 * (size_t)hpb * rope_gpad(G) * dh * sizeof(_Float16)
                                : (size_t)hpb * G * dh * sizeof(float);
  return (size_t)RCH * recon_kld(dh) * sizeof(_Float16) + q;
}

__global__ void __launch_bounds__(256)
rope_scores_kernel(const _Float16* __restrict__ q, const _Float16* __restrict__ khat,
                   const int32_t* __restrict__ seq_len, int32_t capacity, int32_t Hq, int32_t Hkv, int32_t dh,
                   int32_t hpb, float scale, const float2* __restrict__ rope, float* __restrict__ pre) {
  extern __shared__ __attribute__((aligned(16))) uint8_t rs_smem[];
  const int b = blockIdx.y, ch = blockIdx.x, tid = threadIdx.x;
  const int L = min(seq_len[b], capacity);
  const int t0 = ch * RCH;
  if (t0 >= L) return;
  const int tn = min(RCH, L - t0);
  const int G = Hq / Hkv, half = dh >> 1, kld = recon_kld(dh), nkv = Hkv * dh;
  const int g0 = blockIdx.z * hpb, nh = min(hpb, Hkv - g0);
  const bool mf = rope_mfma(G);
  const int GP = mf ? rope_gpad(G) : G;
  _Float16* Ks = reinterpret_cast<_Float16*>(rs_smem);
  _Float16* qhi = Ks + RCH * kld;                                  // MFMA: [nh][GP][dh], zero past G
  _Float16* qlo = qhi + hpb * GP * dh;
  float* qs = reinterpret_cast<float*>(Ks + RCH * kld);            // else: fp32 [nh][G][dh]
  const _Float16* qb = q + (int64_t)b * Hq * dh + (int64_t)g0 * G * dh;
  for (int e = tid; e < nh * GP * dh; e += 256) {
    const int hp = e / dh, c = e - hp * dh, hh = hp / GP, hg = hp - hh * GP, j = c < half ? c : c - half;
    float y = 0.f;
    if (hg < G) {
      const float2 cs = rope[(int64_t)(L - 1) * half + j];
      const _Float16* qr = qb + (hh * G + hg) * dh;
      float ra, rb;
      rope_pair((float)qr[j], (float)qr[j + half], cs.x, cs.y, &ra, &rb);
      y = (c < half ? ra : rb) * scale;
    }
    if (mf) {
      const _Float16 yh = (_Float16)y;
      qhi[e] = yh;
      qlo[e] = (_Float16)(y - (float)yh);
    } else {
      qs[e] = y;
    }
  }
  // staging slot i of this thread: token tl, pairs 8x .. 8x+7 (x < dh/16)
  const int cph = half / 8;
  float4 cs4[kRopeSlots][4];
  f16x8 lo[kRopeSlots], hi[kRopeSlots];
  const _Float16* rows = khat + ((int64_t)b * capacity + t0) * nkv;
  auto load_head = [&](int g) {
#pragma unroll
    for (int i = 0; i < kRopeSlots; ++i) {
      const int e = tid + 256 * i, tl = e / cph, x = e - tl * cph;
      lo[i] = hi[i] = f16x8{};
      if (e < RCH * cph && tl < tn) {
        const _Float16* src = rows + (int64_t)tl * nkv + (int64_t)g * dh + 8 * x;
        lo[i] = *reinterpret_cast<const f16x8*>(src);
        hi[i] = *reinterpret_cast<const f16x8*>(src + half);
      }
    }
  };
#pragma unroll
  for (int i = 0; i < kRopeSlots; ++i) {
    const int e = tid + 256 * i, tl = e / cph, x = e - tl * cph;
    if (e < RCH * cph && tl < tn) {
      const float4* src = reinterpret_cast<const float4*>(rope + (int64_t)(t0 + tl) * half + 8 * x);
#pragma unroll
      for (int k = 0; k < 4; ++k) cs4[i][k] = src[k];
    }
  }
  load_head(g0);
  float* prow = pre + ((int64_t)b * capacity + t0) * kHeadBlk;
  const int lane = tid & 63, wv = tid >> 6, l16 = lane & 15, kq = lane >> 4;
  for (int hh = 0; hh < nh; ++hh) {
#pragma unroll
    for (int i = 0; i < kRopeSlots; ++i) {
      const int e = tid + 256 * i, tl = e / cph, x = e - tl * cph;
      if (e >= RCH * cph) continue;
      f16x8 a = lo[i], c = hi[i];
#pragma unroll
      for (int k = 0; k < 4; ++k) {     // pairs 2k, 2k + 1: (cos, sin, cos, sin)
        float ra, rb;
        rope_pair((float)a[2 * k], (float)c[2 * k], cs4[i][k].x, cs4[i][k].y, &ra, &rb);
        a[2 * k] = to_f16(ra);
        c[2 * k] = to_f16(rb);
        rope_pair((float)a[2 * k + 1], (float)c[2 * k + 1], cs4[i][k].z, cs4[i][k].w, &ra, &rb);
        a[2 * k + 1] = to_f16(ra);
        c[2 * k + 1] = to_f16(rb);
      }
      *reinterpret_cast<f16x8*>(Ks + tl * kld + 8 * x) = a;
      *reinterpret_cast<f16x8*>(Ks + tl * kld + half + 8 * x) = c;
    }
    if (hh + 1 < nh) load_head(g0 + hh + 1);
    __syncthreads();
    if (!mf) {
      // every thread runs G iterations (G * RCH * 4 items, 256 per query
      // head), so the quad reduction is uniform across the wave
      const int dq = dh / 4;
      for (int e = tid; e < G * RCH * 4; e += 256) {
        const int qd = e & 3, tl = (e >> 2) & (RCH - 1), hg = e >> 8;
        const float* qh = qs + (hh * G + hg) * dh + qd * dq;
        const _Float16* kr = Ks + tl * kld + qd * dq;
        float acc = 0.f;
        for (int c = 0; c < dq; c += 8) {
          const f16x8 k8 = *reinterpret_cast<const f16x8*>(kr + c);
#pragma unroll
          for (int i = 0; i < 8; ++i) acc = fmaf(qh[c + i], (float)k8[i], acc);
        }
        acc += __shfl_xor(acc, 1);
        acc += __shfl_xor(acc, 2);
        if (qd == 0 && tl < tn) prow[(int64_t)tl * kHeadBlk + (g0 + hh) * G + hg] = acc;
      }
    }
    // S[token][head]: A = K^ rows (lane: token 16 wv + l16, k 4 kq .. +3 of
    // each 16-wide step), B = the query rows (lane: head 16 hb + l16); lane
    // receives head 16 hb + l16 at tokens 16 wv + 4 kq + v
    for (int hb = 0; mf && hb < GP; hb += 16) {
      f32x4 acc = f32x4{};
      const _Float16* ka = Ks + (16 * wv + l16) * kld + 4 * kq;
      const _Float16* qh = qhi + ((hh * GP) + hb + l16) * dh + 4 * kq;
      const _Float16* ql = qlo + ((hh * GP) + hb + l16) * dh + 4 * kq;
      for (int k0 = 0; k0 < dh; k0 += 16) {
        const f16x4 a = *reinterpret_cast<const f16x4*>(ka + k0);
        acc = __builtin_amdgcn_mfma_f32_16x16x16f16(a, *reinterpret_cast<const f16x4*>(qh + k0), acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_16x16x16f16(a, *reinterpret_cast<const f16x4*>(ql + k0), acc, 0, 0, 0);
      }
      const int hg = hb + l16;
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int tl = 16 * wv + 4 * kq + v;
        if (hg < G && tl < tn) prow[(int64_t)tl * kHeadBlk + (g0 + hh) * G + hg] = acc[v];
      }
    }
    __syncthreads();
  }
  if (blockIdx.z == 0)
    for (int e = tid; e < tn * (kHeadBlk - Hq); e += 256) {
      const int tl = e / (kHeadBlk - Hq), h = Hq + e - tl * (kHeadBlk - Hq);
      prow[(int64_t)tl * kHeadBlk + h] = 0.f;
    }
}

// The turned, scaled queries of the fused rotary scores:
// qrot[b][h][c] = scale * rot(q[b][h], position seq_len[b] - 1)[c], fp32.
__global__ void __launch_bounds__(256)
rope_query_kernel(const _Float16* __restrict__ q, const int32_t* __restrict__ seq_len, int32_t capacity,
                  int32_t batch, int32_t Hq, int32_t dh, float scale, const float2* __restrict__ rope,
                  float* __restrict__ qrot) {
  const int half = dh >> 1;
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;   // one pair (b, h, j)
  if (e >= (int64_t)batch * Hq * half) return;
  const int j = (int)(e % half);
  const int64_t bh = e / half;
  const int b = (int)(bh / Hq);
  const int L = min(seq_len[b], capacity);
  const float2 cs = rope[(int64_t)max(L - 1, 0) * half + j];
  const _Float16* qr = q + bh * dh;
  float ra, rb;
  rope_pair((float)qr[j], (float)qr[j + half], cs.x, cs.y, &ra, &rb);
  qrot[bh * dh + j] = ra * scale;
  qrot[bh * dh + j + half] = rb * scale;
}

struct ReconPlan {
  size_t kv_bytes, opart_bytes, ml_bytes, w16_bytes, rope_bytes;
  int n_chunks, n_hb;       // context chunks of RCH tokens, blocks of 32 query heads
};

// (cos, sin) rows of the rotary table for every position a cache can hold.
static size_t rope_table_bytes(const qsvd_layer& w, const qsvd_cache& c) {
  return (size_t)c.capacity * (w.head_dim / 2) * sizeof(float2);
}

static hipError_t launch_rope_table(const AttnArgs& a, float2* cs, hipStream_t s) {
  const int len = a.c->max_len > 0 ? a.c->max_len : 1;
  const int64_t n = (int64_t)len * (a.w->head_dim / 2);
  KernelScope ks("rope_table", s);
  QSVD_LAUNCH(ks, rope_table_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, cs, len, a.w->head_dim,
              log2((double)a.rope_theta));
  return hipGetLastError();
}

static ReconPlan plan_recon(const qsvd_layer& w, const qsvd_cache& c) {
  ReconPlan p{};
  const int nkv2 = 2 * w.n_kv_heads * w.head_dim;
  p.n_chunks = (c.capacity + RCH - 1) / RCH;
  p.kv_bytes = (size_t)c.batch * c.capacity * nkv2 * sizeof(_Float16);
  p.n_hb = (w.n_q_heads + kHeadBlk - 1) / kHeadBlk;
  p.opart_bytes = (size_t)c.batch * p.n_hb * p.n_chunks * w.head_dim * kHeadBlk * sizeof(_Float16);
  p.ml_bytes = (size_t)c.batch * p.n_hb * p.n_chunks * 64 * sizeof(float);
  p.w16_bytes = c.fmt == QSVD_CACHE_F16 ? (size_t)nkv2 * w.r * sizeof(_Float16) : 0;
  p.rope_bytes = rope_table_bytes(w, c);
  return p;
}

// The rotary variant with the value side in latent space: K^ only, the
// scores, then the latent attention's value half, merge and W^u_v.
bool rope_latent_supported(const qsvd_layer& w, const qsvd_cache& c) {
  int rw, nw;
  return w.n_q_heads <= kHeadBlk && pick_slice(w.r, &rw, &nw);
}

struct RopeLatentPlan {
  size_t khat_bytes, pre_bytes, w16_bytes, rope_bytes;
  AbsorbPlan ap;
};

// The key rebuild with the rotary scores in its epilogue (fp16 caches, and
// int8 caches with per-channel int8 weights; head_dim 32, 64 or 128): the
// turned keys never leave the product, and their workspace holds the turned
// queries instead.
static bool rope_fused_supported(const qsvd_layer& w, const qsvd_cache& c) {
  const bool prod = c.fmt == QSVD_CACHE_F16 || (c.fmt == QSVD_CACHE_I8 && w.w_bits == 8 && !w.w_group);
  return prod && (w.head_dim == 32 || w.head_dim == 64 || w.head_dim == 128);
}

static RopeLatentPlan plan_rope_latent(const qsvd_layer& w, const qsvd_cache& c) {
  RopeLatentPlan p{};
  const int nkv = w.n_kv_heads * w.head_dim;
  p.khat_bytes = rope_fused_supported(w, c) ? (size_t)c.batch * w.n_q_heads * w.head_dim * sizeof(float)
                                             : (size_t)c.batch * c.capacity * nkv * sizeof(_Float16);
  p.pre_bytes = (size_t)c.batch * c.capacity * kHeadBlk * sizeof(float);
  p.w16_bytes = c.fmt == QSVD_CACHE_F16 ? (size_t)nkv * w.r * sizeof(_Float16) : 0;
  p.rope_bytes = rope_table_bytes(w, c);
  p.ap = plan_absorbed(w, c, 1);
  return p;
}

static size_t rope_latent_workspace(const qsvd_layer& w, const qsvd_cache& c) {
  const RopeLatentPlan p = plan_rope_latent(w, c);
  return align256(p.khat_bytes) + align256(p.pre_bytes) + align256(p.w16_bytes) + align256(p.rope_bytes) +
         align256(p.ap.opart_bytes) + align256(p.ap.ml_bytes) + align256(p.ap.olat_bytes);
}

// One workspace size serves both reconstruct-side forms (with and without
// the value side in latent space).
size_t attn_reconstruct_workspace(const qsvd_layer& w, const qsvd_cache& c) {
  const ReconPlan p = plan_recon(w, c);
  const size_t full = align256(p.kv_bytes) + align256(p.opart_bytes) + align256(p.ml_bytes) + align256(p.w16_bytes) +
                      align256(p.rope_bytes);
  const size_t lat = rope_latent_supported(w, c) ? rope_latent_workspace(w, c) : 0;
  return full > lat ? full : lat;
}

// Columns [nq, nq + ncols) of C W^u for the cache rows, fp16 into out (row
// stride ncols): K^ (ncols = Hkv dh) or K^ | V^ (2 Hkv dh).  Rows past a
// sequence's length are rebuilt too when that keeps one launch (at most a
// third of the rows wasted); otherwise one launch per sequence over its first
// max_len rows.
static hipError_t rebuild_rows(const AttnArgs& a, int ncols, _Float16* w16, _Float16* out, hipStream_t s) {
  const qsvd_layer& w = *a.w;
  const qsvd_cache& c = *a.c;
  const int N = (w.n_q_heads + 2 * w.n_kv_heads) * w.head_dim;
  const int nq = w.n_q_heads * w.head_dim;
  const int len = c.max_len > 0 ? c.max_len : 1;
  const bool f16 = c.fmt == QSVD_CACHE_F16, i4 = c.fmt == QSVD_CACHE_I4;
  if (f16) {
    KernelScope ks("recon_weights", s);
    const int64_t runs = (int64_t)ncols * (w.r / 8);
    QSVD_LAUNCH(ks, recon_weights_kernel, dim3((unsigned)((runs + 255) / 256)), dim3(256), 0, s,
                (const uint8_t*)w.b_t, w.s_b, w.r, N, nq, ncols, w.w_bits, w.w_group, w16);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  const size_t row_bytes = f16 ? (size_t)c.r * 2 : i4 ? (size_t)c.r / 2 : (size_t)c.r;
  const bool one = c.batch == 1 || 4 * (int64_t)len >= 3 * (int64_t)c.capacity;
  const int launches = one ? 1 : c.batch;
  for (int i = 0; i < launches; ++i) {
    GemmArgs g{};
    const int64_t r0 = one ? 0 : (int64_t)i * c.capacity;
    g.a = reinterpret_cast<const int8_t*>(reinterpret_cast<const uint8_t*>(c.data) + r0 * row_bytes);
    g.row_scale = f16 ? nullptr : c.scale + r0;
    g.M = one ? (c.batch == 1 ? len : (int64_t)c.batch * c.capacity) : len;
    g.N = ncols;
    g.K = w.r;
    g.seg[0] = OutSeg{out + r0 * ncols, ncols, 0, ncols};
    g.n_seg = 1;
    g.abits = i4 ? 4 : 8;
    hipError_t e;
    if (f16) {
      g.b = reinterpret_cast<const int8_t*>(w16);
      g.col_scale = w.w_group ? nullptr : w.s_b + nq;
      e = launch_gemm_f16(g, s);
    } else {
      g.b = reinterpret_cast<const int8_t*>(w.b_t) + (int64_t)nq * (w.w_bits == 8 ? w.r : w.r / 2);
      g.col_scale = w.s_b + nq;
      e = (!i4 && w.w_bits == 8 && !w.w_group) ? launch_gemm_i8(g, s)
                                               : launch_gemm_q4(g, g.abits, w.w_bits, w.w_group, N, s);
    }
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_attn_reconstruct(const AttnArgs& a, void* ws, hipStream_t s) {
  const qsvd_layer& w = *a.w;
  const qsvd_cache& c = *a.c;
  const ReconPlan p = plan_recon(w, c);
  uint8_t* base = (uint8_t*)ws;
  _Float16* kv = (_Float16*)base;
  base += align256(p.kv_bytes);
  _Float16* opart = (_Float16*)base;
  base += align256(p.opart_bytes);
  float* ml = (float*)base;
  base += align256(p.ml_bytes);
  _Float16* w16 = p.w16_bytes ? (_Float16*)base : nullptr;
  base += align256(p.w16_bytes);
  float2* rope = a.rope_theta > 0.f ? (float2*)base : nullptr;
  const int nkv2 = 2 * w.n_kv_heads * w.head_dim;
  const int len = c.max_len > 0 ? c.max_len : 1;
  hipError_t e = rebuild_rows(a, nkv2, w16, kv, s);
  if (e != hipSuccess) return e;
  if (a.q_len > 1) {
    // several queries per sequence: causal attention of the last q_len
    // positions over the rebuilt rows on the fp16 matrix cores (rotary
    // embeddings turned in that kernel at each row's position)
    const CacheAttnArgs ca{a.q, kv, c.seq_len, c.batch, c.capacity, a.q_len, w.n_q_heads, w.n_kv_heads, w.head_dim,
                           a.sm_scale, a.rope_theta, a.out};
    return launch_cache_attention(ca, s);
  }
  if (rope && (e = launch_rope_table(a, rope, s)) != hipSuccess) return e;
  const int nch = (len + RCH - 1) / RCH;
  const int G = w.n_q_heads / w.n_kv_heads;
  {
    KernelScope ks("recon_attn", s);
    const size_t lds = recon_attn_lds(w.head_dim, G);
    hipError_t ea = hipFuncSetAttribute((const void*)recon_attn_kernel, hipFuncAttributeMaxDynamicSharedMemorySize,
                                        (int)recon_attn_lds(128, kMaxAbsorbedHeads));
    if (ea != hipSuccess) return ea;
    QSVD_LAUNCH(ks, recon_attn_kernel, dim3(nch, c.batch, w.n_kv_heads), dim3(256), lds, s, a.q, kv, c.seq_len,
                c.capacity, w.n_q_heads, w.n_kv_heads, w.head_dim, a.sm_scale * kLog2e, p.n_chunks, p.n_hb, rope,
                opart, ml);
  }
  {
    KernelScope ks("recon_combine", s);
    QSVD_LAUNCH(ks, combine_kernel, dim3((w.head_dim + 63) / 64, c.batch * p.n_hb), dim3(256), 0, s, opart, ml,
                c.seq_len, RCH, p.n_chunks, nch, w.head_dim, w.n_q_heads, p.n_hb, a.out);
  }
  return hipGetLastError();
}

static hipError_t rebuild_rope_scores(const AttnArgs& a, _Float16* w16, float* qrot, const float2* rope, float* pre,
                                      hipStream_t s) {
  const qsvd_layer& w = *a.w;
  const qsvd_cache& c = *a.c;
  const int N = (w.n_q_heads + 2 * w.n_kv_heads) * w.head_dim;
  const int nq = w.n_q_heads * w.head_dim, nkv = w.n_kv_heads * w.head_dim;
  const int len = c.max_len > 0 ? c.max_len : 1;
  const bool f16 = c.fmt == QSVD_CACHE_F16;
  {
    KernelScope ks("rope_query", s);
    const int64_t n = (int64_t)c.batch * w.n_q_heads * (w.head_dim / 2);
    QSVD_LAUNCH(ks, rope_query_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, a.q, c.seq_len,
                c.capacity, c.batch, w.n_q_heads, w.head_dim, a.sm_scale * kLog2e, rope, qrot);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (f16) {
    KernelScope ks("recon_weights", s);
    const int64_t runs = (int64_t)nkv * (w.r / 8);
    QSVD_LAUNCH(ks, recon_weights_kernel, dim3((unsigned)((runs + 255) / 256)), dim3(256), 0, s,
                (const uint8_t*)w.b_t, w.s_b, w.r, N, nq, nkv, w.w_bits, w.w_group, w16);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  const size_t row_bytes = f16 ? (size_t)c.r * 2 : (size_t)c.r;
  const bool one = c.batch == 1 || 4 * (int64_t)len >= 3 * (int64_t)c.capacity;
  const int launches = one ? 1 : c.batch;
  for (int i = 0; i < launches; ++i) {
    GemmArgs g{};
    const int64_t r0 = one ? 0 : (int64_t)i * c.capacity;
    g.a = reinterpret_cast<const int8_t*>(reinterpret_cast<const uint8_t*>(c.data) + r0 * row_bytes);
    g.row_scale = f16 ? nullptr : c.scale + r0;
    g.M = one ? (c.batch == 1 ? len : (int64_t)c.batch * c.capacity) : len;
    g.N = nkv;
    g.K = w.r;
    g.n_seg = 0;
    g.abits = 8;
    if (f16) {
      g.b = reinterpret_cast<const int8_t*>(w16);
      g.col_scale = w.w_group ? nullptr : w.s_b + nq;
    } else {
      g.b = reinterpret_cast<const int8_t*>(w.b_t) + (int64_t)nq * w.r;
      g.col_scale = w.s_b + nq;
    }
    const RopeEpi re{qrot, rope, c.seq_len, pre, r0, c.capacity, w.n_q_heads, w.n_q_heads / w.n_kv_heads,
                     w.head_dim};
    const hipError_t e = launch_gemm_rope_scores(g, re, f16, s);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_attn_rope_latent(const AttnArgs& a, void* ws, hipStream_t s) {
  const qsvd_layer& w = *a.w;
  const qsvd_cache& c = *a.c;
  const RopeLatentPlan p = plan_rope_latent(w, c);
  uint8_t* base = (uint8_t*)ws;
  _Float16* khat = (_Float16*)base;
  base += align256(p.khat_bytes);
  float* pre = (float*)base;
  base += align256(p.pre_bytes);
  _Float16* w16 = p.w16_bytes ? (_Float16*)base : nullptr;
  base += align256(p.w16_bytes);
  float2* rope = (float2*)base;
  base += align256(p.rope_bytes);
  _Float16* opart = (_Float16*)base;
  base += align256(p.ap.opart_bytes);
  float* ml = (float*)base;
  base += align256(p.ap.ml_bytes);
  _Float16* olat = (_Float16*)base;
  const int nkv = w.n_kv_heads * w.head_dim;
  const int len = c.max_len > 0 ? c.max_len : 1;
  hipError_t e;
  if (rope_fused_supported(w, c)) {
    // the turned queries go where the rebuilt keys would be staged
    if ((e = launch_rope_table(a, rope, s)) != hipSuccess) return e;
    if ((e = rebuild_rope_scores(a, w16, reinterpret_cast<float*>(khat), rope, pre, s)) != hipSuccess) return e;
  } else {
    if ((e = rebuild_rows(a, nkv, w16, khat, s)) != hipSuccess) return e;
    if ((e = launch_rope_table(a, rope, s)) != hipSuccess) return e;
    {
      KernelScope ks("rope_scores", s);
      const int G = w.n_q_heads / w.n_kv_heads, nch = (len + RCH - 1) / RCH;
      // runs of up to 8 key/value heads share the (cos, sin) registers, as long
      // as the grid keeps about four workgroups per CU and the staged queries
      // fit the default 64 KB of LDS (one head always does)
      int hpb = std::min(w.n_kv_heads, 8);
      while (hpb > 1 && ((int64_t)nch * c.batch * ((w.n_kv_heads + hpb - 1) / hpb) < 1024 ||
                         rope_scores_lds(w.head_dim, hpb, G) > 65536))
        hpb /= 2;
      const unsigned runs = (unsigned)((w.n_kv_heads + hpb - 1) / hpb);
      QSVD_LAUNCH(ks, rope_scores_kernel, dim3(nch, c.batch, runs), dim3(256), rope_scores_lds(w.head_dim, hpb, G), s,
                  a.q, khat, c.seq_len, c.capacity, w.n_q_heads, w.n_kv_heads, w.head_dim, hpb, a.sm_scale * kLog2e,
                  rope, pre);
      e = hipGetLastError();
      if (e != hipSuccess) return e;
    }
  }
  e = c.fmt == QSVD_CACHE_F16 ? dispatch_latent_pre<QSVD_CACHE_F16>(p.ap, c, pre, opart, ml, s)
      : c.fmt == QSVD_CACHE_I8  ? dispatch_latent_pre<QSVD_CACHE_I8>(p.ap, c, pre, opart, ml, s)
                                : dispatch_latent_pre<QSVD_CACHE_I4>(p.ap, c, pre, opart, ml, s);
  if (e != hipSuccess) return e;
  return merge_and_project(a, p.ap, opart, ml, olat, s);
}

}  // namespace qsvd
