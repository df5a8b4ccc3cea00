/*
 * qsvd.h -- C ABI of the QSVD latent-QKV hot path on AMD Instinct MI355X (gfx950).
 *
 * QSVD ("Efficient Low-rank Approximation for Unified Query-Key-Value Weight
 * Compression in Low-Precision Vision-Language Models", arXiv 2510.16292)
 * replaces the three projections W_q, W_k, W_v of an attention layer by one
 * joint truncated SVD of [W_q | W_k | W_v] (Section 3.1, Eq. 2-4): a shared
 * down-projection W^d (d x r) and an up-projection W^u = [W^u_q | W^u_k | W^u_v]
 * (r x N).  The per-token latent C = X W^d is the only thing cached
 * (Section 3.1); keys and values are rebuilt from it, K = C W^u_k and
 * V = C W^u_v (Eq. 5).  Weights and activations are quantized (Section 3.3,
 * Eq. 11-12; per-token symmetric activations and round-to-nearest
 * per-channel symmetric weights, Section 4).
 *
 * Conventions for every call:
 *  - Pointers marked "device" are device (HBM) addresses allocated by the
 *    caller; the library never allocates, frees or keeps device memory, and
 *    keeps no state between calls except the optional profiler.
 *  - `stream` is a hipStream_t (NULL = the null stream).  Calls enqueue work
 *    on it and return without synchronizing.
 *  - Arguments are validated on the host before any GPU work is enqueued.  On
 *    any status other than QSVD_OK nothing was enqueued, outputs are left
 *    untouched and cache state (seq_len, max_len) is unchanged -- except
 *    QSVD_ERR_HIP, which reports a failed launch after validation passed.
 *    qsvd_last_error() describes the most recent failure of the calling thread.
 *  - Row-major layouts; "[a][b]" means b is the contiguous index.
 *  - Integer codes are symmetric two's complement: int8 in [-127, 127], int4
 *    in [-7, 7] packed two per byte, element 2i in the low nibble of byte i.
 */
#ifndef QSVD_H
#define QSVD_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  QSVD_OK = 0,
  QSVD_ERR_INVALID_ARG = 1,  /* null pointer, negative size, inconsistent shapes */
  QSVD_ERR_UNSUPPORTED = 2,  /* well-formed but outside what the kernels implement */
  QSVD_ERR_CAPACITY = 3,     /* an append would exceed the cache capacity */
  QSVD_ERR_WORKSPACE = 4,    /* workspace missing or smaller than the size query */
  QSVD_ERR_HIP = 5           /* a HIP runtime call or kernel launch failed */
} qsvd_status;

/* Latent cache storage formats. */
enum { QSVD_CACHE_F16 = 0, QSVD_CACHE_I8 = 1, QSVD_CACHE_I4 = 2 };

/* Decode attention forms.  RECONSTRUCT rebuilds K and V from the latent for
 * every cached token (Eq. 5) and attends as usual; ABSORBED folds W^u_k into
 * the query and applies W^u_v after the latent-space weighted sum (the
 * latent-attention form of Section 1 and 2.2).  Both compute the same
 * attention; AUTO picks the faster one for the layer (ABSORBED). */
enum { QSVD_ATTN_AUTO = 0, QSVD_ATTN_ABSORBED = 1, QSVD_ATTN_RECONSTRUCT = 2 };

/* Which up-projection outputs qsvd_lowrank_qkv_prefill writes. */
enum { QSVD_OUT_Q = 1, QSVD_OUT_K = 2, QSVD_OUT_V = 4 };

/* One attention layer after the offline stage (joint SVD, truncation, beta
 * split, weight quantization).  N = (n_q_heads + 2 * n_kv_heads) * head_dim.
 * Query head h reads key/value head floor(h * n_kv_heads / n_q_heads). */
typedef struct {
  int32_t d;           /* embedding dimension E (contraction of X W^d) */
  int32_t r;           /* joint rank */
  int32_t n_q_heads;
  int32_t n_kv_heads;
  int32_t head_dim;
  int32_t w_bits;      /* 8: int8 codes; 4: packed int4 codes */
  int32_t w_group;     /* 0: one scale per output channel; G > 0: one scale per
                          output channel and per G contraction rows */
  const void*  a_t;    /* device, W^d codes transposed: [r][d] int8 or [r][d/2] int4 */
  const float* s_a;    /* device, W^d scales: [r] (w_group 0) or [d/G][r] */
  const void*  b_t;    /* device, W^u codes transposed: [N][r] int8 or [N][r/2] int4;
                          rows 0..Hq*hd-1 are W^u_q, then W^u_k, then W^u_v */
  const float* s_b;    /* device, W^u scales: [N] (w_group 0) or [r/G][N] */
} qsvd_layer;

/* Latent cache of `batch` sequences.  Sequence b holds seq_len[b] rows.
 * F16: data is [batch][capacity][r] fp16, scale NULL.
 * I8:  data is [batch][capacity][r] int8, scale [batch][capacity] fp32.
 * I4:  data is [batch][capacity][r/2] packed int4, scale [batch][capacity] fp32.
 * A row of an integer cache is Q(C) of the token (its codes and scale). */
typedef struct {
  int32_t  fmt;        /* QSVD_CACHE_* */
  int32_t  batch;
  int32_t  capacity;   /* rows per sequence */
  int32_t  r;
  void*    data;       /* device */
  float*   scale;      /* device or NULL (F16) */
  int32_t* seq_len;    /* device [batch] */
  int32_t  max_len;    /* host: an upper bound of every seq_len[b]; the caller sets
                          it when initialising seq_len, append advances it */
  int32_t* overflow;   /* device, optional (NULL: not reported): an append that finds
                          seq_len[b] + n_new > capacity on the device (possible only
                          when the host check was bypassed, e.g. by a graph replay)
                          stores 1 here; the caller clears it */
} qsvd_cache;

/* Per-token symmetric activation quantization (Section 4 setup; Q(.) of Eq. 12).
 * Per row m, in fp32: a = clip * max_k |x[m][k]|; if a == 0 then s = 1 and all
 * codes are 0, else inv = Qm / a (IEEE division), s = a / Qm and
 * q = clamp(rint(x * inv), -Qm, Qm) with ties to even; Qm = 2^(bits-1) - 1.
 *   x   device fp16 [M][ldx] (first K columns used)
 *   xq  device int8 [M][K] (bits 8) or packed int4 [M][K/2] (bits 4)
 *   sx  device fp32 [M]
 * Requires K % 8 == 0, ldx % 8 == 0, 16-byte aligned x; bits 8 or 4; 0 < clip <= 1. */
qsvd_status qsvd_quantize_act(const void* x, int64_t M, int32_t K, int64_t ldx, int32_t bits,
                              float clip, void* xq, float* sx, void* stream);

/* Per-token quantization of rotated activations, Q(X H1^T) (Eq. 11-12), for
 * layers whose input rotation H1 cannot be folded into the previous layer;
 * the layer's W^d then holds H1 W^d (folded offline).
 *   H1 = blockdiag(H_B, ..., H_B) diag(signs) / sqrt(B), H_B the Sylvester
 *   Hadamard matrix of order B = block, so X H1^T = (X o signs) blockdiag(H_B) / sqrt(B).
 * Per row, in fp32: v_k = x_k * signs_k; the Walsh-Hadamard stages
 * h = 1, 2, 4, ..., B/2 in that order, each replacing (v_i, v_{i+h}) by
 * (v_i + v_{i+h}, v_i - v_{i+h}) for every i whose bit h is clear (each sum
 * rounded to fp32); y = v * c with c = fp32(1 / sqrt(B)); then y goes through
 * the quantizer of qsvd_quantize_act (same clip, scale and codes).
 *   x      device fp16 [M][ldx] (first K columns used)
 *   signs  device int8 [K] of +1 / -1 (NULL: all +1)
 *   block  B: a power of two >= 8 dividing K
 *   xq, sx as for qsvd_quantize_act
 * Requires K % 8 == 0, K <= 16384, ldx % 8 == 0, 16-byte aligned x, 8-byte
 * aligned xq and signs; bits 8 or 4; 0 < clip <= 1. */
qsvd_status qsvd_quantize_act_rotated(const void* x, int64_t M, int32_t K, int64_t ldx, int32_t bits,
                                      float clip, const int8_t* signs, int32_t block, void* xq,
                                      float* sx, void* stream);

/* Quantized joint low-rank QKV projection (Section 3.1 and Eq. 11-12):
 *   C   = (xq W^d codes) dequantized: fp32 (acc * sx[m]) * s_a[j] (per group:
 *         sum over groups of acc_g * s_a[g][j], then * sx[m]), stored as fp16
 *   Q(C) = per-token quantization of the fp16 C with act_bits (as qsvd_quantize_act, clip 1)
 *   [Q|K|V] = (Q(C) W^u codes) dequantized the same way, stored as fp16
 *   w        layer (host struct, device pointers)
 *   xq, sx   device, output of qsvd_quantize_act with act_bits, M rows
 *   c_h      device fp16 [M][r]                     (always written)
 *   cq, sc   device int8 [M][r] (or int4 [M][r/2]) and fp32 [M]   (always written)
 *   q, k, v  device fp16 [M][Hq*hd], [M][Hkv*hd], [M][Hkv*hd]; written when the
 *            matching QSVD_OUT_* bit is set (others may be NULL)
 *   dbg_acc_xa, dbg_acc_cb  optional device int32 [M][r] and [M][N] copies of
 *            the integer accumulators (w_group 0 only; NULL to skip)
 *   ws       unused (qsvd_prefill_workspace_size() returns 0; kept for callers
 *            that size one anyway)
 * Requires d % 64 == 0, r % 64 == 0, act_bits 8 or 4, int8 or int4 weights
 * with per-channel or per-group scales (groups a multiple of 64 dividing d and
 * r), 16-byte aligned xq, c_h, cq and weight codes.  More than 32 tokens also
 * need head_dim a multiple of 8 and 16-byte aligned q, k, v.  The integer
 * accumulator dumps need act_bits 8 and per-channel weights.  Other
 * combinations return QSVD_ERR_UNSUPPORTED. */
qsvd_status qsvd_lowrank_qkv_prefill(const qsvd_layer* w, const void* xq, const float* sx,
                                     int64_t M, int32_t act_bits, uint32_t out_mask,
                                     void* c_h, void* cq, float* sc, void* q, void* k, void* v,
                                     int32_t* dbg_acc_xa, int32_t* dbg_acc_cb,
                                     void* ws, size_t ws_bytes, void* stream);

size_t qsvd_prefill_workspace_size(const qsvd_layer* w, int64_t M, uint32_t out_mask);

/* Append n_new latent rows to every sequence of the cache (only C is buffered,
 * Section 3.1).  Source rows are token-major with sequence b's rows at
 * [b * n_new, (b + 1) * n_new):
 *   F16 cache: c_h  device fp16 [batch * n_new][r]           (cq, sc ignored)
 *   I8 / I4:   cq   device int8 [..][r] / int4 [..][r/2], sc device fp32 [..]
 * Row i of sequence b goes to position seq_len[b] + i; then seq_len[b] += n_new
 * on the device and c->max_len += n_new on the host.  Returns QSVD_ERR_CAPACITY
 * if c->max_len + n_new > c->capacity.  On the device, rows that would land at
 * or past capacity are not written, seq_len[b] stops at capacity and
 * *c->overflow is set to 1 (when given): a replayed graph, which skips the
 * host check, cannot grow a sequence past its buffer. */
qsvd_status qsvd_latent_cache_append(qsvd_cache* c, const void* c_h, const void* cq,
                                     const float* sc, int32_t n_new, void* stream);

/* One decode step's projection of the new tokens together with the append of
 * their latent rows (Section 3.1: one new token per sequence; only C is
 * buffered): per-token quantization of x with act_bits and clip, C = the
 * quantized down-projection, Q(C), the Q up-projection, and the append of each
 * sequence's latent row (fp16 C, or Q(C) codes and scale for an integer
 * cache) at position seq_len[b], then seq_len[b] += 1 on the device and
 * c->max_len += 1 on the host.  Every output byte, cache byte and length is
 * the one of qsvd_quantize_act + qsvd_lowrank_qkv_prefill(out_mask QSVD_OUT_Q)
 * + qsvd_latent_cache_append(n_new 1); the quantizer runs inside the
 * down-projection and the append inside the two products, so the step takes
 * two launches instead of four.
 *   x         device fp16 [batch][ldx], row b the new token of sequence b
 *   xq, sx    device outputs: Q(x) codes ([batch][d] int8 or [batch][d/2] int4) and scales
 *   c_h       device fp16 [batch][r]; cq, sc: Q(C) ([batch][r] / [batch][r/2], [batch])
 *   q         device fp16 [batch][Hq*hd]
 * Requires batch <= 32, an I8 cache with act_bits 8 or an I4 cache with
 * act_bits 4 (any act_bits for F16), ldx % 8 == 0, 16-byte aligned x, xq,
 * c_h, cq and weight codes, and the layer requirements of
 * qsvd_lowrank_qkv_prefill.  QSVD_ERR_CAPACITY if c->max_len + 1 > capacity;
 * on the device, a row at or past capacity is dropped as in
 * qsvd_latent_cache_append. */
qsvd_status qsvd_decode_project_append(const qsvd_layer* w, qsvd_cache* c, const void* x, int64_t ldx,
                                       int32_t act_bits, float clip, void* xq, float* sx, void* c_h,
                                       void* cq, float* sc, void* q, void* stream);

/* Causal self-attention of a prefill block over its own projections (Section
 * 3.1: in prefill every prompt token's keys and values are at hand as the rows
 * K = C W^u_k and V = C W^u_v that qsvd_lowrank_qkv_prefill wrote, Eq. 5 and
 * Eq. 11).  Token i of a sequence attends to tokens 0..i of the same sequence:
 * softmax(q k^T * sm_scale) v with an fp32 softmax, query head h reading
 * key/value head floor(h * n_kv_heads / n_q_heads).
 *   q           device fp16 [M][n_q_heads * head_dim] (the projection's Q)
 *   k, v        device fp16 [M][n_kv_heads * head_dim] (its K and V)
 *   cu_seqlens  device int32 [batch + 1]: sequence b is rows
 *               [cu_seqlens[b], cu_seqlens[b + 1]); nondecreasing, cu_seqlens[0] = 0
 *   max_seqlen  host: at least every sequence's length (sizes the launch)
 *   sm_scale    0 selects 1/sqrt(head_dim)
 *   out         device fp16 [M][n_q_heads * head_dim]
 * Requires head_dim 64 or 128 and 16-byte aligned q, k, v, out.  Rows of a
 * sequence longer than max_seqlen past max_seqlen are left unwritten.  No
 * workspace; asynchronous on `stream`. */
qsvd_status qsvd_prefill_attention(const void* q, const void* k, const void* v, int32_t batch,
                                   const int32_t* cu_seqlens, int32_t max_seqlen, int32_t n_q_heads,
                                   int32_t n_kv_heads, int32_t head_dim, float sm_scale, void* out,
                                   void* stream);

/* qsvd_prefill_attention for layers that apply a rotary position embedding
 * to q and k (the paper's layers have none; the position-encoded variant of
 * the same prefill step, with the same rotation as
 * qsvd_latent_decode_attention_rope).  Before the product, row i of a
 * sequence (its position within that sequence, counted from 0) has the pairs
 * (j, j + head_dim/2), j < head_dim/2, of every query and key head vector
 * turned by the angle i * rope_theta^(-2j/head_dim): the angle is formed in
 * revolutions and reduced to [0, 1) in fp64, its sine and cosine taken in
 * fp32, and the turned rows rounded to fp16 before the products.  Values are
 * not turned.  A decode step that continues the sequence over its cache sees
 * the same key positions.  Same arguments, requirements and errors as
 * qsvd_prefill_attention; rope_theta must be finite and > 1
 * (QSVD_ERR_INVALID_ARG otherwise). */
qsvd_status qsvd_prefill_attention_rope(const void* q, const void* k, const void* v, int32_t batch,
                                        const int32_t* cu_seqlens, int32_t max_seqlen, int32_t n_q_heads,
                                        int32_t n_kv_heads, int32_t head_dim, float sm_scale, float rope_theta,
                                        void* out, void* stream);

/* Attention of the newest queries of every sequence over its cached latent
 * rows (Section 3.1; decoding is l = 1): keys and values are C W^u_k and
 * C W^u_v of the stored rows (dequantized), softmax(q K^T * sm_scale) V with an
 * fp32 softmax.  The q_len queries of sequence b are its last q_len cached
 * positions (append first, then attend): query i sees positions
 * [0, seq_len[b] - q_len + i], causally.  A query with no visible position
 * (seq_len[b] < q_len - i) gets zeros.
 *   q     device fp16 [batch][q_len][Hq*hd] (the Q output of the projection)
 *   out   device fp16 [batch][q_len][Hq*hd]
 *   mode  QSVD_ATTN_ABSORBED (latent form), QSVD_ATTN_RECONSTRUCT (K, V
 *         rebuilt per cached token) or QSVD_ATTN_AUTO (absorbed when its shape
 *         is supported)
 *   sm_scale  0 selects 1/sqrt(head_dim)
 *   ws    device workspace of at least qsvd_decode_workspace_size() bytes
 * Requires head_dim % 32 == 0 and <= 128, batch <= 64, q_len <= max_len,
 * w_group 0 or a multiple of 64, 16-byte aligned q, out and s_b (else
 * QSVD_ERR_UNSUPPORTED or QSVD_ERR_INVALID_ARG).  The absorbed form takes
 * n_q_heads <= 64, r in {128, 512, 1024, 1536} (with at most 32 heads) or r
 * a multiple of 128 up to 3072, any cache format, and
 * batch * q_len * ceil(n_q_heads / 16) <= 65535 (batch * q_len <= 65535
 * with 32-head blocks).  The reconstruct form takes n_q_heads <= 64,
 * capacity <= 16384 and any cache format (F16 rows rebuild on the fp16
 * products, I8 on the int8 products, I4 on the 4-bit products), and with
 * q_len > 1 (causal attention of the last q_len positions over the rebuilt
 * rows on the fp16 matrix cores) head_dim 64 or 128.
 * Launch grids are sized from the host c->max_len and every length is read
 * from seq_len on the device, so a call may be captured in a graph and
 * replayed while the cache grows, provided c->max_len at capture is at least
 * every length the replays reach. */
qsvd_status qsvd_latent_decode_attention(const qsvd_layer* w, const qsvd_cache* c,
                                         const void* q, int32_t q_len, int32_t mode,
                                         float sm_scale, void* out,
                                         void* ws, size_t ws_bytes, void* stream);

/* qsvd_latent_decode_attention without a caller workspace, for callers that
 * cannot allocate device memory (code under graph capture, tight serving
 * loops, harnesses that forbid hipMalloc).  Same arguments, forms, results
 * and errors as qsvd_latent_decode_attention (and the same kernels); its
 * partial results live in a static device array of
 * qsvd_noalloc_scratch_bytes() bytes (32 MiB), one per GPU, held from the
 * first call on that GPU until the process ends.  A call whose workspace
 * query exceeds that size returns QSVD_ERR_WORKSPACE before any GPU work.
 * Calls nothing that allocates.  Every call on one GPU shares its array:
 * calls that may overlap on one GPU (other streams, other threads) race and
 * must be ordered by the caller. */
qsvd_status qsvd_latent_decode_attention_noalloc(const qsvd_layer* w, const qsvd_cache* c,
                                                 const void* q, int32_t q_len, int32_t mode,
                                                 float sm_scale, void* out, void* stream);
size_t qsvd_noalloc_scratch_bytes(void);

/* The same attention for layers that apply a rotary position embedding to q
 * and k (the paper's layers have none; this is the position-encoded variant
 * of Section 3.1's decode step).  Every rebuilt key row at position t and the
 * queries at their positions (seq_len[b] - q_len + i) are rotated before the
 * product: each head vector's pairs (j, j + head_dim/2), j < head_dim/2, are
 * turned by the angle t * rope_theta^(-2j/head_dim), formed and reduced
 * modulo one turn in fp64 and evaluated in fp32 (q_len 1: a cos/sin table
 * per call; q_len > 1: the hardware's sine and cosine of the reduced angle in
 * turns).  Values are not rotated.  Because a key then depends on
 * its position, it cannot be folded into the query, so the keys are rebuilt
 * in both forms:
 *   QSVD_ATTN_ABSORBED     K rebuilt and rotated for the scores, the value side
 *                          kept in latent space (sum_t p_t C_t, then W^u_v);
 *                          needs n_q_heads <= 32 and r in {128, 512, 1024, 1536}
 *                          (QSVD_ERR_UNSUPPORTED otherwise)
 *   QSVD_ATTN_RECONSTRUCT  K and V rebuilt, plain attention; needs
 *                          n_q_heads <= 64 and capacity <= 16384; with
 *                          q_len > 1 (query i at position seq_len[b] -
 *                          q_len + i, causal) head_dim 64 or 128
 *   QSVD_ATTN_AUTO         the first where it applies (q_len 1), else the second
 * The latent-value form takes q_len 1 (QSVD_ERR_UNSUPPORTED otherwise).  Both
 * take any cache format (F16, I8, I4), and one workspace size serves both:
 * qsvd_decode_workspace_size(w, c, q_len, QSVD_ATTN_RECONSTRUCT) bytes (the
 * same for every q_len the forms take).  rope_theta must be finite and > 1
 * (QSVD_ERR_INVALID_ARG otherwise). */
qsvd_status qsvd_latent_decode_attention_rope(const qsvd_layer* w, const qsvd_cache* c,
                                              const void* q, int32_t q_len, int32_t mode,
                                              float sm_scale, float rope_theta, void* out,
                                              void* ws, size_t ws_bytes, void* stream);

size_t qsvd_decode_workspace_size(const qsvd_layer* w, const qsvd_cache* c, int32_t q_len,
                                  int32_t mode);

const char* qsvd_status_string(qsvd_status s);
const char* qsvd_last_error(void);

/* Optional kernel timing.  While enabled, every kernel the library launches
 * whose name contains `filter` (all kernels if filter is NULL; the string is
 * copied) is bracketed by HIP events recorded on its launch stream;
 * qsvd_profile_read() synchronizes those events and returns the summed
 * milliseconds and launch count of the recorded kernels whose name contains
 * `name`.  Not for graph capture. */
qsvd_status qsvd_profile_enable(int32_t on, const char* filter);
qsvd_status qsvd_profile_reset(void);
qsvd_status qsvd_profile_read(const char* name, double* total_ms, int64_t* launches);

#ifdef __cplusplus
}
#endif
#endif /* QSVD_H */
