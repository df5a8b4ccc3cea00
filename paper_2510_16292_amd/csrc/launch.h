// Internal host-side launch wrappers (validated arguments only).
#pragma once
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "qsvd.h"

namespace qsvd {

// Kernel timing for the profiler (api.hip): when it is enabled for this name,
// start() and stop() are events that hipExtLaunchKernelGGL stamps with the
// kernel's own start and end times; otherwise they are NULL.  Every profiled
// launch goes through QSVD_LAUNCH.
struct KernelScope {
  KernelScope(const char* name, hipStream_t s);
  ~KernelScope();
  hipEvent_t start();
  hipEvent_t stop();
  int slot_;
  bool used_;
  hipEvent_t start_, stop_;
};

#define QSVD_LAUNCH(ks, kern, grid, block, lds, stream, ...) \
  hipExtLaunchKernelGGL(kern, grid, block, (std::uint32_t)(lds), stream, (ks).start(), (ks).stop(), 0, __VA_ARGS__)

// `name` is the profiler's name of the launch (the latent quantization Q(C)
// inside a projection call is "latent_quant").
hipError_t launch_quantize_rows(const void* x, int64_t M, int32_t K, int64_t ldx, int32_t bits,
                                float clip, void* xq, float* sx, hipStream_t s,
                                const char* name = "quantize_rows");
// Q(X H1^T) for H1 = blockdiag(H_block) diag(signs) / sqrt(block); c = fp32(1/sqrt(block)).
hipError_t launch_quantize_rotated(const void* x, int64_t M, int32_t K, int64_t ldx, int32_t bits, float clip,
                                   const int8_t* signs, int32_t block, float c, void* xq, float* sx,
                                   hipStream_t s);

// C[m][n] = sum_k A[m][k] * B[n][k] for int8 A [M][K] and int8 B [N][K], scaled
// per row and per column, written to up to three fp16 column segments.
struct OutSeg {
  _Float16* ptr;   // NULL: columns of this segment are not stored
  int64_t ld;      // row stride of ptr in elements
  int32_t n0;      // first column of the segment in the full product
  int32_t n;       // columns in the segment
};
struct GemmArgs {
  const int8_t* a;      // [M][K]
  const int8_t* b;      // [N][K] (rows n_begin.. of the weight)
  const float* row_scale;
  const float* col_scale;
  int64_t M;
  int32_t N;            // columns computed
  int32_t K;
  OutSeg seg[3];
  int32_t n_seg;
  int32_t* dbg;         // optional int32 [M][N]
  // Down-projection only: when cq is set, the fp16 result (segment 0, ld == N)
  // is also quantized per row with abits into cq / sc.
  void* cq;
  float* sc;
  int32_t abits;
};
// Rotary scores straight from a key-rebuild product (the fused form of the
// rotary decode's scores): product row m0 + i is cache position t of sequence
// b ((row0 + m) = b * capacity + t); each head's dh columns of the dequantized
// fp16 row are turned at position t with the (cos, sin) table rope[t][dh/2],
// rounded to fp16 and dotted in fp32 with the G turned, scaled queries
// qrot[b][Hq][dh] of its query heads; pre[b][t][32] receives the scores
// (heads Hq .. 31 zero), positions t >= seq_len[b] are skipped.
struct RopeEpi {
  const float* qrot;
  const float2* rope;
  const int32_t* seq_len;
  float* pre;
  int64_t row0;
  int32_t capacity, Hq, G, dh;
};

// Tiled int8 GEMM for M > 32 (prefill); with g.cq set, the fp16 result is also
// quantized per row into g.cq / g.sc.
hipError_t launch_gemm_i8(const GemmArgs& g, hipStream_t s);
// The same pipeline over fp16 operands (a: fp16 [M][K], b: fp16 [N][K], K in
// elements, a multiple of 32), fp32 accumulation, then (acc * row_scale) *
// col_scale with NULL scale vectors read as 1; no accumulator dumps or row
// quantization.
hipError_t launch_gemm_f16(const GemmArgs& g, hipStream_t s);
// The int8 (f16 false) or fp16 product of a key rebuild with the rotary-score
// epilogue instead of stores: N = n_kv_heads * dh, dh dividing the 128- or
// 256-column tile (32, 64 or 128).
hipError_t launch_gemm_rope_scores(const GemmArgs& g, const RopeEpi& re, bool f16, hipStream_t s);

// The same products with 4-bit activations and/or int4 weights, per-channel or
// per-group (group contraction elements, a multiple of 64; scale of group g
// for column n at col_scale[g * sstride + n]).
hipError_t launch_gemm_q4(const GemmArgs& g, int32_t abits, int32_t wbits, int32_t group, int32_t sstride,
                          hipStream_t s);

// Decode-size products (M <= 32): A is int8 codes, or (a_is_f16_latent) the
// fp16 latent quantized per row inside the kernel, which then also writes
// g.cq / g.sc.  Weights int8 or int4 (grouped, scale row stride sstride).
// Whether the decode-size kernel takes M rows over a contraction of K (A from
// int8 codes, or f16q: from the fp16 latent, quantized on the fly).
bool skinny_supported(int64_t M, int32_t K, int32_t group, bool f16q);
hipError_t launch_skinny(const GemmArgs& g, bool a_is_f16_latent, int32_t wbits, int32_t group, int32_t sstride,
                         hipStream_t s);

// The decode step's fused variants (one new row per sequence, M = batch):
// A from fp16 rows quantized in the kernel (the activations X with `clip`,
// row stride lda, codes and scales optionally stored to g.cq / g.sc; or the
// latent C with clip 1), and the latent cache append folded in (mode
// SK_APPEND_* of skinny.hip: the fp16 C row from the down-projection; the
// Q(C) codes and the seq_len advance from the up-projection).
enum { SKA_CODES = 0, SKA_F16_LATENT = 1, SKA_F16_ACT = 2 };
struct SkinnyAppendArgs {
  void* data;
  float* scale;
  int32_t* seq_len;
  int32_t* overflow;
  int32_t capacity;
  int32_t mode;        // 0: none
};
hipError_t launch_skinny_fused(const GemmArgs& g, int32_t asrc, float clip, int64_t lda, int32_t wbits, int32_t group,
                               int32_t sstride, const SkinnyAppendArgs& aa, hipStream_t s);

hipError_t launch_cache_append(const qsvd_cache& c, const void* c_h, const void* cq,
                               const float* sc, int32_t n_new, hipStream_t s);

struct AttnArgs {
  const qsvd_layer* w;
  const qsvd_cache* c;
  const _Float16* q;      // [batch][q_len][Hq * head_dim]
  _Float16* out;          // same layout
  float sm_scale;
  int32_t q_len;          // queries per sequence: the last q_len cached positions, causal among them
  float rope_theta;       // > 0: rotary embedding of q and the rebuilt K (the two reconstruct-side forms)
};
size_t attn_absorbed_workspace(const qsvd_layer& w, const qsvd_cache& c, int32_t q_len);
// Rows of the absorbed attention grid: (sequence, query) rows times head blocks.
int64_t absorbed_grid_rows(const qsvd_layer& w, const qsvd_cache& c, int32_t q_len);
hipError_t launch_attn_absorbed(const AttnArgs& a, void* ws, hipStream_t s);
// Workspace of either reconstruct-side form (the larger of the two).
size_t attn_reconstruct_workspace(const qsvd_layer& w, const qsvd_cache& c);
// K^ and V^ rebuilt for every cached token, plain attention over them.
hipError_t launch_attn_reconstruct(const AttnArgs& a, void* ws, hipStream_t s);
// Rotary layers: K^ rebuilt and rotated for the scores, the value side in
// latent space (32-head plans: n_q_heads <= 32, r in {128, 512, 1024, 1536}).
bool rope_latent_supported(const qsvd_layer& w, const qsvd_cache& c);
hipError_t launch_attn_rope_latent(const AttnArgs& a, void* ws, hipStream_t s);

// Causal prefill attention over the projection's own Q, K, V (token-major,
// sequences back to back at cu_seqlens).
struct PrefillAttnArgs {
  const _Float16* q;        // [M][n_q_heads * head_dim]
  const _Float16* k;        // [M][n_kv_heads * head_dim]
  const _Float16* v;
  const int32_t* cu_seqlens;  // device [batch + 1]
  int32_t batch, max_seqlen, n_q_heads, n_kv_heads, head_dim;
  float sm_scale;
  _Float16* out;            // [M][n_q_heads * head_dim]
  float rope_theta;         // > 0: rotary layer (q and k turned at their positions)
};
bool prefill_attention_supported(int32_t head_dim);
hipError_t launch_prefill_attention(const PrefillAttnArgs& a, hipStream_t s);

struct CacheAttnArgs {
  const _Float16* q;        // [batch][q_len][n_q_heads * head_dim]
  const _Float16* kv;       // rebuilt rows [batch][capacity][2 * n_kv_heads * head_dim]: K^ then V^
  const int32_t* seq_len;   // device [batch]
  int32_t batch, capacity, q_len, n_q_heads, n_kv_heads, head_dim;
  float sm_scale, rope_theta;
  _Float16* out;            // [batch][q_len][n_q_heads * head_dim]
};
hipError_t launch_cache_attention(const CacheAttnArgs& c, hipStream_t s);

}  // namespace qsvd
