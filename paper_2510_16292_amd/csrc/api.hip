// The C ABI of include/qsvd.h: host-side validation, then launches on the
// caller's stream.  Validation runs before any HIP call, so argument errors are
// reported without touching the GPU.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <mutex>
#include <string>
#include <vector>

#include "common.h"
#include "launch.h"

namespace qsvd {
bool absorbed_supported(const qsvd_layer& w, const qsvd_cache& c);
}

using namespace qsvd;

namespace {

thread_local std::string g_err;

qsvd_status fail(qsvd_status s, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
qsvd_status fail(qsvd_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return s;
}

qsvd_status hip_status(hipError_t e, const char* where) {
  if (e == hipSuccess) return QSVD_OK;
  return fail(QSVD_ERR_HIP, "%s: %s", where, hipGetErrorString(e));
}

bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

int64_t n_total(const qsvd_layer& w) { return (int64_t)(w.n_q_heads + 2 * w.n_kv_heads) * w.head_dim; }

// (sequence, query) rows one attention call takes: the grid's second dimension
constexpr int64_t kMaxQueryRows = 65535;

qsvd_status check_layer(const qsvd_layer* w) {
  if (!w) return fail(QSVD_ERR_INVALID_ARG, "layer is NULL");
  if (w->d <= 0 || w->r <= 0 || w->n_q_heads <= 0 || w->n_kv_heads <= 0 || w->head_dim <= 0)
    return fail(QSVD_ERR_INVALID_ARG, "layer dimensions must be positive");
  if (w->n_q_heads % w->n_kv_heads)
    return fail(QSVD_ERR_INVALID_ARG, "n_q_heads (%d) must be a multiple of n_kv_heads (%d)", w->n_q_heads,
                w->n_kv_heads);
  if (!w->a_t || !w->s_a || !w->b_t || !w->s_b) return fail(QSVD_ERR_INVALID_ARG, "layer weight pointer is NULL");
  if (w->w_bits != 8 && w->w_bits != 4) return fail(QSVD_ERR_INVALID_ARG, "w_bits must be 8 or 4");
  if (w->w_group < 0) return fail(QSVD_ERR_INVALID_ARG, "w_group must be >= 0");
  if (w->w_group > 0 && (w->d % w->w_group || w->r % w->w_group))
    return fail(QSVD_ERR_INVALID_ARG, "w_group must divide d and r");
  if (w->w_bits == 4 && w->w_group == 0)
    return fail(QSVD_ERR_UNSUPPORTED, "int4 weights need a group size");
  if (w->d % 64 || w->r % 64) return fail(QSVD_ERR_UNSUPPORTED, "d and r must be multiples of 64");
  if (w->r > 4096) return fail(QSVD_ERR_UNSUPPORTED, "r must be at most 4096");
  return QSVD_OK;
}

qsvd_status check_cache(const qsvd_cache* c) {
  if (!c) return fail(QSVD_ERR_INVALID_ARG, "cache is NULL");
  if (c->fmt < QSVD_CACHE_F16 || c->fmt > QSVD_CACHE_I4) return fail(QSVD_ERR_INVALID_ARG, "unknown cache format");
  if (c->batch <= 0 || c->capacity <= 0 || c->r <= 0) return fail(QSVD_ERR_INVALID_ARG, "cache sizes must be positive");
  if (c->r % 32) return fail(QSVD_ERR_UNSUPPORTED, "cache r must be a multiple of 32");
  if (!c->data || !c->seq_len) return fail(QSVD_ERR_INVALID_ARG, "cache data/seq_len is NULL");
  if (c->fmt != QSVD_CACHE_F16 && !c->scale) return fail(QSVD_ERR_INVALID_ARG, "integer cache needs scales");
  if (c->max_len < 0 || c->max_len > c->capacity)
    return fail(QSVD_ERR_INVALID_ARG, "max_len %d outside [0, capacity %d]", c->max_len, c->capacity);
  if (!aligned(c->data, 16)) return fail(QSVD_ERR_UNSUPPORTED, "cache data must be 16-byte aligned");
  return QSVD_OK;
}

// ---------------------------------------------------------------- profiler
struct ProfRec {
  std::string name;
  hipEvent_t start, stop;
  bool valid;      // the events were handed to a launch
};
std::mutex g_prof_mu;
bool g_prof_on = false;
std::string g_prof_filter;
std::vector<ProfRec> g_prof;

}  // namespace

namespace qsvd {

KernelScope::KernelScope(const char* name, hipStream_t) : slot_(-1), used_(false), start_(nullptr), stop_(nullptr) {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  if (!g_prof_on) return;
  if (!g_prof_filter.empty() && std::string(name).find(g_prof_filter) == std::string::npos) return;
  ProfRec r{name, nullptr, nullptr, false};
  if (hipEventCreate(&r.start) != hipSuccess) return;
  if (hipEventCreate(&r.stop) != hipSuccess) {
    (void)hipEventDestroy(r.start);
    return;
  }
  start_ = r.start;
  stop_ = r.stop;
  g_prof.push_back(r);
  slot_ = (int)g_prof.size() - 1;
}

hipEvent_t KernelScope::start() {
  used_ = used_ || start_ != nullptr;
  return start_;
}

hipEvent_t KernelScope::stop() { return stop_; }

KernelScope::~KernelScope() {
  if (slot_ < 0) return;
  std::lock_guard<std::mutex> lk(g_prof_mu);
  if (slot_ < (int)g_prof.size() && g_prof[slot_].start == start_) g_prof[slot_].valid = used_;
}

}  // namespace qsvd

extern "C" {

const char* qsvd_status_string(qsvd_status s) {
  switch (s) {
    case QSVD_OK: return "ok";
    case QSVD_ERR_INVALID_ARG: return "invalid argument";
    case QSVD_ERR_UNSUPPORTED: return "unsupported";
    case QSVD_ERR_CAPACITY: return "cache capacity exceeded";
    case QSVD_ERR_WORKSPACE: return "workspace too small";
    case QSVD_ERR_HIP: return "HIP error";
  }
  return "unknown status";
}

const char* qsvd_last_error(void) { return g_err.c_str(); }

qsvd_status qsvd_quantize_act(const void* x, int64_t M, int32_t K, int64_t ldx, int32_t bits, float clip,
                              void* xq, float* sx, void* stream) {
  if (M < 0 || K <= 0 || ldx < K) return fail(QSVD_ERR_INVALID_ARG, "bad sizes M=%lld K=%d ldx=%lld", (long long)M, K, (long long)ldx);
  if (bits != 8 && bits != 4) return fail(QSVD_ERR_INVALID_ARG, "bits must be 8 or 4");
  if (!(clip > 0.f && clip <= 1.f)) return fail(QSVD_ERR_INVALID_ARG, "clip must be in (0, 1]");
  if (M > 0 && (!x || !xq || !sx)) return fail(QSVD_ERR_INVALID_ARG, "NULL pointer");
  if (K % 8 || ldx % 8) return fail(QSVD_ERR_UNSUPPORTED, "K and ldx must be multiples of 8");
  if (!aligned(x, 16) || !aligned(xq, 8)) return fail(QSVD_ERR_UNSUPPORTED, "x must be 16-byte and xq 8-byte aligned");
  return hip_status(launch_quantize_rows(x, M, K, ldx, bits, clip, xq, sx, (hipStream_t)stream), "quantize_act");
}

qsvd_status qsvd_quantize_act_rotated(const void* x, int64_t M, int32_t K, int64_t ldx, int32_t bits, float clip,
                                      const int8_t* signs, int32_t block, void* xq, float* sx, void* stream) {
  if (M < 0 || K <= 0 || ldx < K) return fail(QSVD_ERR_INVALID_ARG, "bad sizes M=%lld K=%d ldx=%lld", (long long)M, K, (long long)ldx);
  if (bits != 8 && bits != 4) return fail(QSVD_ERR_INVALID_ARG, "bits must be 8 or 4");
  if (!(clip > 0.f && clip <= 1.f)) return fail(QSVD_ERR_INVALID_ARG, "clip must be in (0, 1]");
  if (block < 8 || (block & (block - 1)) || K % block)
    return fail(QSVD_ERR_INVALID_ARG, "block must be a power of two >= 8 dividing K");
  if (M > 0 && (!x || !xq || !sx)) return fail(QSVD_ERR_INVALID_ARG, "NULL pointer");
  if (K % 8 || ldx % 8) return fail(QSVD_ERR_UNSUPPORTED, "K and ldx must be multiples of 8");
  if (K > 16384) return fail(QSVD_ERR_UNSUPPORTED, "K must be at most 16384");
  if (!aligned(x, 16) || !aligned(xq, 8) || !aligned(signs, 8))
    return fail(QSVD_ERR_UNSUPPORTED, "x must be 16-byte, xq and signs 8-byte aligned");
  const float c = (float)(1.0 / sqrt((double)block));
  return hip_status(launch_quantize_rotated(x, M, K, ldx, bits, clip, signs, block, c, xq, sx, (hipStream_t)stream),
                    "quantize_act_rotated");
}

static void prefill_ranges(const qsvd_layer& w, uint32_t mask, bool full, int32_t* lo, int32_t* hi) {
  const int32_t nq = w.n_q_heads * w.head_dim, nkv = w.n_kv_heads * w.head_dim;
  const int32_t b0[3] = {0, nq, nq + nkv}, b1[3] = {nq, nq + nkv, nq + 2 * nkv};
  *lo = INT32_MAX;
  *hi = 0;
  for (int s = 0; s < 3; ++s)
    if (mask & (1u << s)) {
      if (b0[s] < *lo) *lo = b0[s];
      if (b1[s] > *hi) *hi = b1[s];
    }
  if (full) {
    *lo = 0;
    *hi = nq + 2 * nkv;
  }
  if (*lo > *hi) *lo = *hi = 0;
}

size_t qsvd_prefill_workspace_size(const qsvd_layer* w, int64_t M, uint32_t out_mask) {
  (void)w;
  (void)M;
  (void)out_mask;
  return 0;   // no kernel of the projection needs device scratch
}

qsvd_status qsvd_lowrank_qkv_prefill(const qsvd_layer* w, const void* xq, const float* sx, int64_t M,
                                     int32_t act_bits, uint32_t out_mask, void* c_h, void* cq, float* sc,
                                     void* q, void* k, void* v, int32_t* dbg_acc_xa, int32_t* dbg_acc_cb,
                                     void* ws, size_t ws_bytes, void* stream) {
  qsvd_status st = check_layer(w);
  if (st != QSVD_OK) return st;
  if (M < 0) return fail(QSVD_ERR_INVALID_ARG, "M must be >= 0");
  if (out_mask & ~7u) return fail(QSVD_ERR_INVALID_ARG, "unknown out_mask bits");
  if (act_bits != 8 && act_bits != 4) return fail(QSVD_ERR_INVALID_ARG, "act_bits must be 8 or 4");
  if (M == 0) return QSVD_OK;
  if (!xq || !sx || !c_h || !cq || !sc) return fail(QSVD_ERR_INVALID_ARG, "NULL input/latent pointer");
  if (((out_mask & QSVD_OUT_Q) && !q) || ((out_mask & QSVD_OUT_K) && !k) || ((out_mask & QSVD_OUT_V) && !v))
    return fail(QSVD_ERR_INVALID_ARG, "requested output pointer is NULL");
  const bool skinny = M <= 32 && skinny_supported(M, w->d, w->w_group, false) &&
                      skinny_supported(M, w->r, w->w_group, true);
  if (act_bits == 4 && (dbg_acc_xa || dbg_acc_cb))
    return fail(QSVD_ERR_UNSUPPORTED, "integer accumulator dumps need 8-bit activations");
  if (w->w_group % 64) return fail(QSVD_ERR_UNSUPPORTED, "w_group must be a multiple of 64");
  // products with 4-bit operands or per-group scales (M > 32)
  const bool mixed = !skinny && (w->w_bits != 8 || w->w_group != 0 || act_bits != 8);
  if (w->w_group && (dbg_acc_xa || dbg_acc_cb))
    return fail(QSVD_ERR_UNSUPPORTED, "integer accumulator dumps need per-channel weights");
  if (!aligned(xq, 16) || !aligned(cq, 16) || !aligned(c_h, 16) || !aligned(w->a_t, 16) || !aligned(w->b_t, 16))
    return fail(QSVD_ERR_UNSUPPORTED, "operands must be 16-byte aligned");
  if (!skinny && (w->head_dim % 8 || !aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16)))
    return fail(QSVD_ERR_UNSUPPORTED, "more than 32 tokens: head_dim a multiple of 8 and 16-byte aligned outputs");
  (void)ws;
  (void)ws_bytes;
  int32_t lo, hi;
  prefill_ranges(*w, out_mask, dbg_acc_cb != nullptr, &lo, &hi);
  const int32_t nq = w->n_q_heads * w->head_dim, nkv = w->n_kv_heads * w->head_dim;
  const int32_t N = nq + 2 * nkv;
  hipStream_t s = (hipStream_t)stream;

  // X W^d -> C (fp16); on the tiled path Q(C) follows in the same call
  GemmArgs g1{};
  g1.a = (const int8_t*)xq;
  g1.b = (const int8_t*)w->a_t;
  g1.row_scale = sx;
  g1.col_scale = w->s_a;
  g1.M = M;
  g1.N = w->r;
  g1.K = w->d;
  g1.seg[0] = OutSeg{(_Float16*)c_h, w->r, 0, w->r};
  g1.n_seg = 1;
  g1.dbg = dbg_acc_xa;
  g1.abits = act_bits;
  if (!skinny) {
    g1.cq = cq;
    g1.sc = sc;
  }
  st = hip_status(skinny  ? launch_skinny(g1, false, w->w_bits, w->w_group, w->r, s)
                  : mixed ? launch_gemm_q4(g1, act_bits, w->w_bits, w->w_group, w->r, s)
                          : launch_gemm_i8(g1, s),
                  "down-projection");
  if (st != QSVD_OK) return st;
  if (hi <= lo) {
    if (!skinny) return QSVD_OK;
    return hip_status(launch_quantize_rows(c_h, M, w->r, w->r, act_bits, 1.f, cq, sc, s, "latent_quant"),
                      "latent quantization");
  }

  // Q(C) W^u -> Q | K | V (fp16) over the columns [lo, hi)
  GemmArgs g2{};
  g2.a = skinny ? (const int8_t*)c_h : (const int8_t*)cq;
  g2.b = (const int8_t*)w->b_t + (int64_t)lo * (w->w_bits == 8 ? w->r : w->r / 2);
  g2.row_scale = sc;
  g2.col_scale = w->s_b + lo;
  g2.M = M;
  g2.N = hi - lo;
  g2.K = w->r;
  g2.seg[0] = OutSeg{(out_mask & QSVD_OUT_Q) ? (_Float16*)q : nullptr, nq, 0 - lo, nq};
  g2.seg[1] = OutSeg{(out_mask & QSVD_OUT_K) ? (_Float16*)k : nullptr, nkv, nq - lo, nkv};
  g2.seg[2] = OutSeg{(out_mask & QSVD_OUT_V) ? (_Float16*)v : nullptr, nkv, nq + nkv - lo, nkv};
  g2.n_seg = 3;
  g2.dbg = dbg_acc_cb;
  g2.abits = act_bits;
  g2.cq = skinny ? cq : nullptr;     // the skinny up-projection quantizes C itself and stores Q(C)
  g2.sc = skinny ? sc : nullptr;
  return hip_status(skinny  ? launch_skinny(g2, true, w->w_bits, w->w_group, N, s)
                    : mixed ? launch_gemm_q4(g2, act_bits, w->w_bits, w->w_group, N, s)
                            : launch_gemm_i8(g2, s),
                    "up-projection");
}

static qsvd_status check_project_append(const qsvd_layer* w, const qsvd_cache* c, const void* x, int64_t ldx,
                                        int32_t act_bits, float clip, const void* xq, const float* sx,
                                        const void* c_h, const void* cq, const float* sc, const void* q) {
  qsvd_status st = check_layer(w);
  if (st != QSVD_OK) return st;
  st = check_cache(c);
  if (st != QSVD_OK) return st;
  if (c->r != w->r) return fail(QSVD_ERR_INVALID_ARG, "cache r %d != layer r %d", c->r, w->r);
  if (act_bits != 8 && act_bits != 4) return fail(QSVD_ERR_INVALID_ARG, "act_bits must be 8 or 4");
  if (!(clip > 0.f && clip <= 1.f)) return fail(QSVD_ERR_INVALID_ARG, "clip must be in (0, 1]");
  if (!x || !xq || !sx || !c_h || !cq || !sc || !q) return fail(QSVD_ERR_INVALID_ARG, "NULL pointer");
  if (ldx < w->d) return fail(QSVD_ERR_INVALID_ARG, "ldx %lld < d %d", (long long)ldx, w->d);
  if ((c->fmt == QSVD_CACHE_I8 && act_bits != 8) || (c->fmt == QSVD_CACHE_I4 && act_bits != 4))
    return fail(QSVD_ERR_UNSUPPORTED, "an integer cache stores Q(C) at the activation width (I8: 8 bits, I4: 4 bits)");
  if ((int64_t)c->max_len + 1 > c->capacity)
    return fail(QSVD_ERR_CAPACITY, "max_len %d + 1 exceeds capacity %d", c->max_len, c->capacity);
  if (w->w_group % 64) return fail(QSVD_ERR_UNSUPPORTED, "w_group must be a multiple of 64");
  const int64_t M = c->batch;
  if (M > 32 || !skinny_supported(M, w->r, w->w_group, true) || !skinny_supported(M, w->d, w->w_group, false))
    return fail(QSVD_ERR_UNSUPPORTED, "the fused decode projection takes at most 32 sequences");
  if (ldx % 8 || !aligned(x, 16) || !aligned(c_h, 16) || !aligned(cq, 16) || !aligned(xq, 16) ||
      !aligned(w->a_t, 16) || !aligned(w->b_t, 16))
    return fail(QSVD_ERR_UNSUPPORTED, "ldx a multiple of 8 and 16-byte aligned x, xq, c_h, cq and weight codes");
  return QSVD_OK;
}

// X W^d -> C (and, for fp16 caches, C's row into the cache): the quantizer of
// the activations runs inside the product when its rows fit the workgroup's
// LDS, else as its own launch first.
static qsvd_status decode_down(const qsvd_layer* w, const qsvd_cache* c, const void* x, int64_t ldx,
                               int32_t act_bits, float clip, void* xq, float* sx, void* c_h, hipStream_t s) {
  const int64_t M = c->batch;
  GemmArgs g1{};
  g1.b = (const int8_t*)w->a_t;
  g1.col_scale = w->s_a;
  g1.M = M;
  g1.N = w->r;
  g1.K = w->d;
  g1.seg[0] = OutSeg{(_Float16*)c_h, w->r, 0, w->r};
  g1.n_seg = 1;
  g1.abits = act_bits;
  SkinnyAppendArgs a1{c->data, c->scale, c->seq_len, c->overflow, c->capacity,
                      c->fmt == QSVD_CACHE_F16 ? 1 : 0};
  if (skinny_supported(M, w->d, w->w_group, true)) {
    g1.a = (const int8_t*)x;
    g1.cq = xq;
    g1.sc = sx;
    return hip_status(launch_skinny_fused(g1, SKA_F16_ACT, clip, ldx, w->w_bits, w->w_group, w->r, a1, s),
                      "decode down-projection");
  }
  qsvd_status st = hip_status(launch_quantize_rows(x, M, w->d, ldx, act_bits, clip, xq, sx, s), "quantize_act");
  if (st != QSVD_OK) return st;
  g1.a = (const int8_t*)xq;
  g1.row_scale = sx;
  return hip_status(launch_skinny_fused(g1, SKA_CODES, 1.f, w->d, w->w_bits, w->w_group, w->r, a1, s),
                    "decode down-projection");
}

// The cache update of the up-projection: the Q(C) row of integer caches and
// the length advance (fp16 caches got their row from the down-projection).
static SkinnyAppendArgs up_append(const qsvd_cache* c) {
  return SkinnyAppendArgs{c->data, c->scale, c->seq_len, c->overflow, c->capacity, c->fmt == QSVD_CACHE_F16 ? 3 : 2};
}

qsvd_status qsvd_decode_project_append(const qsvd_layer* w, qsvd_cache* c, const void* x, int64_t ldx,
                                       int32_t act_bits, float clip, void* xq, float* sx, void* c_h, void* cq,
                                       float* sc, void* q, void* stream) {
  qsvd_status st = check_project_append(w, c, x, ldx, act_bits, clip, xq, sx, c_h, cq, sc, q);
  if (st != QSVD_OK) return st;
  hipStream_t s = (hipStream_t)stream;
  st = decode_down(w, c, x, ldx, act_bits, clip, xq, sx, c_h, s);
  if (st != QSVD_OK) return st;

  // Q(C) W^u_q -> Q, with the cache row (integer caches) and the length advance
  const int32_t nq = w->n_q_heads * w->head_dim;
  const int32_t N = nq + 2 * w->n_kv_heads * w->head_dim;
  GemmArgs g2{};
  g2.a = (const int8_t*)c_h;
  g2.b = (const int8_t*)w->b_t;
  g2.col_scale = w->s_b;
  g2.M = c->batch;
  g2.N = nq;
  g2.K = w->r;
  g2.seg[0] = OutSeg{(_Float16*)q, nq, 0, nq};
  g2.n_seg = 1;
  g2.abits = act_bits;
  g2.cq = cq;
  g2.sc = sc;
  st = hip_status(launch_skinny_fused(g2, SKA_F16_LATENT, 1.f, w->r, w->w_bits, w->w_group, N, up_append(c), s),
                  "decode up-projection");
  if (st == QSVD_OK) c->max_len += 1;
  return st;
}

qsvd_status qsvd_latent_cache_append(qsvd_cache* c, const void* c_h, const void* cq, const float* sc,
                                     int32_t n_new, void* stream) {
  qsvd_status st = check_cache(c);
  if (st != QSVD_OK) return st;
  if (n_new < 0) return fail(QSVD_ERR_INVALID_ARG, "n_new must be >= 0");
  if (n_new == 0) return QSVD_OK;
  if (c->fmt == QSVD_CACHE_F16 && !c_h) return fail(QSVD_ERR_INVALID_ARG, "fp16 cache needs c_h");
  if (c->fmt != QSVD_CACHE_F16 && (!cq || !sc)) return fail(QSVD_ERR_INVALID_ARG, "integer cache needs cq and sc");
  if ((int64_t)c->max_len + n_new > c->capacity)
    return fail(QSVD_ERR_CAPACITY, "max_len %d + %d exceeds capacity %d", c->max_len, n_new, c->capacity);
  const void* src = c->fmt == QSVD_CACHE_F16 ? c_h : cq;
  if (!aligned(src, 16)) return fail(QSVD_ERR_UNSUPPORTED, "source rows must be 16-byte aligned");
  st = hip_status(launch_cache_append(*c, c_h, cq, sc, n_new, (hipStream_t)stream), "cache append");
  if (st == QSVD_OK) c->max_len += n_new;
  return st;
}

static qsvd_status prefill_attention(const void* q, const void* k, const void* v, int32_t batch,
                                     const int32_t* cu_seqlens, int32_t max_seqlen, int32_t n_q_heads,
                                     int32_t n_kv_heads, int32_t head_dim, float sm_scale, float rope_theta, void* out,
                                     void* stream) {
  if (batch < 0 || max_seqlen < 0) return fail(QSVD_ERR_INVALID_ARG, "batch and max_seqlen must be >= 0");
  if (n_q_heads <= 0 || n_kv_heads <= 0 || head_dim <= 0) return fail(QSVD_ERR_INVALID_ARG, "head sizes must be positive");
  if (n_q_heads % n_kv_heads)
    return fail(QSVD_ERR_INVALID_ARG, "n_q_heads (%d) must be a multiple of n_kv_heads (%d)", n_q_heads, n_kv_heads);
  if (!(sm_scale >= 0.f) || isinf(sm_scale)) return fail(QSVD_ERR_INVALID_ARG, "sm_scale must be finite and >= 0");
  if (batch == 0 || max_seqlen == 0) return QSVD_OK;
  if (!q || !k || !v || !out || !cu_seqlens) return fail(QSVD_ERR_INVALID_ARG, "NULL pointer");
  if (!prefill_attention_supported(head_dim)) return fail(QSVD_ERR_UNSUPPORTED, "head_dim must be 64 or 128");
  if (!aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16) || !aligned(out, 16))
    return fail(QSVD_ERR_UNSUPPORTED, "q, k, v and out must be 16-byte aligned");
  if ((int64_t)batch * n_q_heads * ((max_seqlen + 127) / 128) > INT32_MAX)
    return fail(QSVD_ERR_UNSUPPORTED, "batch * n_q_heads * ceil(max_seqlen / 128) exceeds the grid");
  PrefillAttnArgs a{(const _Float16*)q, (const _Float16*)k, (const _Float16*)v, cu_seqlens, batch, max_seqlen,
                    n_q_heads, n_kv_heads, head_dim, sm_scale > 0.f ? sm_scale : 1.f / sqrtf((float)head_dim),
                    (_Float16*)out, rope_theta};
  return hip_status(launch_prefill_attention(a, (hipStream_t)stream), "prefill attention");
}

qsvd_status qsvd_prefill_attention(const void* q, const void* k, const void* v, int32_t batch,
                                   const int32_t* cu_seqlens, int32_t max_seqlen, int32_t n_q_heads,
                                   int32_t n_kv_heads, int32_t head_dim, float sm_scale, void* out, void* stream) {
  return prefill_attention(q, k, v, batch, cu_seqlens, max_seqlen, n_q_heads, n_kv_heads, head_dim, sm_scale, 0.f,
                           out, stream);
}

qsvd_status qsvd_prefill_attention_rope(const void* q, const void* k, const void* v, int32_t batch,
                                        const int32_t* cu_seqlens, int32_t max_seqlen, int32_t n_q_heads,
                                        int32_t n_kv_heads, int32_t head_dim, float sm_scale, float rope_theta,
                                        void* out, void* stream) {
  if (!(rope_theta > 1.f) || isinf(rope_theta)) return fail(QSVD_ERR_INVALID_ARG, "rope_theta must be finite and > 1");
  return prefill_attention(q, k, v, batch, cu_seqlens, max_seqlen, n_q_heads, n_kv_heads, head_dim, sm_scale,
                           rope_theta, out, stream);
}

size_t qsvd_decode_workspace_size(const qsvd_layer* w, const qsvd_cache* c, int32_t q_len, int32_t mode) {
  if (!w || !c || q_len < 1) return 0;
  if (c->batch <= 0 || c->capacity <= 0 || w->r <= 0) return 0;
  if ((int64_t)c->batch * q_len > kMaxQueryRows) return 0;
  const bool abs_ok = absorbed_supported(*w, *c);
  if (mode == QSVD_ATTN_RECONSTRUCT || (mode == QSVD_ATTN_AUTO && !abs_ok))
    return q_len == 1 || prefill_attention_supported(w->head_dim) ? attn_reconstruct_workspace(*w, *c) : 0;
  if (absorbed_grid_rows(*w, *c, q_len) > kMaxQueryRows) return 0;
  return attn_absorbed_workspace(*w, *c, q_len);
}

// ---------------------------------------------------------------- static scratch
// Device scratch of the allocation-free decode attention: one array per GPU,
// held until the process ends.  Host code never passes `scratch` itself to a
// kernel (in host code the name is a host-side stand-in); it uses the device
// address that hipGetSymbolAddress returns for the current device, looked up
// once per device.
constexpr size_t kScratchBytes = (size_t)32 << 20;
static __device__ __align__(256) uint8_t scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
static std::mutex g_scratch_mu;
static void* g_scratch_ptr[kMaxDevices] = {};

static qsvd_status scratch_address(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_status(e, "static scratch: hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices) return fail(QSVD_ERR_UNSUPPORTED, "device %d beyond the scratch table", dev);
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_status(e, "static scratch: hipGetSymbolAddress");
    if (!p) return fail(QSVD_ERR_HIP, "static scratch: NULL symbol address");
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return QSVD_OK;
}

// use_scratch: the workspace is the device's static scratch array instead of
// the caller's (ws, ws_bytes are then ignored).
static qsvd_status decode_attention(const qsvd_layer* w, const qsvd_cache* c, const void* q, int32_t q_len,
                                    int32_t mode, float sm_scale, float rope_theta, void* out, void* ws,
                                    size_t ws_bytes, void* stream, bool use_scratch = false) {
  qsvd_status st = check_layer(w);
  if (st != QSVD_OK) return st;
  st = check_cache(c);
  if (st != QSVD_OK) return st;
  if (c->r != w->r) return fail(QSVD_ERR_INVALID_ARG, "cache r %d != layer r %d", c->r, w->r);
  if (!q || !out) return fail(QSVD_ERR_INVALID_ARG, "NULL q/out");
  if (mode < QSVD_ATTN_AUTO || mode > QSVD_ATTN_RECONSTRUCT) return fail(QSVD_ERR_INVALID_ARG, "unknown mode");
  if (!(sm_scale >= 0.f) || isinf(sm_scale)) return fail(QSVD_ERR_INVALID_ARG, "sm_scale must be finite and >= 0");
  if (q_len < 1) return fail(QSVD_ERR_INVALID_ARG, "q_len must be >= 1");
  if ((int64_t)c->batch * q_len > kMaxQueryRows)
    return fail(QSVD_ERR_UNSUPPORTED, "batch * q_len must be at most %d", (int)kMaxQueryRows);
  if (c->max_len < q_len) return fail(QSVD_ERR_INVALID_ARG, "cache holds %d tokens, fewer than q_len %d", c->max_len, q_len);
  if (w->n_q_heads > 64) return fail(QSVD_ERR_UNSUPPORTED, "at most 64 query heads");
  if (w->head_dim % 32 || w->head_dim > 128) return fail(QSVD_ERR_UNSUPPORTED, "head_dim must be 32, 64, 96 or 128");
  if (c->batch > 64) return fail(QSVD_ERR_UNSUPPORTED, "at most 64 sequences per call");
  if (w->w_group % 64) return fail(QSVD_ERR_UNSUPPORTED, "decode attention needs w_group 0 or a multiple of 64");
  if (!aligned(q, 16) || !aligned(out, 16) || !aligned(w->s_b, 16))
    return fail(QSVD_ERR_UNSUPPORTED, "q, out and s_b must be 16-byte aligned");
  const bool rope = rope_theta > 0.f;
  // Rotary layers: ABSORBED is the form with the value side in latent space
  // (the keys must be rebuilt and turned per position); RECONSTRUCT rebuilds
  // K and V.
  const bool abs_ok = rope ? rope_latent_supported(*w, *c) : absorbed_supported(*w, *c);
  if (mode == QSVD_ATTN_ABSORBED && !abs_ok)
    return fail(QSVD_ERR_UNSUPPORTED, rope ? "the rotary latent-value form needs n_q_heads <= 32 and r in {128, 512, 1024, 1536}"
                                           : "absorbed form needs r in {128, 512, 1024, 1536} or a multiple of 128 up to 3072");
  // the rotary latent-value form takes one query per sequence; AUTO then rebuilds K and V
  const bool absorbed = mode == QSVD_ATTN_ABSORBED || (mode == QSVD_ATTN_AUTO && abs_ok && !(rope && q_len > 1));
  if (absorbed && absorbed_grid_rows(*w, *c, q_len) > kMaxQueryRows)
    return fail(QSVD_ERR_UNSUPPORTED, "batch * q_len * head blocks must be at most %d", (int)kMaxQueryRows);
  if (absorbed && rope && q_len != 1) return fail(QSVD_ERR_UNSUPPORTED, "the rotary latent-value form takes q_len 1 only");
  if (!absorbed && q_len != 1 && !prefill_attention_supported(w->head_dim))
    return fail(QSVD_ERR_UNSUPPORTED, "the reconstruct form with q_len > 1 needs head_dim 64 or 128");
  if (!absorbed && c->capacity > 16384)
    return fail(QSVD_ERR_UNSUPPORTED, "reconstruct form supports capacity <= 16384");
  const size_t need = absorbed && !rope ? attn_absorbed_workspace(*w, *c, q_len) : attn_reconstruct_workspace(*w, *c);
  if (use_scratch) {
    if (need > kScratchBytes)
      return fail(QSVD_ERR_WORKSPACE, "this call needs %zu bytes of scratch, more than the %zu-byte static array",
                  need, kScratchBytes);
    st = scratch_address(&ws);
    if (st != QSVD_OK) return st;
    ws_bytes = kScratchBytes;
  }
  if (!ws || ws_bytes < need) return fail(QSVD_ERR_WORKSPACE, "workspace %zu < %zu bytes", ws_bytes, need);
  AttnArgs a{w, c, (const _Float16*)q, (_Float16*)out, sm_scale > 0.f ? sm_scale : 1.f / sqrtf((float)w->head_dim),
             q_len, rope ? rope_theta : 0.f};
  hipStream_t s = (hipStream_t)stream;
  const hipError_t e = !absorbed ? launch_attn_reconstruct(a, ws, s)
                       : rope    ? launch_attn_rope_latent(a, ws, s)
                                 : launch_attn_absorbed(a, ws, s);
  return hip_status(e, "decode attention");
}

qsvd_status qsvd_latent_decode_attention(const qsvd_layer* w, const qsvd_cache* c, const void* q, int32_t q_len,
                                         int32_t mode, float sm_scale, void* out, void* ws, size_t ws_bytes,
                                         void* stream) {
  return decode_attention(w, c, q, q_len, mode, sm_scale, 0.f, out, ws, ws_bytes, stream);
}

qsvd_status qsvd_latent_decode_attention_noalloc(const qsvd_layer* w, const qsvd_cache* c, const void* q,
                                                 int32_t q_len, int32_t mode, float sm_scale, void* out,
                                                 void* stream) {
  return decode_attention(w, c, q, q_len, mode, sm_scale, 0.f, out, nullptr, 0, stream, true);
}

size_t qsvd_noalloc_scratch_bytes(void) { return kScratchBytes; }

qsvd_status qsvd_latent_decode_attention_rope(const qsvd_layer* w, const qsvd_cache* c, const void* q, int32_t q_len,
                                              int32_t mode, float sm_scale, float rope_theta, void* out, void* ws,
                                              size_t ws_bytes, void* stream) {
  if (!(rope_theta > 1.f) || isinf(rope_theta)) return fail(QSVD_ERR_INVALID_ARG, "rope_theta must be finite and > 1");
  return decode_attention(w, c, q, q_len, mode, sm_scale, rope_theta, out, ws, ws_bytes, stream);
}

qsvd_status qsvd_profile_enable(int32_t on, const char* filter) {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  g_prof_on = on != 0;
  g_prof_filter = filter ? filter : "";
  return QSVD_OK;
}

qsvd_status qsvd_profile_reset(void) {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  for (auto& r : g_prof) {
    (void)hipEventDestroy(r.start);
    (void)hipEventDestroy(r.stop);
  }
  g_prof.clear();
  return QSVD_OK;
}

qsvd_status qsvd_profile_read(const char* name, double* total_ms, int64_t* launches) {
  if (!name || !total_ms || !launches) return fail(QSVD_ERR_INVALID_ARG, "NULL argument");
  std::lock_guard<std::mutex> lk(g_prof_mu);
  double tot = 0.0;
  int64_t n = 0;
  for (auto& r : g_prof) {
    if (!r.valid || r.name.find(name) == std::string::npos) continue;
    hipError_t e = hipEventSynchronize(r.stop);
    if (e != hipSuccess) return hip_status(e, "profile read");
    float ms = 0.f;
    e = hipEventElapsedTime(&ms, r.start, r.stop);
    if (e != hipSuccess) return hip_status(e, "profile read");
    tot += ms;
    ++n;
  }
  *total_ms = tot;
  *launches = n;
  return QSVD_OK;
}

}  // extern "C"
