// Latent cache append: only the per-token latent C is buffered (Section 3.1).
#include "common.h"
#include "launch.h"

namespace qsvd {

// One workgroup per (new row, sequence): copy `row_bytes` bytes (a multiple of
// 16) of source row b*n_new + i to position seq_len[b] + i, and its scale.
__global__ void __launch_bounds__(128)
cache_append_kernel(const uint8_t* __restrict__ src, const float* __restrict__ src_scale,
                    uint8_t* __restrict__ dst, float* __restrict__ dst_scale,
                    const int32_t* __restrict__ seq_len, int32_t capacity, int32_t n_new,
                    int32_t row_bytes) {
  const int i = blockIdx.x, b = blockIdx.y;
  const int32_t pos = seq_len[b] + i;
  if (pos < 0 || pos >= capacity) return;
  const int64_t srow = (int64_t)b * n_new + i;
  const int64_t drow = (int64_t)b * capacity + pos;
  const uint4* s = reinterpret_cast<const uint4*>(src + srow * row_bytes);
  uint4* d = reinterpret_cast<uint4*>(dst + drow * row_bytes);
  for (int e = threadIdx.x; e < row_bytes / 16; e += blockDim.x) d[e] = s[e];
  if (dst_scale && threadIdx.x == 0) dst_scale[drow] = src_scale[srow];
}

// New length of a sequence after an append: rows at or past capacity were
// not written, so the length stops at capacity and the overflow flag (if the
// caller gave one) records that rows were dropped.
__device__ __forceinline__ int32_t advanced_len(int32_t base, int32_t n_new, int32_t capacity,
                                                int32_t* __restrict__ overflow) {
  const int64_t want = (int64_t)base + n_new;
  if (want > capacity && overflow) *overflow = 1;
  return want > capacity ? capacity : (int32_t)want;
}

// Decode-sized appends (few rows per sequence): one workgroup per sequence
// copies its rows, then advances seq_len[b] itself after a barrier, so no
// second launch is needed.
__global__ void __launch_bounds__(256)
cache_append_fused_kernel(const uint8_t* __restrict__ src, const float* __restrict__ src_scale,
                          uint8_t* __restrict__ dst, float* __restrict__ dst_scale,
                          int32_t* __restrict__ seq_len, int32_t capacity, int32_t n_new, int32_t row_bytes,
                          int32_t* __restrict__ overflow) {
  const int b = blockIdx.x;
  const int32_t base = seq_len[b];
  const int per_row = row_bytes / 16;
  for (int e = threadIdx.x; e < n_new * per_row; e += blockDim.x) {
    const int i = e / per_row, k = e - i * per_row;
    const int32_t pos = base + i;
    if (pos < 0 || pos >= capacity) continue;
    const int64_t srow = (int64_t)b * n_new + i;
    const int64_t drow = (int64_t)b * capacity + pos;
    reinterpret_cast<uint4*>(dst + drow * row_bytes)[k] = reinterpret_cast<const uint4*>(src + srow * row_bytes)[k];
    if (dst_scale && k == 0) dst_scale[drow] = src_scale[srow];
  }
  __syncthreads();
  if (threadIdx.x == 0) seq_len[b] = advanced_len(base, n_new, capacity, overflow);
}

__global__ void seq_len_advance_kernel(int32_t* __restrict__ seq_len, int32_t batch, int32_t n_new,
                                       int32_t capacity, int32_t* __restrict__ overflow) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b < batch) seq_len[b] = advanced_len(seq_len[b], n_new, capacity, overflow);
}

hipError_t launch_cache_append(const qsvd_cache& c, const void* c_h, const void* cq,
                               const float* sc, int32_t n_new, hipStream_t s) {
  if (n_new == 0 || c.batch == 0) return hipSuccess;
  int32_t row_bytes;
  const void* src;
  if (c.fmt == QSVD_CACHE_F16) {
    row_bytes = c.r * 2;
    src = c_h;
  } else if (c.fmt == QSVD_CACHE_I8) {
    row_bytes = c.r;
    src = cq;
  } else {
    row_bytes = c.r / 2;
    src = cq;
  }
  if (n_new <= 16) {
    KernelScope ks("cache_append", s);
    QSVD_LAUNCH(ks, cache_append_fused_kernel, dim3(c.batch), dim3(256), 0, s, (const uint8_t*)src,
                       c.fmt == QSVD_CACHE_F16 ? nullptr : sc, (uint8_t*)c.data,
                       c.fmt == QSVD_CACHE_F16 ? nullptr : c.scale, c.seq_len, c.capacity, n_new, row_bytes,
                       c.overflow);
    return hipGetLastError();
  }
  {
    KernelScope ks("cache_append", s);
    QSVD_LAUNCH(ks, cache_append_kernel, dim3(n_new, c.batch), dim3(128), 0, s, (const uint8_t*)src,
                       c.fmt == QSVD_CACHE_F16 ? nullptr : sc, (uint8_t*)c.data,
                       c.fmt == QSVD_CACHE_F16 ? nullptr : c.scale, c.seq_len, c.capacity, n_new,
                       row_bytes);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  {
    KernelScope ks("seq_len_advance", s);
    QSVD_LAUNCH(ks, seq_len_advance_kernel, dim3((c.batch + 255) / 256), dim3(256), 0, s, c.seq_len,
                       c.batch, n_new, c.capacity, c.overflow);
  }
  return hipGetLastError();
}

}  // namespace qsvd
