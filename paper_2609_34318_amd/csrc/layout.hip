// Rank-local halves of the Ulysses exchanges and the zigzag ring shard (hydra_layout.h).
//
// All four calls are permutations of 16-byte chunks, bound by HBM bandwidth: every chunk
// is read once and written once.  Each thread moves four chunks per step of a grid-stride
// loop (loads first, then stores) so that enough memory traffic is in flight; consecutive
// threads touch consecutive 16-byte chunks of the destination, and the source runs are
// contiguous for a whole head group (pack / unpack) or a whole chunk of rows (zigzag).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "hydra_layout.h"
#include "prof.h"

namespace hydra {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
constexpr int kUnroll = 4;
constexpr int kThreads = 256;

// Streaming 16-byte accesses: every chunk is touched once, so they bypass cache retention
// (non-temporal), which measured 6.3 against 5.9 TB/s for a plain device copy.
__device__ __forceinline__ u32x4 ld_stream(const u32x4* p) { return __builtin_nontemporal_load(p); }
__device__ __forceinline__ void st_stream(u32x4* p, u32x4 v) { __builtin_nontemporal_store(v, p); }

// Chunk q of the packed side [cp_u][T][g*hb16] <-> chunk of the token side [T][H*hb16].
// INV = false: pack (token side -> packed side), true: unpack.
unsigned grid_for(uint64_t total) {
  const uint64_t per_block = (uint64_t)kThreads * kUnroll;
  const uint64_t want = (total + per_block - 1) / per_block;
  const uint64_t cap = 256ull * 256;  // enough blocks to fill 256 CUs many times over
  return (unsigned)(want < cap ? want : cap);
}

// IDX is the index type: 32-bit divisions whenever the tensor has fewer than 2^32 chunks.
template <bool INV, class IDX>
__global__ __launch_bounds__(kThreads) void pack_heads_kernel(const u32x4* __restrict__ src, u32x4* __restrict__ dst,
                                                              IDX total, uint32_t row16, uint32_t T, uint32_t tok16) {
  // row16 = g*hb16 (one head group of one token), tok16 = H*hb16 (one token, all heads)
  const IDX stride = (IDX)gridDim.x * kThreads * kUnroll;
  for (IDX base = (IDX)blockIdx.x * kThreads * kUnroll + threadIdx.x; base < total; base += stride) {
    u32x4 v[kUnroll];
    IDX other[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const IDX q = base + (IDX)u * kThreads;  // index on the packed side
      const IDX rest = q / row16;
      const uint32_t c = (uint32_t)(q - rest * row16);
      const IDX j = rest / T;
      const uint32_t t = (uint32_t)(rest - j * T);
      other[u] = (IDX)t * tok16 + j * row16 + c;  // index on the token side
      if (q < total) v[u] = ld_stream(src + (INV ? q : other[u]));
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const IDX q = base + (IDX)u * kThreads;
      if (q < total) st_stream(dst + (INV ? other[u] : q), v[u]);
    }
  }
}

template <bool INV>
void launch_pack(const void* src, void* dst, uint64_t total, uint32_t row16, uint32_t T, uint32_t tok16,
                 hipStream_t s) {
  // (total + one grid stride) must stay below 2^32 for the 32-bit form
  if (total + (uint64_t)256 * 256 * kThreads * kUnroll < (uint64_t(1) << 32))
    hipLaunchKernelGGL((pack_heads_kernel<INV, uint32_t>), dim3(grid_for(total)), dim3(kThreads), 0, s,
                       static_cast<const u32x4*>(src), static_cast<u32x4*>(dst), (uint32_t)total, row16, T, tok16);
  else
    hipLaunchKernelGGL((pack_heads_kernel<INV, uint64_t>), dim3(grid_for(total)), dim3(kThreads), 0, s,
                       static_cast<const u32x4*>(src), static_cast<u32x4*>(dst), total, row16, T, tok16);
}

// Two contiguous segments: dst[d_k + i] = src[s_k + i] for i < len (16-byte units),
// segment 0 first, then segment 1.
__global__ __launch_bounds__(kThreads) void copy2_kernel(const u32x4* __restrict__ src, u32x4* __restrict__ dst,
                                                         uint64_t len, uint64_t s0, uint64_t d0, uint64_t s1,
                                                         uint64_t d1) {
  const uint64_t total = 2 * len;
  const uint64_t stride = (uint64_t)gridDim.x * kThreads * kUnroll;
  for (uint64_t base = (uint64_t)blockIdx.x * kThreads * kUnroll + threadIdx.x; base < total; base += stride) {
    u32x4 v[kUnroll];
    uint64_t to[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const uint64_t q = base + (uint64_t)u * kThreads;
      const bool second = q >= len;
      const uint64_t i = second ? q - len : q;
      to[u] = (second ? d1 : d0) + i;
      if (q < total) v[u] = ld_stream(src + (second ? s1 : s0) + i);
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const uint64_t q = base + (uint64_t)u * kThreads;
      if (q < total) st_stream(dst + to[u], v[u]);
    }
  }
}


bool aligned16(const void* p) { return p && (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

// [a, a + alen) and [b, b + blen) share a byte
bool overlap(const void* a, uint64_t alen, const void* b, uint64_t blen) {
  const uintptr_t x = reinterpret_cast<uintptr_t>(a), y = reinterpret_cast<uintptr_t>(b);
  return x < y + blen && y < x + alen;
}

int pack_common(bool inv, int64_t n_tokens, int32_t n_heads, int32_t head_bytes, int32_t cp_u, const void* src,
                void* dst, void* stream) {
  if (n_tokens < 0 || n_heads <= 0 || head_bytes <= 0 || cp_u <= 0) return HYDRA_ERR_INVALID;
  if (n_heads % cp_u != 0 || head_bytes % 16 != 0) return HYDRA_ERR_INVALID;
  // one token with every head, in 16-byte units, must fit 32 bits
  if (n_tokens > (int64_t(1) << 31) || (uint64_t)n_heads * (uint64_t)head_bytes > (uint64_t(1) << 34))
    return HYDRA_ERR_INVALID;
  if (!src || !dst) return HYDRA_ERR_INVALID;
  if (!aligned16(src) || !aligned16(dst)) return HYDRA_ERR_ALIGN;
  const uint64_t bytes = (uint64_t)n_tokens * n_heads * head_bytes;
  if (overlap(src, bytes, dst, bytes)) return HYDRA_ERR_INVALID;
  if (n_tokens == 0) return HYDRA_OK;
  const uint32_t hb16 = head_bytes / 16, g = n_heads / cp_u;
  const uint64_t total = bytes / 16;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int tok = prof_begin(inv ? "unpack_heads" : "pack_heads", s);
  if (inv) launch_pack<true>(src, dst, total, g * hb16, (uint32_t)n_tokens, (uint32_t)n_heads * hb16, s);
  else launch_pack<false>(src, dst, total, g * hb16, (uint32_t)n_tokens, (uint32_t)n_heads * hb16, s);
  prof_end(tok, s);
  return hipGetLastError() == hipSuccess ? HYDRA_OK : HYDRA_ERR_HIP;
}

int zigzag_common(bool scatter, int64_t n_rows, int64_t row_bytes, int32_t cp_r, int32_t r, const void* src,
                  void* dst, void* stream) {
  if (n_rows < 0 || row_bytes <= 0 || cp_r <= 0 || r < 0 || r >= cp_r) return HYDRA_ERR_INVALID;
  if (row_bytes % 16 != 0 || n_rows % (2 * (int64_t)cp_r) != 0) return HYDRA_ERR_INVALID;
  if (n_rows > (int64_t(1) << 40) || row_bytes > (int64_t(1) << 30) || (uint64_t)n_rows * (uint64_t)row_bytes >> 50)
    return HYDRA_ERR_INVALID;
  if (!src || !dst) return HYDRA_ERR_INVALID;
  if (!aligned16(src) || !aligned16(dst)) return HYDRA_ERR_ALIGN;
  const uint64_t shard_bytes = (uint64_t)(n_rows / cp_r) * row_bytes, full_bytes = (uint64_t)n_rows * row_bytes;
  if (overlap(src, scatter ? shard_bytes : full_bytes, dst, scatter ? full_bytes : shard_bytes)) return HYDRA_ERR_INVALID;
  if (n_rows == 0) return HYDRA_OK;
  const uint64_t c16 = (uint64_t)(n_rows / (2 * cp_r)) * (row_bytes / 16);  // one chunk, 16-byte units
  const uint64_t nat0 = (uint64_t)r * c16, nat1 = (uint64_t)(2 * cp_r - 1 - r) * c16;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int tok = prof_begin(scatter ? "zigzag_scatter" : "zigzag_gather", s);
  if (scatter)
    hipLaunchKernelGGL(copy2_kernel, dim3(grid_for(2 * c16)), dim3(kThreads), 0, s, static_cast<const u32x4*>(src),
                       static_cast<u32x4*>(dst), c16, (uint64_t)0, nat0, c16, nat1);
  else
    hipLaunchKernelGGL(copy2_kernel, dim3(grid_for(2 * c16)), dim3(kThreads), 0, s, static_cast<const u32x4*>(src),
                       static_cast<u32x4*>(dst), c16, nat0, (uint64_t)0, nat1, c16);
  prof_end(tok, s);
  return hipGetLastError() == hipSuccess ? HYDRA_OK : HYDRA_ERR_HIP;
}

}  // namespace
}  // namespace hydra

extern "C" {

int hydra_pack_heads(int64_t n_tokens, int32_t n_heads, int32_t head_bytes, int32_t cp_u, const void* src, void* dst,
                     void* stream) {
  return hydra::pack_common(false, n_tokens, n_heads, head_bytes, cp_u, src, dst, stream);
}

int hydra_unpack_heads(int64_t n_tokens, int32_t n_heads, int32_t head_bytes, int32_t cp_u, const void* src,
                       void* dst, void* stream) {
  return hydra::pack_common(true, n_tokens, n_heads, head_bytes, cp_u, src, dst, stream);
}

int hydra_zigzag_gather(int64_t n_rows, int64_t row_bytes, int32_t cp_r, int32_t r, const void* src, void* dst,
                        void* stream) {
  return hydra::zigzag_common(false, n_rows, row_bytes, cp_r, r, src, dst, stream);
}

int hydra_zigzag_scatter(int64_t n_rows, int64_t row_bytes, int32_t cp_r, int32_t r, const void* src, void* dst,
                         void* stream) {
  return hydra::zigzag_common(true, n_rows, row_bytes, cp_r, r, src, dst, stream);
}

}  // extern "C"
