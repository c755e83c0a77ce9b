// The gated attention output fused with the reverse Ulysses exchange (hydra_gate.h).
//
// Both calls are elementwise over the [T][H][d_v] output, bound by HBM bandwidth: every
// byte is read once and written once (forward 6 bytes per element with a per-channel gate,
// backward 10).  The loop walks the packed side [cp_u][T][H/cp_u][d_v] in 16-byte chunks
// of 8 bf16, as the plain pack / unpack do; consecutive threads touch consecutive chunks,
// and the token-side runs are contiguous for a whole head group.  With one logit per
// (token, head) the d_v/8 chunks of a head sit in consecutive lanes of one wave, so the
// backward's sum over the channels is a butterfly over those lanes.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "hydra_gate.h"
#include "prof.h"

namespace hydra {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8v __attribute__((ext_vector_type(8)));
constexpr int kUnroll = 4;
constexpr int kThreads = 256;

// Streaming 16-byte accesses: every chunk is touched once, so they bypass cache retention
// (non-temporal).
__device__ __forceinline__ u32x4 ld_stream(const u32x4* p) { return __builtin_nontemporal_load(p); }
__device__ __forceinline__ void st_stream(u32x4* p, u32x4 v) { __builtin_nontemporal_store(v, p); }

unsigned grid_for(uint64_t total) {
  const uint64_t per_block = (uint64_t)kThreads * kUnroll;
  const uint64_t want = (total + per_block - 1) / per_block;
  const uint64_t cap = 256ull * 256;
  return (unsigned)(want < cap ? want : cap);
}

// 8 bf16 -> 8 fp32 (exact)
__device__ __forceinline__ f32x8 widen(u32x4 v) {
  f32x8 r;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    r[2 * i] = __uint_as_float(v[i] << 16);
    r[2 * i + 1] = __uint_as_float(v[i] & 0xffff0000u);
  }
  return r;
}

// 8 fp32 -> 8 bf16, round to nearest even (v_cvt_pk_bf16_f32)
__device__ __forceinline__ u32x4 narrow(f32x8 x) { return __builtin_bit_cast(u32x4, __builtin_convertvector(x, bf16x8v)); }

__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float(uint32_t(h) << 16); }

// s = 1 / (1 + e^-g) and 1 - s without overflow or cancellation: with e = e^-|g| in (0, 1],
// the pair is (1/(1+e), e/(1+e)) for g >= 0 and swapped for g < 0.
__device__ __forceinline__ void logistic(float g, float& s, float& om) {
  const float e = __builtin_amdgcn_exp2f(-fabsf(g) * 1.4426950408889634f);
  const float r = __builtin_amdgcn_rcpf(1.f + e);
  const float er = e * r;
  s = g >= 0.f ? r : er;
  om = g >= 0.f ? er : r;
}

// BWD = false: out[token side] = in[packed side] * s.
// BWD = true:  out[packed side] = in[token side] * s, and the gate gradient.
// HEADWISE: one logit per (token, head); lg16 = log2(d_v / 8) chunks per head.
template <bool BWD, bool HEADWISE, class IDX>
__global__ __launch_bounds__(kThreads) void gate_kernel(const u32x4* __restrict__ in, const u32x4* __restrict__ yg,
                                                        const void* __restrict__ gate, u32x4* __restrict__ out,
                                                        void* __restrict__ dgate, IDX total, uint32_t row16,
                                                        uint32_t T, uint32_t tok16, uint32_t lg16) {
  const IDX stride = (IDX)gridDim.x * kThreads * kUnroll;
  const uint32_t hb16 = 1u << lg16;
  for (IDX base = (IDX)blockIdx.x * kThreads * kUnroll + threadIdx.x; base < total; base += stride) {
    u32x4 a[kUnroll], b[kUnroll], gv[kUnroll];
    IDX other[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const IDX q = base + (IDX)u * kThreads;  // index on the packed side
      const IDX rest = q / row16;
      const uint32_t c = (uint32_t)(q - rest * row16);
      const IDX j = rest / T;
      const uint32_t t = (uint32_t)(rest - j * T);
      other[u] = (IDX)t * tok16 + j * row16 + c;  // index on the token side
      if (q < total) {
        a[u] = ld_stream(in + (BWD ? other[u] : q));
        if (BWD) b[u] = ld_stream(yg + other[u]);
        if (HEADWISE) gv[u][0] = static_cast<const uint16_t*>(gate)[other[u] >> lg16];
        else gv[u] = ld_stream(static_cast<const u32x4*>(gate) + other[u]);
      } else {
        a[u] = u32x4{0, 0, 0, 0};
        b[u] = a[u];
        gv[u] = a[u];
      }
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const IDX q = base + (IDX)u * kThreads;
      const f32x8 x = widen(a[u]);
      f32x8 s8, om8;
      if (HEADWISE) {
        float s, om;
        logistic(bf16_to_f32((uint16_t)gv[u][0]), s, om);
#pragma unroll
        for (int i = 0; i < 8; ++i) s8[i] = s, om8[i] = om;
      } else {
        const f32x8 g = widen(gv[u]);
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          float s, om;
          logistic(g[i], s, om);
          s8[i] = s;
          om8[i] = om;
        }
      }
      const u32x4 res = narrow(x * s8);
      if (!BWD) {
        if (q < total) st_stream(out + other[u], res);
        continue;
      }
      if (q < total) st_stream(out + q, res);
      const f32x8 p = x * widen(b[u]);  // dY' * Y'
      if (HEADWISE) {
        // The chunks of one head are hb16 consecutive lanes starting at a multiple of hb16
        // (q = lane mod 256, and total is a multiple of hb16), all in range or all out.
        float sum = ((p[0] + p[1]) + (p[2] + p[3])) + ((p[4] + p[5]) + (p[6] + p[7]));
        for (uint32_t m = 1; m < hb16; m <<= 1) sum += __shfl_xor(sum, (int)m, 64);
        if (q < total && (q & (hb16 - 1)) == 0) {
          const __bf16 r = (__bf16)(sum * om8[0]);
          static_cast<__bf16*>(dgate)[other[u] >> lg16] = r;
        }
      } else if (q < total) {
        st_stream(static_cast<u32x4*>(dgate) + other[u], narrow(p * om8));
      }
    }
  }
}

template <bool BWD, bool HEADWISE>
void launch(const void* in, const void* yg, const void* gate, void* out, void* dgate, uint64_t total, uint32_t row16,
            uint32_t T, uint32_t tok16, uint32_t lg16, hipStream_t s) {
  const dim3 grid(grid_for(total)), block(kThreads);
  const u32x4* i4 = static_cast<const u32x4*>(in);
  const u32x4* y4 = static_cast<const u32x4*>(yg);
  u32x4* o4 = static_cast<u32x4*>(out);
  if (total + (uint64_t)256 * 256 * kThreads * kUnroll < (uint64_t(1) << 32))
    hipLaunchKernelGGL((gate_kernel<BWD, HEADWISE, uint32_t>), grid, block, 0, s, i4, y4, gate, o4, dgate,
                       (uint32_t)total, row16, T, tok16, lg16);
  else
    hipLaunchKernelGGL((gate_kernel<BWD, HEADWISE, uint64_t>), grid, block, 0, s, i4, y4, gate, o4, dgate, total,
                       row16, T, tok16, lg16);
}

bool aligned16(const void* p) { return p && (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

struct Span {
  const void* p;
  uint64_t n;
};

bool overlap(Span a, Span b) {
  const uintptr_t x = reinterpret_cast<uintptr_t>(a.p), y = reinterpret_cast<uintptr_t>(b.p);
  return x < y + b.n && y < x + a.n;
}

int gate_common(bool bwd, int64_t n_tokens, int32_t n_heads, int32_t d_v, int32_t gate_dim, int32_t cp_u,
                const void* in, const void* yg, const void* gate, void* out, void* dgate, void* stream) {
  if (n_tokens < 0 || n_heads <= 0 || cp_u <= 0 || n_heads % cp_u != 0) return HYDRA_ERR_INVALID;
  if (d_v < 8 || d_v > 512 || (d_v & (d_v - 1)) != 0) return HYDRA_ERR_INVALID;
  if (gate_dim != 1 && gate_dim != d_v) return HYDRA_ERR_INVALID;
  if (n_tokens > (int64_t(1) << 31) || n_heads > 65536) return HYDRA_ERR_INVALID;
  if (n_tokens == 0) return HYDRA_OK;
  if (!in || !gate || !out || (bwd && (!yg || !dgate))) return HYDRA_ERR_INVALID;
  if (!aligned16(in) || !aligned16(gate) || !aligned16(out) || (bwd && (!aligned16(yg) || !aligned16(dgate))))
    return HYDRA_ERR_ALIGN;
  const uint64_t elems = (uint64_t)n_tokens * n_heads * d_v;
  const Span s_in{in, elems * 2}, s_gate{gate, (uint64_t)n_tokens * n_heads * gate_dim * 2}, s_out{out, elems * 2};
  if (overlap(s_in, s_out) || overlap(s_gate, s_out)) return HYDRA_ERR_INVALID;
  if (bwd) {
    const Span s_y{yg, elems * 2}, s_dg{dgate, s_gate.n};
    if (overlap(s_y, s_out) || overlap(s_in, s_dg) || overlap(s_y, s_dg) || overlap(s_gate, s_dg) ||
        overlap(s_out, s_dg))
      return HYDRA_ERR_INVALID;
  }
  uint32_t lg16 = 0;
  while ((8u << lg16) < (uint32_t)d_v) ++lg16;
  const uint32_t hb16 = (uint32_t)d_v / 8, g = (uint32_t)(n_heads / cp_u);
  const uint64_t total = elems / 8;
  const uint32_t row16 = g * hb16, tok16 = (uint32_t)n_heads * hb16, T = (uint32_t)n_tokens;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const bool hw = gate_dim == 1;
  const int tok = prof_begin(bwd ? "pack_gated_bwd" : "unpack_gated", s);
  if (bwd && hw) launch<true, true>(in, yg, gate, out, dgate, total, row16, T, tok16, lg16, s);
  else if (bwd) launch<true, false>(in, yg, gate, out, dgate, total, row16, T, tok16, lg16, s);
  else if (hw) launch<false, true>(in, nullptr, gate, out, nullptr, total, row16, T, tok16, lg16, s);
  else launch<false, false>(in, nullptr, gate, out, nullptr, total, row16, T, tok16, lg16, s);
  prof_end(tok, s);
  return hipGetLastError() == hipSuccess ? HYDRA_OK : HYDRA_ERR_HIP;
}

}  // namespace
}  // namespace hydra

extern "C" {

int hydra_unpack_heads_gated(int64_t n_tokens, int32_t n_heads, int32_t d_v, int32_t gate_dim, int32_t cp_u,
                             const void* recv, const void* gate, void* y, void* stream) {
  return hydra::gate_common(false, n_tokens, n_heads, d_v, gate_dim, cp_u, recv, nullptr, gate, y, nullptr, stream);
}

int hydra_pack_heads_gated_bwd(int64_t n_tokens, int32_t n_heads, int32_t d_v, int32_t gate_dim, int32_t cp_u,
                               const void* y, const void* gate, const void* d_y, void* d_send, void* d_gate,
                               void* stream) {
  return hydra::gate_common(true, n_tokens, n_heads, d_v, gate_dim, cp_u, d_y, y, gate, d_send, d_gate, stream);
}

}  // extern "C"
