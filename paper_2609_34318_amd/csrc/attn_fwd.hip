// Forward partial of one ring step: O = softmax(scale * Q K^T, masked) V and its LSE.
//
// One workgroup = 4 waves = 128 query rows of one head; each wave owns 32 rows and keeps
// them in registers as MFMA B operands for the whole key loop.  Key/value tiles of 64
// rows are staged through LDS.  Scores are computed transposed (S^T = K Q^T), so every
// lane holds one query and the softmax row reductions stay in-lane plus one exchange
// with the lane 32 away.  The running max / sum update is the standard online softmax
// that FlashAttention uses (named in Sec. 1 and Sec. 3.5); the result is exact up to
// rounding.  Only tiles that straddle a document start, the causal diagonal or the end
// of a range evaluate the mask (Sec. 2.2); every other visited tile is fully visible.
#include "kernels.h"
#include "prof.h"

namespace hydra {

constexpr int FWD_BK = 64;

__global__ __launch_bounds__(256, 2) void attn_fwd_kernel(AttnArgs a, uint16_t* __restrict__ o_bf16) {
  __shared__ __attribute__((aligned(16))) __bf16 Ks[FWD_BK * PITCH_QK];
  __shared__ __attribute__((aligned(16))) __bf16 Vs[FWD_BK * PITCH_V];

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int m = lane & 31, hh = lane >> 5, g = lane >> 4, gi = lane & 15;
  const int head = blockIdx.x % a.H;
  const int* it = a.items + (blockIdx.x / a.H) * ITEM_INTS;
  const int q_row0 = it[0], q_pos0 = it[1], q_n = it[2], n_ranges = it[3];

  const int qi = wave * 32 + m;
  const bool q_valid = qi < q_n;
  const int pos_q = q_valid ? q_pos0 + qi : -1;
  const int lo_q = q_valid ? a.cu[doc_of(a.cu, a.n_docs, pos_q)] : 0;
  const int lo_last = a.cu[doc_of(a.cu, a.n_docs, q_pos0 + q_n - 1)];
  const float sl2 = a.scale * LOG2E;

  bf16x8 qf[DQK / 16];
  {
    const uint16_t* qrow = a.q + ((int64_t)(q_row0 + (q_valid ? qi : 0)) * a.H + head) * DQK + 8 * hh;
#pragma unroll
    for (int t = 0; t < DQK / 16; ++t) {
      u32x4 u = {0u, 0u, 0u, 0u};
      if (q_valid) u = ldg16(qrow + 16 * t);
      qf[t] = __builtin_bit_cast(bf16x8, u);
    }
  }

  f32x16 acc[DV / 32];
#pragma unroll
  for (int d = 0; d < DV / 32; ++d) acc[d] = f32x16{};
  float m_run = NEG_BIG, l_run = 0.f;

  for (int r = 0; r < n_ranges; ++r) {
    const int k_row0 = it[4 + 3 * r], k_pos0 = it[5 + 3 * r], k_cnt = it[6 + 3 * r];
    for (int kt = 0; kt < k_cnt; kt += FWD_BK) {
      const int kn = min(FWD_BK, k_cnt - kt);
      const int kpos = k_pos0 + kt;
      __syncthreads();
      stage_rows<DQK, PITCH_QK, FWD_BK, 256>(Ks, a.k, k_row0 + kt, kn, a.H, head, tid);
      stage_rows<DV, PITCH_V, FWD_BK, 256>(Vs, a.v, k_row0 + kt, kn, a.H, head, tid);
      __syncthreads();

      f32x16 s[2];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        s[kb] = f32x16{};
        const __bf16* krow = Ks + (kb * 32 + pi_row(m)) * PITCH_QK + 8 * hh;
#pragma unroll
        for (int t = 0; t < DQK / 16; ++t) s[kb] = mfma(lds_read8(krow + 16 * t), qf[t], s[kb]);
      }

      const bool full = (kn == FWD_BK) && (lo_last <= kpos) && (kpos + FWD_BK - 1 <= q_pos0);
      float mx = m_run;
      if (full) {
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int e = 0; e < 16; ++e) {
            s[kb][e] *= sl2;
            mx = fmax2(mx, s[kb][e]);
          }
      } else {
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int e = 0; e < 16; ++e) {
            const int key = kb * 32 + 16 * (e >> 3) + 8 * hh + (e & 7);
            const int kp = kpos + key;
            const bool vis = (key < kn) && (kp <= pos_q) && (kp >= lo_q);
            s[kb][e] = vis ? s[kb][e] * sl2 : -INFINITY;
            mx = fmax2(mx, s[kb][e]);
          }
      }
      mx = xhalf_max(mx);
      const float alpha = __builtin_amdgcn_exp2f(m_run - mx);
      m_run = mx;
      l_run *= alpha;
#pragma unroll
      for (int d = 0; d < DV / 32; ++d) acc[d] *= alpha;

      bf16x8 pf[4];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        float p[16];
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          p[e] = __builtin_amdgcn_exp2f(s[kb][e] - mx);
          l_run += p[e];
        }
        pf[2 * kb] = to_bf16x8(p);
        pf[2 * kb + 1] = to_bf16x8(p + 8);
      }

      // O^T[dv][q] += V^T[dv][key] * P^T[key][q]; V^T fragments via LDS transpose reads.
#pragma unroll
      for (int st = 0; st < 4; ++st) {
        const int vr = 16 * st + 8 * hh + (gi >> 2);
#pragma unroll
        for (int d = 0; d < DV / 32; ++d) {
          const int vc = 32 * d + 16 * (g & 1) + 4 * (gi & 3);
          const bf16x8 va = lds_read8_tr(Vs + vr * PITCH_V + vc, Vs + (vr + 4) * PITCH_V + vc);
          acc[d] = mfma(va, pf[st], acc[d]);
        }
      }
    }
  }

  const float l_tot = xhalf_sum(l_run);
  if (q_valid) {
    const float inv = l_tot > 0.f ? 1.0f / l_tot : 0.f;
    const int64_t base = ((int64_t)(q_row0 + qi) * a.H + head) * DV + 4 * hh;
    float* orow = a.out_o + base;
#pragma unroll
    for (int d = 0; d < DV / 32; ++d)
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        f32x4 val = {acc[d][4 * rr] * inv, acc[d][4 * rr + 1] * inv, acc[d][4 * rr + 2] * inv,
                     acc[d][4 * rr + 3] * inv};
        *reinterpret_cast<f32x4*>(orow + 32 * d + 8 * rr) = val;
        if (o_bf16) {
          uint32_t lo = pack_bf16x2(val[0], val[1]), hi = pack_bf16x2(val[2], val[3]);
          *reinterpret_cast<uint2*>(o_bf16 + base + 32 * d + 8 * rr) = make_uint2(lo, hi);
        }
      }
    if (hh == 0)
      a.out_lse[(int64_t)head * a.nq + q_row0 + qi] =
          l_tot > 0.f ? (m_run + __builtin_log2f(l_tot)) * LN2 : -INFINITY;
  }
}

hipError_t launch_attn_fwd(const AttnArgs& a, uint16_t* o_bf16, hipStream_t stream) {
  if (a.n_items == 0) return hipSuccess;
  const int tok = prof_begin("attn_fwd", stream);
  hipLaunchKernelGGL(attn_fwd_kernel, dim3(a.n_items * a.H), dim3(256), 0, stream, a, o_bf16);
  prof_end(tok, stream);
  return hipGetLastError();
}

}  // namespace hydra
