// Backward of one ring step, differentiating with the final merged O and LSE of each row:
//   D_i = <dO_i, O_i>,  P = exp(S - LSE),  dV += P^T dO,  dS = P o (dO V^T - D),
//   dK += scale dS^T Q,  dQ += scale dS K.
// Three kernels:
//   bwd_pre   D = rowsum(dO o O)                                  (HBM-bound)
//   bwd_dq    query-stationary: recomputes S^T and dP^T per key tile, accumulates dQ^T
//   bwd_dkdv  key-stationary: recomputes S and dP per query tile, accumulates dK^T, dV^T
// Splitting dQ from dK/dV recomputes S and dP once more but needs no atomics and is
// deterministic: every output row is owned by exactly one workgroup.
#include "kernels.h"
#include "prof.h"

namespace hydra {

// ------------------------------------------------------------------ D = rowsum(dO * O)
__global__ __launch_bounds__(256) void bwd_pre_kernel(const uint16_t* __restrict__ o,
                                                      const uint16_t* __restrict__ dO,
                                                      float* __restrict__ D, int nq, int H) {
  const int64_t gid = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t rh = gid >> 4;  // (row, head) pair, 16 lanes each
  const int sub = threadIdx.x & 15;
  const bool ok = rh < (int64_t)nq * H;
  float acc = 0.f;
  if (ok) {
    const u32x4 uo = ldg16(o + rh * DV + sub * 8);
    const u32x4 ud = ldg16(dO + rh * DV + sub * 8);
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      acc += __uint_as_float(uo[w] << 16) * __uint_as_float(ud[w] << 16);
      acc += __uint_as_float(uo[w] & 0xffff0000u) * __uint_as_float(ud[w] & 0xffff0000u);
    }
  }
  acc += __shfl_xor(acc, 8, 16);
  acc += __shfl_xor(acc, 4, 16);
  acc += __shfl_xor(acc, 2, 16);
  acc += __shfl_xor(acc, 1, 16);
  if (ok && sub == 0) {
    const int row = (int)(rh / H), head = (int)(rh % H);
    D[(int64_t)head * nq + row] = acc;
  }
}

// ------------------------------------------------------------------ dQ (query-stationary)
constexpr int DQ_BK = 64;

__global__ __launch_bounds__(256, 1) void bwd_dq_kernel(AttnArgs a) {
  __shared__ __attribute__((aligned(16))) __bf16 Ks[DQ_BK * PITCH_QK];
  __shared__ __attribute__((aligned(16))) __bf16 Vs[DQ_BK * PITCH_V];

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int m = lane & 31, hh = lane >> 5, g = lane >> 4, gi = lane & 15;
  const int head = blockIdx.x % a.H;
  const int* it = a.items + (blockIdx.x / a.H) * ITEM_INTS;
  const int q_row0 = it[0], q_pos0 = it[1], q_n = it[2], n_ranges = it[3];
  if (n_ranges == 0) return;  // uniform over the workgroup

  const int qi = wave * 32 + m;
  const bool q_valid = qi < q_n;
  const int pos_q = q_valid ? q_pos0 + qi : -1;
  const int lo_q = q_valid ? a.cu[doc_of(a.cu, a.n_docs, pos_q)] : 0;
  const int lo_last = a.cu[doc_of(a.cu, a.n_docs, q_pos0 + q_n - 1)];
  const float sl2 = a.scale * LOG2E;
  const int64_t qrow = q_row0 + (q_valid ? qi : 0);
  // invalid rows: LSE = +inf makes P = 0, D = 0 keeps dS = 0
  const float lse2 = q_valid ? a.lse[(int64_t)head * a.nq + qrow] * LOG2E : INFINITY;
  const float Dq = q_valid ? a.Dvec[(int64_t)head * a.nq + qrow] : 0.f;

  bf16x8 qf[DQK / 16], df[DV / 16];
  {
    const uint16_t* qp = a.q + (qrow * a.H + head) * DQK + 8 * hh;
    const uint16_t* dp = a.dO + (qrow * a.H + head) * DV + 8 * hh;
#pragma unroll
    for (int t = 0; t < DQK / 16; ++t) {
      u32x4 u = {0u, 0u, 0u, 0u};
      if (q_valid) u = ldg16(qp + 16 * t);
      qf[t] = __builtin_bit_cast(bf16x8, u);
    }
#pragma unroll
    for (int t = 0; t < DV / 16; ++t) {
      u32x4 u = {0u, 0u, 0u, 0u};
      if (q_valid) u = ldg16(dp + 16 * t);
      df[t] = __builtin_bit_cast(bf16x8, u);
    }
  }

  f32x16 acc[DQK / 32];
#pragma unroll
  for (int c = 0; c < DQK / 32; ++c) acc[c] = f32x16{};

  for (int r = 0; r < n_ranges; ++r) {
    const int k_row0 = it[4 + 3 * r], k_pos0 = it[5 + 3 * r], k_cnt = it[6 + 3 * r];
    for (int kt = 0; kt < k_cnt; kt += DQ_BK) {
      const int kn = min(DQ_BK, k_cnt - kt);
      const int kpos = k_pos0 + kt;
      __syncthreads();
      stage_rows<DQK, PITCH_QK, DQ_BK, 256>(Ks, a.k, k_row0 + kt, kn, a.H, head, tid);
      stage_rows<DV, PITCH_V, DQ_BK, 256>(Vs, a.v, k_row0 + kt, kn, a.H, head, tid);
      __syncthreads();
      const bool full = (kn == DQ_BK) && (lo_last <= kpos) && (kpos + DQ_BK - 1 <= q_pos0);

#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        f32x16 s = f32x16{}, dp = f32x16{};
        const __bf16* krow = Ks + (kb * 32 + pi_row(m)) * PITCH_QK + 8 * hh;
        const __bf16* vrow = Vs + (kb * 32 + pi_row(m)) * PITCH_V + 8 * hh;
#pragma unroll
        for (int t = 0; t < DQK / 16; ++t) s = mfma(lds_read8(krow + 16 * t), qf[t], s);
#pragma unroll
        for (int t = 0; t < DV / 16; ++t) dp = mfma(lds_read8(vrow + 16 * t), df[t], dp);

        float ds[16];
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          float p = __builtin_amdgcn_exp2f(s[e] * sl2 - lse2);
          if (!full) {
            const int key = kb * 32 + 16 * (e >> 3) + 8 * hh + (e & 7);
            const int kp = kpos + key;
            const bool vis = (key < kn) && (kp <= pos_q) && (kp >= lo_q);
            p = vis ? p : 0.f;
          }
          ds[e] = p * (dp[e] - Dq);
        }
        const bf16x8 dsf0 = to_bf16x8(ds), dsf1 = to_bf16x8(ds + 8);

        // dQ^T[c][q] += K^T[c][key] dS^T[key][q]; K^T fragments via LDS transpose reads.
#pragma unroll
        for (int half = 0; half < 2; ++half) {
          const int kr = kb * 32 + 16 * half + 8 * hh + (gi >> 2);
#pragma unroll
          for (int c = 0; c < DQK / 32; ++c) {
            const int kc = 32 * c + 16 * (g & 1) + 4 * (gi & 3);
            const bf16x8 ka = lds_read8_tr(Ks + kr * PITCH_QK + kc, Ks + (kr + 4) * PITCH_QK + kc);
            acc[c] = mfma(ka, half ? dsf1 : dsf0, acc[c]);
          }
        }
      }
    }
  }

  if (q_valid) {
    float* dq = a.dq + (qrow * a.H + head) * DQK + 4 * hh;
#pragma unroll
    for (int c = 0; c < DQK / 32; ++c)
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        f32x4* p = reinterpret_cast<f32x4*>(dq + 32 * c + 8 * rr);
        f32x4 old = *p;
        old[0] += a.scale * acc[c][4 * rr];
        old[1] += a.scale * acc[c][4 * rr + 1];
        old[2] += a.scale * acc[c][4 * rr + 2];
        old[3] += a.scale * acc[c][4 * rr + 3];
        *p = old;
      }
  }
}

// ------------------------------------------------------------------ dK, dV (key-stationary)
constexpr int KV_BQ = 32;

__global__ __launch_bounds__(256, 1) void bwd_dkdv_kernel(AttnArgs a) {
  __shared__ __attribute__((aligned(16))) __bf16 Qs[KV_BQ * PITCH_QK];
  __shared__ __attribute__((aligned(16))) __bf16 dOs[KV_BQ * PITCH_V];
  __shared__ __attribute__((aligned(16))) float lse_s[KV_BQ];
  __shared__ __attribute__((aligned(16))) float D_s[KV_BQ];

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int m = lane & 31, hh = lane >> 5, g = lane >> 4, gi = lane & 15;
  const int head = blockIdx.x % a.H;
  const int* it = a.items + (blockIdx.x / a.H) * ITEM_INTS;
  const int k_row0 = it[0], k_pos0 = it[1], k_n = it[2], n_ranges = it[3];
  if (n_ranges == 0) return;  // uniform over the workgroup

  const int kj = wave * 32 + m;
  const bool k_valid = kj < k_n;
  const int pos_k = k_valid ? k_pos0 + kj : 0x7fffffff;
  const int hi_k = k_valid ? a.cu[doc_of(a.cu, a.n_docs, pos_k) + 1] : 0;
  const int kn_w = min(32, max(0, k_n - wave * 32));  // valid keys of this wave
  const int wk_first = k_pos0 + wave * 32;
  const int wk_last = wk_first + kn_w - 1;
  const int hi_first = kn_w > 0 ? a.cu[doc_of(a.cu, a.n_docs, wk_first) + 1] : 0;
  const float sl2 = a.scale * LOG2E;
  const int64_t krow = k_row0 + (k_valid ? kj : 0);

  bf16x8 kf[DQK / 16], vf[DV / 16];
  {
    const uint16_t* kp = a.k + (krow * a.H + head) * DQK + 8 * hh;
    const uint16_t* vp = a.v + (krow * a.H + head) * DV + 8 * hh;
#pragma unroll
    for (int t = 0; t < DQK / 16; ++t) {
      u32x4 u = {0u, 0u, 0u, 0u};
      if (k_valid) u = ldg16(kp + 16 * t);
      kf[t] = __builtin_bit_cast(bf16x8, u);
    }
#pragma unroll
    for (int t = 0; t < DV / 16; ++t) {
      u32x4 u = {0u, 0u, 0u, 0u};
      if (k_valid) u = ldg16(vp + 16 * t);
      vf[t] = __builtin_bit_cast(bf16x8, u);
    }
  }

  f32x16 accK[DQK / 32], accV[DV / 32];
#pragma unroll
  for (int c = 0; c < DQK / 32; ++c) accK[c] = f32x16{};
#pragma unroll
  for (int d = 0; d < DV / 32; ++d) accV[d] = f32x16{};

  for (int r = 0; r < n_ranges; ++r) {
    const int q_row0 = it[4 + 3 * r], q_pos0 = it[5 + 3 * r], q_cnt = it[6 + 3 * r];
    for (int qt = 0; qt < q_cnt; qt += KV_BQ) {
      const int qn = min(KV_BQ, q_cnt - qt);
      const int qpos = q_pos0 + qt;
      __syncthreads();
      stage_rows<DQK, PITCH_QK, KV_BQ, 256>(Qs, a.q, q_row0 + qt, qn, a.H, head, tid);
      stage_rows<DV, PITCH_V, KV_BQ, 256>(dOs, a.dO, q_row0 + qt, qn, a.H, head, tid);
      if (tid < KV_BQ) {
        const int64_t row = q_row0 + qt + tid;
        lse_s[tid] = tid < qn ? a.lse[(int64_t)head * a.nq + row] * LOG2E : INFINITY;
        D_s[tid] = tid < qn ? a.Dvec[(int64_t)head * a.nq + row] : 0.f;
      }
      __syncthreads();
      if (kn_w == 0) continue;  // wave-uniform; barriers above are still reached

      f32x16 s = f32x16{}, dp = f32x16{};
      {
        const __bf16* qr = Qs + pi_row(m) * PITCH_QK + 8 * hh;
        const __bf16* dr = dOs + pi_row(m) * PITCH_V + 8 * hh;
#pragma unroll
        for (int t = 0; t < DQK / 16; ++t) s = mfma(lds_read8(qr + 16 * t), kf[t], s);
#pragma unroll
        for (int t = 0; t < DV / 16; ++t) dp = mfma(lds_read8(dr + 16 * t), vf[t], dp);
      }
      const bool full = (kn_w == 32) && (qn == KV_BQ) && (wk_last <= qpos) && (qpos + KV_BQ - 1 < hi_first);
      float p[16], ds[16];
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int qq = 16 * (e >> 3) + 8 * hh + (e & 7);
        float pv = __builtin_amdgcn_exp2f(s[e] * sl2 - lse_s[qq]);
        if (!full) {
          const int pq = qpos + qq;
          const bool vis = (qq < qn) && (pq >= pos_k) && (pq < hi_k);
          pv = vis ? pv : 0.f;
        }
        p[e] = pv;
        ds[e] = pv * (dp[e] - D_s[qq]);
      }
      const bf16x8 pf0 = to_bf16x8(p), pf1 = to_bf16x8(p + 8);
      const bf16x8 sf0 = to_bf16x8(ds), sf1 = to_bf16x8(ds + 8);

#pragma unroll
      for (int half = 0; half < 2; ++half) {
        const int qr = 16 * half + 8 * hh + (gi >> 2);
        // dV^T[dv][key] += dO^T[dv][q] P[q][key]
#pragma unroll
        for (int d = 0; d < DV / 32; ++d) {
          const int dc = 32 * d + 16 * (g & 1) + 4 * (gi & 3);
          const bf16x8 da = lds_read8_tr(dOs + qr * PITCH_V + dc, dOs + (qr + 4) * PITCH_V + dc);
          accV[d] = mfma(da, half ? pf1 : pf0, accV[d]);
        }
        // dK^T[c][key] += Q^T[c][q] dS[q][key]
#pragma unroll
        for (int c = 0; c < DQK / 32; ++c) {
          const int qc = 32 * c + 16 * (g & 1) + 4 * (gi & 3);
          const bf16x8 qa = lds_read8_tr(Qs + qr * PITCH_QK + qc, Qs + (qr + 4) * PITCH_QK + qc);
          accK[c] = mfma(qa, half ? sf1 : sf0, accK[c]);
        }
      }
    }
  }

  if (k_valid) {
    float* dk = a.dk + (krow * a.H + head) * DQK + 4 * hh;
    float* dv = a.dv + (krow * a.H + head) * DV + 4 * hh;
#pragma unroll
    for (int c = 0; c < DQK / 32; ++c)
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        f32x4* p = reinterpret_cast<f32x4*>(dk + 32 * c + 8 * rr);
        f32x4 old = *p;
        old[0] += a.scale * accK[c][4 * rr];
        old[1] += a.scale * accK[c][4 * rr + 1];
        old[2] += a.scale * accK[c][4 * rr + 2];
        old[3] += a.scale * accK[c][4 * rr + 3];
        *p = old;
      }
#pragma unroll
    for (int d = 0; d < DV / 32; ++d)
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        f32x4* p = reinterpret_cast<f32x4*>(dv + 32 * d + 8 * rr);
        f32x4 old = *p;
        old[0] += accV[d][4 * rr];
        old[1] += accV[d][4 * rr + 1];
        old[2] += accV[d][4 * rr + 2];
        old[3] += accV[d][4 * rr + 3];
        *p = old;
      }
  }
}

hipError_t launch_attn_bwd(const AttnArgs& a, int n_qitems, int n_kitems, const int* kitems,
                           hipStream_t stream) {
  const int64_t pairs = (int64_t)a.nq * a.H;
  const int64_t blocks = (pairs * 16 + 255) / 256;
  int tok = prof_begin("bwd_pre", stream);
  hipLaunchKernelGGL(bwd_pre_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, a.o, a.dO, a.Dvec,
                     a.nq, a.H);
  prof_end(tok, stream);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (n_qitems > 0) {
    AttnArgs b = a;
    b.n_items = n_qitems;
    tok = prof_begin("bwd_dq", stream);
    hipLaunchKernelGGL(bwd_dq_kernel, dim3(n_qitems * a.H), dim3(256), 0, stream, b);
    prof_end(tok, stream);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (n_kitems > 0) {
    AttnArgs b = a;
    b.items = kitems;
    b.n_items = n_kitems;
    tok = prof_begin("bwd_dkdv", stream);
    hipLaunchKernelGGL(bwd_dkdv_kernel, dim3(n_kitems * a.H), dim3(256), 0, stream, b);
    prof_end(tok, stream);
    e = hipGetLastError();
  }
  return e;
}

}  // namespace hydra
