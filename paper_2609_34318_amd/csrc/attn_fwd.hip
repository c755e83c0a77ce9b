// Forward partial of one ring step: O = softmax(scale * Q K^T, masked) V and its LSE.
//
// One workgroup = 8 waves = 256 query rows of one head; each wave owns 32 rows and keeps
// them in registers as MFMA B operands for the whole key loop.  Key/value tiles of 64 rows
// stream through two swizzled LDS stages (80 KB) filled by direct global->LDS copies:
// the copies of tile t+1 are in flight while tile t is computed, one barrier per
// tile.  Eight waves share every tile, which halves the L2->LDS traffic per FLOP against a
// 128-row workgroup; two waves per SIMD let one's softmax overlap the other's matrix work.
// Scores are computed transposed (S^T = K Q^T), so every lane holds one query and the
// softmax row reductions stay in-lane plus one exchange with the lane 32 away.
//
// The running max / sum update is the online softmax that FlashAttention uses (named in
// Sec. 1 and Sec. 3.5), with one liberty: the reference max m only moves when a tile's max
// exceeds it by more than 8 (log2 units), so O is rescaled rarely.  Every term is still
// exp2(s - m) for the same m in numerator and denominator, so the result is unchanged up to
// rounding (terms stay <= 2^8).  Only tiles that straddle a document start, the causal
// diagonal or the end of a range evaluate the mask (Sec. 2.2).
#include "kernels.h"
#include "prof.h"

namespace hydra {

constexpr int FWD_BK = 64;
constexpr int FWD_KBYTES = FWD_BK * DQK * 2;             // 24 KB
constexpr int FWD_STAGE = FWD_KBYTES + FWD_BK * DV * 2;  // 40 KB
constexpr int FWD_NSTAGE = 2;  // measured faster than three stages
constexpr int FWD_WAVES = 8;
// Copy instructions one fwd_issue adds per wave: 3 (K) + 2 (V).  With three stages,
// waiting for vmcnt <= 5 completes tile t while tile t+1 may stay in flight; with two,
// tile t's copies are the only ones in flight.
constexpr int FWD_VMCNT_ONE_TILE = 5;
constexpr float RESCALE_SLACK = 8.0f;

// Starts the copy of key/value tile t into LDS stage t % FWD_NSTAGE.
__device__ __forceinline__ void fwd_issue(lds_char* smem, const AttnArgs& a, const TileRanges kr, int t, int koff,
                                          int voff, int head, int wave) {
  int row0, pos0, n;
  tile_at(kr, t, FWD_BK, row0, pos0, n);
  lds_char* dst = smem + (t % FWD_NSTAGE) * FWD_STAGE;
  dma_tile<DQK, FWD_BK, FWD_WAVES>(dst, tile_rsrc(a.k, row0, n, a.k_s), koff, a.k_s, wave);
  dma_tile<DV, FWD_BK, FWD_WAVES>(dst + FWD_KBYTES, tile_rsrc(a.v, row0, n, a.v_s), voff, a.v_s, wave);
}

__global__ __launch_bounds__(64 * FWD_WAVES, 1) void attn_fwd_kernel(AttnArgs a, uint16_t* __restrict__ o_bf16) {
  __shared__ __attribute__((aligned(1024))) char smem_raw[FWD_NSTAGE * FWD_STAGE];
  lds_char* smem = (lds_char*)smem_raw;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform, known to the compiler
  const int m = lane & 31, hh = lane >> 5;
  int head, item;
  xcd_head_item(blockIdx.x, a.H, a.n_items, head, item);
  const Item it(a.items, item);
  const int q_row0 = it.row0, q_pos0 = it.pos0, q_n = it.n;
  const TileRanges kr = tile_ranges(it, FWD_BK);
  const int n_tiles = kr.nt;

  lds_clear<64 * FWD_WAVES>(smem, FWD_NSTAGE * FWD_STAGE, tid);

  const int qi = wave * 32 + m;
  const bool q_valid = qi < q_n;
  const int pos_q = q_valid ? q_pos0 + qi : -1;
  int lo_q = q_valid ? a.cu[doc_of(a.cu, a.n_docs, pos_q)] : 0;
  // finish this load here: left pending, the tile loop would wait for all copies in flight
  asm volatile("s_waitcnt vmcnt(0)" : "+v"(lo_q)::"memory");
  const int lo_last = a.cu[doc_of(a.cu, a.n_docs, q_pos0 + q_n - 1)];
  const float sl2 = a.scale * LOG2E;
  const int kv_head = head / a.grp;  // grouped K/V heads: contiguous groups of query heads
  const int koff = dma_lane_off<DQK>(a.k_s, kv_head, wave, lane);
  const int voff = dma_lane_off<DV>(a.v_s, kv_head, wave, lane);

  bf16x8 qf[DQK / 16];
  {
    const uint16_t* qrow = a.q + (int64_t)(q_row0 + (q_valid ? qi : 0)) * a.q_s + head * DQK + 8 * hh;
#pragma unroll
    for (int t = 0; t < DQK / 16; ++t) {
      u32x4 u = {0u, 0u, 0u, 0u};
      if (q_valid) u = ldg16(qrow + 16 * t);
      settle(u);
      qf[t] = __builtin_bit_cast(bf16x8, u);
    }
  }
  __syncthreads();  // LDS cleared before the first copy lands

  for (int t = 0; t < FWD_NSTAGE - 1 && t < n_tiles; ++t) fwd_issue(smem, a, kr, t, koff, voff, head, wave);

  f32x16 acc[DV / 32];
#pragma unroll
  for (int d = 0; d < DV / 32; ++d) acc[d] = f32x16{};
  float m_run = NEG_BIG, l_run[4] = {0.f, 0.f, 0.f, 0.f};

  OperandOffsets o = operand_offsets(lane);

  for (int t = 0; t < n_tiles; ++t) {
    refresh(o);
    int k_row0, kpos, kn;
    tile_at(kr, t, FWD_BK, k_row0, kpos, kn);
    // copies of tile t are done once at most the later tiles' copies issued so far (with
    // two stages: none) are still in flight
    if (FWD_NSTAGE > 2 && t + 1 < n_tiles) asm volatile("s_waitcnt vmcnt(%0)" ::"n"(FWD_VMCNT_ONE_TILE) : "memory");
    else wait_dma();
    barrier_lds();
    if (t + FWD_NSTAGE - 1 < n_tiles) fwd_issue(smem, a, kr, t + FWD_NSTAGE - 1, koff, voff, head, wave);
    const lds_char* Ks = smem + (t % FWD_NSTAGE) * FWD_STAGE;
    const lds_char* Vs = Ks + FWD_KBYTES;

    f32x16 s[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      s[kb] = f32x16{};
#pragma unroll
      for (int t2 = 0; t2 < DQK / 16; ++t2)
        s[kb] = mfma(op_b128<FWD_BK>(Ks, o, 32 * kb, t2), qf[t2], s[kb]);
    }

    const bool full = (kn == FWD_BK) && (lo_last <= kpos) && (kpos + FWD_BK - 1 <= q_pos0);
    if (!full) {
      // key kpos + key(e) is visible iff lo_q <= it <= pos_q and key(e) < kn, i.e. iff
      // 0 <= base + c(e) < lim with base = kpos - lo_q + 8*hh
      const int base = kpos - lo_q + 8 * hh;
      const int lim = q_valid ? max(0, min(pos_q + 1, kpos + kn) - lo_q) : 0;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int r = base + 32 * kb + 16 * (e >> 3) + (e & 7);
          s[kb][e] = (unsigned)r < (unsigned)lim ? s[kb][e] : -INFINITY;
        }
    }
    // row max as four independent chains that take two new values per step (one
    // three-input maximum each)
    float mx4[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const f32x16& v = s[j >> 1];
      const int e0 = 8 * (j & 1);
      float t = fmax2(fmax2(v[e0], v[e0 + 1]), v[e0 + 2]);
      t = fmax2(fmax2(t, v[e0 + 3]), v[e0 + 4]);
      mx4[j] = fmax2(fmax2(t, v[e0 + 5]), v[e0 + 6]);
    }
    float mx = fmax2(fmax2(mx4[0], s[0][7]), s[0][15]);
    mx = fmax2(fmax2(mx, mx4[1]), s[1][7]);
    mx = fmax2(fmax2(mx, mx4[2]), s[1][15]);
    mx = fmax2(mx, mx4[3]);
    const float mxs = xhalf_max(mx) * sl2;  // -inf when nothing is visible
    if (__builtin_amdgcn_ballot_w64(mxs > m_run + RESCALE_SLACK) != 0) {
      const float m_new = mxs > m_run + RESCALE_SLACK ? mxs : m_run;
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
      m_run = m_new;
#pragma unroll
      for (int j = 0; j < 4; ++j) l_run[j] *= alpha;
#pragma unroll
      for (int d = 0; d < DV / 32; ++d) acc[d] *= alpha;
    }
    const float neg_m = -m_run;

    // P = exp2(s*scale*log2e - m); the row sum is kept as four partial sums
    bf16x8 pf[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      float p[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) p[e] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[j >> 1][8 * (j & 1) + e], sl2, neg_m));
      l_run[j] += ((p[0] + p[1]) + (p[2] + p[3])) + ((p[4] + p[5]) + (p[6] + p[7]));
      pf[j] = to_bf16x8(p);
    }

    // O^T[dv][q] += V^T[dv][key] * P^T[key][q]; V^T fragments via LDS transpose reads.  The
    // products of key step st are issued before the fragments of step st+1 load.
    bf16x8 vf[2][DV / 32];
    op_tr_x4<FWD_BK, 0, 0>(Vs, o, vf[0]);
    static_for<4>([&](auto st_) {
      constexpr int st = decltype(st_)::value;
#pragma unroll
      for (int d = 0; d < DV / 32; ++d) acc[d] = mfma(vf[st & 1][d], pf[st], acc[d]);
      if constexpr (st + 1 < 4) op_tr_x4<FWD_BK, 16 * (st + 1), 0>(Vs, o, vf[(st + 1) & 1]);
    });
  }

  const float l_tot = xhalf_sum((l_run[0] + l_run[1]) + (l_run[2] + l_run[3]));
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
  hipLaunchKernelGGL(attn_fwd_kernel, dim3(a.n_items * a.H), dim3(64 * FWD_WAVES), 0, stream, a, o_bf16);
  prof_end(tok, stream);
  return hipGetLastError();
}

}  // namespace hydra
