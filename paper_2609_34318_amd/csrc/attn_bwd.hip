// Backward of one ring step, differentiating with the final merged O and LSE of each row:
//   D_i = <dO_i, O_i>,  P = exp(S - LSE),  dV += P^T dO,  dS = P o (dO V^T - D),
//   dK += scale dS^T Q,  dQ += scale dS K.
// Three kernels:
//   bwd_pre   D = rowsum(dO o O) and LSE * log2(e)                  (HBM-bound)
//   bwd_dq    query-stationary: recomputes S^T and dP^T per key tile, accumulates dQ^T
//   bwd_dkdv  key-stationary: recomputes S and dP per query tile, accumulates dK^T, dV^T
// Splitting dQ from dK/dV recomputes S and dP once more but needs no atomics and is
// deterministic: every output row is owned by exactly one workgroup.  Both main kernels
// stream their other-side tiles through swizzled LDS stages filled by direct
// buffer->LDS copies issued ahead of use.
#include "kernels.h"
#include "prof.h"

namespace hydra {

// ------------------------------------------------------------------ D = rowsum(dO * O)
__global__ __launch_bounds__(256) void bwd_pre_kernel(const uint16_t* __restrict__ o,
                                                      const uint16_t* __restrict__ dO,
                                                      const float* __restrict__ lse,
                                                      float* __restrict__ D, float* __restrict__ lse2,
                                                      int nq, int H) {
  const int sub = threadIdx.x & 15;
  const int64_t total = (int64_t)nq * H;
  // (row, head) pairs, 16 lanes each, strided over a capped grid; the 16 lanes of a pair
  // stay together, so the reduction below always has all of them
  for (int64_t rh = (int64_t)blockIdx.x * 16 + (threadIdx.x >> 4); rh < total; rh += (int64_t)gridDim.x * 16) {
    const u32x4 uo = ldg16(o + rh * DV + sub * 8);
    const u32x4 ud = ldg16(dO + rh * DV + sub * 8);
    float acc = 0.f;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      acc += __uint_as_float(uo[w] << 16) * __uint_as_float(ud[w] << 16);
      acc += __uint_as_float(uo[w] & 0xffff0000u) * __uint_as_float(ud[w] & 0xffff0000u);
    }
    acc += __shfl_xor(acc, 8, 16);
    acc += __shfl_xor(acc, 4, 16);
    acc += __shfl_xor(acc, 2, 16);
    acc += __shfl_xor(acc, 1, 16);
    if (sub == 0) {
      const int row = (int)(rh / H), head = (int)(rh % H);
      const int64_t li = (int64_t)head * nq + row;
      D[li] = acc;
      lse2[li] = lse[li] * LOG2E;
    }
  }
}

// ------------------------------------------------------------------ dQ (query-stationary)
constexpr int DQ_BK = 96;  // keys per tile: measured faster than 64 and 128
constexpr int DQ_KBYTES = DQ_BK * DQK * 2;            // 36 KB
constexpr int DQ_STAGE = DQ_KBYTES + DQ_BK * DV * 2;  // 60 KB
constexpr int DQ_NSTAGE = 2;  // measured faster than three stages
constexpr int DQ_WAVES = 8;                           // 256 query rows per workgroup
constexpr int DQ_COPY_WAVES = 4;                      // the 12 copies per column block split evenly over 4
// copies per tile per copying wave: (3 (K) + 2 (V) column blocks) x 3
constexpr int DQ_VMCNT_ONE_TILE = (DQK / 64 + DV / 64) * (DQ_BK / 8 / DQ_COPY_WAVES);

__device__ __forceinline__ void dq_issue(lds_char* smem, const AttnArgs& a, const TileRanges kr, int t, int koff,
                                         int voff, int wave) {
  int row0, pos0, n;
  tile_at(kr, t, DQ_BK, row0, pos0, n);
  lds_char* dst = smem + (t % DQ_NSTAGE) * DQ_STAGE;
  if (wave >= DQ_COPY_WAVES) return;  // wave-uniform
  dma_tile<DQK, DQ_BK, DQ_COPY_WAVES>(dst, tile_rsrc(a.k, row0, n, a.k_s), koff, a.k_s, wave);
  dma_tile<DV, DQ_BK, DQ_COPY_WAVES>(dst + DQ_KBYTES, tile_rsrc(a.v, row0, n, a.v_s), voff, a.v_s, wave);
}

__global__ __launch_bounds__(64 * DQ_WAVES, 1) void bwd_dq_kernel(AttnArgs a) {
  __shared__ __attribute__((aligned(1024))) char smem_raw[DQ_NSTAGE * DQ_STAGE];
  lds_char* smem = (lds_char*)smem_raw;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform, known to the compiler
  const int m = lane & 31, hh = lane >> 5;
  int hl, item;
  xcd_head_item(blockIdx.x, a.q_heads, a.n_items, hl, item);
  const int head = a.q_head0 + hl;
  const Item it(a.items, item);
  const TileRanges kr = tile_ranges(it, DQ_BK);
  const int n_tiles = kr.nt;
  if (n_tiles == 0) return;  // uniform over the workgroup
  const int q_row0 = it.row0, q_pos0 = it.pos0, q_n = it.n;

  lds_clear<64 * DQ_WAVES>(smem, DQ_NSTAGE * DQ_STAGE, tid);
  const int qi = wave * 32 + m;
  const bool q_valid = qi < q_n;
  const int pos_q = q_valid ? q_pos0 + qi : -1;
  int lo_q = q_valid ? a.cu[doc_of(a.cu, a.n_docs, pos_q)] : 0;
  // finish this load here: left pending, the tile loop would wait for all copies in flight
  asm volatile("s_waitcnt vmcnt(0)" : "+v"(lo_q)::"memory");
  const int lo_last = a.cu[doc_of(a.cu, a.n_docs, q_pos0 + q_n - 1)];
  const float sl2 = a.scale * LOG2E;
  const int64_t qrow = q_row0 + (q_valid ? qi : 0);
  // invalid rows: LSE = +inf makes P = 0, D = 0 keeps dS = 0
  float lse2 = q_valid ? a.lse2[(int64_t)head * a.nq + qrow] : INFINITY;
  float Dq = q_valid ? a.Dvec[(int64_t)head * a.nq + qrow] : 0.f;
  settle(lse2);
  settle(Dq);
  const int kv_head = head / a.grp;  // grouped K/V heads: contiguous groups of query heads
  const int koff = dma_lane_off<DQK>(a.k_s, kv_head, wave, lane);
  const int voff = dma_lane_off<DV>(a.v_s, kv_head, wave, lane);

  bf16x8 qf[DQK / 16], df[DV / 16];
  {
    const uint16_t* qp = a.q + qrow * a.q_s + head * DQK + 8 * hh;
    const uint16_t* dp = a.dO + (qrow * a.H + head) * DV + 8 * hh;
#pragma unroll
    for (int t = 0; t < DQK / 16; ++t) {
      u32x4 u = {0u, 0u, 0u, 0u};
      if (q_valid) u = ldg16(qp + 16 * t);
      settle(u);
      qf[t] = __builtin_bit_cast(bf16x8, u);
    }
#pragma unroll
    for (int t = 0; t < DV / 16; ++t) {
      u32x4 u = {0u, 0u, 0u, 0u};
      if (q_valid) u = ldg16(dp + 16 * t);
      settle(u);
      df[t] = __builtin_bit_cast(bf16x8, u);
    }
  }
  __syncthreads();  // LDS cleared before the first copy lands
  for (int t = 0; t < DQ_NSTAGE - 1 && t < n_tiles; ++t) dq_issue(smem, a, kr, t, koff, voff, wave);

  f32x16 acc[DQK / 32];
#pragma unroll
  for (int c = 0; c < DQK / 32; ++c) acc[c] = f32x16{};

  OperandOffsets o = operand_offsets(lane);

  for (int t = 0; t < n_tiles; ++t) {
    refresh(o);
    int k_row0, kpos, kn;
    tile_at(kr, t, DQ_BK, k_row0, kpos, kn);
    // copies of tile t are done once at most the later tiles' copies issued so far (with
    // two stages: none) are still in flight
    if (DQ_NSTAGE > 2 && t + 1 < n_tiles) asm volatile("s_waitcnt vmcnt(%0)" ::"n"(DQ_VMCNT_ONE_TILE) : "memory");
    else wait_dma();
    barrier_lds();
    if (t + DQ_NSTAGE - 1 < n_tiles) dq_issue(smem, a, kr, t + DQ_NSTAGE - 1, koff, voff, wave);
    const lds_char* Ks = smem + (t % DQ_NSTAGE) * DQ_STAGE;
    const lds_char* Vs = Ks + DQ_KBYTES;
    const bool full = (kn == DQ_BK) && (lo_last <= kpos) && (kpos + DQ_BK - 1 <= q_pos0);

    static_for<DQ_BK / 32>([&](auto kb_) {
      constexpr int kb = decltype(kb_)::value;
      f32x16 s = f32x16{}, dp = f32x16{};
#pragma unroll
      for (int t2 = 0; t2 < DQK / 16; ++t2) s = mfma(op_b128<DQ_BK>(Ks, o, 32 * kb, t2), qf[t2], s);
#pragma unroll
      for (int t2 = 0; t2 < DV / 16; ++t2) dp = mfma(op_b128<DQ_BK>(Vs, o, 32 * kb, t2), df[t2], dp);

      float ds[16];
      if (full) {
#pragma unroll
        for (int e = 0; e < 16; ++e) ds[e] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[e], sl2, -lse2)) * (dp[e] - Dq);
      } else {
        // key kpos + key(e) is visible iff lo_q <= it <= pos_q and key(e) < kn, i.e. iff
        // 0 <= base + c(e) < lim with base = kpos - lo_q + 32*kb + 8*hh; masked entries get
        // exp2(-inf) = 0
        const int base = kpos - lo_q + 32 * kb + 8 * hh;
        const int lim = q_valid ? max(0, min(pos_q + 1, kpos + kn) - lo_q) : 0;
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int r = base + 16 * (e >> 3) + (e & 7);
          const bool vis = (unsigned)r < (unsigned)lim;
          ds[e] = __builtin_amdgcn_exp2f(vis ? __builtin_fmaf(s[e], sl2, -lse2) : -INFINITY) * (dp[e] - Dq);
        }
      }
      const bf16x8 dsf[2] = {to_bf16x8(ds), to_bf16x8(ds + 8)};

      // dQ^T[c][q] += K^T[c][key] dS^T[key][q]; K^T fragments by LDS transpose reads, three
      // column blocks per group; a group's products are issued before the next group loads.
      bf16x8 f[2][3];
      op_tr_x3<DQ_BK, 32 * kb, 0>(Ks, o, f[0]);
      static_for<4>([&](auto g_) {
        constexpr int gq = decltype(g_)::value, half = gq >> 1, c0 = 3 * (gq & 1);
#pragma unroll
        for (int j = 0; j < 3; ++j) acc[c0 + j] = mfma(f[gq & 1][j], dsf[half], acc[c0 + j]);
        if constexpr (gq + 1 < 4)
          op_tr_x3<DQ_BK, 32 * kb + 16 * ((gq + 1) >> 1), 3 * ((gq + 1) & 1)>(Ks, o, f[(gq + 1) & 1]);
        sched_fence();
      });
    });
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
// Eight waves share 128 keys as four pairs, one pair per SIMD, 32 keys per pair.  The two
// waves of a pair split the work so that each fits in 256 registers (two waves per SIMD,
// whose matrix and vector work then overlap):
//   wave A: S = Q K^T, P = exp(S - LSE) (masked), dV^T += dO^T P
//   wave B: dP = dO V^T, dS = P o (dP - D), dK^T += Q^T dS
// P crosses from A to B through LDS (rounded to bf16, the value the dV product uses).  Per
// 96-query tile: barrier, start the copy of the next tile (LDS holds two), phase 1 (A: S
// and P, B: dP), barrier, phase 2 (A: dV, B: dS and dK).
constexpr int KV_BQ = KV_QTILE_ROWS;                             // query rows per tile
constexpr int KV_NSB = KV_BQ / 32;                               // 32-row sub-blocks per tile
constexpr int KV_VEC = 128;                                      // LDS slots per vector (LSE2, D)
constexpr int KV_QBYTES = KV_BQ * DQK * 2;                       // 36 KB
constexpr int KV_OBYTES = KV_BQ * DV * 2;                        // 24 KB
constexpr int KV_STAGE = KV_QBYTES + KV_OBYTES + 2 * KV_VEC * 4;  // + LSE2 and D
constexpr int KV_NSTAGE = 2;  // measured faster than three stages
constexpr int KV_PBYTES = 4 * KV_NSB * 2048;                     // P: 4 pairs x sub-blocks x 32x32 bf16
// The copies are issued by the four role-B waves only (role A's first phase is the longer
// one).  Vector-memory instructions one kv_issue adds per issuing wave: (3 + 2) column
// blocks x KV_BQ/32 copies of 1 KB (Q, dO), plus one vector copy (LSE2 or D) on each wave
// that has one.  With three stages, waiting for vmcnt <= KV_VMCNT_ONE_TILE completes tile
// t while tile t+1 may stay in flight; with two, tile t's copies are the only ones in flight.
constexpr int KV_VMCNT_ONE_TILE = (DQK / 64 + DV / 64) * (KV_BQ / 32);

// The query tile of flat tile index t = member * nt + i (member: query head of the group):
// each member's tiles are walked last first.  Every range of a key item ends where its
// document or segment ends, which is the same row for most items, so the workgroups running
// together start at the same query tiles and stream them through the L2 together (walked
// first to last, they would start at their own key positions, each on its own tiles).
__device__ __forceinline__ int kv_tile(const TileRanges& qr, int t, int member) { return qr.nt - 1 - (t - member * qr.nt); }

// Flat tile index t covers (query head of the group, query tile): t = member * nt + tile.
// wave_b: 0 .. 3, the issuing wave among the role-B waves.
__device__ __forceinline__ void kv_issue(lds_char* smem, const AttnArgs& a, const TileRanges qr, int t, int qoff,
                                         int ooff, int head0, int wave_b, int lane) {
  const int member = t / qr.nt, qt = kv_tile(qr, t, member);
  int row0, pos0, n;
  tile_at(qr, qt, KV_BQ, row0, pos0, n);
  lds_char* dst = smem + (t % KV_NSTAGE) * KV_STAGE;
  dma_tile<DQK, KV_BQ, 4>(dst, tile_rsrc(a.q, row0, n, a.q_s), qoff + member * (DQK * 2), a.q_s, wave_b);
  dma_tile<DV, KV_BQ, 4>(dst + KV_QBYTES, tile_rsrc(a.dO, row0, n, a.H * DV), ooff + member * (DV * 2), a.H * DV,
                         wave_b);
  const int64_t li = (int64_t)(head0 + member) * a.nq + row0;
  // LSE2 and D of the tile's rows, 64 per copy; rows past the tile's end read as zero
  static_assert(KV_BQ <= 2 * 64 && KV_BQ <= KV_VEC, "two 64-row copies per vector");
  lds_char* vec = dst + KV_QBYTES + KV_OBYTES;
  if (wave_b == 0) dma_vec64(vec, a.lse2 + li, min(n, 64), lane);
  if (wave_b == 1) dma_vec64(vec + KV_VEC * 4, a.Dvec + li, min(n, 64), lane);
  if constexpr (KV_BQ > 64) {
    if (wave_b == 2) dma_vec64(vec + 256, a.lse2 + li + 64, max(n - 64, 0), lane);
    if (wave_b == 3) dma_vec64(vec + KV_VEC * 4 + 256, a.Dvec + li + 64, max(n - 64, 0), lane);
  }
}

// STORE_DS: also store dS (bf16, as the MFMA operand registers hold it) for the query-
// stationary dQ kernel that reads it back instead of recomputing S and dP.
template <bool STORE_DS>
__global__ __launch_bounds__(512, 1) void bwd_dkdv_kernel(AttnArgs a) {
  __shared__ __attribute__((aligned(1024))) char smem_raw[KV_NSTAGE * KV_STAGE + KV_PBYTES];
  lds_char* smem = (lds_char*)smem_raw;
  lds_char* pbuf = smem + KV_NSTAGE * KV_STAGE;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform, known to the compiler
  const int pair = wave & 3, role = wave >> 2;  // role 0: S, P, dV   role 1: dP, dS, dK
  const int m = lane & 31, hh = lane >> 5;
  // one K/V head per workgroup; its dK/dV sum over the group's query heads head0 ..
  int kvl, item_idx;
  xcd_head_item(blockIdx.x, a.kv_heads, a.n_items, kvl, item_idx);
  const int kv_head = a.kv_head0 + kvl;
  const int head0 = kv_head * a.grp;
  const Item it(a.items, item_idx);
  const TileRanges qr = tile_ranges(it, KV_BQ);
  const int n_tiles = qr.nt * a.grp;  // (query head, query tile) pairs
  if (n_tiles == 0) return;  // uniform over the workgroup
  const int k_row0 = it.row0, k_pos0 = it.pos0, k_n = it.n;

  lds_clear<512>(smem, KV_NSTAGE * KV_STAGE + KV_PBYTES, tid);
  const int kj = pair * 32 + m;
  const bool k_valid = kj < k_n;
  const int pos_k = k_valid ? k_pos0 + kj : 0x7fffffff;
  int hi_k = k_valid ? a.cu[doc_of(a.cu, a.n_docs, pos_k) + 1] : 0;
  // finish these loads here: left pending, the tile loop would wait for all copies in flight
  asm volatile("s_waitcnt vmcnt(0)" : "+v"(hi_k)::"memory");
  const int kn_w = min(32, max(0, k_n - pair * 32));  // valid keys of this pair
  const int wk_first = k_pos0 + pair * 32;
  const int wk_last = wk_first + kn_w - 1;
  const int hi_first =
      __builtin_amdgcn_readfirstlane(kn_w > 0 ? a.cu[doc_of(a.cu, a.n_docs, wk_first) + 1] : 0);
  const float sl2 = a.scale * LOG2E;
  const int64_t krow = k_row0 + (k_valid ? kj : 0);
  const int qoff = dma_lane_off<DQK>(a.q_s, head0, pair, lane);  // role B's copy lanes (wave b = pair)
  const int ooff = dma_lane_off<DV>(a.H * DV, head0, pair, lane);
  const int poff = pair * (KV_NSB * 2048) + lane * 16;  // this lane's P slot: + sb*2048 + half*1024
  const bool active = kn_w > 0;               // uniform over the pair
  // first dS slot of this key item (stored-dS backward only)
  const int ds_slot0 = STORE_DS ? __builtin_amdgcn_readfirstlane(a.kbase[item_idx]) : 0;

  // The two roles run separate copies of the tile loop, with the same copies and the same
  // two barriers per tile: each copy keeps only its own role's operands and accumulators
  // live, which leaves registers for reading LDS operands well ahead of their products.
  auto run = [&](auto role_c) {
    constexpr int ROLE = decltype(role_c)::value;
    // role A keeps K^T fragments (B operand of S) and dV^T; role B V^T fragments (B operand
    // of dP) and dK^T
    constexpr int NF = ROLE == 0 ? DQK / 16 : DV / 16;
    constexpr int NACC = ROLE == 0 ? DV / 32 : DQK / 32;
    bf16x8 bf[NF];
    {
      const uint16_t* src = ROLE == 0 ? a.k + krow * a.k_s + kv_head * DQK + 8 * hh
                                      : a.v + krow * a.v_s + kv_head * DV + 8 * hh;
      u32x4 u[12];
#pragma unroll
      for (int t = 0; t < 12; ++t) u[t] = u32x4{0u, 0u, 0u, 0u};
      if (k_valid) {
        ldg_x4(src, u[0], u[1], u[2], u[3]);
        ldg_x4(src + 64, u[4], u[5], u[6], u[7]);
        if (ROLE == 0) ldg_x4(src + 128, u[8], u[9], u[10], u[11]);
      }
#pragma unroll
      for (int t = 0; t < NF; ++t) bf[t] = __builtin_bit_cast(bf16x8, u[t]);
    }
    __syncthreads();  // LDS cleared before the first copies land
    if constexpr (ROLE == 1)
      for (int t = 0; t < KV_NSTAGE - 1 && t < n_tiles; ++t) kv_issue(smem, a, qr, t, qoff, ooff, head0, pair, lane);

    f32x16 acc[NACC];
#pragma unroll
    for (int c = 0; c < NACC; ++c) acc[c] = f32x16{};
    OperandOffsets o = operand_offsets(lane);

    for (int t = 0; t < n_tiles; ++t) {
      refresh(o);
      int q_row0, qpos, qn;
      tile_at(qr, kv_tile(qr, t, t / qr.nt), KV_BQ, q_row0, qpos, qn);
      // copies of tile t are done once at most the later tiles' copies issued so far (with
      // two stages: none) are still in flight
      if constexpr (ROLE == 1) {
        if (KV_NSTAGE > 2 && t + 1 < n_tiles) asm volatile("s_waitcnt vmcnt(%0)" ::"n"(KV_VMCNT_ONE_TILE) : "memory");
        else wait_dma();
      }
      barrier_lds();
      if constexpr (ROLE == 1)
        if (t + KV_NSTAGE - 1 < n_tiles) kv_issue(smem, a, qr, t + KV_NSTAGE - 1, qoff, ooff, head0, pair, lane);
      const lds_char* Qs = smem + (t % KV_NSTAGE) * KV_STAGE;
      const lds_char* Os = lds_opaque(Qs + KV_QBYTES);
      const lds_char* vec_s = lds_opaque(Qs + KV_QBYTES + KV_OBYTES);  // LSE2 then D, KV_VEC slots each

      if constexpr (ROLE == 0) {
        // ---------------- phase 1: S, P = exp(S - LSE) (masked), P to LDS for role B
        bf16x8 pk[KV_BQ / 16];  // P of this tile, bf16: rows 16*g .. 16*g+15 in pk[g]
        if (active) {
          // S of the 32-row sub-blocks.  Left to itself the compiler issues each read just
          // before its product and waits for it there; instead sub-block 0's reads are all
          // issued first, and each next sub-block's as the current one's products free
          // their registers.
          const RowBases qr_b = row_bases(Qs, o);
          bf16x8 qa[DQK / 16];
#pragma unroll
          for (int t2 = 0; t2 < DQK / 16; ++t2) qa[t2] = op_b128<KV_BQ>(qr_b, 0, t2);
          sched_fence();
          f32x16 sc[KV_NSB];
          static_for<KV_NSB>([&](auto sb_) {
            constexpr int sb = decltype(sb_)::value;
            sc[sb] = f32x16{};
#pragma unroll
            for (int t2 = 0; t2 < DQK / 16; ++t2) {
              sc[sb] = mfma(qa[t2], bf[t2], sc[sb]);
              if constexpr (sb + 1 < KV_NSB) qa[t2] = op_b128<KV_BQ>(qr_b, 32 * (sb + 1), t2);
            }
            sched_fence();
          });
          static_for<KV_BQ / 32>([&](auto sb_) {
            constexpr int sb = decltype(sb_)::value;
            const int qb = qpos + 32 * sb;
            const f32x16& s = sc[sb];
            // this lane's query rows are 32*sb + 8*hh + {0..7, 16..23}
            f32x4 l0, l1, l2, l3;
            lds_x4_f32<128 * sb, 128 * sb + 16, 128 * sb + 64, 128 * sb + 80>(vec_s, 32 * hh, l0, l1, l2, l3);
            const float lse_r[16] = {l0[0], l0[1], l0[2], l0[3], l1[0], l1[1], l1[2], l1[3],
                                     l2[0], l2[1], l2[2], l2[3], l3[0], l3[1], l3[2], l3[3]};
            const bool full = (kn_w == 32) && (qn >= 32 * (sb + 1)) && (wk_last <= qb) && (qb + 31 < hi_first);
            float p[16];
            if (full) {
#pragma unroll
              for (int e = 0; e < 16; ++e) p[e] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[e], sl2, -lse_r[e]));
            } else {
              // query row qq = base + c(e) is visible iff lo <= base + c(e) < lim, where base
              // is this lane's first row relative to its key position; masked entries get
              // exp2(-inf)
              const int base = qpos - pos_k + 32 * sb + 8 * hh;
              const int lim = k_valid ? max(0, min(qpos + qn, hi_k) - pos_k) : 0;
#pragma unroll
              for (int e = 0; e < 16; ++e) {
                const int r = base + 16 * (e >> 3) + (e & 7);
                const bool vis = (unsigned)r < (unsigned)lim;
                p[e] = __builtin_amdgcn_exp2f(vis ? __builtin_fmaf(s[e], sl2, -lse_r[e]) : -INFINITY);
              }
            }
            pk[2 * sb] = to_bf16x8(p);
            pk[2 * sb + 1] = to_bf16x8(p + 8);
            lds_st16<2048 * sb>(pbuf, poff, pk[2 * sb]);
            lds_st16<2048 * sb + 1024>(pbuf, poff, pk[2 * sb + 1]);
          });
        }
        barrier_lds();  // P of this tile is in LDS
        // ---------------- phase 2: dV^T[dv][key] += dO^T[dv][q] P[q][key]; groups of four
        // dO^T fragments, one per 16 query rows; a group's products are issued before the
        // next group loads
        if (active) {
          bf16x8 f[2][4];
          op_tr_x4<KV_BQ, 0, 0>(Os, o, f[0]);
          static_for<KV_BQ / 16>([&](auto g_) {
            constexpr int gq = decltype(g_)::value;
#pragma unroll
            for (int d = 0; d < DV / 32; ++d) acc[d] = mfma(f[gq & 1][d], pk[gq], acc[d]);
            if constexpr (gq + 1 < KV_BQ / 16) op_tr_x4<KV_BQ, 16 * (gq + 1), 0>(Os, o, f[(gq + 1) & 1]);
            sched_fence();
          });
        }
      } else {
        // ---------------- phase 1: dP = dO V^T of both sub-blocks
        f32x16 dp[KV_NSB];
        if (active) {
          // reads issued ahead as in role A's S
          const RowBases or_b = row_bases(Os, o);
          bf16x8 ob[DV / 16];
#pragma unroll
          for (int t2 = 0; t2 < DV / 16; ++t2) ob[t2] = op_b128<KV_BQ>(or_b, 0, t2);
          sched_fence();
          static_for<KV_NSB>([&](auto sb_) {
            constexpr int sb = decltype(sb_)::value;
            dp[sb] = f32x16{};
#pragma unroll
            for (int t2 = 0; t2 < DV / 16; ++t2) {
              dp[sb] = mfma(ob[t2], bf[t2], dp[sb]);
              if constexpr (sb + 1 < KV_NSB) ob[t2] = op_b128<KV_BQ>(or_b, 32 * (sb + 1), t2);
            }
            sched_fence();
          });
        }
        barrier_lds();  // P of this tile is in LDS
        // ---------------- phase 2: dS = P o (dP - D) of every sub-block first (its vector
        // work overlaps role A's dV products), then dK^T[c][key] += Q^T[c][q] dS[q][key]
        if (active) {
          bf16x8 sf[KV_NSB][2];
          static_for<KV_BQ / 32>([&](auto sb_) {
            constexpr int sb = decltype(sb_)::value;
            bf16x8 p0, p1;
            lds_x2_bf16<2048 * sb, 2048 * sb + 1024>(pbuf, poff, p0, p1);
            f32x4 d0, d1, d2, d3;
            lds_x4_f32<KV_VEC * 4 + 128 * sb, KV_VEC * 4 + 128 * sb + 16, KV_VEC * 4 + 128 * sb + 64,
                       KV_VEC * 4 + 128 * sb + 80>(vec_s, 32 * hh, d0, d1, d2, d3);
            const float D_r[16] = {d0[0], d0[1], d0[2], d0[3], d1[0], d1[1], d1[2], d1[3],
                                   d2[0], d2[1], d2[2], d2[3], d3[0], d3[1], d3[2], d3[3]};
            float ds[16];
#pragma unroll
            for (int e = 0; e < 16; ++e) {
              const float pv = (float)(e < 8 ? p0[e] : p1[e - 8]);
              ds[e] = pv * (dp[sb][e] - D_r[e]);
            }
            sf[sb][0] = to_bf16x8(ds);
            sf[sb][1] = to_bf16x8(ds + 8);
            if constexpr (STORE_DS) {
              // this pair's 32 keys x sub-block sb's 32 queries, 2 KB: two 1 KB stores in the
              // register layout (lane 32h + m: key m, queries 16*half + 8h .. +7), non-temporal
              // (read once, by the dQ kernel)
              typedef __attribute__((address_space(1))) u32x4 gu32x4;
              const int member = t / qr.nt, tl = kv_tile(qr, t, member);
              char* dst = a.ds + (int64_t)((kv_head - a.kv_head0) * a.grp + member) * a.ds_head_bytes +
                          (int64_t)(ds_slot0 + tl) * DS_TILE_BYTES + (sb * 4 + pair) * DS_BLOCK_BYTES + lane * 16;
              __builtin_nontemporal_store(__builtin_bit_cast(u32x4, sf[sb][0]), (gu32x4*)(dst));
              __builtin_nontemporal_store(__builtin_bit_cast(u32x4, sf[sb][1]), (gu32x4*)(dst + DS_BLOCK_BYTES / 2));
            }
          });
          static_for<KV_BQ / 32>([&](auto sb_) {
            constexpr int sb = decltype(sb_)::value;
            // groups of three Q^T column blocks
            bf16x8 f[2][3];
            op_tr_x3<KV_BQ, 32 * sb, 0>(Qs, o, f[0]);
            static_for<4>([&](auto g_) {
              constexpr int gq = decltype(g_)::value, half = gq >> 1, c0 = 3 * (gq & 1);
#pragma unroll
              for (int j = 0; j < 3; ++j) acc[c0 + j] = mfma(f[gq & 1][j], sf[sb][half], acc[c0 + j]);
              if constexpr (gq + 1 < 4)
                op_tr_x3<KV_BQ, 32 * sb + 16 * ((gq + 1) >> 1), 3 * ((gq + 1) & 1)>(Qs, o, f[(gq + 1) & 1]);
              sched_fence();
            });
          });
        }
      }
    }

    if (k_valid) {
      if constexpr (ROLE == 0) {
        float* dv = a.dv + (krow * a.Hkv + kv_head) * DV + 4 * hh;
#pragma unroll
        for (int d = 0; d < DV / 32; ++d)
#pragma unroll
          for (int rr = 0; rr < 4; ++rr) {
            f32x4* p = reinterpret_cast<f32x4*>(dv + 32 * d + 8 * rr);
            f32x4 old = *p;
            old[0] += acc[d][4 * rr];
            old[1] += acc[d][4 * rr + 1];
            old[2] += acc[d][4 * rr + 2];
            old[3] += acc[d][4 * rr + 3];
            *p = old;
          }
      } else {
        float* dk = a.dk + (krow * a.Hkv + kv_head) * DQK + 4 * hh;
#pragma unroll
        for (int c = 0; c < DQK / 32; ++c)
#pragma unroll
          for (int rr = 0; rr < 4; ++rr) {
            f32x4* p = reinterpret_cast<f32x4*>(dk + 32 * c + 8 * rr);
            f32x4 old = *p;
            old[0] += a.scale * acc[c][4 * rr];
            old[1] += a.scale * acc[c][4 * rr + 1];
            old[2] += a.scale * acc[c][4 * rr + 2];
            old[3] += a.scale * acc[c][4 * rr + 3];
            *p = old;
          }
      }
    }
  };
  if (role == 0) run(IntC<0>{});
  else run(IntC<1>{});
}

// ------------------------------------------------------------------ dQ from stored dS
// Query-stationary like bwd_dq, but reading the dS that bwd_dkdv<true> stored instead of
// recomputing S and dP: dQ^T[c][q] += K^T[c][key] dS^T[key][q], 384 of bwd_dq's 1024 FLOP
// per visible pair, and 2 bytes of dS read per pair (HBM-bound).  Eight waves x 32 query
// rows; keys walk the key items that the query tile's visible ranges touch, 64 keys (half
// an item) per tile.  Every 32-row query block coincides with one 32-row sub-block of each
// key item's query tiling (segments are 32-aligned on this path), so a wave finds its dS
// block from the item's ranges.
constexpr int DQS_BK = 64;                               // keys per tile
constexpr int DQS_KBYTES = DQS_BK * DQK * 2;             // 24 KB
constexpr int DQS_WAVE_BYTES = 2 * DS_BLOCK_BYTES;       // a wave's 32 queries x 64 keys of dS
constexpr int DQS_DBYTES = 8 * DQS_WAVE_BYTES;           // 32 KB
// K tiles (mostly L2 hits) are copied one tile ahead, the dS (read once, from HBM) two
// tiles ahead: 2 x 24 KB + 3 x 32 KB of LDS
constexpr int DQS_KSTAGES = 2, DQS_DSTAGES = 3;
constexpr int DQS_LDS = DQS_KSTAGES * DQS_KBYTES + DQS_DSTAGES * DQS_DBYTES;

// One tile of the walk (scalars): 64 keys of a key item, and where the wave's dS block for
// them sits (off < 0: the wave's rows do not see the item).  valid = 0 once the walk is over.
struct DsTile {
  int valid, krow0, kn;
  int64_t off;
};

// The walk over the key items that a query item's ranges touch, in row order, 64 keys at a
// time.  The item records live in row order, so within a range the next item's record is
// the next one; they are read through the constant address space, which makes them scalar
// loads that the compiler waits for where they are used (never together with the copies in
// flight, as vector loads after the copies' memory-clobbering assembly would be).
struct DsWalk {
  int rr, r, j;
  i32x16 rec;
};

typedef const __attribute__((address_space(4))) int cint;
typedef const __attribute__((address_space(4))) i32x16 crec16;

__device__ __forceinline__ DsTile ds_next(const AttnArgs& a, const Item& it, DsWalk& w, bool wave_rows, int qrow) {
  DsTile d;
  d.valid = 0;
  bool jump = w.j < 0;
  while (w.rr < it.nr) {
    const int kr = w.rr == 0 ? it.r0 : w.rr == 1 ? it.r1 : w.rr == 2 ? it.r2 : it.r3;
    const int kc = w.rr == 0 ? it.c0 : w.rr == 1 ? it.c1 : w.rr == 2 ? it.c2 : it.c3;
    if (w.r < kr) {
      w.r = kr;
      jump = true;
    }
    if (w.r < kr + kc) break;
    ++w.rr;
  }
  if (w.rr >= it.nr) return d;
  if (jump) {
    w.j = ((cint*)a.kmap32)[w.r >> 5];
    w.rec = *(crec16*)(a.krec + w.j * ITEM_INTS);
  } else if (w.r >= w.rec[0] + w.rec[1]) {  // past this item: the next one in row order
    ++w.j;
    w.rec = *(crec16*)(a.krec + w.j * ITEM_INTS);
  }
  const int half = (w.r - w.rec[0]) >> 6;
  d.valid = 1;
  d.krow0 = w.rec[0] + 64 * half;
  d.kn = min(DQS_BK, w.rec[1] - 64 * half);
  w.r = d.krow0 + DQS_BK;
  // the sub-block of the item's query tiling that holds the wave's rows [qrow, qrow + 32)
  d.off = -1;
  if (wave_rows) {
    int slot = w.rec[3];
#pragma unroll
    for (int k = 0; k < MAX_RANGES; ++k) {
      if (k >= w.rec[2]) break;
      const int row = w.rec[4 + 2 * k], cnt = w.rec[5 + 2 * k];
      if (qrow >= row && qrow < row + cnt) {
        const int u = (qrow - row) >> 5;
        const int sb = u % (KV_QTILE_ROWS / 32);
        d.off = (int64_t)(slot + u / (KV_QTILE_ROWS / 32)) * DS_TILE_BYTES + (sb * 4 + 2 * half) * DS_BLOCK_BYTES;
        break;
      }
      slot += (cnt + KV_QTILE_ROWS - 1) / KV_QTILE_ROWS;
    }
  }
  return d;
}

__global__ __launch_bounds__(512, 1) void bwd_dq_ds_kernel(AttnArgs a) {
  __shared__ __attribute__((aligned(1024))) char smem_raw[DQS_LDS];
  lds_char* smem = (lds_char*)smem_raw;
  lds_char* dsmem = smem + DQS_KSTAGES * DQS_KBYTES;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int m = lane & 31, hh = lane >> 5;
  int hl, item;
  xcd_head_item(blockIdx.x, a.q_heads, a.n_items, hl, item);
  const int head = a.q_head0 + hl;
  const Item it(a.items, item);
  const bool wave_rows = 32 * wave < it.n;  // the wave's 32 query rows (all valid or none)
  const int qrow0 = it.row0 + 32 * wave;
  DsWalk walk;
  walk.rr = 0;
  walk.r = 0;
  walk.j = -1;
  DsTile t0 = ds_next(a, it, walk, wave_rows, qrow0);
  if (!t0.valid) return;  // uniform over the workgroup
  const int kv_head = head / a.grp;
  const char* ds_head = a.ds + (int64_t)(head - a.q_head0) * a.ds_head_bytes;
  const int koff = dma_lane_off<DQK>(a.k_s, kv_head, wave, lane);
  // dS copy: LDS unit u = 4k + q8 (key k, queries 8*q8 .. +7) fetched from the stored
  // register layout (half q8/2, lane 32*(q8%2) + k)
  const int ds_voff = 1024 * ((lane >> 1) & 1) + 512 * (lane & 1) + 16 * (lane >> 2);
  // transpose read of the B operand: keys 8h' + 4v + j at query 16*(g%2) + i
  const int ds_rd = 512 * (lane >> 5) + 32 * ((lane >> 4) & 1) + 64 * ((lane >> 2) & 3) + 8 * (lane & 3);

  lds_clear<512>(smem, DQS_LDS, tid);
  __syncthreads();  // LDS cleared before the first copy lands

  // copies of tile d's K rows into K stage st (every wave its share)
  auto issue_k = [&](const DsTile& d, int st) {
    dma_tile<DQK, DQS_BK, 8>(smem + st * DQS_KBYTES, tile_rsrc(a.k, d.krow0, d.kn, a.k_s), koff, a.k_s, wave);
  };
  // this wave's dS block of tile d into dS stage st; returns the copy instructions issued
  // (0: the wave's rows do not see the tile's keys)
  auto issue_ds = [&](const DsTile& d, int st) -> int {
    if (d.off < 0) return 0;
    const int bytes = d.kn > 32 ? 2 * DS_BLOCK_BYTES : DS_BLOCK_BYTES;
    const u32x4 desc = tile_desc(ds_head, d.off, bytes);
    const uint32_t m0 = __builtin_amdgcn_readfirstlane(lds_addr(dsmem + st * DQS_DBYTES + wave * DQS_WAVE_BYTES));
    dma16_stream(m0, desc, ds_voff, 0);
    dma16_stream(m0 + 1024, desc, ds_voff, 256);
    if (d.kn <= 32) return 2;
    dma16_stream(m0 + 2048, desc, ds_voff, 2048);
    dma16_stream(m0 + 3072, desc, ds_voff, 2048 + 256);
    return 4;
  };

  f32x16 acc[DQK / 32];
#pragma unroll
  for (int c = 0; c < DQK / 32; ++c) acc[c] = f32x16{};
  OperandOffsets o = operand_offsets(lane);

  // issue order per wave: K(0) D(0) D(1) | K(1) D(2) | K(2) D(3) | ...: at the top of tile u
  // only D(u+1) (issued after K(u)) may still be in flight
  DsTile t1 = ds_next(a, it, walk, wave_rows, qrow0);
  issue_k(t0, 0);
  int n_cur = issue_ds(t0, 0);
  int n_1 = t1.valid ? issue_ds(t1, 1) : 0;
  DsTile t2;
  t2.valid = 0;
  if (t1.valid) t2 = ds_next(a, it, walk, wave_rows, qrow0);
  for (int u = 0;; ++u) {
    refresh(o);
    if (n_1 == 4) asm volatile("s_waitcnt vmcnt(4)" ::: "memory");
    else if (n_1 == 2) asm volatile("s_waitcnt vmcnt(2)" ::: "memory");
    else wait_dma();
    barrier_lds();
    int n_2 = 0;
    if (t1.valid) issue_k(t1, (u + 1) % DQS_KSTAGES);
    if (t2.valid) n_2 = issue_ds(t2, (u + 2) % DQS_DSTAGES);
    if (n_cur > 0) {
      const lds_char* Ks = smem + (u % DQS_KSTAGES) * DQS_KBYTES;
      const lds_char* Ds = dsmem + (u % DQS_DSTAGES) * DQS_DBYTES + wave * DQS_WAVE_BYTES + ds_rd;
      auto kstep = [&](auto s_) {
        constexpr int s = decltype(s_)::value;
        constexpr int base = 2048 * (s >> 1) + 1024 * (s & 1);
        const bf16x8 b = join(lds_tr8(Ds + base), lds_tr8(Ds + base + 256));
        bf16x8 f[2][3];
        op_tr_x3<DQS_BK, 16 * s, 0>(Ks, o, f[0]);
        op_tr_x3<DQS_BK, 16 * s, 3>(Ks, o, f[1]);
#pragma unroll
        for (int j = 0; j < 3; ++j) acc[j] = mfma(f[0][j], b, acc[j]);
#pragma unroll
        for (int j = 0; j < 3; ++j) acc[3 + j] = mfma(f[1][j], b, acc[3 + j]);
      };
      kstep(IntC<0>{});
      kstep(IntC<1>{});
      if (n_cur == 4) {
        kstep(IntC<2>{});
        kstep(IntC<3>{});
      }
    }
    if (!t1.valid) break;
    t1 = t2;
    n_cur = n_1;
    n_1 = n_2;
    if (t2.valid) t2 = ds_next(a, it, walk, wave_rows, qrow0);
  }

  if (wave_rows) {
    float* dq = a.dq + ((int64_t)(qrow0 + m) * a.H + head) * DQK + 4 * hh;
#pragma unroll
    for (int c = 0; c < DQK / 32; ++c)
#pragma unroll
      for (int rr2 = 0; rr2 < 4; ++rr2) {
        f32x4* p = reinterpret_cast<f32x4*>(dq + 32 * c + 8 * rr2);
        f32x4 old = *p;
        old[0] += a.scale * acc[c][4 * rr2];
        old[1] += a.scale * acc[c][4 * rr2 + 1];
        old[2] += a.scale * acc[c][4 * rr2 + 2];
        old[3] += a.scale * acc[c][4 * rr2 + 3];
        *p = old;
      }
  }
}

// kv_heads_per_pass = 0: recompute path (bwd_dq + bwd_dkdv over all heads).  Otherwise the
// stored-dS path, in passes of that many K/V heads (the dS of one pass's query heads fits
// a.ds): bwd_dkdv<true> stores dS, then bwd_dq_ds reads it back.
hipError_t launch_attn_bwd(const AttnArgs& a, int n_qitems, int n_kitems, const int* kitems, int kv_heads_per_pass,
                           hipStream_t stream) {
  const int64_t pairs = (int64_t)a.nq * a.H;
  const int64_t blocks = (pairs + 15) / 16 < (1 << 20) ? (pairs + 15) / 16 : (1 << 20);
  int tok = prof_begin("bwd_pre", stream);
  hipLaunchKernelGGL(bwd_pre_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, a.o, a.dO, a.lse, a.Dvec,
                     a.lse2, a.nq, a.H);
  prof_end(tok, stream);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (kv_heads_per_pass > 0) {
    if (n_qitems == 0 || n_kitems == 0) return hipSuccess;
    for (int g0 = 0; g0 < a.Hkv; g0 += kv_heads_per_pass) {
      const int G = min(kv_heads_per_pass, a.Hkv - g0);
      AttnArgs b = a;
      b.items = kitems;
      b.n_items = n_kitems;
      b.kv_head0 = g0;
      b.kv_heads = G;
      b.q_head0 = g0 * a.grp;
      b.q_heads = G * a.grp;
      tok = prof_begin("bwd_dkdv_ds", stream);
      hipLaunchKernelGGL(bwd_dkdv_kernel<true>, dim3(n_kitems * G), dim3(512), 0, stream, b);
      prof_end(tok, stream);
      if ((e = hipGetLastError()) != hipSuccess) return e;
      AttnArgs c = b;
      c.items = a.items;
      c.n_items = n_qitems;
      tok = prof_begin("bwd_dq_ds", stream);
      hipLaunchKernelGGL(bwd_dq_ds_kernel, dim3(n_qitems * G * a.grp), dim3(512), 0, stream, c);
      prof_end(tok, stream);
      if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    return hipSuccess;
  }
  if (n_qitems > 0) {
    AttnArgs b = a;
    b.n_items = n_qitems;
    tok = prof_begin("bwd_dq", stream);
    hipLaunchKernelGGL(bwd_dq_kernel, dim3(n_qitems * a.H), dim3(64 * DQ_WAVES), 0, stream, b);
    prof_end(tok, stream);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (n_kitems > 0) {
    AttnArgs b = a;
    b.items = kitems;
    b.n_items = n_kitems;
    tok = prof_begin("bwd_dkdv", stream);
    hipLaunchKernelGGL(bwd_dkdv_kernel<false>, dim3(n_kitems * a.Hkv), dim3(512), 0, stream, b);
    prof_end(tok, stream);
    e = hipGetLastError();
  }
  return e;
}

}  // namespace hydra
