// Device-side building blocks shared by the gfx950 attention kernels.
//
// Matrix-core conventions (v_mfma_f32_32x32x16_bf16, wave64), lane l = 32*h + m:
//   A operand (32 x 16): lane holds A[m][8h .. 8h+7]
//   B operand (16 x 32): lane holds B[8h .. 8h+7][m]
//   C (32 x 32, 16 fp32 per lane): reg r holds C[8*(r/4) + 4h + r%4][m]
// A tile whose rows are read from LDS in the order pi(row) (bits 2 and 3 of the row
// index swapped) therefore produces C rows with reg r <-> row 16*(r/8) + 8h + r%8: each
// lane holds two runs of 8 consecutive rows, which is exactly the k-slice layout of the
// next contraction's B operand.  Scores computed that way feed P*V (and dS*K, dS*Q,
// P*dO) straight from registers, with no shuffle.
//
// ds_read_b64_tr_b16 (LDS transpose read): within each 16-lane group, lane i receives
// element (i % 4) of the 8-byte words addressed by lanes 4j + i/4, j = 0..3.  Pointing
// lane i at row (base_row + i/4), column (base_col + 4*(i%4)) of a row-major bf16 tile
// gives lane i the column (base_col + i) for rows base_row .. base_row+3: a transposed
// operand fragment without a transposed copy in memory.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace hydra {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) char lds_char;

constexpr int DQK = 192;
constexpr int DV = 128;
constexpr int ITEM_INTS = 16;
constexpr int MAX_RANGES = 4;
constexpr float LOG2E = 1.4426950408889634f;
constexpr float LN2 = 0.6931471805599453f;
constexpr float NEG_BIG = -1.0e30f;  // finite running-max floor: keeps exp2 arguments NaN-free

// LDS row pitches (bf16 elements): 16 bytes of padding per row spreads consecutive rows
// over different banks for 16-byte reads.
constexpr int PITCH_QK = DQK + 8;  // 400 bytes
constexpr int PITCH_V = DV + 8;    // 272 bytes

__device__ __forceinline__ int pi_row(int m) { return (m & ~12) | ((m & 4) << 1) | ((m & 8) >> 1); }

__device__ __forceinline__ f32x16 mfma(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float fmax2(float a, float b) { return a > b ? a : b; }

// Value held by the lane 32 positions away (m stays, h flips) and the max / sum with it.
__device__ __forceinline__ float xhalf_max(float v) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmax2(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float xhalf_sum(float v) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

__device__ __forceinline__ bf16x8 lds_read8(const __bf16* p) {
  return *reinterpret_cast<const bf16x8*>(p);
}

// Two transpose reads: rows r0..r0+3 and r0+4..r0+7 (see the header comment).
__device__ __forceinline__ bf16x8 lds_read8_tr(const __bf16* p0, const __bf16* p1) {
  i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) i16x4*)(
      (lds_char*)(p0)));
  i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) i16x4*)(
      (lds_char*)(p1)));
  typedef short i16x8 __attribute__((ext_vector_type(8)));
  i16x8 v = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
  return __builtin_bit_cast(bf16x8, v);
}

__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  __bf16 x = (__bf16)a, y = (__bf16)b;
  return uint32_t(__builtin_bit_cast(uint16_t, x)) | (uint32_t(__builtin_bit_cast(uint16_t, y)) << 16);
}

// Eight fp32 values -> one bf16 operand fragment (round to nearest even).
__device__ __forceinline__ bf16x8 to_bf16x8(const float* v) {
  u32x4 u;
  u[0] = pack_bf16x2(v[0], v[1]);
  u[1] = pack_bf16x2(v[2], v[3]);
  u[2] = pack_bf16x2(v[4], v[5]);
  u[3] = pack_bf16x2(v[6], v[7]);
  return __builtin_bit_cast(bf16x8, u);
}

__device__ __forceinline__ u32x4 ldg16(const void* p) { return *reinterpret_cast<const u32x4*>(p); }

// Largest d with cu[d] <= pos (cu has n_docs + 1 entries, pos inside the window).
__device__ __forceinline__ int doc_of(const int* __restrict__ cu, int n_docs, int pos) {
  int lo = 0, hi = n_docs;
  while (hi - lo > 1) {
    int mid = (lo + hi) >> 1;
    if (cu[mid] <= pos) lo = mid; else hi = mid;
  }
  return lo;
}

// Stage `rows` rows (of at most 32*n_sub) of a [token][head][dim] bf16 tensor into an LDS
// tile with the given pitch; rows beyond `valid` are zero-filled.
template <int DIM, int PITCH, int ROWS, int THREADS>
__device__ __forceinline__ void stage_rows(__bf16* lds, const uint16_t* __restrict__ g, int64_t row0,
                                           int valid, int H, int head, int tid) {
  constexpr int CH = DIM / 8;  // 16-byte chunks per row
  constexpr int TOTAL = ROWS * CH;
  static_assert(TOTAL % THREADS == 0, "tile must split evenly over the workgroup");
#pragma unroll
  for (int i = 0; i < TOTAL / THREADS; ++i) {
    const int c = tid + i * THREADS;
    const int r = c / CH, col = (c % CH) * 8;
    u32x4 val = {0u, 0u, 0u, 0u};
    if (r < valid) val = ldg16(g + ((row0 + r) * H + head) * (int64_t)DIM + col);
    *reinterpret_cast<u32x4*>(lds + r * PITCH + col) = val;
  }
}

struct AttnArgs {
  const uint16_t* q;   // [nq][H][192]
  const uint16_t* k;   // [nk][H][192]
  const uint16_t* v;   // [nk][H][128]
  const uint16_t* o;   // bwd: final O bf16 [nq][H][128]
  const uint16_t* dO;  // bwd: [nq][H][128]
  const float* lse;    // bwd: final LSE [H][nq]
  float* out_o;        // fwd: O partial fp32
  float* out_lse;      // fwd: LSE partial
  float* dq;           // bwd accumulators
  float* dk;
  float* dv;
  float* Dvec;         // bwd: [H][nq] rowsum(dO * O)
  const int* items;    // work items
  const int* cu;       // document boundaries
  int n_docs;
  int n_items;
  int H;
  int nq, nk;
  float scale;         // softmax scale
};

}  // namespace hydra
