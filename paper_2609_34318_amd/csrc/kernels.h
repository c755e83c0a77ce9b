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

// 16-byte global load as inline assembly, for operands loaded once before a tile loop whose
// copies are waited for with partial vmcnt counts: the compiler's wait insertion would
// otherwise keep such registers "possibly pending" across the loop back edge and wait for
// every copy in flight before each use.  Complete them with wait_vmem_all() before use.
__device__ __forceinline__ u32x4 ldg16_asm(const void* p) {
  u32x4 v;
  asm volatile("global_load_dwordx4 %0, %1, off" : "=v"(v) : "v"(p) : "memory");
  return v;
}

// Largest d with cu[d] <= pos (cu has n_docs + 1 entries, pos inside the window).
__device__ __forceinline__ int doc_of(const int* __restrict__ cu, int n_docs, int pos) {
  int lo = 0, hi = n_docs;
  while (hi - lo > 1) {
    int mid = (lo + hi) >> 1;
    if (cu[mid] <= pos) lo = mid; else hi = mid;
  }
  return lo;
}

// ------------------------------------------------------------------ swizzled LDS tiles
// Tiles are stored unpadded.  d = 128 tiles: ROWS rows of 256 B.  d = 192 tiles: three
// column blocks of 64 elements, each ROWS rows of 128 B, so that one 1 KB direct-to-LDS
// instruction always covers whole rows (4 or 8).  Within a row the 16-byte chunk c lives at
// chunk c ^ swz(r); the XOR spreads both the 16-byte operand reads (16 rows, one chunk) and
// the transpose reads (4 rows x 4 chunks) over all 64 LDS banks.
__device__ __forceinline__ int swz256(int r) { return ((r & 3) << 2) | ((r >> 2) & 3); }
__device__ __forceinline__ int swz128(int r) { return (((r >> 1) & 1) << 2) | ((r >> 2) & 3); }

// Byte offset of logical 16-byte chunk `c` of row `r` in a tile of ROWS rows.
template <int DIM, int ROWS> __device__ __forceinline__ int tile_off(int r, int c);
template <> __device__ __forceinline__ int tile_off<128, 64>(int r, int c) { return r * 256 + ((c ^ swz256(r)) << 4); }
template <> __device__ __forceinline__ int tile_off<128, 32>(int r, int c) { return r * 256 + ((c ^ swz256(r)) << 4); }
template <> __device__ __forceinline__ int tile_off<192, 64>(int r, int c) {
  return (c >> 3) * (64 * 128) + r * 128 + (((c & 7) ^ swz128(r)) << 4);
}
template <> __device__ __forceinline__ int tile_off<192, 32>(int r, int c) {
  return (c >> 3) * (32 * 128) + r * 128 + (((c & 7) ^ swz128(r)) << 4);
}

__device__ __forceinline__ bf16x8 lds_ld16(const lds_char* base, int off) {
  return *reinterpret_cast<const __attribute__((address_space(3))) bf16x8*>(base + off);
}

__device__ __forceinline__ i16x4 lds_tr8(const lds_char* base, int off) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) i16x4*)(base + off));
}

// Transposed operand fragment: each lane points at row `row` (and row + 4) and element
// column `col`; the transpose read hands lane i of each 16-lane group one column of the
// 4 x 16 block its group addressed (see the header comment).
template <int DIM, int ROWS>
__device__ __forceinline__ bf16x8 lds_tr_frag(const lds_char* base, int row, int col) {
  const int c = col >> 3, w = (col & 7) << 1;
  i16x4 lo = lds_tr8(base, tile_off<DIM, ROWS>(row, c) + w);
  i16x4 hi = lds_tr8(base, tile_off<DIM, ROWS>(row + 4, c) + w);
  typedef short i16x8 __attribute__((ext_vector_type(8)));
  i16x8 v = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
  return __builtin_bit_cast(bf16x8, v);
}

// The same transpose read issued as inline assembly.  The compiler's wait insertion treats
// the builtin as a possible alias of every direct-to-LDS copy still in flight (including
// the prefetch into the other stage) and waits for all of them first; the asm form is not
// tracked by that pass, so the caller must wait for it explicitly with lds_wait(), which
// also ties the fragments to the wait so their consumers cannot move above it.
__device__ __forceinline__ i16x4 lds_tr8_asm(const lds_char* base, int off) {
  i16x4 v;
  const uint32_t addr = (uint32_t)(uintptr_t)(base + off);
  asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(v) : "v"(addr) : "memory");
  return v;
}

template <int DIM, int ROWS>
__device__ __forceinline__ bf16x8 lds_tr_frag_async(const lds_char* base, int row, int col) {
  const int c = col >> 3, w = (col & 7) << 1;
  i16x4 lo = lds_tr8_asm(base, tile_off<DIM, ROWS>(row, c) + w);
  i16x4 hi = lds_tr8_asm(base, tile_off<DIM, ROWS>(row + 4, c) + w);
  typedef short i16x8 __attribute__((ext_vector_type(8)));
  i16x8 v = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
  return __builtin_bit_cast(bf16x8, v);
}

// Four floats from LDS as inline assembly (same reason as lds_tr8_asm); wait with lds_wait4.
__device__ __forceinline__ f32x4 lds_f4_asm(const lds_char* base, int off) {
  f32x4 v;
  const uint32_t addr = (uint32_t)(uintptr_t)(base + off);
  asm volatile("ds_read_b128 %0, %1" : "=v"(v) : "v"(addr) : "memory");
  return v;
}
__device__ __forceinline__ void lds_wait4(f32x4& a, f32x4& b, f32x4& c, f32x4& d) {
  asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(a), "+v"(b), "+v"(c), "+v"(d)::"memory");
}

// Waits for every outstanding LDS read and marks the fragments as produced here.
__device__ __forceinline__ void lds_wait(bf16x8& a, bf16x8& b, bf16x8& c, bf16x8& d) {
  asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(a), "+v"(b), "+v"(c), "+v"(d)::"memory");
}
__device__ __forceinline__ void lds_wait(bf16x8& a, bf16x8& b) {
  asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(a), "+v"(b)::"memory");
}
__device__ __forceinline__ void lds_wait(bf16x8& a, bf16x8& b, bf16x8& c) {
  asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(a), "+v"(b), "+v"(c)::"memory");
}

// ------------------------------------------------------------------ direct global -> LDS copies
// A buffer resource is built per tile with its base at the tile's first row and its record
// count ending at the tile's last valid row, so rows past the end are out of range for the
// hardware bounds check and never touch memory (all of the offset travels in the VGPR
// operand, which is what the check covers) (the kernels mask those rows and clear LDS
// once at start, so whatever the copy leaves there is finite).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t tile_rsrc(const uint16_t* g, int64_t row0, int valid, int H,
                                                            int dim) {
  const uint16_t* base = g + row0 * H * (int64_t)dim;
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(base), (short)0, valid * H * dim * 2, 0x00020000);
}

// Per-lane byte offset (tile-independent) for dma_tile with 4 waves.  Lane L of wave w writes
// bytes [16L, 16L+16) of each 1 KB instruction, which holds rows 4j..4j+3 (d = 128) or
// 8j..8j+7 of one column block (d = 192), j = w + 4i; it fetches the logical chunk the
// swizzle places there.
template <int DIM> __device__ __forceinline__ int dma_lane_off(int H, int head, int wave, int lane);
template <> __device__ __forceinline__ int dma_lane_off<128>(int H, int head, int wave, int lane) {
  const int q = lane >> 4;
  const int lc = (lane & 15) ^ ((q << 2) | (wave & 3));
  return (((4 * wave + q) * H + head) * 128 + lc * 8) * 2;
}
template <> __device__ __forceinline__ int dma_lane_off<192>(int H, int head, int wave, int lane) {
  const int q = lane >> 3;
  const int lc = (lane & 7) ^ ((((q >> 1) & 1) << 2) | ((wave & 1) << 1) | (q >> 2));
  return (((8 * wave + q) * H + head) * 192 + lc * 8) * 2;
}

// voff + inc, computed where it is used: the compiler would otherwise hoist one VGPR per
// copy instruction out of the tile loop and, under register pressure, spill them (the
// reloads then wait on every copy in flight).
__device__ __forceinline__ int add_here(int voff, int inc) {
  int o;
  asm volatile("v_add_u32 %0, %1, %2" : "=v"(o) : "s"(inc), "v"(voff));
  return o;
}

template <int DIM, int ROWS>
__device__ __forceinline__ void dma_tile(lds_char* lds, __amdgpu_buffer_rsrc_t rs, int voff, int H, int wave) {
  typedef __attribute__((address_space(3))) void lds_void;
  if constexpr (DIM == 128) {
    constexpr int NINS = ROWS / 4;
    static_assert(NINS % 4 == 0, "tile must split evenly over 4 waves");
#pragma unroll
    for (int i = 0; i < NINS / 4; ++i)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_void*)(lds + (wave + 4 * i) * 1024), 16,
                                               i == 0 ? voff : add_here(voff, 16 * i * H * 256), 0, 0, 0);
  } else {
    constexpr int NINS = ROWS / 8;  // per column block
    static_assert(NINS % 4 == 0, "tile must split evenly over 4 waves");
#pragma unroll
    for (int b = 0; b < 3; ++b)
#pragma unroll
      for (int i = 0; i < NINS / 4; ++i)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_void*)(lds + b * ROWS * 128 + (wave + 4 * i) * 1024), 16,
                                                 (b == 0 && i == 0) ? voff : add_here(voff, 32 * i * H * 384 + b * 128),
                                                 0, 0, 0);
  }
}

// 64 consecutive floats (one per lane) into LDS; entries past `valid` are out of range.
__device__ __forceinline__ void dma_vec64(lds_char* lds, const float* g, int valid, int lane) {
  typedef __attribute__((address_space(3))) void lds_void;
  __amdgpu_buffer_rsrc_t rs =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(g), (short)0, valid * 4, 0x00020000);
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_void*)lds, 4, lane * 4, 0, 0, 0);
}

__device__ __forceinline__ void wait_dma() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// Workgroup barrier for the tile loops: this wave's LDS reads are finished and every wave
// has arrived.  Copies into LDS are waited for explicitly (wait_dma / vmcnt) before it;
// unlike __syncthreads it does not also wait for the copies still in flight for later tiles.
__device__ __forceinline__ void barrier_lds() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// Clears `bytes` (multiple of 16 * threads) of LDS.
template <int THREADS>
__device__ __forceinline__ void lds_clear(lds_char* lds, int bytes, int tid) {
  for (int o = tid * 16; o < bytes; o += THREADS * 16)
    *reinterpret_cast<__attribute__((address_space(3))) u32x4*>(lds + o) = u32x4{0u, 0u, 0u, 0u};
}

// A work item (16 ints, see the plan), read once into scalar registers.  Plain scalar
// members only: an array here would be placed in scratch memory and indexed dynamically.
struct Item {
  int row0, pos0, n, nr;
  int r0, p0, c0, r1, p1, c1, r2, p2, c2, r3, p3, c3;

  __device__ __forceinline__ Item(const int* items, int idx) {
    const int* s = items + idx * ITEM_INTS;
    row0 = __builtin_amdgcn_readfirstlane(s[0]);
    pos0 = __builtin_amdgcn_readfirstlane(s[1]);
    n = __builtin_amdgcn_readfirstlane(s[2]);
    nr = __builtin_amdgcn_readfirstlane(s[3]);
    r0 = __builtin_amdgcn_readfirstlane(s[4]);
    p0 = __builtin_amdgcn_readfirstlane(s[5]);
    c0 = nr > 0 ? __builtin_amdgcn_readfirstlane(s[6]) : 0;
    r1 = __builtin_amdgcn_readfirstlane(s[7]);
    p1 = __builtin_amdgcn_readfirstlane(s[8]);
    c1 = nr > 1 ? __builtin_amdgcn_readfirstlane(s[9]) : 0;
    r2 = __builtin_amdgcn_readfirstlane(s[10]);
    p2 = __builtin_amdgcn_readfirstlane(s[11]);
    c2 = nr > 2 ? __builtin_amdgcn_readfirstlane(s[12]) : 0;
    r3 = __builtin_amdgcn_readfirstlane(s[13]);
    p3 = __builtin_amdgcn_readfirstlane(s[14]);
    c3 = nr > 3 ? __builtin_amdgcn_readfirstlane(s[15]) : 0;
  }
};

// The ranges of a work item cut into tiles of B rows (the last tile of a range may be short).
// A value type of scalars: pass it by value and never take its address, so that it stays in
// scalar registers (a select between fields of a struct in memory becomes a scratch load
// with a dynamic index).
struct TileRanges {
  int r0, p0, c0, r1, p1, c1, r2, p2, c2, r3, p3, c3;
  int f1, f2, f3, nt;  // first tile of ranges 1..3, total tiles
};

__device__ __forceinline__ TileRanges tile_ranges(const Item& it, int B) {
  TileRanges R;
  R.r0 = it.r0; R.p0 = it.p0; R.c0 = it.c0;
  R.r1 = it.r1; R.p1 = it.p1; R.c1 = it.c1;
  R.r2 = it.r2; R.p2 = it.p2; R.c2 = it.c2;
  R.r3 = it.r3; R.p3 = it.p3; R.c3 = it.c3;
  R.f1 = (R.c0 + B - 1) / B;
  R.f2 = R.f1 + (R.c1 + B - 1) / B;
  R.f3 = R.f2 + (R.c2 + B - 1) / B;
  R.nt = R.f3 + (R.c3 + B - 1) / B;
  return R;
}

// Rows [row0, row0 + n) at global positions [pos0, pos0 + n) of tile t < R.nt.
__device__ __forceinline__ void tile_at(const TileRanges R, int t, int B, int& row0, int& pos0, int& n) {
  int rr = R.r0, pp = R.p0, cc = R.c0, ff = 0;
  if (t >= R.f1) { rr = R.r1; pp = R.p1; cc = R.c1; ff = R.f1; }
  if (t >= R.f2) { rr = R.r2; pp = R.p2; cc = R.c2; ff = R.f2; }
  if (t >= R.f3) { rr = R.r3; pp = R.p3; cc = R.c3; ff = R.f3; }
  const int off = (t - ff) * B;
  row0 = rr + off;
  pos0 = pp + off;
  n = min(B, cc - off);
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
  float* lse2;         // bwd: [H][nq] final LSE * log2(e)
  const int* items;    // work items
  const int* cu;       // document boundaries
  int n_docs;
  int n_items;
  int H;
  int nq, nk;
  float scale;         // softmax scale
};

}  // namespace hydra
