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

#include <utility>

#include "tiles.h"

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

__device__ __forceinline__ int pi_row(int m) { return (m & ~12) | ((m & 4) << 1) | ((m & 8) >> 1); }

__device__ __forceinline__ f32x16 mfma(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// IEEE 754-2019 maximum (a NaN operand gives NaN; scores never are NaN).  Unlike fmax it
// needs no canonicalising v_max of each operand first: nested calls become v_maximum3_f32.
__device__ __forceinline__ float fmax2(float a, float b) { return __builtin_elementwise_maximum(a, b); }

// Value held by the lane 32 positions away (m stays, h flips) and the max / sum with it.
__device__ __forceinline__ float xhalf_max(float v) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmax2(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float xhalf_sum(float v) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  __bf16 x = (__bf16)a, y = (__bf16)b;
  return uint32_t(__builtin_bit_cast(uint16_t, x)) | (uint32_t(__builtin_bit_cast(uint16_t, y)) << 16);
}

// Eight fp32 values -> one bf16 operand fragment (round to nearest even, v_cvt_pk_bf16_f32).
__device__ __forceinline__ bf16x8 to_bf16x8(const float* v) {
  typedef float f32x8 __attribute__((ext_vector_type(8)));
  const f32x8 x = {v[0], v[1], v[2], v[3], v[4], v[5], v[6], v[7]};
  return __builtin_convertvector(x, bf16x8);
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

// ------------------------------------------------------------------ swizzled LDS tiles
// A tile of ROWS rows and DIM (128 or 192) bf16 columns is stored as DIM/64 column blocks of
// 64 elements; each block is ROWS rows of 128 bytes, unpadded, so that one 1 KB direct-to-LDS
// instruction covers 8 whole rows.  Within a row the 16-byte chunk c (0..7) lives at chunk
// c ^ swz(r), which spreads both the 16-byte operand reads (16 rows, one chunk) and the
// transpose reads (4 rows x 4 chunks) over all 64 LDS banks.  swz(r) only looks at bits
// 1..3 of r, so every read below is a per-lane constant plus a compile-time offset.
__device__ __forceinline__ int swz(int r) { return (((r >> 1) & 1) << 2) | ((r >> 2) & 3); }

template <int ROWS> constexpr int block_bytes() { return ROWS * 128; }

// Lane-constant parts of the operand reads of a 32x32x16 MFMA from such tiles.
//   b128[j]: 16-byte read of row pi(m), chunk 2j + h within a column block (k-step t uses
//            j = t & 3, block t >> 2)
//   tr[v][k]: transpose read at row (v ? 4 : 0) + 8h + i/4, column 32*cb + 16*(g&1) + 4*(i&3)
//            with k = cb & 1 (block cb >> 1)
// Callers add row_block*128 (row_block a multiple of 16) and block*block_bytes as immediates.
struct OperandOffsets {
  int b128[4];
  int tr[2][2];
};

__device__ __forceinline__ OperandOffsets operand_offsets(int lane) {
  const int m = lane & 31, h = lane >> 5, g = lane >> 4, gi = lane & 15;
  OperandOffsets o;
  const int ra = pi_row(m);
#pragma unroll
  for (int j = 0; j < 4; ++j) o.b128[j] = ra * 128 + (((2 * j + h) ^ swz(ra)) << 4);
  const int rt = 8 * h + (gi >> 2);
  const int cl = 2 * (g & 1) + ((gi & 3) >> 1);  // chunk within 4, plus the 8-byte half below
  const int w = (gi & 1) << 3;
#pragma unroll
  for (int v = 0; v < 2; ++v)
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      const int r = rt + 4 * v;
      o.tr[v][k] = r * 128 + (((4 * k + cl) ^ swz(r)) << 4) + w;
    }
  return o;
}

// Makes the offsets opaque at the top of each tile iteration, in place: otherwise the
// compiler hoists every (offset + immediate) sum out of the tile loop, one register each,
// instead of folding the immediate into the read's offset field.  In place, so that no
// second copy of the offsets stays live across the loop.
__device__ __forceinline__ void refresh(OperandOffsets& o) {
#pragma unroll
  for (int j = 0; j < 4; ++j) asm volatile("" : "+v"(o.b128[j]));
#pragma unroll
  for (int v = 0; v < 2; ++v)
#pragma unroll
    for (int k = 0; k < 2; ++k) asm volatile("" : "+v"(o.tr[v][k]));
}

__device__ __forceinline__ bf16x8 lds_ld16(const lds_char* base, int off) {
  return *reinterpret_cast<const __attribute__((address_space(3))) bf16x8*>(base + off);
}

// This lane's four read addresses of b128 operands in a tile (row pi(m), one per 16-byte
// chunk of a 64-column block), opaque to the compiler: every read is then base + an
// immediate offset (column block, row block), with no address add per read.  Left to
// itself the compiler addresses the reads of a phase from its last read, with negative
// offsets that the unsigned offset field of an LDS read cannot hold.
struct RowBases {
  const lds_char* p[4];
};

__device__ __forceinline__ RowBases row_bases(const lds_char* tile, const OperandOffsets& o) {
  RowBases r;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    r.p[j] = tile + o.b128[j];
    asm volatile("" : "+v"(r.p[j]));
  }
  return r;
}

// k-step t of a b128 operand at rows row_block + pi(m) of a ROWS-row tile.
template <int ROWS>
__device__ __forceinline__ bf16x8 op_b128(const lds_char* tile, const OperandOffsets& o, int row_block, int t) {
  return lds_ld16(tile, o.b128[t & 3] + (t >> 2) * block_bytes<ROWS>() + row_block * 128);
}

// The same read from opaque bases.
template <int ROWS>
__device__ __forceinline__ bf16x8 op_b128(const RowBases& r, int row_block, int t) {
  return lds_ld16(r.p[t & 3], (t >> 2) * block_bytes<ROWS>() + row_block * 128);
}

// ------------------------------------------------------------------ LDS operand reads
// Plain LDS loads and the transpose-read builtin: the compiler schedules them ahead of their
// uses and waits for exactly the reads it needs.  It never sees the direct-to-LDS copies
// (those are inline assembly, below), so it never waits for a copy still in flight; the
// kernels wait for their copies explicitly and publish them with a barrier.

template <int N> struct IntC { static constexpr int value = N; };

// Calls f(IntC<0>{}) .. f(IntC<N-1>{}) (compile-time loop index).
template <class F, int... I>
__device__ __forceinline__ void static_for_impl(F&& f, std::integer_sequence<int, I...>) {
  (f(IntC<I>{}), ...);
}
template <int N, class F> __device__ __forceinline__ void static_for(F&& f) {
  static_for_impl(f, std::make_integer_sequence<int, N>{});
}

__device__ __forceinline__ uint32_t lds_addr(const lds_char* p) { return (uint32_t)(uintptr_t)p; }

// The same (wave-uniform) LDS address, opaque to the compiler.  Without it the compiler
// addresses one tile's reads as offsets from another tile's base, and the negative ones do
// not fit the unsigned offset field of an LDS read, so each costs its own address add.
__device__ __forceinline__ const lds_char* lds_opaque(const lds_char* p) {
  asm volatile("" : "+s"(p));
  return p;
}

__device__ __forceinline__ bf16x8 join(i16x4 lo, i16x4 hi) {
  typedef short i16x8 __attribute__((ext_vector_type(8)));
  i16x8 v = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
  return __builtin_bit_cast(bf16x8, v);
}

__device__ __forceinline__ i16x4 lds_tr8(const lds_char* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) i16x4*)(p));
}

// Transposed operand fragments for column blocks CB0 .. CB0+N-1 of rows ROWB .. ROWB+15 of
// a ROWS-row tile (lane pattern of OperandOffsets::tr).
template <int ROWS, int ROWB, int CB0, int N>
__device__ __forceinline__ void op_tr(const lds_char* tile, const OperandOffsets& o, bf16x8 (&f)[N]) {
#pragma unroll
  for (int n = 0; n < N; ++n) {
    const lds_char* b = tile + ((CB0 + n) >> 1) * block_bytes<ROWS>() + ROWB * 128;
    f[n] = join(lds_tr8(b + o.tr[0][(CB0 + n) & 1]), lds_tr8(b + o.tr[1][(CB0 + n) & 1]));
  }
}
template <int ROWS, int ROWB, int CB0>
__device__ __forceinline__ void op_tr_x4(const lds_char* tile, const OperandOffsets& o, bf16x8 (&f)[4]) {
  op_tr<ROWS, ROWB, CB0, 4>(tile, o, f);
}
template <int ROWS, int ROWB, int CB0>
__device__ __forceinline__ void op_tr_x3(const lds_char* tile, const OperandOffsets& o, bf16x8 (&f)[3]) {
  op_tr<ROWS, ROWB, CB0, 3>(tile, o, f);
}

// Four 16-byte LDS reads at base + lane_off + I0..I3.
template <int I0, int I1, int I2, int I3>
__device__ __forceinline__ void lds_x4_f32(const lds_char* base, int lane_off, f32x4& a, f32x4& b, f32x4& c,
                                           f32x4& d) {
  typedef const __attribute__((address_space(3))) f32x4* P;
  const lds_char* p = base + lane_off;
  a = *reinterpret_cast<P>(p + I0);
  b = *reinterpret_cast<P>(p + I1);
  c = *reinterpret_cast<P>(p + I2);
  d = *reinterpret_cast<P>(p + I3);
}

// Two 16-byte LDS reads at base + lane_off + I0, I1.
template <int I0, int I1>
__device__ __forceinline__ void lds_x2_bf16(const lds_char* base, int lane_off, bf16x8& a, bf16x8& b) {
  a = lds_ld16(base + lane_off, I0);
  b = lds_ld16(base + lane_off, I1);
}

// 16-byte LDS store of an operand fragment.
template <int I0>
__device__ __forceinline__ void lds_st16(lds_char* base, int lane_off, bf16x8 v) {
  *reinterpret_cast<__attribute__((address_space(3))) bf16x8*>(base + lane_off + I0) = v;
}

// Keeps the instruction scheduler from moving anything across this point (used between
// the groups of a software-pipelined loop so that reads are not all hoisted to its top,
// which would need registers for every group at once).
__device__ __forceinline__ void sched_fence() { __builtin_amdgcn_sched_barrier(0); }

// Makes the compiler treat x as freshly produced here: a value loaded before a tile loop
// and passed through settle() right after its load is waited for at that point, not at its
// first use inside the loop (where the wait would also cover every copy in flight).
template <class T> __device__ __forceinline__ void settle(T& x) { asm volatile("" : "+v"(x)); }

// Four 16-byte global loads from p + 0, 32, 64, 96 bytes, issued and completed in one
// statement (operands loaded once before a tile loop).
__device__ __forceinline__ void ldg_x4(const uint16_t* p, u32x4& a, u32x4& b, u32x4& c, u32x4& d) {
  asm volatile(
      "global_load_dwordx4 %0, %4, off\n\t"
      "global_load_dwordx4 %1, %4, off offset:32\n\t"
      "global_load_dwordx4 %2, %4, off offset:64\n\t"
      "global_load_dwordx4 %3, %4, off offset:96\n\t"
      "s_waitcnt vmcnt(0)"
      : "=&v"(a), "=&v"(b), "=&v"(c), "=&v"(d)
      : "v"(p)
      : "memory");
}

typedef int i32x16 __attribute__((ext_vector_type(16)));

// ------------------------------------------------------------------ direct global -> LDS copies
// Copies are inline assembly, invisible to the compiler's wait insertion (see above).  A
// buffer descriptor is built per tile with its base at the tile's first row and its record
// count ending at the tile's last valid row, so rows past the end are out of range for the
// hardware bounds check and never touch memory (all of the offset travels in the VGPR
// operand, which is what the check covers) (the kernels mask those rows and clear LDS
// once at start, so whatever the copy leaves there is finite).  Each copy instruction
// writes 16 (or 4) bytes per lane at LDS address M0 + 16*lane (4*lane).
__device__ __forceinline__ u32x4 tile_desc(const void* base, int64_t byte_off, int bytes) {
  const uint64_t b = (uint64_t)(uintptr_t)base + (uint64_t)byte_off;
  u32x4 d;
  d[0] = __builtin_amdgcn_readfirstlane((uint32_t)b);
  d[1] = __builtin_amdgcn_readfirstlane((uint32_t)(b >> 32)) & 0xffffu;  // stride 0
  d[2] = __builtin_amdgcn_readfirstlane((uint32_t)bytes);                // record count (bytes)
  d[3] = 0x00020000u;
  return d;
}
// Rows [row0, row0 + valid) of a token-major tensor whose rows are `pitch` elements apart.
__device__ __forceinline__ u32x4 tile_rsrc(const uint16_t* g, int64_t row0, int valid, int pitch) {
  return tile_desc(g, row0 * pitch * 2, valid * pitch * 2);
}

// One 16-byte-per-lane copy at voff + inc (s_nop: M0 and the descriptor are written by the
// compiler just before; 5 wait states cover both the M0 and the SGPR-write hazards).
__device__ __forceinline__ void dma16(uint32_t m0v, u32x4 desc, int voff, int inc) {
  int tmp;
  asm volatile(
      "v_add_u32 %0, %1, %2\n\t"
      "s_mov_b32 m0, %3\n\t"
      "s_nop 4\n\t"
      "buffer_load_dwordx4 %0, %4, 0 offen lds"
      : "=&v"(tmp)
      : "s"(inc), "v"(voff), "s"(m0v), "s"(desc)
      : "memory", "m0");
}
// dma16 for bytes read exactly once (the stored dS): the non-temporal hint keeps them from
// displacing lines that other workgroups read again (the K tiles of the same head).
__device__ __forceinline__ void dma16_stream(uint32_t m0v, u32x4 desc, int voff, int inc) {
  int tmp;
  asm volatile(
      "v_add_u32 %0, %1, %2\n\t"
      "s_mov_b32 m0, %3\n\t"
      "s_nop 4\n\t"
      "buffer_load_dwordx4 %0, %4, 0 offen nt lds"
      : "=&v"(tmp)
      : "s"(inc), "v"(voff), "s"(m0v), "s"(desc)
      : "memory", "m0");
}
__device__ __forceinline__ void dma4(uint32_t m0v, u32x4 desc, int voff) {
  asm volatile(
      "s_mov_b32 m0, %1\n\t"
      "s_nop 4\n\t"
      "buffer_load_dword %0, %2, 0 offen lds"
      :
      : "v"(voff), "s"(m0v), "s"(desc)
      : "memory", "m0");
}

// Per-lane byte offset (tile-independent) for dma_tile with NW = 4 or 8 waves.  Lane L of
// wave w writes bytes [16L, 16L+16) of each 1 KB instruction, which holds rows 8j..8j+7 of
// one column block, j = w + NW*i; it fetches the logical chunk the swizzle places there
// (rows 8j + L/8 have bits 1..3 = (L/8 >> 1) and (j & 1) == (w & 1) for every i).
template <int DIM> __device__ __forceinline__ int dma_lane_off(int pitch, int head, int wave, int lane) {
  const int q = lane >> 3;
  const int lc = (lane & 7) ^ ((((q >> 1) & 1) << 2) | ((wave & 1) << 1) | (q >> 2));
  return ((8 * wave + q) * pitch + head * DIM + lc * 8) * 2;
}

// Copies a ROWS x DIM tile (NW waves, rows 8j .. 8j+7 of each column block per 1 KB
// instruction, j = wave + NW*i).  `wave` must be wave-uniform.
template <int DIM, int ROWS, int NW = 4>
__device__ __forceinline__ void dma_tile(lds_char* lds, u32x4 desc, int voff, int pitch, int wave) {
  constexpr int NINS = ROWS / 8;  // per column block
  static_assert(NINS % NW == 0, "tile must split evenly over the waves");
  const uint32_t base = __builtin_amdgcn_readfirstlane(lds_addr(lds) + wave * 1024);
#pragma unroll
  for (int b = 0; b < DIM / 64; ++b)
#pragma unroll
    for (int i = 0; i < NINS / NW; ++i)
      dma16(base + b * block_bytes<ROWS>() + NW * i * 1024, desc, voff, 8 * NW * i * pitch * 2 + b * 128);
}

// 64 fp32 values (valid of them in range) -> LDS, one wave.
__device__ __forceinline__ void dma_vec64(lds_char* lds, const float* g, int valid, int lane) {
  dma4(__builtin_amdgcn_readfirstlane(lds_addr(lds)), tile_desc(g, 0, valid * 4), lane * 4);
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

// Workgroups are dispatched round-robin over the 8 XCDs (workgroup b runs on XCD b % 8), each
// with its own L2.  When the heads of a launch are a multiple of 8, each XCD takes whole heads
// one after another (its j-th workgroup: head (b % 8) * H / 8 + j / n_items, item j % n_items,
// heaviest first), so the workgroups running together on an XCD stream the same head's
// other-side tiles through its L2.  Otherwise the items of a head alternate over the XCDs
// (head b % H, item b / H).
constexpr int N_XCD = 8;
__device__ __forceinline__ void xcd_head_item(int b, int n_heads, int n_items, int& head, int& item) {
  if (n_heads % N_XCD == 0) {
    const int x = b % N_XCD, j = b / N_XCD;
    head = x * (n_heads / N_XCD) + j / n_items;
    item = j % n_items;
  } else {
    head = b % n_heads;
    item = b / n_heads;
  }
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

struct AttnArgs {
  const uint16_t* q;   // [nq][H][192]
  const uint16_t* k;   // [nk][Hkv][192]
  const uint16_t* v;   // [nk][Hkv][128]
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
  int H;               // query heads
  int Hkv;             // K/V heads; query head h uses K/V head h / grp
  int grp;             // H / Hkv
  int nq, nk;
  int q_s, k_s, v_s;   // elements between consecutive token rows of q, k, v (dO, O: dense)
  float scale;         // softmax scale
  // heads of one launch: K/V heads kv_head0 .. +kv_heads (key-stationary kernel), query heads
  // q_head0 .. +q_heads (query-stationary kernels)
  int kv_head0, kv_heads;
  int q_head0, q_heads;
  // stored-dS backward: dS blocks of the launch's query heads, ds_head_bytes apart; per key
  // item (launch order) its first tile slot; the key items in row order as records (row0,
  // rows, ranges, first slot) and the record index of each 32-row key block
  char* ds;
  int64_t ds_head_bytes;
  const int* kbase;
  const int* kmap32;
  const int* krec;
  const int* kitems;   // key-stationary items
};

}  // namespace hydra
