// Host-side argument checks and work planning for one ring step (no HIP calls).
#pragma once
#include <cstddef>
#include <cstdint>
#include <vector>

#include "hydra_attn.h"

namespace hydra {

constexpr int kDqk = 192;
constexpr int kDv = 128;
constexpr int kQTile = 256;    // query rows per query-stationary workgroup (8 waves x 32)
constexpr int kKvTile = 128;   // key rows per key-stationary workgroup (4 waves x 32)
constexpr int kItemInts = 16;  // int32 per work item

// Checked and normalised view of a hydra_problem_t.
struct Problem {
  int H = 0;
  int Hkv = 0;  // K/V heads (divides H)
  float scale = 0.f;
  std::vector<int32_t> cu;     // n_docs + 1 boundaries
  hydra_chunk_t q{}, kv{};
  int64_t nq = 0, nk = 0;
  int q_s = 0, k_s = 0, v_s = 0;  // token-row strides of q, k, v in elements
};

// Returns HYDRA_OK or an error status; fills `out` on success.
int check_problem(const hydra_problem_t* p, Problem* out);

// Work items (kItemInts each), heaviest first.  which = 0: query-stationary tiles of
// kQTile rows with their visible key ranges; which = 1: key-stationary tiles of kKvTile
// rows with their visible query ranges.
void plan_items(const Problem& pr, int which, std::vector<int32_t>* items);

int64_t visible_pairs(const Problem& pr);

// Byte offsets of the workspace regions.
struct WsLayout {
  size_t cu_off, qitems_off, kitems_off, kbase_off, kmap_off, krec_off, d_off, lse2_off, total;
  int64_t n_qitems, n_kitems, n_kblocks;
};
WsLayout ws_layout(const Problem& pr);

// The stored-dS backward applies when every segment of both chunks starts and ends on a
// multiple of 32 positions: the key-stationary tiles then cut the query rows into 32-row
// blocks that coincide with the query-stationary kernel's per-wave blocks.
bool ds_path_applies(const Problem& pr);

// For the stored-dS backward, from the key items in launch order: kbase[i] = first tile
// slot of item i (slots of 24 KB, one per query tile of the item); the items again in
// row order as records of kItemInts ints, krec[j] = {row0, n, n_ranges, first slot, then
// (first row, rows) of each query range}; kmap32[b] = the row-order index of the item
// holding local key rows [32b, 32b + 32).  Returns the slots per query head.
int64_t ds_tables(const Problem& pr, const std::vector<int32_t>& kitems, std::vector<int32_t>* kbase,
                  std::vector<int32_t>* kmap32, std::vector<int32_t>* krec);

}  // namespace hydra
