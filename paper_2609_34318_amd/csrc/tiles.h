// Tile geometry that the host plan and the kernels must agree on (no HIP types here: the
// plan is also built as plain host C++).
#pragma once

namespace hydra {

// Query rows per tile of the key-stationary backward kernel (three 32-row sub-blocks).  The
// plan lays out the stored dS with it: one slot per (key item, query tile), each slot
// holding the 3 x 4 blocks of 32 queries x 32 keys.
constexpr int KV_QTILE_ROWS = 96;
constexpr int DS_BLOCK_BYTES = 32 * 32 * 2;                               // bf16
constexpr int DS_TILE_BYTES = (KV_QTILE_ROWS / 32) * 4 * DS_BLOCK_BYTES;  // 24 KB

}  // namespace hydra
