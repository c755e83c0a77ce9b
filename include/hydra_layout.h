/*
 * hydra_layout.h -- the data-layout steps around one rank's attention share on AMD MI355X.
 *
 * A CP degree P is factored into an inner Ulysses group over heads and an outer ring over
 * the sequence, P = cp_u * cp_r with cp_u = min(P, h) (Sec. 5.2.1, Eq. (usp)).  Ulysses
 * moves from a token split to a head split with an all-to-all inside each group
 * (Sec. 3.5) and back again for the output.  These calls are the rank-local halves of
 * those exchanges plus the assignment of sequence chunks to ring ranks:
 *
 *   hydra_pack_heads     token shard [T][H][*] -> cp_u send buffers [cp_u][T][H/cp_u][*]
 *                        (buffer j goes to group rank j)
 *   hydra_unpack_heads   cp_u receive buffers [cp_u][T][H/cp_u][*] -> [T][H][*]
 *                        (the inverse, after the reverse exchange)
 *   hydra_zigzag_gather  natural-order rows [S][*] -> ring rank r's rows [S/cp_r][*]
 *   hydra_zigzag_scatter the inverse (rank r's rows back into natural order)
 *
 * Which rows a ring rank holds is not printed in the paper; these calls use the usual
 * causal load balancing: the S rows are cut into 2*cp_r equal chunks and ring rank r holds
 * chunks r and 2*cp_r-1-r, in that order.  After the forward exchange a group's token
 * slices arrive in rank order, which is already the contiguous [cp_u*T][H/cp_u][*] layout
 * the attention calls take, so that side needs no kernel.
 *
 * The all-to-all itself (RCCL over xGMI) is the caller's; these calls never communicate.
 *
 * Conventions: device pointers, 16-byte aligned; row and head sizes in bytes, multiples
 * of 16; src and dst must not overlap; the caller owns every buffer.  Arguments are
 * checked on the host before any HIP call (status codes and hydra_strerror are those of
 * hydra_attn.h).  Calls enqueue one kernel on `stream` and return; they allocate nothing.
 */
#ifndef HYDRA_LAYOUT_H
#define HYDRA_LAYOUT_H

#include <stdint.h>

#include "hydra_attn.h"

#ifdef __cplusplus
extern "C" {
#endif

/* dst[j][t][k] = src[t][j*(n_heads/cp_u) + k] for j < cp_u, t < n_tokens, k < n_heads/cp_u,
 * each element head_bytes bytes.  n_heads must be a multiple of cp_u; n_tokens <= 2^31 and
 * n_heads * head_bytes <= 2^34.  n_tokens == 0 is a no-op.  Errors: HYDRA_ERR_INVALID (sizes, NULL, overlap), HYDRA_ERR_ALIGN, HYDRA_ERR_HIP. */
int hydra_pack_heads(int64_t n_tokens, int32_t n_heads, int32_t head_bytes, int32_t cp_u,
                     const void* src, void* dst, void* stream);

/* dst[t][j*(n_heads/cp_u) + k] = src[j][t][k]: the inverse of hydra_pack_heads. */
int hydra_unpack_heads(int64_t n_tokens, int32_t n_heads, int32_t head_bytes, int32_t cp_u,
                       const void* src, void* dst, void* stream);

/* dst[i] = src[z(i)] for i < n_rows / cp_r, rows of row_bytes bytes, where with
 * c = n_rows / (2*cp_r):  z(i) = r*c + i for i < c,  (2*cp_r-1-r)*c + (i-c) otherwise.
 * n_rows must be a multiple of 2*cp_r; 0 <= r < cp_r. */
int hydra_zigzag_gather(int64_t n_rows, int64_t row_bytes, int32_t cp_r, int32_t r,
                        const void* src, void* dst, void* stream);

/* dst[z(i)] = src[i]: ring rank r's rows written back to their natural positions (the
 * other ranks' rows of dst are untouched). */
int hydra_zigzag_scatter(int64_t n_rows, int64_t row_bytes, int32_t cp_r, int32_t r,
                         const void* src, void* dst, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* HYDRA_LAYOUT_H */
