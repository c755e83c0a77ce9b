/*
 * hydra_gate.h -- the gated attention output, fused with the rank-local half of the
 * reverse Ulysses exchange, on AMD MI355X.
 *
 * The paper's model uses gated MLA (Sec. 5.2.2 and the figure of its asynchronous
 * all-to-all schedule, citing Qiu et al. 2025): beside Q, K and V a gate projection of
 * the layer input is computed, and that projection needs no context-parallel
 * communication.  The paper prints no gate formula; these calls take the cited work's
 * gate, the attention output multiplied elementwise by the logistic sigmoid of gate
 * logits G:
 *
 *   Y'[t][h][d] = Y[t][h][d] * s[t][h][e],   s = 1 / (1 + exp(-G)),
 *
 * with one logit per (token, head, channel) (gate_dim = d_v, e = d) or one per (token,
 * head) (gate_dim = 1, e = 0).  Since G is computed on the rank's own tokens with every
 * head, the product is taken where the attention output is back in that layout: right
 * after the reverse (head -> sequence) exchange, fused with its unpack.  The backward is
 * fused with the pack that starts the backward exchange, and needs only the gated output
 * Y' (which the next projection keeps for its own backward), because Y * s = Y':
 *
 *   dY = dY' * s  (sent back through the exchange to the attention backward),
 *   dG = dY' * Y' * (1 - s)   (gate_dim = d_v)   or   (1 - s) * sum_d dY' * Y'  (gate_dim = 1).
 *
 * With cp_u = 1 (no Ulysses exchange) the calls are the plain gated epilogue.
 *
 * Conventions: device pointers, 16-byte aligned; all tensors bf16 (raw 16-bit patterns),
 * token-major; products in fp32, each output rounded once to nearest even.  The exchange
 * itself (RCCL over xGMI) is the caller's.  Inputs and outputs must not overlap.
 * Arguments are checked on the host before any HIP call (status codes and hydra_strerror
 * are those of hydra_attn.h); each call enqueues one kernel on `stream`, allocates
 * nothing and keeps no pointer.
 */
#ifndef HYDRA_GATE_H
#define HYDRA_GATE_H

#include <stdint.h>

#include "hydra_attn.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Forward: recv [cp_u][T][H/cp_u][d_v] holds, in buffer j, this rank's T tokens of head
 * group j (what the reverse exchange delivered); gate [T][H][gate_dim] the gate logits.
 * Writes y [T][H][d_v]:
 *   y[t][j*(H/cp_u) + k][d] = bf16(recv[j][t][k][d] * s[t][j*(H/cp_u) + k][e]).
 * n_tokens = T in [0, 2^31] (0 is a no-op; the pointers may then be NULL), n_heads = H in
 * [1, 65536] and a multiple of cp_u, d_v a power of two in [8, 512], gate_dim 1 or d_v.
 * Errors: HYDRA_ERR_INVALID (sizes, NULL, overlap), HYDRA_ERR_ALIGN, HYDRA_ERR_HIP. */
int hydra_unpack_heads_gated(int64_t n_tokens, int32_t n_heads, int32_t d_v, int32_t gate_dim,
                             int32_t cp_u, const void* recv, const void* gate, void* y,
                             void* stream);

/* Backward: y [T][H][d_v] the gated output of the forward, gate [T][H][gate_dim] its
 * logits, d_y [T][H][d_v] the gradient of y.  Writes
 *   d_send [cp_u][T][H/cp_u][d_v]: d_send[j][t][k][d] = bf16(d_y[t][h][d] * s[t][h][e]),
 *          h = j*(H/cp_u) + k (buffer j goes to group rank j),
 *   d_gate [T][H][gate_dim]: bf16(d_y * y * (1 - s)), summed over d in fp32 when
 *          gate_dim = 1.
 * Same size rules and errors as hydra_unpack_heads_gated. */
int hydra_pack_heads_gated_bwd(int64_t n_tokens, int32_t n_heads, int32_t d_v, int32_t gate_dim,
                               int32_t cp_u, const void* y, const void* gate, const void* d_y,
                               void* d_send, void* d_gate, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* HYDRA_GATE_H */
