/*
 * hydra_attn.h -- one context-parallel (CP) rank's attention share on AMD MI355X (gfx950).
 *
 * What the library computes (arxiv 2609.34318, "HyDra"):
 *   - Documents are packed into one window and attention is masked across their
 *     boundaries (Sec. 2.2): a query at global position p attends to the keys of its
 *     own document at positions <= p (causal, the diagonal included).
 *   - A CP degree P is factored into an inner Ulysses group over heads and an outer
 *     ring over the sequence, P = cp_u * cp_r (Sec. 5.2.1, Eq. (usp)).  A rank therefore
 *     holds h / cp_u heads ("n_heads" below) and a chunk of the sequence; K/V chunks
 *     circulate around the ring (Sec. 2.1, Sec. 3.5) and each ring step is one call here.
 *   - Every step yields a partial output plus its log-sum-exp; partials combine exactly
 *     as in standard ring CP (Sec. 5.2.2, last paragraph): hydra_lse_merge.
 *   - Under MLA every head has its own K and V (Sec. 1); this library supports
 *     d_qk = 192 and d_v = 128.
 *
 * Conventions shared by every call:
 *   - Tensors are token-major and contiguous: X[token][head][dim], last dim fastest.
 *     bf16 tensors are passed as raw 16-bit patterns.  LSE and D are [head][token] fp32,
 *     natural logarithm.  "Token" is the rank-local row index; its global position comes
 *     from the chunk's segments (hydra_chunk_t).
 *   - Device pointers unless marked HOST.  Every device pointer must be 16-byte aligned.
 *   - `stream` is a hipStream_t (NULL = the default stream).  Compute calls enqueue work
 *     and return; kernel faults surface at the caller's next synchronisation.
 *   - Compute calls never allocate device memory.  They upload a small work plan into the
 *     caller's workspace with hipMemcpyAsync from host memory; that upload may wait for
 *     work already queued on `stream`.
 *   - The caller owns every buffer.  The library keeps no pointer after a call returns.
 *   - All arguments are validated on the host before any HIP call; on error nothing is
 *     written and no HIP call is made.  No C++ exception crosses this interface.
 *   - Calls are thread-safe; two calls that write the same buffers must not overlap.
 */
#ifndef HYDRA_ATTN_H
#define HYDRA_ATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes (returned as int). */
#define HYDRA_OK                 0
#define HYDRA_ERR_INVALID       -1  /* malformed argument: sizes, cu_seqlens, segments, NULL */
#define HYDRA_ERR_UNSUPPORTED   -2  /* well-formed but not supported (d_qk != 192, d_v != 128) */
#define HYDRA_ERR_ALIGN         -3  /* a device pointer is not 16-byte aligned */
#define HYDRA_ERR_WORKSPACE     -4  /* workspace NULL or smaller than hydra_workspace_size() */
#define HYDRA_ERR_HIP           -5  /* a HIP runtime call or kernel launch failed */
#define HYDRA_ERR_TOO_LARGE     -6  /* beyond the no-allocation call's scratch (see below) */

#define HYDRA_MAX_SEGS 4

/* A chunk of the packed sequence held by this rank: up to HYDRA_MAX_SEGS segments of
 * consecutive global positions, laid out one after another as local rows.  One segment
 * is a contiguous ring chunk; two segments express a zigzag (head + tail) chunk.
 * Segments must lie inside [0, cu_seqlens[n_docs]); lengths may be 0. */
typedef struct {
  int32_t n_segs;                   /* 0..HYDRA_MAX_SEGS                                 */
  int32_t start[HYDRA_MAX_SEGS];    /* global position of the segment's first token      */
  int32_t len[HYDRA_MAX_SEGS];      /* tokens in the segment                              */
} hydra_chunk_t;

/* One ring step of one rank (Sec. 5.2.1: per-rank Q chunk, KV chunk, document boundaries,
 * chunk global offsets, head shard). */
typedef struct {
  int32_t n_heads;                  /* head shard on this rank, h / cp_u; > 0            */
  int32_t d_qk;                     /* must be 192                                       */
  int32_t d_v;                      /* must be 128                                       */
  float   softmax_scale;            /* <= 0 selects 1/sqrt(d_qk)                         */
  const int32_t* cu_seqlens;        /* HOST int32[n_docs+1]: document boundaries in global
                                       positions, cu[0] = 0, nondecreasing; read only
                                       during the call                                   */
  int32_t n_docs;                   /* >= 1                                              */
  hydra_chunk_t q;                  /* this rank's query chunk                           */
  hydra_chunk_t kv;                 /* this ring step's key/value chunk                  */
  int32_t n_kv_heads;               /* K/V heads held (Sec. 3.5: h_kv <= h); 0 means
                                       n_heads (MLA).  Must divide n_heads: query head i
                                       uses K/V head i / (n_heads / n_kv_heads)            */
  int32_t q_tok_stride;             /* elements from one token row of q to the next; 0 =
                                       dense (n_heads * 192).  Otherwise at least that, a
                                       multiple of 8 and below 2^22 (heads stay contiguous
                                       within a row, e.g. views into a fused QKV buffer)  */
  int32_t k_tok_stride;             /* the same for k (dense: Hkv * 192)                 */
  int32_t v_tok_stride;             /* the same for v (dense: Hkv * 128)                 */
} hydra_problem_t;

/* Size limits (HYDRA_ERR_INVALID beyond them): n_heads <= 4096; Nq, Nk <= 2^30 rows;
 * Nq * n_heads * 192, Nk * n_heads * 192, Nq * q_tok_stride and Nk * k_tok_stride below
 * 2^40 elements; and, because every
 * attention launch holds one 512-lane workgroup per (tile, head) and a dispatch fewer than
 * 2^32 lanes, (sum over the query segments of ceil(len / 256)) * n_heads and (sum over the
 * K/V segments of ceil(len / 128)) * n_kv_heads below 2^23.
 *
 * Bytes of device workspace the compute calls need for `p` (host only, no GPU needed).
 * Returns 0 if `p` is invalid. */
size_t hydra_workspace_size(const hydra_problem_t* p);

/* Forward partial of one ring step (Sec. 5.2.2; Sec. 2.2 for the masking):
 *   q [Nq][H][192] bf16, k [Nk][Hkv][192] bf16, v [Nk][Hkv][128] bf16   (inputs;
 *   Hkv = n_kv_heads, or H when that is 0; token rows q_tok_stride / k_tok_stride /
 *   v_tok_stride elements apart, every other tensor dense)
 *   o_part  [Nq][H][128] fp32   softmax(QK^T * scale, masked) V over this chunk's keys
 *   lse_part [H][Nq] fp32       natural-log sum of exp of the visible scores
 *   o_part_bf16: NULL, or [Nq][H][128] bf16 that also receives O (for a ring of one step,
 *                whose partial is already final)
 * A row that sees no key of this chunk gets O = 0 and LSE = -inf (the merge identity).
 * Every row of o_part and lse_part is written.  Outputs (o_part, lse_part, o_part_bf16 and
 * the workspace) must not overlap each other or the inputs: checked, HYDRA_ERR_INVALID. */
int hydra_attn_fwd(const hydra_problem_t* p, const void* q, const void* k, const void* v,
                   float* o_part, float* lse_part, void* o_part_bf16,
                   void* workspace, size_t workspace_bytes, void* stream);

/* Backward of one ring step, given the FINAL merged output and LSE of the rows (the same
 * function is differentiated at every step):
 *   o_final [Nq][H][128] bf16, lse_final [H][Nq] fp32, d_o [Nq][H][128] bf16
 *   dq_acc [Nq][H][192] fp32 += this step's dQ        (caller zero-initialises once)
 *   dk_acc [Nk][Hkv][192] fp32 += dK of this KV chunk   from this rank's queries
 *   dv_acc [Nk][Hkv][128] fp32 += dV of this KV chunk   from this rank's queries
 *          (with Hkv < H each K/V head sums the gradients of its query-head group)
 * Outputs (the three gradient buffers and the workspace) must not overlap each other or
 * the inputs: checked, HYDRA_ERR_INVALID. */
int hydra_attn_bwd(const hydra_problem_t* p, const void* q, const void* k, const void* v,
                   const void* o_final, const float* lse_final, const void* d_o,
                   float* dq_acc, float* dk_acc, float* dv_acc,
                   void* workspace, size_t workspace_bytes, void* stream);

/* Backward of one ring step without the dQ kernel's recomputation of S and dP (Sec. 3.5:
 * the rank's cost is its S^2 h / P attention work, so work done twice is what to cut): the
 * key-stationary kernel also stores dS (bf16, 2 bytes per visible (query, key) pair and
 * query head) into ds_buf, and a query-stationary kernel reads it back for
 * dQ += scale dS K.  Same arguments, results and checks as hydra_attn_bwd, plus
 *   ds_buf   device scratch, 16-byte aligned, written and read by this call only (its
 *            contents are meaningless afterwards); must not overlap any other argument
 *   ds_bytes its size.  The heads are processed in passes of the largest number of K/V
 *            heads whose query heads' dS fits: hydra_bwd_ds_bytes(p, g) bytes for g K/V
 *            heads per pass (one pass holds all heads when ds_bytes >= hydra_bwd_ds_bytes(
 *            p, n_kv_heads)).
 * The path applies when every segment of both chunks starts at, and has a length that is, a
 * multiple of 32 positions.  Otherwise, or when ds_bytes is below one K/V head's need, or
 * ds_buf is NULL, the call computes exactly what hydra_attn_bwd computes, the same way.  The
 * results are hydra_attn_bwd's up to rounding: dK and dV bit for bit, dQ from the dS that the
 * dK/dV products use (formed from the bf16-rounded P) instead of a recomputed one. */
int hydra_attn_bwd_ds(const hydra_problem_t* p, const void* q, const void* k, const void* v,
                      const void* o_final, const float* lse_final, const void* d_o,
                      float* dq_acc, float* dk_acc, float* dv_acc, void* ds_buf, size_t ds_bytes,
                      void* workspace, size_t workspace_bytes, void* stream);

/* Bytes of ds_buf that hydra_attn_bwd_ds needs to process `kv_heads_per_pass` K/V heads (and
 * their query heads) per pass; 0 when `p` is invalid or the stored-dS path does not apply
 * (host only). */
size_t hydra_bwd_ds_bytes(const hydra_problem_t* p, int32_t kv_heads_per_pass);

/* For callers that cannot allocate device memory (code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc): hydra_attn_bwd without the workspace
 * argument.  The workspace (plan, D, LSE*log2(e)) lives in a device array of the library,
 * one per GPU, of hydra_noalloc_scratch_bytes() = 32 MiB, held until the process ends; the
 * call allocates nothing.  Problems whose hydra_workspace_size() exceeds it are refused with
 * HYDRA_ERR_TOO_LARGE before any HIP call (32 MiB covers n_heads x Nq up to about 4M, e.g.
 * 16 heads x 256K rows).  Every call on a GPU uses that GPU's one array: calls that overlap
 * on one GPU (other streams, other threads) race and must be serialised by the caller.
 * Everything else (arguments, checks, results) is hydra_attn_bwd's, bit for bit. */
int hydra_attn_bwd_noalloc(const hydra_problem_t* p, const void* q, const void* k, const void* v,
                           const void* o_final, const float* lse_final, const void* d_o,
                           float* dq_acc, float* dk_acc, float* dv_acc, void* stream);
size_t hydra_noalloc_scratch_bytes(void);

/* For callers that record the calls into a HIP graph (stream capture), where the plan's
 * host-to-device copy cannot be recorded: hydra_attn_plan uploads the complete work plan of
 * `p` (both sides) into `workspace` once, outside the capture; the *_planned calls then take
 * exactly the arguments of hydra_attn_fwd / hydra_attn_bwd, check them the same way on the
 * host, and only launch kernels (no copy, no host-side wait), reading the plan from the
 * workspace.  The workspace must hold the plan of this same problem (same cu_seqlens,
 * chunks and head counts; strides may differ) and must not be reused for another problem
 * while a recorded graph still uses it; one workspace per ring step.  The backward writes
 * D and LSE*log2(e) into the workspace as before.  The library remembers, per workspace
 * address, which problem its last upload was for (hydra_attn_plan, or the upload inside
 * hydra_attn_fwd / hydra_attn_bwd, where the forward's holds only the query-side items):
 * a planned call on a workspace whose recorded plan is another problem's, or lacks the
 * key-side items the backward needs, returns HYDRA_ERR_WORKSPACE before any HIP call.  A
 * workspace freed and reallocated at the same address must be planned again. */
int hydra_attn_plan(const hydra_problem_t* p, void* workspace, size_t workspace_bytes, void* stream);
int hydra_attn_fwd_planned(const hydra_problem_t* p, const void* q, const void* k, const void* v,
                           float* o_part, float* lse_part, void* o_part_bf16,
                           void* workspace, size_t workspace_bytes, void* stream);
int hydra_attn_bwd_planned(const hydra_problem_t* p, const void* q, const void* k, const void* v,
                           const void* o_final, const float* lse_final, const void* d_o,
                           float* dq_acc, float* dk_acc, float* dv_acc,
                           void* workspace, size_t workspace_bytes, void* stream);

/* Exact merge of two partials of the same rows (ring CP, Sec. 5.2.2):
 *   L = log(e^La + e^Lb),  O = e^(La-L) O_a + e^(Lb-L) O_b, in place into (o_acc, lse_acc).
 * (0, -inf) is the identity; two empty rows stay (0, -inf) with no NaN.
 *   o_acc/o_part [n_rows][n_heads][d_v] fp32, lse_acc/lse_part [n_heads][n_rows] fp32.
 *   o_out_bf16: NULL, or [n_rows][n_heads][d_v] bf16 that also receives the merged O.
 * d_v must be 128.  n_rows = 0 is a no-op.  The outputs (o_acc, lse_acc, o_out_bf16) must
 * not overlap each other or the partial: checked, HYDRA_ERR_INVALID. */
int hydra_lse_merge(int64_t n_rows, int32_t n_heads, int32_t d_v,
                    float* o_acc, float* lse_acc, const float* o_part, const float* lse_part,
                    void* o_out_bf16, void* stream);

/* Text for a status code (static storage). */
const char* hydra_strerror(int status);

/* Exact number of visible (query, key) pairs per head for `p` (host only).  The
 * benchmark's FLOP count is this times 2*(d_qk+d_v) forward and 2*(3*d_qk+2*d_v)
 * backward.  Returns -1 if `p` is invalid. */
int64_t hydra_visible_pairs(const hydra_problem_t* p);

/* Host-only view of the work plan, for tests.  which = 0: query-stationary items (forward
 * and dQ), which = 1: key-stationary items (dK/dV).  Each item is 16 int32:
 *   [0] first local row  [1] its global position  [2] rows in the tile  [3] n_ranges
 *   [4+3r] first local row of range r on the other side, [5+3r] its global position,
 *   [6+3r] rows in range r   (r < n_ranges <= HYDRA_MAX_SEGS)
 * Items come in launch order (heaviest first).  Writes min(cap, n) items to `out` (may be
 * NULL when cap = 0) and returns n, or a negative status. */
int64_t hydra_plan_items(const hydra_problem_t* p, int32_t which, int32_t* out, int64_t cap);

/* Tile sizes of the plan: rows per query-stationary tile, rows per key-stationary tile. */
void hydra_tile_rows(int32_t* q_tile_rows, int32_t* kv_tile_rows);

/* Per-kernel timing (a tracing aid for benchmarks; off by default).  While recording, every
 * kernel this library launches is bracketed by two hipEvents on its launch stream.
 * hydra_profile_start() clears earlier records and starts recording.
 * hydra_profile_stop() waits for the recorded events, stops recording, writes up to `cap`
 * per-kernel summaries to `out` and returns the number of distinct kernels (or a negative
 * status).  Names: "attn_fwd", "bwd_pre", "bwd_dq", "bwd_dkdv", "lse_merge", and for the
 * calls of hydra_layout.h and hydra_gate.h "pack_heads", "unpack_heads", "zigzag_gather",
 * "zigzag_scatter", "unpack_gated", "pack_gated_bwd". */
typedef struct {
  char    name[32];
  int64_t launches;
  double  total_ms;
  double  min_ms;
  double  max_ms;
} hydra_kernel_stat_t;

int hydra_profile_start(void);
int hydra_profile_stop(hydra_kernel_stat_t* out, int32_t cap);

#ifdef __cplusplus
}
#endif
#endif /* HYDRA_ATTN_H */
