/*
 * hydra_sched.h -- the load-driven dynamic-CP scheduler (host only, no GPU).
 *
 * Given the sequence lengths of a global batch, decides every sequence's context-parallel
 * degree and places it in a micro-batch (MB) and a group of ranks of the HDP pool
 * (Sec. 5.1):
 *   - targets (Sec. 5.1.1): W = sum s_i^2; CP-degree cap
 *       C_mem = ceil2(s_max / B),  C_hat = s_max^2 sqrt((pp-1) (theta/c) G / W),
 *       C* = min(G, ceil2(max(C_mem, C_hat)))                    (Eq. (cstar-cont), (cstar))
 *     per-rank load target Lambda* = s_max^2 / C* (Eq. (load-target)), MB count target
 *     M* = ceil(C* W / (s_max^2 G)) (Eq. (mstar)), and per sequence
 *       cp(s) = min(C*, ceil2(max(s^2 / Lambda*, s / B)))            (Eq. (cp))
 *     where ceil2(x) is the smallest power of two >= x;
 *   - placement (Alg. 1): longest first, one MB at a time over all G ranks: a sequence of
 *     degree k opens a new k-aligned group on free ranks, else piggybacks on the smallest
 *     feasible open group of size >= k (least loaded on ties), else the MB closes; closed
 *     MBs backfill idle ranks by doubling their smallest groups;
 *   - heap-accelerated search (Sec. 5.1.3): open groups are kept per size class in a lazy
 *     min-heap by load plus a max-heap by remaining token capacity for groups that failed
 *     the token test; classes whose least loaded group already reached the target are
 *     pruned; a min-heap drives backfill; the pool maximum for the balance test is kept
 *     incrementally.  O(N log G) per batch; the placement is identical to linear scans.
 *
 * Readings where the paper is silent:
 *   1. A new group needs a free k-aligned block of ranks; the lowest one is taken.  G must
 *      be a multiple of C*.
 *   2. Equal lengths keep their input order; among equally small, equally loaded feasible
 *      groups the one starting at the lowest rank wins.
 *   3. "k has shrunk and MB balanced": k is below the degree of the sequence that opened
 *      the MB, no rank is free, and the least loaded group carries at least balance_ratio
 *      of the most loaded one's load.
 *   4. Backfill repeatedly doubles the smallest group (size, then start) whose aligned
 *      buddy block is free and whose doubled size stays <= C*; per-rank load and tokens
 *      halve.
 *   5. theta/c is an input (the paper measures it); pp = 1 drops the bubble term.  A fixed
 *      cap may be given instead of Eq. (cstar).
 *   6. Loads and tokens are tracked exactly, as integers multiplied by C*.
 *
 * Conventions: HOST pointers; the caller owns every buffer; nothing is kept after return.
 * Arguments are validated first (status codes of hydra_attn.h).  Thread-safe.
 */
#ifndef HYDRA_SCHED_H
#define HYDRA_SCHED_H

#include <stdint.h>

#include "hydra_attn.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct {
  int32_t n_ranks;        /* G: ranks of the HDP pool, 1 .. 65536, a multiple of the cap */
  int64_t token_budget;   /* B: tokens one rank can hold, >= 1                            */
  int32_t pp;             /* pipeline stages, >= 1                                         */
  double  theta_over_c;   /* measured cost ratio (time per unit load / cost per MB), >= 0 */
  int32_t cap;            /* 0: C* from Eq. (cstar); else a power of two dividing G that
                             is >= C_mem                                                   */
  double  balance_ratio;  /* balance test of reading 3; 0 selects 0.9; in (0, 1]           */
} hydra_sched_config_t;

typedef struct {
  int64_t w_hi, w_lo;     /* W = sum s_i^2 as w_hi * 2^62 + w_lo                          */
  int64_t s_max;
  int32_t c_mem;
  double  c_hat;
  int32_t cap;            /* C*                                                            */
  int64_t m_target;       /* M*                                                            */
  int32_t n_mbs;          /* realized micro-batch count                                    */
  int64_t max_load_x_cap; /* heaviest per-rank load over all MBs, times C* (<= s_max^2)    */
} hydra_sched_summary_t;

/* Places n_docs sequences (lengths in tokens, 1 .. 2^21).  Writes, per input sequence i,
 * its micro-batch mb[i], and the first rank and size of its group, group_start[i] and
 * group_size[i] (the sequence is split over ranks group_start .. group_start+group_size-1
 * of that micro-batch).  summary may be NULL.  Errors: HYDRA_ERR_INVALID (arguments, or the
 * longest sequence cannot fit the pool under the budget). */
int hydra_schedule(const int64_t* lengths, int64_t n_docs, const hydra_sched_config_t* cfg, int32_t* mb,
                   int32_t* group_start, int32_t* group_size, hydra_sched_summary_t* summary);

#ifdef __cplusplus
}
#endif

#endif /* HYDRA_SCHED_H */
