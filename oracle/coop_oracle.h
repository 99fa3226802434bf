/*
 * coop_oracle.h -- CPU oracle for the Coop sliding-window eviction search.
 *
 * TEST INFRASTRUCTURE ONLY.  This library is the correctness reference that
 * the GPU path is compared against.  It is called by the test suite, by the
 * smoke check and by the benchmark's CPU-baseline leg, and by nothing else.
 * It shares no code, header, table or helper with the GPU library: it defines
 * its own constants and reads plain host arrays.
 *
 * What it computes (Coop, "Memory is not a Commodity", section 3.1 Eq. (1)
 * and section 3.3):
 *
 *   A pool snapshot is an address-sorted list of N blocks.  Block k has a
 *   byte size size[k], a kind (0 = free chunk, 1 = evictable tensor,
 *   any value >= 2 = unevictable/pinned tensor) and a cost cost[k].  Free
 *   chunks count as zero-cost entries (section 3.3: free chunks are tensors
 *   whose heuristic is zero); the stored cost of free and pinned blocks is
 *   ignored.  Pinned blocks can never be evicted (Fig. 1 caption).
 *
 *   For a request of S bytes the result is the window [start, end), a run of
 *   adjacent blocks containing no pinned block, whose byte total is >= S and
 *   whose summed evictable cost is minimal.  Ties are broken by the smaller
 *   byte total, then the lower start (the paper does not fix a tie-break;
 *   this one makes the answer unique).  S == 0 yields the empty window
 *   {0, 0, 0}.  No qualifying window yields {~0, ~0, ~0}.
 *
 * Batch layout (all host memory, caller-owned):
 *   size[num_blocks], cost[num_blocks], kind[num_blocks]: blocks of all
 *     snapshots, concatenated.
 *   seg_offsets[num_segments + 1]: snapshot b is blocks
 *     [seg_offsets[b], seg_offsets[b+1]); seg_offsets[0] == 0, non-decreasing,
 *     seg_offsets[num_segments] == num_blocks.
 *   req_sizes[num_requests], req_offsets[num_segments + 1]: the requests of
 *     snapshot b are [req_offsets[b], req_offsets[b+1]), same rules, last
 *     entry == num_requests.
 *   out[3 * num_requests]: (start, end, cost) per request, start/end local to
 *     the request's snapshot.
 *
 * Return codes: 0 ok, -1 invalid arguments, -4 a run's size or effective-cost
 * total does not fit in 64 bits (the precondition the GPU path relies on),
 * -5 input too large for a brute-force enumerator, -6 an invalid real-valued
 * heuristic.
 */
#ifndef COOP_ORACLE_H
#define COOP_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define COOP_ORACLE_OK 0
#define COOP_ORACLE_ERR_INVALID (-1)
#define COOP_ORACLE_ERR_OVERFLOW (-4)
#define COOP_ORACLE_ERR_TOO_LARGE (-5)
#define COOP_ORACLE_ERR_VALUE (-6)

/* Linear two-pointer sweep per run (section 3.3), one request at a time,
 * requests spread over num_threads POSIX threads (<= 0 means 1). */
int coop_oracle_window_search(const uint64_t *size, const uint64_t *cost,
                              const uint8_t *kind, uint64_t num_blocks,
                              const uint64_t *seg_offsets, uint64_t num_segments,
                              const uint64_t *req_sizes, const uint64_t *req_offsets,
                              uint64_t num_requests, uint64_t *out, int num_threads);

/* Brute force over every window [i, j) of every snapshot, keyed by
 * (cost, bytes, i, j).  O(N^3) per request; snapshots must have <= 512
 * blocks.  Same arguments and output as coop_oracle_window_search. */
int coop_oracle_brute_windows(const uint64_t *size, const uint64_t *cost,
                              const uint8_t *kind, uint64_t num_blocks,
                              const uint64_t *seg_offsets, uint64_t num_segments,
                              const uint64_t *req_sizes, const uint64_t *req_offsets,
                              uint64_t num_requests, uint64_t *out);

/* Eq. (1) taken literally: enumerate every subset of the evictable blocks of
 * the snapshot, evict it, measure the largest contiguous run of available
 * bytes (free chunks plus evicted blocks), and keep the cheapest subset whose
 * run reaches S.  Writes the minimal cost per request to out_cost, or ~0 when
 * no subset qualifies.  At most 20 evictable blocks per snapshot. */
int coop_oracle_brute_eq1(const uint64_t *size, const uint64_t *cost,
                          const uint8_t *kind, uint64_t num_blocks,
                          const uint64_t *seg_offsets, uint64_t num_segments,
                          const uint64_t *req_sizes, const uint64_t *req_offsets,
                          uint64_t num_requests, uint64_t *out_cost);

/* First fit (section 2.1; find_free_block_not_less_than in Algorithm 1):
 * for every request, the lowest snapshot-local index k of a free chunk
 * (kind[k] == 0) with size[k] >= S, or ~0 when the snapshot holds none.
 * S == 0 takes the first free chunk.  out[num_requests].  Same batch layout
 * as above, without costs; requests over num_threads POSIX threads. */
int coop_oracle_first_fit(const uint64_t *size, const uint8_t *kind, uint64_t num_blocks,
                          const uint64_t *seg_offsets, uint64_t num_segments,
                          const uint64_t *req_sizes, const uint64_t *req_offsets,
                          uint64_t num_requests, uint64_t *out, int num_threads);

/* The search with real-valued heuristics (section 3.3: h = c / s).  h[k]
 * (binary64) replaces cost[k]; a window costs the exact sum of its h values:
 * each h is rounded to a multiple of 2^-64 (to nearest, ties to even; exact
 * for h >= 2^-12) and summed in 128-bit fixed point, so the answer does not
 * depend on any summation order.  Ranking and tie-breaks as above.  Per
 * request out[4] = (start, end, low and high 64 bits of the exact sum in
 * units of 2^-64) and out_cost = that sum rounded to the nearest binary64
 * (ties to even).  S == 0: (0, 0, 0, 0) and 0.0; infeasible: all ~0 and
 * +inf.  Returns -6 if an evictable block's h is NaN, negative or >= 2^64,
 * -4 if a run's byte total or h total reaches 2^64.  Must run under the
 * default floating-point rounding mode. */
int coop_oracle_window_search_real(const uint64_t *size, const double *h, const uint8_t *kind,
                                   uint64_t num_blocks, const uint64_t *seg_offsets,
                                   uint64_t num_segments, const uint64_t *req_sizes,
                                   const uint64_t *req_offsets, uint64_t num_requests,
                                   uint64_t *out, double *out_cost, int num_threads);

/* Replay of Algorithm 1 (allocate: first fit, else evict the sliding
 * window's tensors, merge the window into one free chunk and fit again;
 * expensive operations placed at the left end of the chunk, others at the
 * right end as in section 3.4) and of releases, on num_pools independent
 * pools.  Pool b occupies slots [b * capacity, (b + 1) * capacity) of
 * size/cost/kind/id (tensor ids, 0 for free chunks); len[b] blocks are in
 * use.  All are updated in place.  Operations: num_ops per pool, pool b's at
 * [b * num_ops, (b + 1) * num_ops): op 0 = allocate(op_id, op_size,
 * op_cost, op_flags: 1 expensive, 2 unevictable), op 1 = release(op_id).
 * Outputs per operation: out_block (the tensor's block, the merged free
 * chunk of a release, ~0 for a failed allocation or a release of an evicted
 * tensor), out_window[2] (evicted window, pre-eviction indices, or ~0),
 * out_cost (its eviction cost), out_free (free bytes just before an
 * eviction, else ~0).  Returns -5 if a pool would exceed its capacity.
 *
 * policy 0 is Coop's (the sliding window).  policy 1 is the DTR-style greedy
 * baseline: while no chunk fits, evict the evictable tensor of least
 * h = cost / (size * staleness), staleness being op_id minus the tensor's
 * id (ids are issued in allocation order), ties to the lower index; each
 * eviction frees and merges one block.  out_window[0] then holds the number
 * of tensors evicted for the operation (out_window[1] ~0), out_cost their
 * summed cost, out_free the free bytes before the first of them.  If the
 * pool runs out of evictable tensors the allocation fails, the evictions
 * staying done. */
int coop_oracle_replay(uint64_t *size, uint64_t *cost, uint8_t *kind, uint32_t *id, uint64_t *len,
                       uint64_t num_pools, uint64_t capacity, const uint8_t *op,
                       const uint32_t *op_id, const uint64_t *op_size, const uint64_t *op_cost,
                       const uint8_t *op_flags, uint64_t num_ops, uint64_t *out_block,
                       uint64_t *out_window, uint64_t *out_cost, uint64_t *out_free,
                       int policy, int num_threads);

#ifdef __cplusplus
}
#endif

#endif /* COOP_ORACLE_H */
