/*
 * coop.h -- C ABI of the MI355X (gfx950) batched sliding-window eviction
 * search of Coop ("Memory is not a Commodity", section 3.3).
 *
 * The problem (section 3.1 Eq. (1), restated for windows in section 3.3):
 * a pool snapshot is the address-sorted list of the blocks of a memory pool.
 * Each block is a free chunk (cost 0), an evictable tensor with an eviction
 * cost, or a pinned (unevictable) tensor.  For a request of S bytes, find the
 * window [start, end) of adjacent blocks that contains no pinned block, holds
 * at least S bytes in total, and has the smallest summed cost of its
 * evictable blocks.  Ties are broken by the smaller byte total, then by the
 * lower start, which makes the answer unique.  S == 0 gives the empty window
 * {0, 0, 0}; a request no window satisfies gives {~0, ~0, ~0}.
 *
 * The library is stateless apart from a per-process call counter, allocates
 * nothing, never synchronises the stream, and may be called from several
 * host threads (with distinct workspaces).  It needs no HIP header: streams
 * are passed as void* (a hipStream_t; NULL is the default stream).
 *
 * Every entry point may be called on a stream that is capturing a HIP graph,
 * and the graph replayed any number of times: each replay recomputes the
 * outputs from whatever the input buffers hold at that point.  No entry point
 * records a memset node.
 *
 * Debug checks: with COOP_DEBUG=1 in the environment (read on every call),
 * coop_window_search, coop_first_fit and coop_window_search_real first copy
 * the batch's offset arrays (and, where the entry point sums, its blocks)
 * back on the call's stream, synchronise the stream, and reject a batch that
 * breaks a device-resident rule: COOP_ERR_INVALID for an offset rule,
 * COOP_ERR_OVERFLOW for a run whose byte total, or the cost total of its
 * evictable blocks, exceeds 2^64 - 1.  Nothing is launched then.  Calls made
 * while the stream is capturing a graph skip the checks (a capture cannot
 * synchronise).  The checks cost a copy of the arrays per call.
 */
#ifndef COOP_H
#define COOP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Block kinds stored in the kind[] array.  Every value >= COOP_PINNED is
 * pinned: it can never be part of a window (Fig. 1 caption: parameters and
 * buffers are unevictable).  A free chunk is a zero-cost entry whatever its
 * stored cost (section 3.3). */
typedef enum {
    COOP_FREE = 0,
    COOP_EVICTABLE = 1,
    COOP_PINNED = 2
} coop_kind_t;

/* One result: the window [start, end), indices local to the request's
 * snapshot, and its summed eviction cost.  Infeasible: all three ~0. */
typedef struct {
    uint64_t start;
    uint64_t end;
    uint64_t cost;
} coop_window_t;

typedef enum {
    COOP_OK = 0,
    COOP_ERR_INVALID = -1,   /* null pointer with a nonzero count, bad sizes */
    COOP_ERR_WORKSPACE = -2, /* workspace missing or smaller than required */
    COOP_ERR_HIP = -3,       /* a HIP launch failed; the HIP error is cleared */
    COOP_ERR_OVERFLOW = -4,  /* debug checks only: a run's total exceeds 2^64 - 1 */
    COOP_ERR_TOO_LARGE = -5  /* coop_window_search_static: the batch needs more
                                scratch than the library's static array holds */
} coop_status_t;

/* Version of this ABI; bumped on any incompatible change. */
#define COOP_ABI_VERSION 4
int coop_abi_version(void);

/* Human-readable text for a status code (static storage, never NULL). */
const char *coop_status_string(int status);

/* Bytes of device workspace coop_window_search needs for a batch of these
 * dimensions.  Depends only on the three counts.  Returns COOP_ERR_INVALID
 * if bytes_out is NULL or the batch is too large to launch. */
coop_status_t coop_window_search_workspace_size(uint64_t num_blocks,
                                                uint64_t num_segments,
                                                uint64_t num_requests,
                                                size_t *bytes_out);

/* How coop_window_search splits a batch of these dimensions: host-side
 * planning only, for diagnostics and tests.  A unit is one tile of up to
 * 4096 blocks of a snapshot for one slice of that snapshot's requests.  Each
 * of the `workgroups` persistent workgroups first sweeps a chunk of
 * first_chunk_units consecutive units (all of them lie below first_units);
 * the units from first_units on are claimed from a queue in chunks of at
 * least queued_chunk_units units, which the kernel lengthens until no
 * snapshot spans more than partial_slots - 2 chunks.  chunks_max bounds the
 * number of chunks; partial_slots is the number of partial results kept per
 * request.  Returns COOP_ERR_INVALID if plan_out is NULL or the batch is too
 * large to launch. */
typedef struct {
    uint64_t workgroups;
    uint64_t slices;
    uint64_t units;
    uint64_t first_chunk_units;
    uint64_t first_units;
    uint64_t queued_chunk_units;
    uint64_t chunks_max;
    uint64_t partial_slots;
} coop_plan_t;

coop_status_t coop_window_search_plan(uint64_t num_blocks, uint64_t num_segments,
                                      uint64_t num_requests, coop_plan_t *plan_out);

/*
 * coop_window_search -- enqueue the search for every request of a batch.
 *
 * Blocks (device memory, structure of arrays, num_blocks entries each; the
 * snapshots are concatenated):
 *   size[k]  block size in bytes;
 *   cost[k]  eviction cost, used only when kind[k] == COOP_EVICTABLE;
 *   kind[k]  coop_kind_t (any value >= 2 is pinned).
 * Snapshots (device): seg_offsets[num_segments + 1]; snapshot b is blocks
 *   [seg_offsets[b], seg_offsets[b+1]).  seg_offsets[0] == 0, the entries
 *   never decrease, seg_offsets[num_segments] == num_blocks.  Empty
 *   snapshots are allowed.
 * Requests (device): req_sizes[num_requests] in bytes;
 *   req_offsets[num_segments + 1] with the same rules (last entry ==
 *   num_requests); the requests of snapshot b are
 *   [req_offsets[b], req_offsets[b+1]).
 * out (device): num_requests results, in request order.
 * workspace (device): at least coop_window_search_workspace_size() bytes,
 *   256-byte aligned, owned by the caller; its contents need not be
 *   initialised and are meaningless afterwards.  Two calls in flight at the
 *   same time must not share a workspace.  The kernels tell one call's
 *   cross-workgroup counters from an earlier call's by a tag: an eager call
 *   takes it from the per-process call counter; a call made while the stream
 *   is capturing a graph records one single-thread kernel ahead of the search
 *   that advances a tag word kept in the workspace, and the search reads its
 *   tag from there, so every replay gets a fresh one.
 * stream: hipStream_t the work is enqueued on; out is valid once the
 *   stream has reached this point.
 *
 * Preconditions that live in device memory are not checked by the kernels
 * (only by the debug checks above): the offset rules above, and that within
 * every run (a maximal stretch of unpinned blocks) the byte total and the
 * total cost of evictable blocks fit in 64 bits.  When they fail the results
 * are unspecified (but every memory access stays inside the arrays described
 * by the counts).
 *
 * Returns COOP_OK once the work is enqueued (and immediately, enqueuing
 * nothing, when num_requests == 0); COOP_ERR_INVALID for a NULL pointer
 * whose array is non-empty, requests without snapshots, or a batch too large
 * to launch; COOP_ERR_WORKSPACE for a missing or too small workspace;
 * COOP_ERR_HIP when the launch fails; under the debug checks also
 * COOP_ERR_INVALID for a broken offset rule and COOP_ERR_OVERFLOW.
 */
coop_status_t coop_window_search(const uint64_t *size, const uint64_t *cost,
                                 const uint8_t *kind, uint64_t num_blocks,
                                 const uint64_t *seg_offsets, uint64_t num_segments,
                                 const uint64_t *req_sizes, const uint64_t *req_offsets,
                                 uint64_t num_requests, coop_window_t *out,
                                 void *workspace, size_t workspace_bytes, void *stream);

/*
 * coop_window_search_static -- coop_window_search for callers that cannot
 * allocate device memory: code under HIP graph capture that may not call
 * hipMalloc, tight serving loops, harnesses that forbid allocation.  Same
 * arguments, results and status codes as coop_window_search, without the
 * workspace: the cross-workgroup state (partial keys, arrival counters, the
 * chunk queue, the graph tag word, the list of jobs left to the second
 * kernel and its claim word, per-tile records and deferral bits) lives in a static device array of the
 * library, 32 MiB on every GPU the library runs on, held until the process
 * ends.  Its address is looked up on the first call on a device (with the
 * stream's device current) and kept; the call then allocates nothing and
 * never synchronises.
 *
 * The array holds coop_window_search_static_capacity() bytes of workspace.
 * The search is planned with the largest partial-key budget whose workspace
 * fits (fewer partial slots only make the kernel's chunks longer; the
 * results are the same).  A batch that fits no plan -- roughly more than
 * 500,000 requests, or more than 4 million snapshots -- is rejected with
 * COOP_ERR_TOO_LARGE before anything is enqueued.  The debug checks are not
 * run (they copy the batch back to host memory).
 *
 * Every call on one GPU shares that GPU's array, and the array keeps the
 * last call's contents (no call needs it cleared: every counter carries the
 * call's tag).  Calls that overlap in time on one GPU -- on different
 * streams, or from different host threads without ordering -- race on it
 * and give undefined results; calls ordered on one stream are safe.
 */
size_t coop_window_search_static_capacity(void);

coop_status_t coop_window_search_static(const uint64_t *size, const uint64_t *cost,
                                        const uint8_t *kind, uint64_t num_blocks,
                                        const uint64_t *seg_offsets, uint64_t num_segments,
                                        const uint64_t *req_sizes,
                                        const uint64_t *req_offsets, uint64_t num_requests,
                                        coop_window_t *out, void *stream);

/*
 * First fit (section 2.1; Algorithm 1's find_free_block_not_less_than, the
 * step before any eviction): for every request of S bytes, the leftmost free
 * chunk (kind == COOP_FREE) of its snapshot holding at least S bytes, where
 * a first-fit allocator places the tensor.  Evictable and pinned blocks are
 * occupied whatever their size.  S == 0 takes the first free chunk.
 *
 * Same batch layout as coop_window_search (cost is not needed); out
 * (device) receives num_requests snapshot-local block indices, ~0 where the
 * snapshot has no such chunk.  workspace (device, caller-owned, contents
 * need not be initialised) holds per-group and per-tile summaries of the
 * free chunk sizes: coop_first_fit_workspace_size() bytes, which depend on
 * num_blocks only (0 for an empty batch; workspace may then be NULL).  Two
 * launches are enqueued on `stream`; nothing is allocated or synchronised.
 * Status codes and unchecked device preconditions as for
 * coop_window_search.
 */
coop_status_t coop_first_fit_workspace_size(uint64_t num_blocks, size_t *bytes_out);

coop_status_t coop_first_fit(const uint64_t *size, const uint8_t *kind, uint64_t num_blocks,
                             const uint64_t *seg_offsets, uint64_t num_segments,
                             const uint64_t *req_sizes, const uint64_t *req_offsets,
                             uint64_t num_requests, uint64_t *out,
                             void *workspace, size_t workspace_bytes, void *stream);

/*
 * The search with real-valued heuristics (section 3.3 defines a tensor's
 * heuristic as h = c / s, projected cost over staleness, a real number).
 * Same batch layout and window rules as coop_window_search, with h[k]
 * (binary64, device) in place of cost[k].  A window costs the exact real sum
 * of its evictable blocks' h: each h is rounded once to a multiple of 2^-64
 * (to nearest, ties to even; exact for every h >= 2^-12) and the sums are
 * taken in 128-bit fixed point, so no summation order can change the answer.
 * Ranking and tie-breaks as in coop_window_search.
 *
 * out (device) receives num_requests coop_window_real_t: start, end, the
 * exact cost in units of 2^-64 (cost_lo, cost_hi) and that cost rounded to
 * the nearest binary64 (ties to even).  S == 0 gives all zeros; an
 * infeasible request start = end = cost_lo = cost_hi = ~0 and cost = +inf.
 * status (device u32) is set to 0, then bit 0 if an evictable block's h is
 * NaN, infinite, negative (other than -0) or at least 2^64; results for
 * such a batch are unspecified.  The h of free and pinned blocks is
 * ignored.  Precondition: within every run each snapshot's byte total and
 * h total stay below 2^64 (the debug checks cover the offsets and the byte
 * totals, not the h totals).
 *
 * workspace: coop_window_search_real_workspace_size() bytes (device,
 * caller-owned, contents need not be initialised): about 26 bytes per block
 * (tile-local prefix sums) plus partial results.  Four launches are
 * enqueued on `stream`; nothing is allocated or synchronised.  Status codes
 * as for coop_window_search.
 */
typedef struct {
    uint64_t start;
    uint64_t end;
    uint64_t cost_lo; /* exact cost in units of 2^-64, low 64 bits */
    uint64_t cost_hi; /* high 64 bits */
    double cost;      /* the exact cost rounded to the nearest binary64 */
} coop_window_real_t;

coop_status_t coop_window_search_real_workspace_size(uint64_t num_blocks, uint64_t num_segments,
                                                     uint64_t num_requests, size_t *bytes_out);

coop_status_t coop_window_search_real(const uint64_t *size, const double *h, const uint8_t *kind,
                                      uint64_t num_blocks, const uint64_t *seg_offsets,
                                      uint64_t num_segments, const uint64_t *req_sizes,
                                      const uint64_t *req_offsets, uint64_t num_requests,
                                      coop_window_real_t *out, uint32_t *status,
                                      void *workspace, size_t workspace_bytes, void *stream);

/* Eviction policies of coop_replay. */
typedef enum {
    COOP_POLICY_WINDOW = 0, /* Coop: the sliding window (section 3.3) */
    COOP_POLICY_GREEDY = 1  /* DTR's heuristic, one tensor at a time (section 3.3) */
} coop_policy_t;

/*
 * Replay of Algorithm 1 on num_pools independent pools, all in lockstep.
 * For every operation of a pool's trace, in order: an allocation runs first
 * fit; when no free chunk holds S bytes, the sliding-window search for S,
 * evicts the window's tensors, merges the window and its free neighbours
 * into one free chunk and fits again; the tensor goes to the chunk's left
 * end when the operation is expensive and to its right end otherwise
 * (section 3.4).  With no window the allocation fails and nothing changes.
 * A release frees the tensor's block and merges it with free neighbours; a
 * tensor already evicted is skipped.
 *
 * policy COOP_POLICY_WINDOW is the above.  COOP_POLICY_GREEDY is the
 * baseline Coop is compared against: while first fit finds no chunk, evict
 * the evictable tensor of least h = c / (m * s), cost over size times
 * staleness (op_id minus the tensor's id, modulo 2^32; ids are issued in
 * allocation order), a zero size or staleness counting as 1, ties to the
 * lower block index, comparing exactly; each eviction frees and merges one
 * block.  Placement is the same.  With nothing left to evict the allocation
 * fails and the evictions stay done.  Any other value: COOP_ERR_INVALID.
 *
 * Pools (device, updated in place): pool b occupies slots
 *   [b * capacity, (b + 1) * capacity) of size, cost (u64), kind (u8) and id
 *   (u32 tensor ids, 0 for free chunks); len[b] (u64) blocks are in use,
 *   never two free chunks side by side, and unused slots must hold empty
 *   pinned blocks (size 0, kind COOP_PINNED), which the replay keeps so.
 * Operations (device): num_ops per pool, pool b's at [b * num_ops, +num_ops):
 *   op 0 allocate (op_id != 0, op_size > 0, op_cost, op_flags bit 0
 *   expensive, bit 1 unevictable tensor), op 1 release op_id.
 * Outputs (device), per operation: out_block (the tensor's block, or the
 *   merged free chunk of a release; ~0 for a failed allocation or a
 *   skipped release), out_window[2] (the evicted window, indices before the
 *   eviction, or ~0; greedy: {number of tensors evicted, ~0}), out_cost (the
 *   evicted cost, modulo 2^64), out_free (free bytes just before an
 *   eviction, else ~0: the fragmentation-rate sample of section 4.2, free
 *   memory over the memory the allocator holds).
 * status (device u32): set to 0, then bit 0 if a pool ran out of slots (that
 *   allocation is skipped), bit 1 for an invalid operation.
 * workspace: coop_replay_workspace_size() bytes (device, caller-owned).
 * Pools of up to about 5250 slots (31 bytes of LDS a slot, within 160 KiB)
 * are replayed by two launches, a workgroup per pool holding the pool in
 * LDS; larger ones step by step, about five launches per operation (the
 * greedy policy skips the window search's).  Either way everything is enqueued on `stream`; nothing is
 * allocated or synchronised.
 */
coop_status_t coop_replay_workspace_size(uint64_t num_pools, uint64_t capacity,
                                         size_t *bytes_out);

coop_status_t coop_replay(uint64_t *size, uint64_t *cost, uint8_t *kind, uint32_t *id,
                          uint64_t *len, uint64_t num_pools, uint64_t capacity,
                          const uint8_t *op, const uint32_t *op_id, const uint64_t *op_size,
                          const uint64_t *op_cost, const uint8_t *op_flags, uint64_t num_ops,
                          int32_t policy, uint64_t *out_block, uint64_t *out_window,
                          uint64_t *out_cost, uint64_t *out_free, uint32_t *status,
                          void *workspace, size_t workspace_bytes, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* COOP_H */
