/*
 * coop_oracle.c -- plain, slow, obviously correct CPU reference for the Coop
 * sliding-window eviction search (section 3.1 Eq. (1), section 3.3).
 *
 * TEST INFRASTRUCTURE ONLY: called by the tests, the smoke check and the
 * benchmark's CPU-baseline leg.  It shares nothing with the GPU library.
 *
 * Everything is unsigned 64-bit integer arithmetic; no rounding is involved,
 * so any correct implementation must agree with this one bit for bit.
 */
#include "coop_oracle.h"

#include <math.h>
#include <pthread.h>
#include <stdatomic.h>
#include <stdlib.h>
#include <string.h>

#define NONE UINT64_MAX

/* Kinds (section 3.3 and the Fig. 1 caption): free chunk, evictable tensor,
 * unevictable tensor.  Any kind value of 2 or more is unevictable. */
#define KIND_FREE 0
#define KIND_EVICTABLE 1

static int is_pinned(uint8_t k) { return k >= 2; }

/* Cost of evicting one block: a free chunk is a zero-heuristic entry
 * (section 3.3), a pinned block is never part of a window. */
static uint64_t eviction_cost(uint8_t k, uint64_t c) {
    return k == KIND_EVICTABLE ? c : 0;
}

/* Lexicographic order on (cost, bytes, start). */
static int key_less(uint64_t c1, uint64_t b1, uint64_t s1,
                    uint64_t c2, uint64_t b2, uint64_t s2) {
    if (c1 != c2) return c1 < c2;
    if (b1 != b2) return b1 < b2;
    return s1 < s2;
}

/* Checks the CSR offsets of one batch dimension. */
static int offsets_ok(const uint64_t *off, uint64_t n, uint64_t total) {
    if (!off || off[0] != 0 || off[n] != total) return 0;
    for (uint64_t b = 0; b < n; ++b)
        if (off[b + 1] < off[b]) return 0;
    return 1;
}

static int batch_ok(const uint64_t *size, const uint64_t *cost, const uint8_t *kind,
                    uint64_t num_blocks, const uint64_t *seg_offsets,
                    uint64_t num_segments, const uint64_t *req_sizes,
                    const uint64_t *req_offsets, uint64_t num_requests,
                    const void *out) {
    if (num_blocks && (!size || !cost || !kind)) return 0;
    if (num_requests && (!req_sizes || !out)) return 0;
    if (num_segments == 0) return num_blocks == 0 && num_requests == 0;
    return offsets_ok(seg_offsets, num_segments, num_blocks) &&
           offsets_ok(req_offsets, num_segments, num_requests);
}

/* The precondition every implementation relies on: within each run (a
 * maximal stretch of unpinned blocks) the byte total and the effective-cost
 * total fit in 64 bits.  Then every window sum fits as well. */
static int runs_fit(const uint64_t *size, const uint64_t *cost, const uint8_t *kind,
                    uint64_t n) {
    uint64_t bytes = 0, c = 0;
    for (uint64_t k = 0; k < n; ++k) {
        if (is_pinned(kind[k])) { bytes = 0; c = 0; continue; }
        if (__builtin_add_overflow(bytes, size[k], &bytes)) return 0;
        if (__builtin_add_overflow(c, eviction_cost(kind[k], cost[k]), &c)) return 0;
    }
    return 1;
}

/* ---------------------------------------------------------------------------
 * Linear sweep (section 3.3).  The list is cut into runs at pinned blocks.
 * Inside a run two indices, st and e, bound the window [st, e).  For each
 * start st the end e is pushed right until the window holds at least S
 * bytes; that is the shortest window beginning at st, and any longer one
 * costs no less and holds no fewer bytes, so it is the only candidate for
 * st.  Moving st one block right never moves the shortest end left, so e
 * only ever advances and one pass over the run suffices.
 * ------------------------------------------------------------------------- */
static void sweep_one(const uint64_t *size, const uint64_t *cost, const uint8_t *kind,
                      uint64_t n, uint64_t S, uint64_t res[3]) {
    res[0] = res[1] = res[2] = NONE;
    if (S == 0) { res[0] = res[1] = res[2] = 0; return; }

    int found = 0;
    uint64_t best_c = 0, best_b = 0, best_s = 0, best_e = 0;
    uint64_t i = 0;
    while (i < n) {
        if (is_pinned(kind[i])) { ++i; continue; }
        uint64_t r = i;                       /* the run is [i, r) */
        while (r < n && !is_pinned(kind[r])) ++r;

        uint64_t e = i, bytes = 0, c = 0;     /* window [st, e) */
        for (uint64_t st = i; st < r; ++st) {
            while (e < r && bytes < S) {
                bytes += size[e];
                c += eviction_cost(kind[e], cost[e]);
                ++e;
            }
            if (bytes < S) break;             /* no later start can reach S */
            if (!found || key_less(c, bytes, st, best_c, best_b, best_s)) {
                found = 1;
                best_c = c; best_b = bytes; best_s = st; best_e = e;
            }
            bytes -= size[st];
            c -= eviction_cost(kind[st], cost[st]);
        }
        i = r;
    }
    if (found) { res[0] = best_s; res[1] = best_e; res[2] = best_c; }
}

/* Request q belongs to the snapshot b with req_offsets[b] <= q < req_offsets[b+1]. */
static uint64_t owner_segment(const uint64_t *req_offsets, uint64_t num_segments,
                              uint64_t q) {
    uint64_t lo = 0, hi = num_segments;       /* answer in [lo, hi) */
    while (hi - lo > 1) {
        uint64_t mid = lo + (hi - lo) / 2;
        if (req_offsets[mid] <= q) lo = mid; else hi = mid;
    }
    return lo;
}

struct sweep_job {
    const uint64_t *size, *cost;
    const uint8_t *kind;
    const uint64_t *seg_offsets, *req_sizes, *req_offsets;
    uint64_t num_segments, num_requests;
    uint64_t *out;
    _Atomic uint64_t next;
};

#define SWEEP_CHUNK 16

static void *sweep_worker(void *arg) {
    struct sweep_job *job = (struct sweep_job *)arg;
    for (;;) {
        uint64_t q0 = atomic_fetch_add(&job->next, SWEEP_CHUNK);
        if (q0 >= job->num_requests) break;
        uint64_t q1 = q0 + SWEEP_CHUNK < job->num_requests ? q0 + SWEEP_CHUNK
                                                           : job->num_requests;
        for (uint64_t q = q0; q < q1; ++q) {
            uint64_t b = owner_segment(job->req_offsets, job->num_segments, q);
            uint64_t s0 = job->seg_offsets[b], n = job->seg_offsets[b + 1] - s0;
            sweep_one(job->size + s0, job->cost + s0, job->kind + s0, n,
                      job->req_sizes[q], job->out + 3 * q);
        }
    }
    return NULL;
}

int coop_oracle_window_search(const uint64_t *size, const uint64_t *cost,
                              const uint8_t *kind, uint64_t num_blocks,
                              const uint64_t *seg_offsets, uint64_t num_segments,
                              const uint64_t *req_sizes, const uint64_t *req_offsets,
                              uint64_t num_requests, uint64_t *out, int num_threads) {
    if (!batch_ok(size, cost, kind, num_blocks, seg_offsets, num_segments, req_sizes,
                  req_offsets, num_requests, out))
        return COOP_ORACLE_ERR_INVALID;
    if (num_requests == 0) return COOP_ORACLE_OK;
    for (uint64_t b = 0; b < num_segments; ++b) {
        uint64_t s0 = seg_offsets[b];
        if (!runs_fit(size + s0, cost + s0, kind + s0, seg_offsets[b + 1] - s0))
            return COOP_ORACLE_ERR_OVERFLOW;
    }

    struct sweep_job job;
    job.size = size; job.cost = cost; job.kind = kind;
    job.seg_offsets = seg_offsets; job.req_sizes = req_sizes;
    job.req_offsets = req_offsets; job.num_segments = num_segments;
    job.num_requests = num_requests; job.out = out;
    atomic_init(&job.next, 0);

    if (num_threads <= 1) {
        sweep_worker(&job);
        return COOP_ORACLE_OK;
    }
    pthread_t *tid = (pthread_t *)calloc((size_t)num_threads, sizeof(pthread_t));
    if (!tid) return COOP_ORACLE_ERR_INVALID;
    int started = 0;
    for (int t = 0; t < num_threads; ++t) {
        if (pthread_create(&tid[t], NULL, sweep_worker, &job) != 0) break;
        ++started;
    }
    if (started == 0) sweep_worker(&job);
    for (int t = 0; t < started; ++t) pthread_join(tid[t], NULL);
    free(tid);
    return COOP_ORACLE_OK;
}

/* ---------------------------------------------------------------------------
 * Real-valued heuristic.  Section 3.3 defines a tensor's heuristic as
 * h(t) = c(t) / s(t), projected cost over staleness: a real number.  Here
 * each evictable block carries h as a binary64 value and a window costs the
 * exact real sum of its h values, so that no summation order can change
 * which window wins.  To add exactly, each h becomes a 128-bit fixed-point
 * number with 64 fraction bits (Q64.64), rounded to the nearest multiple of
 * 2^-64, ties to even.  That rounding is exact for every h >= 2^-12, whose
 * binary64 spacing is at least 2^-64.  h must be finite, >= 0 and < 2^64;
 * the stored h of free and pinned blocks is ignored.  Each run's total must
 * stay below 2^64 (its fixed-point sum fits 128 bits).
 * ------------------------------------------------------------------------- */
typedef unsigned __int128 u128;

#define U128_NONE (~(u128)0)

/* h to Q64.64: 2^64 * h is exact in binary64 (a power-of-two scaling well
 * inside the exponent range); nearbyint rounds it to an integer under the
 * default rounding mode, to nearest with ties to even; that integer (below
 * 2^128, at most 53 significant bits) is split into two exact halves. */
static int real_to_q(double h, u128 *q) {
    if (!(h >= 0.0) || !(h < 0x1p64)) return 0;
    const double x = nearbyint(ldexp(h, 64));
    const double hi = floor(ldexp(x, -64));
    const double lo = x - ldexp(hi, 64);
    *q = ((u128)(uint64_t)hi << 64) | (u128)(uint64_t)lo;
    return 1;
}

/* Q64.64 to the nearest binary64, ties to even: the compiler's unsigned
 * 128-bit conversion rounds to nearest, and the scaling by 2^-64 is exact. */
static double q_to_real(u128 q) { return ldexp((double)q, -64); }

static u128 real_cost(uint8_t k, u128 q) { return k == KIND_EVICTABLE ? q : 0; }

static int key_less_real(u128 c1, uint64_t b1, uint64_t s1, u128 c2, uint64_t b2,
                         uint64_t s2) {
    if (c1 != c2) return c1 < c2;
    if (b1 != b2) return b1 < b2;
    return s1 < s2;
}

/* The same linear sweep as above, on fixed-point costs. */
static void sweep_one_real(const uint64_t *size, const u128 *q, const uint8_t *kind,
                           uint64_t n, uint64_t S, uint64_t res[4], double *res_cost) {
    res[0] = res[1] = res[2] = res[3] = NONE;
    *res_cost = INFINITY;
    if (S == 0) {
        res[0] = res[1] = res[2] = res[3] = 0;
        *res_cost = 0.0;
        return;
    }
    int found = 0;
    u128 best_c = 0;
    uint64_t best_b = 0, best_s = 0, best_e = 0;
    uint64_t i = 0;
    while (i < n) {
        if (is_pinned(kind[i])) { ++i; continue; }
        uint64_t r = i;
        while (r < n && !is_pinned(kind[r])) ++r;
        uint64_t e = i, bytes = 0;
        u128 c = 0;
        for (uint64_t st = i; st < r; ++st) {
            while (e < r && bytes < S) {
                bytes += size[e];
                c += real_cost(kind[e], q[e]);
                ++e;
            }
            if (bytes < S) break;
            if (!found || key_less_real(c, bytes, st, best_c, best_b, best_s)) {
                found = 1;
                best_c = c; best_b = bytes; best_s = st; best_e = e;
            }
            bytes -= size[st];
            c -= real_cost(kind[st], q[st]);
        }
        i = r;
    }
    if (found) {
        res[0] = best_s;
        res[1] = best_e;
        res[2] = (uint64_t)best_c;
        res[3] = (uint64_t)(best_c >> 64);
        *res_cost = q_to_real(best_c);
    }
}

struct real_job {
    const uint64_t *size;
    const u128 *q;
    const uint8_t *kind;
    const uint64_t *seg_offsets, *req_sizes, *req_offsets;
    uint64_t num_segments, num_requests;
    uint64_t *out;
    double *out_cost;
    _Atomic uint64_t next;
};

static void *real_worker(void *arg) {
    struct real_job *job = (struct real_job *)arg;
    for (;;) {
        uint64_t q0 = atomic_fetch_add(&job->next, SWEEP_CHUNK);
        if (q0 >= job->num_requests) break;
        uint64_t q1 = q0 + SWEEP_CHUNK < job->num_requests ? q0 + SWEEP_CHUNK
                                                           : job->num_requests;
        for (uint64_t r = q0; r < q1; ++r) {
            uint64_t b = owner_segment(job->req_offsets, job->num_segments, r);
            uint64_t s0 = job->seg_offsets[b], n = job->seg_offsets[b + 1] - s0;
            sweep_one_real(job->size + s0, job->q + s0, job->kind + s0, n, job->req_sizes[r],
                           job->out + 4 * r, job->out_cost + r);
        }
    }
    return NULL;
}

int coop_oracle_window_search_real(const uint64_t *size, const double *h, const uint8_t *kind,
                                   uint64_t num_blocks, const uint64_t *seg_offsets,
                                   uint64_t num_segments, const uint64_t *req_sizes,
                                   const uint64_t *req_offsets, uint64_t num_requests,
                                   uint64_t *out, double *out_cost, int num_threads) {
    if (!batch_ok(size, (const uint64_t *)h, kind, num_blocks, seg_offsets, num_segments,
                  req_sizes, req_offsets, num_requests, out) ||
        (num_requests && !out_cost))
        return COOP_ORACLE_ERR_INVALID;
    u128 *q = (u128 *)malloc((num_blocks ? num_blocks : 1) * sizeof(u128));
    if (!q) return COOP_ORACLE_ERR_INVALID;
    int rc = COOP_ORACLE_OK;
    for (uint64_t k = 0; k < num_blocks && rc == COOP_ORACLE_OK; ++k) {
        q[k] = 0;
        if (kind[k] == KIND_EVICTABLE && !real_to_q(h[k], &q[k])) rc = COOP_ORACLE_ERR_VALUE;
    }
    /* every run's byte total below 2^64, its h total below 2^64 */
    for (uint64_t b = 0; b < num_segments && rc == COOP_ORACLE_OK; ++b) {
        uint64_t bytes = 0;
        u128 c = 0;
        for (uint64_t k = seg_offsets[b]; k < seg_offsets[b + 1]; ++k) {
            if (is_pinned(kind[k])) { bytes = 0; c = 0; continue; }
            if (__builtin_add_overflow(bytes, size[k], &bytes) ||
                __builtin_add_overflow(c, q[k], &c)) {
                rc = COOP_ORACLE_ERR_OVERFLOW;
                break;
            }
        }
    }
    if (rc != COOP_ORACLE_OK || num_requests == 0) {
        free(q);
        return rc;
    }
    struct real_job job;
    job.size = size; job.q = q; job.kind = kind;
    job.seg_offsets = seg_offsets; job.req_sizes = req_sizes;
    job.req_offsets = req_offsets; job.num_segments = num_segments;
    job.num_requests = num_requests; job.out = out; job.out_cost = out_cost;
    atomic_init(&job.next, 0);
    pthread_t *tid = num_threads > 1 ? (pthread_t *)calloc((size_t)num_threads,
                                                           sizeof(pthread_t)) : NULL;
    int started = 0;
    for (int t = 0; tid && t < num_threads; ++t) {
        if (pthread_create(&tid[t], NULL, real_worker, &job) != 0) break;
        ++started;
    }
    if (started == 0) real_worker(&job);
    for (int t = 0; t < started; ++t) pthread_join(tid[t], NULL);
    free(tid);
    free(q);
    return COOP_ORACLE_OK;
}

/* ---------------------------------------------------------------------------
 * Brute force over windows: every [i, j) with no pinned block inside and at
 * least S bytes is a candidate; each sum is recomputed from scratch.  The
 * minimum of (cost, bytes, i, j) is the answer.
 * ------------------------------------------------------------------------- */
#define BRUTE_WINDOWS_MAX_N 512

static void brute_windows_one(const uint64_t *size, const uint64_t *cost,
                              const uint8_t *kind, uint64_t n, uint64_t S,
                              uint64_t res[3]) {
    res[0] = res[1] = res[2] = NONE;
    if (S == 0) { res[0] = res[1] = res[2] = 0; return; }
    int found = 0;
    uint64_t bc = 0, bb = 0, bi = 0, bj = 0;
    for (uint64_t i = 0; i < n; ++i) {
        for (uint64_t j = i + 1; j <= n; ++j) {
            int blocked = 0;
            uint64_t bytes = 0, c = 0;
            for (uint64_t k = i; k < j; ++k) {
                if (is_pinned(kind[k])) { blocked = 1; break; }
                bytes += size[k];
                c += eviction_cost(kind[k], cost[k]);
            }
            if (blocked || bytes < S) continue;
            int better = !found || c < bc || (c == bc && bytes < bb) ||
                         (c == bc && bytes == bb && i < bi) ||
                         (c == bc && bytes == bb && i == bi && j < bj);
            if (better) { found = 1; bc = c; bb = bytes; bi = i; bj = j; }
        }
    }
    if (found) { res[0] = bi; res[1] = bj; res[2] = bc; }
}

int coop_oracle_brute_windows(const uint64_t *size, const uint64_t *cost,
                              const uint8_t *kind, uint64_t num_blocks,
                              const uint64_t *seg_offsets, uint64_t num_segments,
                              const uint64_t *req_sizes, const uint64_t *req_offsets,
                              uint64_t num_requests, uint64_t *out) {
    if (!batch_ok(size, cost, kind, num_blocks, seg_offsets, num_segments, req_sizes,
                  req_offsets, num_requests, out))
        return COOP_ORACLE_ERR_INVALID;
    for (uint64_t b = 0; b < num_segments; ++b) {
        uint64_t s0 = seg_offsets[b], n = seg_offsets[b + 1] - s0;
        if (n > BRUTE_WINDOWS_MAX_N) return COOP_ORACLE_ERR_TOO_LARGE;
        if (!runs_fit(size + s0, cost + s0, kind + s0, n)) return COOP_ORACLE_ERR_OVERFLOW;
    }
    for (uint64_t b = 0; b < num_segments; ++b) {
        uint64_t s0 = seg_offsets[b], n = seg_offsets[b + 1] - s0;
        for (uint64_t q = req_offsets[b]; q < req_offsets[b + 1]; ++q)
            brute_windows_one(size + s0, cost + s0, kind + s0, n, req_sizes[q],
                              out + 3 * q);
    }
    return COOP_ORACLE_OK;
}

/* ---------------------------------------------------------------------------
 * Eq. (1) by exhaustion (section 3.3 names this 2^N enumeration as the naive
 * approach).  For a subset E of the evictable blocks, M(E, L) is the largest
 * byte total of adjacent available blocks, where a block is available when
 * it is a free chunk or belongs to E.  The answer is min over E with
 * M(E, L) >= S of the summed cost of E.
 * ------------------------------------------------------------------------- */
#define BRUTE_EQ1_MAX_EVICTABLE 20

static uint64_t brute_eq1_one(const uint64_t *size, const uint64_t *cost,
                              const uint8_t *kind, uint64_t n, uint64_t S,
                              const uint64_t *evictable, unsigned m) {
    uint64_t best = NONE;
    for (uint64_t mask = 0; mask < (1ull << m); ++mask) {
        uint64_t c = 0;
        for (unsigned t = 0; t < m; ++t)
            if (mask >> t & 1) c += cost[evictable[t]];
        /* Largest contiguous available memory after evicting the subset. */
        uint64_t largest = 0, run = 0;
        unsigned t = 0;
        for (uint64_t k = 0; k < n; ++k) {
            int available;
            if (kind[k] == KIND_FREE) {
                available = 1;
            } else if (kind[k] == KIND_EVICTABLE) {
                while (t < m && evictable[t] < k) ++t;
                available = (t < m && evictable[t] == k) ? (int)(mask >> t & 1) : 0;
            } else {
                available = 0;
            }
            run = available ? run + size[k] : 0;
            if (run > largest) largest = run;
        }
        if (largest >= S && c < best) best = c;
    }
    return best;
}

int coop_oracle_brute_eq1(const uint64_t *size, const uint64_t *cost,
                          const uint8_t *kind, uint64_t num_blocks,
                          const uint64_t *seg_offsets, uint64_t num_segments,
                          const uint64_t *req_sizes, const uint64_t *req_offsets,
                          uint64_t num_requests, uint64_t *out_cost) {
    if (!batch_ok(size, cost, kind, num_blocks, seg_offsets, num_segments, req_sizes,
                  req_offsets, num_requests, out_cost))
        return COOP_ORACLE_ERR_INVALID;
    uint64_t evictable[BRUTE_EQ1_MAX_EVICTABLE];
    for (uint64_t b = 0; b < num_segments; ++b) {
        uint64_t s0 = seg_offsets[b], n = seg_offsets[b + 1] - s0;
        unsigned m = 0;
        for (uint64_t k = 0; k < n; ++k) {
            if (kind[s0 + k] != KIND_EVICTABLE) continue;
            if (m == BRUTE_EQ1_MAX_EVICTABLE) return COOP_ORACLE_ERR_TOO_LARGE;
            evictable[m++] = k;
        }
        if (!runs_fit(size + s0, cost + s0, kind + s0, n)) return COOP_ORACLE_ERR_OVERFLOW;
        for (uint64_t q = req_offsets[b]; q < req_offsets[b + 1]; ++q)
            out_cost[q] = brute_eq1_one(size + s0, cost + s0, kind + s0, n,
                                        req_sizes[q], evictable, m);
    }
    return COOP_ORACLE_OK;
}

/* ---------------------------------------------------------------------------
 * First fit (section 2.1, and find_free_block_not_less_than in Algorithm 1):
 * the allocator places a tensor of S bytes at the left end of a free chunk
 * of at least S bytes, the leftmost such chunk.  The answer is that chunk's
 * index in its snapshot, found by walking the list from the left.
 * ------------------------------------------------------------------------- */
static uint64_t first_fit_one(const uint64_t *size, const uint8_t *kind, uint64_t n,
                              uint64_t S) {
    for (uint64_t k = 0; k < n; ++k)
        if (kind[k] == KIND_FREE && size[k] >= S) return k;
    return NONE;
}

struct fit_job {
    const uint64_t *size;
    const uint8_t *kind;
    const uint64_t *seg_offsets, *req_sizes, *req_offsets;
    uint64_t num_segments, num_requests;
    uint64_t *out;
    _Atomic uint64_t next;
};

static void *fit_worker(void *arg) {
    struct fit_job *job = (struct fit_job *)arg;
    for (;;) {
        uint64_t q0 = atomic_fetch_add(&job->next, SWEEP_CHUNK);
        if (q0 >= job->num_requests) break;
        uint64_t q1 = q0 + SWEEP_CHUNK < job->num_requests ? q0 + SWEEP_CHUNK
                                                           : job->num_requests;
        for (uint64_t q = q0; q < q1; ++q) {
            uint64_t b = owner_segment(job->req_offsets, job->num_segments, q);
            uint64_t s0 = job->seg_offsets[b], n = job->seg_offsets[b + 1] - s0;
            job->out[q] = first_fit_one(job->size + s0, job->kind + s0, n, job->req_sizes[q]);
        }
    }
    return NULL;
}

int coop_oracle_first_fit(const uint64_t *size, const uint8_t *kind, uint64_t num_blocks,
                          const uint64_t *seg_offsets, uint64_t num_segments,
                          const uint64_t *req_sizes, const uint64_t *req_offsets,
                          uint64_t num_requests, uint64_t *out, int num_threads) {
    if (num_blocks && (!size || !kind)) return COOP_ORACLE_ERR_INVALID;
    if (num_requests && (!req_sizes || !out)) return COOP_ORACLE_ERR_INVALID;
    if (num_segments == 0) {
        if (num_blocks || num_requests) return COOP_ORACLE_ERR_INVALID;
        return COOP_ORACLE_OK;
    }
    if (!offsets_ok(seg_offsets, num_segments, num_blocks) ||
        !offsets_ok(req_offsets, num_segments, num_requests))
        return COOP_ORACLE_ERR_INVALID;
    if (num_requests == 0) return COOP_ORACLE_OK;

    struct fit_job job;
    job.size = size; job.kind = kind;
    job.seg_offsets = seg_offsets; job.req_sizes = req_sizes;
    job.req_offsets = req_offsets; job.num_segments = num_segments;
    job.num_requests = num_requests; job.out = out;
    atomic_init(&job.next, 0);

    if (num_threads <= 1) {
        fit_worker(&job);
        return COOP_ORACLE_OK;
    }
    pthread_t *tid = (pthread_t *)calloc((size_t)num_threads, sizeof(pthread_t));
    if (!tid) return COOP_ORACLE_ERR_INVALID;
    int started = 0;
    for (int t = 0; t < num_threads; ++t) {
        if (pthread_create(&tid[t], NULL, fit_worker, &job) != 0) break;
        ++started;
    }
    if (started == 0) fit_worker(&job);
    for (int t = 0; t < started; ++t) pthread_join(tid[t], NULL);
    free(tid);
    return COOP_ORACLE_OK;
}

/* ---------------------------------------------------------------------------
 * Replay of Algorithm 1 on independent pools.  A pool is its address-sorted
 * block list, holding a fixed number of bytes; no two free chunks are ever
 * adjacent (section 2.1: a released chunk merges with its free neighbours).
 * Each operation of a pool's trace is applied in order:
 *
 *   allocate(id, S, flags): first fit; if no free chunk holds S bytes, the
 *     sliding-window search for S (section 3.3), the window's evictable
 *     tensors are evicted and the whole window becomes one free chunk, merged
 *     with free neighbours, and first fit runs again (Algorithm 1).  The
 *     tensor goes to the left end of the chunk when the operation is
 *     expensive and to the right end otherwise (section 3.4, applied to
 *     every placement).  No window: the allocation fails and nothing
 *     changes.
 *   release(id): the tensor's block becomes free and merges with free
 *     neighbours; a tensor that was evicted is already gone (no-op).
 *
 * Per operation the replay records the block the tensor went to (or the
 * merged free chunk of a release; ~0 for a failure or a no-op), the evicted
 * window [start, end) in pre-eviction indices (~0 when nothing was evicted),
 * its eviction cost, and, for an eviction, the free bytes of the pool just
 * before it (the fragmentation-rate sample of section 4.2: free memory over
 * the memory the allocator holds).
 * ------------------------------------------------------------------------- */
#define OP_ALLOC 0
#define OP_FREE 1
#define FLAG_LEFT 1u   /* an expensive operation: placed at the left end */
#define FLAG_PINNED 2u /* an unevictable tensor */
#define POLICY_WINDOW 0 /* Coop: evict the sliding window (section 3.3) */
#define POLICY_GREEDY 1 /* DTR-style: evict the least h = c / (m * s), one by one */

/* 160-bit products c * m * s for the greedy comparison (c, m < 2^64,
 * s < 2^32), as (hi, lo) with hi holding bits 128 and up. */
struct u160 { uint64_t hi; unsigned __int128 lo; };

static struct u160 mul3(uint64_t c, uint64_t m, uint32_t st) {
    unsigned __int128 cm = (unsigned __int128)c * m;
    unsigned __int128 lo64 = (unsigned __int128)(uint64_t)cm * st;
    unsigned __int128 hi64 = (unsigned __int128)(uint64_t)(cm >> 64) * st;
    /* cm * st = hi64 * 2^64 + lo64 */
    unsigned __int128 mid = (lo64 >> 64) + (uint64_t)hi64;
    struct u160 r;
    r.lo = (mid << 64) | (uint64_t)lo64;
    r.hi = (uint64_t)(hi64 >> 64) + (uint64_t)(mid >> 64);
    return r;
}

static int u160_less(struct u160 a, struct u160 b) {
    return a.hi != b.hi ? a.hi < b.hi : a.lo < b.lo;
}

/* DTR's heuristic h = c / (m * s) (section 3.3 restates it): cost over
 * size times staleness.  Staleness counts allocations since the tensor's
 * own, read off the trace's tensor ids, which are issued in allocation
 * order (op_id - id, modulo 2^32).  A zero size or staleness counts as 1, so
 * that h is always a finite ratio.  h_a < h_b iff
 * c_a * m_b * s_b < c_b * m_a * s_a, compared exactly; ties go to the lower
 * block index. */
static int greedy_less(uint64_t ca, uint64_t ma, uint32_t sa, uint64_t cb, uint64_t mb,
                       uint32_t sb) {
    ma = ma ? ma : 1; mb = mb ? mb : 1;
    sa = sa ? sa : 1; sb = sb ? sb : 1;
    return u160_less(mul3(ca, mb, sb), mul3(cb, ma, sa));
}

struct replay_pool {
    uint64_t *size, *cost;
    uint8_t *kind;
    uint32_t *id;
    uint64_t len, cap;
};

/* Replaces blocks [lo, hi) by the m blocks given (m <= 2). */
static void pool_replace(struct replay_pool *p, uint64_t lo, uint64_t hi, uint64_t m,
                         const uint64_t *ns, const uint64_t *nc, const uint8_t *nk,
                         const uint32_t *ni) {
    uint64_t tail = p->len - hi;
    memmove(p->size + lo + m, p->size + hi, tail * sizeof(uint64_t));
    memmove(p->cost + lo + m, p->cost + hi, tail * sizeof(uint64_t));
    memmove(p->kind + lo + m, p->kind + hi, tail * sizeof(uint8_t));
    memmove(p->id + lo + m, p->id + hi, tail * sizeof(uint32_t));
    for (uint64_t j = 0; j < m; ++j) {
        p->size[lo + j] = ns[j]; p->cost[lo + j] = nc[j];
        p->kind[lo + j] = nk[j]; p->id[lo + j] = ni[j];
    }
    p->len = p->len - (hi - lo) + m;
}

/* Turns blocks [lo, hi) into one free chunk merged with free neighbours;
 * returns its index. */
static uint64_t pool_free_range(struct replay_pool *p, uint64_t lo, uint64_t hi) {
    while (lo > 0 && p->kind[lo - 1] == KIND_FREE) --lo;
    while (hi < p->len && p->kind[hi] == KIND_FREE) ++hi;
    uint64_t total = 0;
    for (uint64_t k = lo; k < hi; ++k) total += p->size[k];
    uint64_t s = total, c = 0;
    uint8_t kd = KIND_FREE;
    uint32_t i = 0;
    pool_replace(p, lo, hi, 1, &s, &c, &kd, &i);
    return lo;
}

static int replay_one(struct replay_pool *p, const uint8_t *op, const uint32_t *op_id,
                      const uint64_t *op_size, const uint64_t *op_cost, const uint8_t *op_flags,
                      uint64_t num_ops, uint64_t *out_block, uint64_t *out_window,
                      uint64_t *out_cost, uint64_t *out_free, int policy) {
    for (uint64_t t = 0; t < num_ops; ++t) {
        out_block[t] = NONE;
        out_window[2 * t] = out_window[2 * t + 1] = NONE;
        out_cost[t] = 0;
        out_free[t] = NONE;
        if (op[t] == OP_FREE) {
            for (uint64_t k = 0; k < p->len; ++k) {
                if (p->kind[k] != KIND_FREE && p->id[k] == op_id[t]) {
                    out_block[t] = pool_free_range(p, k, k + 1);
                    break;
                }
            }
            continue;
        }
        if (op[t] != OP_ALLOC || op_size[t] == 0 || op_id[t] == 0)
            return COOP_ORACLE_ERR_INVALID;
        const uint64_t S = op_size[t];
        uint64_t k = first_fit_one(p->size, p->kind, p->len, S);
        if (k == NONE && policy == POLICY_GREEDY) {
            /* evict the least-h tensor until a chunk fits or none is left */
            uint64_t free_bytes = 0, count = 0, evcost = 0;
            for (uint64_t j = 0; j < p->len; ++j)
                if (p->kind[j] == KIND_FREE) free_bytes += p->size[j];
            while (k == NONE) {
                uint64_t v = NONE;
                for (uint64_t j = 0; j < p->len; ++j) {
                    if (p->kind[j] != KIND_EVICTABLE) continue;
                    const uint32_t st = op_id[t] - p->id[j];
                    if (v == NONE || greedy_less(p->cost[j], p->size[j], st, p->cost[v],
                                                 p->size[v], op_id[t] - p->id[v]))
                        v = j;
                }
                if (v == NONE) break;
                ++count;
                evcost += p->cost[v];
                pool_free_range(p, v, v + 1);
                k = first_fit_one(p->size, p->kind, p->len, S);
            }
            if (count) {
                out_free[t] = free_bytes;
                out_window[2 * t] = count;
                out_cost[t] = evcost;
            }
            if (k == NONE) continue; /* the allocation fails (evictions stay done) */
        }
        if (k == NONE) {
            uint64_t win[3];
            if (!runs_fit(p->size, p->cost, p->kind, p->len)) return COOP_ORACLE_ERR_OVERFLOW;
            sweep_one(p->size, p->cost, p->kind, p->len, S, win);
            if (win[0] == NONE) continue; /* the allocation fails */
            uint64_t free_bytes = 0;
            for (uint64_t j = 0; j < p->len; ++j)
                if (p->kind[j] == KIND_FREE) free_bytes += p->size[j];
            out_free[t] = free_bytes;
            out_window[2 * t] = win[0];
            out_window[2 * t + 1] = win[1];
            out_cost[t] = win[2];
            pool_free_range(p, win[0], win[1]);
            k = first_fit_one(p->size, p->kind, p->len, S);
            if (k == NONE) return COOP_ORACLE_ERR_INVALID; /* cannot happen */
        }
        if (p->len + 1 > p->cap) return COOP_ORACLE_ERR_TOO_LARGE;
        const uint64_t F = p->size[k];
        const uint8_t tk = (op_flags[t] & FLAG_PINNED) ? 2 : KIND_EVICTABLE;
        uint64_t ns[2], nc[2];
        uint8_t nk[2];
        uint32_t ni[2];
        uint64_t m = 1, at = k;
        if (F == S) {
            ns[0] = S; nc[0] = op_cost[t]; nk[0] = tk; ni[0] = op_id[t];
        } else if (op_flags[t] & FLAG_LEFT) {
            ns[0] = S; nc[0] = op_cost[t]; nk[0] = tk; ni[0] = op_id[t];
            ns[1] = F - S; nc[1] = 0; nk[1] = KIND_FREE; ni[1] = 0;
            m = 2;
        } else {
            ns[0] = F - S; nc[0] = 0; nk[0] = KIND_FREE; ni[0] = 0;
            ns[1] = S; nc[1] = op_cost[t]; nk[1] = tk; ni[1] = op_id[t];
            m = 2;
            at = k + 1;
        }
        pool_replace(p, k, k + 1, m, ns, nc, nk, ni);
        out_block[t] = at;
    }
    return COOP_ORACLE_OK;
}

struct replay_job {
    uint64_t *size, *cost;
    uint8_t *kind;
    uint32_t *id;
    uint64_t *len;
    uint64_t cap, num_pools, num_ops;
    const uint8_t *op;
    const uint32_t *op_id;
    const uint64_t *op_size, *op_cost;
    const uint8_t *op_flags;
    uint64_t *out_block, *out_window, *out_cost, *out_free;
    int policy;
    _Atomic uint64_t next;
    _Atomic int status;
};

static void *replay_worker(void *arg) {
    struct replay_job *j = (struct replay_job *)arg;
    for (;;) {
        uint64_t b = atomic_fetch_add(&j->next, 1);
        if (b >= j->num_pools) break;
        struct replay_pool p = {j->size + b * j->cap, j->cost + b * j->cap, j->kind + b * j->cap,
                                j->id + b * j->cap, j->len[b], j->cap};
        const uint64_t o = b * j->num_ops;
        int rc = replay_one(&p, j->op + o, j->op_id + o, j->op_size + o, j->op_cost + o,
                            j->op_flags + o, j->num_ops, j->out_block + o, j->out_window + 2 * o,
                            j->out_cost + o, j->out_free + o, j->policy);
        j->len[b] = p.len;
        if (rc != COOP_ORACLE_OK) atomic_store(&j->status, rc);
    }
    return NULL;
}

int coop_oracle_replay(uint64_t *size, uint64_t *cost, uint8_t *kind, uint32_t *id, uint64_t *len,
                       uint64_t num_pools, uint64_t capacity, const uint8_t *op,
                       const uint32_t *op_id, const uint64_t *op_size, const uint64_t *op_cost,
                       const uint8_t *op_flags, uint64_t num_ops, uint64_t *out_block,
                       uint64_t *out_window, uint64_t *out_cost, uint64_t *out_free,
                       int policy, int num_threads) {
    if (num_pools == 0) return COOP_ORACLE_OK;
    if (policy != POLICY_WINDOW && policy != POLICY_GREEDY) return COOP_ORACLE_ERR_INVALID;
    if (!size || !cost || !kind || !id || !len || capacity == 0) return COOP_ORACLE_ERR_INVALID;
    if (num_ops && (!op || !op_id || !op_size || !op_cost || !op_flags || !out_block ||
                    !out_window || !out_cost || !out_free))
        return COOP_ORACLE_ERR_INVALID;
    for (uint64_t b = 0; b < num_pools; ++b)
        if (len[b] > capacity) return COOP_ORACLE_ERR_INVALID;
    struct replay_job job;
    job.size = size; job.cost = cost; job.kind = kind; job.id = id; job.len = len;
    job.cap = capacity; job.num_pools = num_pools; job.num_ops = num_ops;
    job.op = op; job.op_id = op_id; job.op_size = op_size; job.op_cost = op_cost;
    job.op_flags = op_flags; job.out_block = out_block; job.out_window = out_window;
    job.out_cost = out_cost; job.out_free = out_free; job.policy = policy;
    atomic_init(&job.next, 0);
    atomic_init(&job.status, COOP_ORACLE_OK);
    if (num_threads <= 1) {
        replay_worker(&job);
        return atomic_load(&job.status);
    }
    pthread_t *tid = (pthread_t *)calloc((size_t)num_threads, sizeof(pthread_t));
    if (!tid) return COOP_ORACLE_ERR_INVALID;
    int started = 0;
    for (int t = 0; t < num_threads; ++t) {
        if (pthread_create(&tid[t], NULL, replay_worker, &job) != 0) break;
        ++started;
    }
    if (started == 0) replay_worker(&job);
    for (int t = 0; t < started; ++t) pthread_join(tid[t], NULL);
    free(tid);
    return atomic_load(&job.status);
}
