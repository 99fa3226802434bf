// Replay of Algorithm 1 (Coop, section 3) on many independent pools at once.
//
// Each pool is an address-sorted block list in a fixed-capacity slot range,
// unused slots holding empty unevictable blocks, so the batch is a plain
// batch of snapshots for the search kernels.  Every operation of a pool's
// trace is applied in order, all pools in lockstep, one step per operation:
//
//   1. first fit for every pool's allocation (coop_first_fit);
//   2. a gate: pools whose allocation found no chunk ask for a window, the
//      others ask for nothing (S = 0 answers at once);
//   3. the sliding-window search for those requests (coop_window_search);
//   4. the update, one workgroup per pool: a release frees the tensor's
//      block and merges it with free neighbours; an allocation that found
//      no chunk evicts the window's tensors, merges the window (and free
//      neighbours) into one free chunk and fits again, which can only pick
//      that chunk; the tensor goes to the chunk's left end for an expensive
//      operation and its right end otherwise (section 3.4).  The rest of the
//      pool moves by one or more slots, and the request of the next
//      operation is written for step 1.
//
// Per operation the update records the tensor's block (or the merged chunk
// of a release; ~0 for a failure or for releasing an evicted tensor), the
// evicted window and its cost, and for an eviction the pool's free bytes
// just before it (the fragmentation-rate sample: free memory over the
// memory the allocator holds).
//
// The greedy policy replaces steps 2-3 and the window eviction by the
// baseline Coop is measured against (DTR's heuristic, restated in section
// 3.3): while no chunk fits, evict the evictable tensor of least
// h = c / (m * s) (cost over size times staleness) and merge its block with
// free neighbours.  The update then records the number of tensors evicted
// and their summed cost instead of a window.

#include <hip/hip_runtime.h>

#include <stdint.h>

#include "coop.h"
#include "coop_host.h"

namespace {

constexpr uint32_t kThreads = 256;
constexpr uint64_t kNone = ~0ull;
constexpr uint8_t kOpAlloc = 0, kOpFree = 1;
constexpr uint8_t kFlagLeft = 1, kFlagPinned = 2;
constexpr uint32_t kErrCapacity = 1, kErrOperation = 2;

// ---------------------------------------------------------------------------
// Greedy victim choice.  h_a < h_b iff c_a * m_b * s_b < c_b * m_a * s_a;
// both sides are products of two u64 and a u32 (below 2^160), compared
// exactly in three words.  A zero size or staleness counts as 1.  Ties go to
// the lower block index, which makes the choice unique, so any reduction
// order gives the same victim.
// ---------------------------------------------------------------------------
struct Prod {
    uint64_t lo, mid, hi;
};

__device__ __forceinline__ Prod mul3(uint64_t c, uint64_t m, uint32_t st) {
    const uint64_t cm_lo = c * m, cm_hi = __umul64hi(c, m);
    // (cm_hi * 2^64 + cm_lo) * st
    const uint64_t a_lo = cm_lo * st, a_hi = __umul64hi(cm_lo, st);
    const uint64_t b_lo = cm_hi * st, b_hi = __umul64hi(cm_hi, st);
    const uint64_t mid = a_hi + b_lo;
    return Prod{a_lo, mid, b_hi + (mid < a_hi ? 1u : 0u)};
}

__device__ __forceinline__ bool prod_less(const Prod& a, const Prod& b) {
    if (a.hi != b.hi) return a.hi < b.hi;
    if (a.mid != b.mid) return a.mid < b.mid;
    return a.lo < b.lo;
}

struct Victim {
    uint64_t c, m;  // cost, size (at least 1)
    uint32_t s, j;  // staleness (at least 1), block index; j == ~0u: none
};

__device__ __forceinline__ bool victim_less(const Victim& a, const Victim& b) {
    if (b.j == ~0u) return a.j != ~0u;
    if (a.j == ~0u) return false;
    const Prod pa = mul3(a.c, b.m, b.s), pb = mul3(b.c, a.m, a.s);
    if (prod_less(pa, pb)) return true;
    if (prod_less(pb, pa)) return false;
    return a.j < b.j;
}

__device__ __forceinline__ Victim shfl_xor_victim(const Victim& v, int o) {
    Victim x;
    x.c = (static_cast<uint64_t>(__shfl_xor(static_cast<uint32_t>(v.c >> 32), o, 64)) << 32) |
          __shfl_xor(static_cast<uint32_t>(v.c), o, 64);
    x.m = (static_cast<uint64_t>(__shfl_xor(static_cast<uint32_t>(v.m >> 32), o, 64)) << 32) |
          __shfl_xor(static_cast<uint32_t>(v.m), o, 64);
    x.s = __shfl_xor(v.s, o, 64);
    x.j = __shfl_xor(v.j, o, 64);
    return x;
}

// The evictable block of least h among blocks [0, n) for operation id oid
// (staleness oid - id, modulo 2^32), or ~0u.  The arrays may live in LDS or
// global memory; every thread of the 256-thread workgroup calls it and gets
// the same answer.  vred holds 4 entries.
__device__ __forceinline__ uint32_t greedy_victim(const uint64_t* sz, const uint64_t* co,
                                                  const uint8_t* kd, const uint32_t* id,
                                                  uint64_t n, uint32_t oid, Victim* vred) {
    const uint32_t tid = threadIdx.x;
    Victim best{0, 1, 1, ~0u};
    for (uint64_t k = tid; k < n; k += 256) {
        if (kd[k] != COOP_EVICTABLE) continue;
        const uint64_t m = sz[k];
        const uint32_t st = oid - id[k];
        const Victim v{co[k], m ? m : 1, st ? st : 1u, static_cast<uint32_t>(k)};
        if (victim_less(v, best)) best = v;
    }
    for (int o = 32; o >= 1; o >>= 1) {
        const Victim x = shfl_xor_victim(best, o);
        if (victim_less(x, best)) best = x;
    }
    if ((tid & 63u) == 0) vred[tid >> 6] = best;
    __syncthreads();
    Victim m = vred[0];
    for (uint32_t w = 1; w < 4; ++w)
        if (victim_less(vred[w], m)) m = vred[w];
    __syncthreads();
    return m.j;
}

// Sets the fixed batch layout (pool b is slots [b * cap, (b + 1) * cap) and
// owns request b) and the requests of the first operation.
__global__ void replay_init_kernel(uint64_t num_pools, uint64_t cap, uint64_t* seg,
                                   uint64_t* req_off, uint64_t* req_ff, const uint8_t* op,
                                   const uint64_t* op_size, uint64_t num_ops, uint32_t* status) {
    const uint64_t i = static_cast<uint64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (i <= num_pools) {
        seg[i] = i * cap;
        req_off[i] = i;
    }
    if (i < num_pools) req_ff[i] = num_ops && op[i * num_ops] == kOpAlloc ? op_size[i * num_ops] : 0;
    if (i == 0) *status = 0;
}

// Clears the status word (a kernel rather than a memset, so that the call
// can be captured in a graph).
__global__ void replay_status_kernel(uint32_t* status) { *status = 0; }

// Step 2: a window is wanted only where an allocation found no chunk.
__global__ void replay_gate_kernel(uint64_t num_pools, const uint64_t* req_ff, const uint64_t* ff,
                                   uint64_t* req_win) {
    const uint64_t b = static_cast<uint64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (b < num_pools) req_win[b] = ff[b] == kNone ? req_ff[b] : 0;
}

struct Pool {
    uint64_t* size;
    uint64_t* cost;
    uint8_t* kind;
    uint32_t* id;
};

// Sum over the workgroup (every thread calls it).
__device__ uint64_t block_sum(uint64_t v, uint64_t* red) {
    for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
    const uint32_t tid = threadIdx.x;
    if ((tid & 63u) == 0) red[tid >> 6] = v;
    __syncthreads();
    uint64_t s = 0;
    for (uint32_t w = 0; w < kThreads / 64; ++w) s += red[w];
    __syncthreads();
    return s;
}

// Replaces slots [lo, hi) of a pool of `len` blocks by the m <= 2 blocks in
// ns/nc/nk/ni (uniform), moving the tail [hi, len) to start at lo + m; when
// the pool shrinks, the freed slots at its end become empty unevictable
// blocks again.  Every thread calls it.
__device__ void pool_replace(Pool p, uint64_t len, uint64_t lo, uint64_t hi, uint32_t m,
                             const uint64_t* ns, const uint64_t* nc, const uint8_t* nk,
                             const uint32_t* ni) {
    const uint32_t tid = threadIdx.x;
    const uint64_t tail = len - hi, dst = lo + m;
    if (dst > hi) {
        // moving right: chunks from the end, each read before it is written
        for (uint64_t c = tail; c > 0;) {
            const uint64_t c0 = c > kThreads ? c - kThreads : 0;
            const uint64_t k = c0 + tid;
            const bool act = k < c;
            uint64_t s = 0, co = 0;
            uint8_t kd = 0;
            uint32_t i = 0;
            if (act) {
                s = p.size[hi + k]; co = p.cost[hi + k]; kd = p.kind[hi + k]; i = p.id[hi + k];
            }
            __syncthreads();
            if (act) {
                p.size[dst + k] = s; p.cost[dst + k] = co; p.kind[dst + k] = kd; p.id[dst + k] = i;
            }
            __syncthreads();
            c = c0;
        }
    } else if (dst < hi) {
        // moving left: chunks from the start
        for (uint64_t c0 = 0; c0 < tail; c0 += kThreads) {
            const uint64_t k = c0 + tid;
            const bool act = k < tail;
            uint64_t s = 0, co = 0;
            uint8_t kd = 0;
            uint32_t i = 0;
            if (act) {
                s = p.size[hi + k]; co = p.cost[hi + k]; kd = p.kind[hi + k]; i = p.id[hi + k];
            }
            __syncthreads();
            if (act) {
                p.size[dst + k] = s; p.cost[dst + k] = co; p.kind[dst + k] = kd; p.id[dst + k] = i;
            }
            __syncthreads();
        }
        // vacated slots at the end
        const uint64_t nl = dst + tail;
        for (uint64_t k = nl + tid; k < len; k += kThreads) {
            p.size[k] = 0; p.cost[k] = 0; p.kind[k] = COOP_PINNED; p.id[k] = 0;
        }
    }
    if (tid < m) {
        p.size[lo + tid] = ns[tid]; p.cost[lo + tid] = nc[tid];
        p.kind[lo + tid] = nk[tid]; p.id[lo + tid] = ni[tid];
    }
    __syncthreads();
}

// Step 4.  Workgroup b updates pool b with operation t.
__global__ __launch_bounds__(kThreads) void replay_update_kernel(
    uint64_t* size, uint64_t* cost, uint8_t* kind, uint32_t* id, uint64_t* len, uint64_t cap,
    const uint8_t* op, const uint32_t* op_id, const uint64_t* op_size, const uint64_t* op_cost,
    const uint8_t* op_flags, uint64_t num_ops, uint64_t t, int32_t policy, const uint64_t* ff,
    const coop_window_t* win, uint64_t* req_ff, uint64_t* out_block, uint64_t* out_window,
    uint64_t* out_cost, uint64_t* out_free, uint32_t* status) {
    __shared__ uint64_t red[kThreads / 64];
    __shared__ Victim vred[kThreads / 64];
    __shared__ uint64_t found;
    const uint32_t tid = threadIdx.x;
    const uint64_t b = blockIdx.x;
    Pool p{size + b * cap, cost + b * cap, kind + b * cap, id + b * cap};
    const uint64_t n = len[b];
    const uint64_t o = b * num_ops + t;
    const uint8_t kop = op[o];
    uint64_t r_block = kNone, r_w0 = kNone, r_w1 = kNone, r_cost = 0, r_free = kNone;
    uint64_t nl = n;
    if (kop == kOpFree) {
        if (tid == 0) found = kNone;
        __syncthreads();
        const uint32_t want = op_id[o];
        for (uint64_t k = tid; k < n; k += kThreads)
            if (p.kind[k] != COOP_FREE && p.id[k] == want) found = k;  // ids are unique
        __syncthreads();
        const uint64_t j = found;
        if (j != kNone) {
            const uint64_t lo = j > 0 && p.kind[j - 1] == COOP_FREE ? j - 1 : j;
            const uint64_t hi = j + 1 < n && p.kind[j + 1] == COOP_FREE ? j + 2 : j + 1;
            uint64_t total = 0;
            for (uint64_t k = lo; k < hi; ++k) total += p.size[k];
            __syncthreads();
            const uint64_t ns[1] = {total}, nc[1] = {0};
            const uint8_t nk[1] = {COOP_FREE};
            const uint32_t ni[1] = {0};
            pool_replace(p, n, lo, hi, 1, ns, nc, nk, ni);
            nl = n - (hi - lo) + 1;
            r_block = lo;
        }
    } else if (kop == kOpAlloc && op_size[o] != 0 && op_id[o] != 0) {
        const uint64_t S = op_size[o];
        uint64_t k = ff[b];
        bool ok = true;
        if (k == kNone && policy == COOP_POLICY_GREEDY) {
            uint64_t fb = 0;
            for (uint64_t j = tid; j < n; j += kThreads)
                if (p.kind[j] == COOP_FREE) fb += p.size[j];
            const uint64_t free0 = block_sum(fb, red);
            uint64_t count = 0, evc = 0;
            while (k == kNone) {
                const uint32_t v = greedy_victim(p.size, p.cost, p.kind, p.id, nl, op_id[o], vred);
                if (v == ~0u) break;
                ++count;
                evc += p.cost[v];
                const uint64_t lo = v > 0 && p.kind[v - 1] == COOP_FREE ? v - 1 : v;
                const uint64_t hi = v + 1 < nl && p.kind[v + 1] == COOP_FREE ? v + 2 : v + 1;
                uint64_t total = 0;
                for (uint64_t j = lo; j < hi; ++j) total += p.size[j];
                __syncthreads();
                const uint64_t ns[1] = {total}, nc[1] = {0};
                const uint8_t nk[1] = {COOP_FREE};
                const uint32_t ni[1] = {0};
                pool_replace(p, nl, lo, hi, 1, ns, nc, nk, ni);
                nl = nl - (hi - lo) + 1;
                // no chunk held S bytes before, so only the merged one can now
                if (total >= S) k = lo;
            }
            if (count) {
                r_free = free0;
                r_w0 = count;
                r_cost = evc;
            }
            ok = k != kNone;  // out of evictable tensors: fails, evictions stay
        } else if (k == kNone) {
            const coop_window_t w = win[b];
            if (w.start == kNone) {
                ok = false;  // no window: the allocation fails, nothing changes
            } else {
                uint64_t fb = 0;
                for (uint64_t j = tid; j < n; j += kThreads)
                    if (p.kind[j] == COOP_FREE) fb += p.size[j];
                r_free = block_sum(fb, red);
                r_w0 = w.start;
                r_w1 = w.end;
                r_cost = w.cost;
                uint64_t lo = w.start, hi = w.end;
                if (lo > 0 && p.kind[lo - 1] == COOP_FREE) --lo;
                if (hi < n && p.kind[hi] == COOP_FREE) ++hi;
                uint64_t tot = 0;
                for (uint64_t j = lo + tid; j < hi; j += kThreads) tot += p.size[j];
                const uint64_t total = block_sum(tot, red);
                const uint64_t ns[1] = {total}, nc[1] = {0};
                const uint8_t nk[1] = {COOP_FREE};
                const uint32_t ni[1] = {0};
                pool_replace(p, n, lo, hi, 1, ns, nc, nk, ni);
                nl = n - (hi - lo) + 1;
                k = lo;  // the only free chunk of at least S bytes
            }
        }
        if (ok && nl + 1 > cap) {
            if (tid == 0) atomicOr(status, kErrCapacity);
            ok = false;
        }
        if (ok) {
            const uint64_t F = p.size[k];
            const uint8_t fl = op_flags[o];
            const uint8_t tk = (fl & kFlagPinned) ? COOP_PINNED : COOP_EVICTABLE;
            uint64_t ns[2], nc[2];
            uint8_t nk[2];
            uint32_t ni[2];
            uint32_t m = 1;
            uint64_t at = k;
            if (F == S) {
                ns[0] = S; nc[0] = op_cost[o]; nk[0] = tk; ni[0] = op_id[o];
            } else if (fl & kFlagLeft) {
                ns[0] = S; nc[0] = op_cost[o]; nk[0] = tk; ni[0] = op_id[o];
                ns[1] = F - S; nc[1] = 0; nk[1] = COOP_FREE; ni[1] = 0;
                m = 2;
            } else {
                ns[0] = F - S; nc[0] = 0; nk[0] = COOP_FREE; ni[0] = 0;
                ns[1] = S; nc[1] = op_cost[o]; nk[1] = tk; ni[1] = op_id[o];
                m = 2;
                at = k + 1;
            }
            __syncthreads();
            pool_replace(p, nl, k, k + 1, m, ns, nc, nk, ni);
            nl = nl + m - 1;
            r_block = at;
        }
    } else if (kop == kOpAlloc) {
        if (tid == 0) atomicOr(status, kErrOperation);
    }
    if (tid == 0) {
        len[b] = nl;
        out_block[o] = r_block;
        out_window[2 * o] = r_w0;
        out_window[2 * o + 1] = r_w1;
        out_cost[o] = r_cost;
        out_free[o] = r_free;
        // the next operation's request for first fit
        const uint64_t on = o + 1;
        req_ff[b] = t + 1 < num_ops && op[on] == kOpAlloc ? op_size[on] : 0;
    }
}

// ---------------------------------------------------------------------------
// Resident replay: one workgroup per pool keeps the pool in LDS and applies
// all of its operations itself, with no launch per step.  Used when a pool's
// slots fit in LDS; the same operations as above, in the same order, with
// the searches done by the workgroup:
//   first fit  the lowest free slot of at least S bytes (a workgroup min);
//   window     plain prefix sums P (bytes), C (eviction cost) and R (pinned
//              count) over the pool; for each start i the first end k with
//              P[k] - P[i] >= S, valid iff R[k] == R[i] (no pinned block in
//              between); each thread takes a run of consecutive starts, finds
//              the first end by bisection and the later ones by walking on
//              (ends never move left); then the lexicographic minimum of
//              (cost, bytes, start) over the workgroup.
// ---------------------------------------------------------------------------
constexpr uint32_t kResThreads = 256;
constexpr uint32_t kResWaves = kResThreads / 64;

// LDS bytes for a pool of cap slots, 31 a slot: size (which holds the byte
// prefix sums during a window search), cost and cost prefix (u64), tensor id
// (u32), pinned-count prefix (u16), kind (u8); plus one prefix entry and
// padding to 8 bytes.  A pool of 2072 slots takes 64 KB, so two pools share
// a CU.
__host__ __device__ constexpr size_t resident_lds_bytes(uint64_t cap) {
    return ((cap + 1) * 8) * 2 + cap * 8 + ((cap * 4 + 7) & ~7ull) +
           (((cap + 1) * 2 + 7) & ~7ull) + ((cap + 7) & ~7ull);
}

struct Lds {
    uint64_t* sz;  // sizes; byte prefix sums while res_window runs
    uint64_t* co;
    uint64_t* C;
    uint32_t* id;
    uint16_t* R;
    uint8_t* kd;
};

__device__ Lds lds_layout(char* base, uint64_t cap) {
    Lds l;
    size_t at = 0;
    l.sz = reinterpret_cast<uint64_t*>(base + at); at += (cap + 1) * 8;
    l.co = reinterpret_cast<uint64_t*>(base + at); at += cap * 8;
    l.C = reinterpret_cast<uint64_t*>(base + at); at += (cap + 1) * 8;
    l.id = reinterpret_cast<uint32_t*>(base + at); at += (cap * 4 + 7) & ~7ull;
    l.R = reinterpret_cast<uint16_t*>(base + at); at += ((cap + 1) * 2 + 7) & ~7ull;
    l.kd = reinterpret_cast<uint8_t*>(base + at);
    return l;
}

struct WinKey {
    uint64_t cost, bytes, start, end;
};

__device__ __forceinline__ bool win_less(const WinKey& a, const WinKey& b) {
    if (a.cost != b.cost) return a.cost < b.cost;
    if (a.bytes != b.bytes) return a.bytes < b.bytes;
    return a.start < b.start;
}

__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t v, int m) {
    const uint32_t lo = __shfl_xor(static_cast<uint32_t>(v), m, 64);
    const uint32_t hi = __shfl_xor(static_cast<uint32_t>(v >> 32), m, 64);
    return (static_cast<uint64_t>(hi) << 32) | lo;
}

__device__ __forceinline__ uint64_t shfl_up_u64(uint64_t v, int d) {
    const uint32_t lo = __shfl_up(static_cast<uint32_t>(v), d, 64);
    const uint32_t hi = __shfl_up(static_cast<uint32_t>(v >> 32), d, 64);
    return (static_cast<uint64_t>(hi) << 32) | lo;
}

// Workgroup sum and minimum (every thread calls them; `red` holds kResWaves).
__device__ uint64_t res_sum(uint64_t v, uint64_t* red) {
    for (int o = 32; o >= 1; o >>= 1) v += shfl_xor_u64(v, o);
    if ((threadIdx.x & 63u) == 0) red[threadIdx.x >> 6] = v;
    __syncthreads();
    uint64_t s = 0;
    for (uint32_t w = 0; w < kResWaves; ++w) s += red[w];
    __syncthreads();
    return s;
}

__device__ uint64_t res_min(uint64_t v, uint64_t* red) {
    for (int o = 32; o >= 1; o >>= 1) {
        const uint64_t x = shfl_xor_u64(v, o);
        v = x < v ? x : v;
    }
    if ((threadIdx.x & 63u) == 0) red[threadIdx.x >> 6] = v;
    __syncthreads();
    uint64_t m = red[0];
    for (uint32_t w = 1; w < kResWaves; ++w) m = red[w] < m ? red[w] : m;
    __syncthreads();
    return m;
}

// Replaces slots [lo, hi) of a pool of n blocks by m <= 2 new blocks (uniform
// values), moving the tail in LDS.  Every thread calls it.
__device__ void res_replace(const Lds& l, uint64_t n, uint64_t lo, uint64_t hi, uint32_t m,
                            const uint64_t* ns, const uint64_t* nc, const uint8_t* nk,
                            const uint32_t* ni) {
    const uint32_t tid = threadIdx.x;
    const uint64_t tail = n - hi, dst = lo + m;
    if (dst != hi) {
        const bool right = dst > hi;
        for (uint64_t c0 = 0; c0 < tail; c0 += kResThreads) {
            // moving right, the chunks go from the end
            const uint64_t base = right ? (tail - c0 > kResThreads ? tail - c0 - kResThreads : 0) : c0;
            const uint64_t cend = right ? tail - c0 : (c0 + kResThreads < tail ? c0 + kResThreads : tail);
            const uint64_t k = base + tid;
            const bool act = k < cend;
            uint64_t s = 0, c = 0;
            uint32_t i = 0;
            uint8_t kd = 0;
            if (act) {
                s = l.sz[hi + k]; c = l.co[hi + k]; i = l.id[hi + k]; kd = l.kd[hi + k];
            }
            __syncthreads();
            if (act) {
                l.sz[dst + k] = s; l.co[dst + k] = c; l.id[dst + k] = i; l.kd[dst + k] = kd;
            }
            __syncthreads();
        }
    }
    if (tid < m) {
        l.sz[lo + tid] = ns[tid]; l.co[lo + tid] = nc[tid];
        l.id[lo + tid] = ni[tid]; l.kd[lo + tid] = nk[tid];
    }
    __syncthreads();
}

// The window search for S > 0 over a pool of n blocks held in LDS.  The
// byte prefix sums P overwrite the sizes for the search (P[k] in sz[k],
// P[n] in sz[n]); the sizes are put back before it returns.
__device__ WinKey res_window(const Lds& l, uint64_t n, uint64_t S, uint64_t* red, WinKey* wred) {
    const uint32_t tid = threadIdx.x, lane = tid & 63u, w = tid >> 6;
    // each thread owns blocks [a, a1): local sums, then a workgroup scan
    const uint64_t per = (n + kResThreads - 1) / kResThreads;
    const uint64_t a = tid * per < n ? tid * per : n;
    const uint64_t a1 = a + per < n ? a + per : n;
    uint64_t ps = 0, pc = 0, pr = 0;
    for (uint64_t k = a; k < a1; ++k) {
        ps += l.sz[k];
        pc += l.kd[k] == COOP_EVICTABLE ? l.co[k] : 0;
        pr += l.kd[k] >= COOP_PINNED ? 1 : 0;
    }
    // inclusive scans over the wavefront
    uint64_t is = ps, ic = pc, ir = pr;
    for (int d = 1; d < 64; d <<= 1) {
        const uint64_t xs = shfl_up_u64(is, d), xc = shfl_up_u64(ic, d), xr = shfl_up_u64(ir, d);
        if (lane >= static_cast<uint32_t>(d)) {
            is += xs; ic += xc; ir += xr;
        }
    }
    if (lane == 63) {
        red[w] = is;
        wred[w] = WinKey{ic, ir, 0, 0};
    }
    __syncthreads();
    uint64_t bs = 0, bc = 0, br = 0;
    for (uint32_t v = 0; v < w; ++v) {
        bs += red[v]; bc += wred[v].cost; br += wred[v].bytes;
    }
    __syncthreads();
    uint64_t xs = bs + is - ps, xc = bc + ic - pc, xr = br + ir - pr;
    for (uint64_t k = a; k < a1; ++k) {  // each thread rewrites only its own blocks
        const uint64_t szk = l.sz[k];
        l.sz[k] = xs; l.C[k] = xc; l.R[k] = static_cast<uint16_t>(xr);
        xs += szk;
        xc += l.kd[k] == COOP_EVICTABLE ? l.co[k] : 0;
        xr += l.kd[k] >= COOP_PINNED ? 1 : 0;
    }
    if (a1 == n && a < a1) {
        l.sz[n] = xs; l.C[n] = xc; l.R[n] = static_cast<uint16_t>(xr);
    }
    if (n == 0 && tid == 0) {
        l.sz[0] = 0; l.C[0] = 0; l.R[0] = 0;
    }
    __syncthreads();
    const uint64_t* const P = l.sz;
    // starts [a, a1): the first end by bisection, later ends by walking on
    WinKey best{kNone, kNone, kNone, kNone};
    uint64_t k = 0;
    for (uint64_t i = a; i < a1; ++i) {
        const uint64_t pi = P[i];
        if (i == a) {
            uint64_t lo = i + 1, hi = n + 1;  // first k in [i + 1, n] with P[k] - P[i] >= S, or n + 1
            while (lo < hi) {
                const uint64_t mid = (lo + hi) >> 1;
                if (P[mid] - pi >= S) hi = mid; else lo = mid + 1;
            }
            k = lo;
        } else {
            if (k < i + 1) k = i + 1;
            while (k <= n && P[k] - pi < S) ++k;
        }
        if (k > n) break;  // no later start of this thread reaches S either
        if (l.R[k] == l.R[i]) {
            const WinKey c{l.C[k] - l.C[i], P[k] - pi, i, k};
            if (win_less(c, best)) best = c;
        }
    }
    // workgroup lexicographic minimum
    for (int o = 32; o >= 1; o >>= 1) {
        WinKey x{shfl_xor_u64(best.cost, o), shfl_xor_u64(best.bytes, o), shfl_xor_u64(best.start, o),
                 shfl_xor_u64(best.end, o)};
        if (win_less(x, best)) best = x;
    }
    if (lane == 0) wred[w] = best;
    __syncthreads();  // also: every read of P is done
    WinKey m = wred[0];
    for (uint32_t v = 1; v < kResWaves; ++v)
        if (win_less(wred[v], m)) m = wred[v];
    // sizes back from the prefixes: sz[k] = P[k + 1] - P[k], each thread over
    // its own blocks, last to first, after reading the prefix just past them
    uint64_t nxt = a < a1 ? P[a1] : 0;
    __syncthreads();
    for (uint64_t k = a1; k > a;) {
        --k;
        const uint64_t pk = l.sz[k];
        l.sz[k] = nxt - pk;
        nxt = pk;
    }
    __syncthreads();
    return m;
}

__global__ __launch_bounds__(kResThreads) void replay_resident_kernel(
    uint64_t* size, uint64_t* cost, uint8_t* kind, uint32_t* id, uint64_t* len, uint64_t cap,
    const uint8_t* op, const uint32_t* op_id, const uint64_t* op_size, const uint64_t* op_cost,
    const uint8_t* op_flags, uint64_t num_ops, int32_t policy, uint64_t* out_block,
    uint64_t* out_window, uint64_t* out_cost, uint64_t* out_free, uint32_t* status) {
    extern __shared__ __align__(16) char lds_raw[];
    __shared__ uint64_t red[kResWaves];
    __shared__ WinKey wred[kResWaves];
    __shared__ Victim vred[kResWaves];
    __shared__ uint32_t hit;
    const uint32_t tid = threadIdx.x;
    const uint64_t b = blockIdx.x;
    const Lds l = lds_layout(lds_raw, cap);
    const uint64_t g = b * cap;
    uint64_t n = len[b];
    if (n > cap) n = cap;
    for (uint64_t k = tid; k < n; k += kResThreads) {
        l.sz[k] = size[g + k]; l.co[k] = cost[g + k]; l.id[k] = id[g + k]; l.kd[k] = kind[g + k];
    }
    __syncthreads();
    for (uint64_t t = 0; t < num_ops; ++t) {
        const uint64_t o = b * num_ops + t;
        const uint8_t kop = op[o];
        const uint32_t oid = op_id[o];
        uint64_t r_block = kNone, r_w0 = kNone, r_w1 = kNone, r_cost = 0, r_free = kNone;
        if (kop == kOpFree) {
            if (tid == 0) hit = ~0u;
            __syncthreads();
            for (uint64_t k = tid; k < n; k += kResThreads)
                if (l.kd[k] != COOP_FREE && l.id[k] == oid) hit = static_cast<uint32_t>(k);
            __syncthreads();
            const uint32_t j = hit;
            if (j != ~0u) {
                const uint64_t lo = j > 0 && l.kd[j - 1] == COOP_FREE ? j - 1 : j;
                const uint64_t hi = j + 1 < n && l.kd[j + 1] == COOP_FREE ? j + 2 : j + 1;
                uint64_t total = 0;
                for (uint64_t k = lo; k < hi; ++k) total += l.sz[k];
                __syncthreads();
                const uint64_t ns[1] = {total}, nc[1] = {0};
                const uint8_t nk[1] = {COOP_FREE};
                const uint32_t ni[1] = {0};
                res_replace(l, n, lo, hi, 1, ns, nc, nk, ni);
                n = n - (hi - lo) + 1;
                r_block = lo;
            }
        } else if (kop == kOpAlloc && op_size[o] != 0 && oid != 0) {
            const uint64_t S = op_size[o];
            uint64_t mine = kNone;
            for (uint64_t k = tid; k < n; k += kResThreads) {
                if (l.kd[k] == COOP_FREE && l.sz[k] >= S) {
                    mine = k;
                    break;
                }
            }
            uint64_t k = res_min(mine, red);
            bool ok = true;
            if (k == kNone && policy == COOP_POLICY_GREEDY) {
                uint64_t fb = 0;
                for (uint64_t j = tid; j < n; j += kResThreads)
                    if (l.kd[j] == COOP_FREE) fb += l.sz[j];
                const uint64_t free0 = res_sum(fb, red);
                uint64_t count = 0, evc = 0;
                while (k == kNone) {
                    const uint32_t v = greedy_victim(l.sz, l.co, l.kd, l.id, n, oid, vred);
                    if (v == ~0u) break;
                    ++count;
                    evc += l.co[v];
                    const uint64_t lo = v > 0 && l.kd[v - 1] == COOP_FREE ? v - 1 : v;
                    const uint64_t hi = v + 1 < n && l.kd[v + 1] == COOP_FREE ? v + 2 : v + 1;
                    uint64_t total = 0;
                    for (uint64_t j = lo; j < hi; ++j) total += l.sz[j];
                    __syncthreads();
                    const uint64_t ns[1] = {total}, nc[1] = {0};
                    const uint8_t nk[1] = {COOP_FREE};
                    const uint32_t ni[1] = {0};
                    res_replace(l, n, lo, hi, 1, ns, nc, nk, ni);
                    n = n - (hi - lo) + 1;
                    // no chunk held S bytes before, so only the merged one can now
                    if (total >= S) k = lo;
                }
                if (count) {
                    r_free = free0;
                    r_w0 = count;
                    r_cost = evc;
                }
                ok = k != kNone;  // out of evictable tensors: fails, evictions stay
            } else if (k == kNone) {
                const WinKey wk = res_window(l, n, S, red, wred);
                if (wk.start == kNone) {
                    ok = false;  // no window: the allocation fails, nothing changes
                } else {
                    uint64_t fb = 0;
                    for (uint64_t j = tid; j < n; j += kResThreads)
                        if (l.kd[j] == COOP_FREE) fb += l.sz[j];
                    r_free = res_sum(fb, red);
                    r_w0 = wk.start;
                    r_w1 = wk.end;
                    r_cost = wk.cost;
                    uint64_t lo = wk.start, hi = wk.end;
                    if (lo > 0 && l.kd[lo - 1] == COOP_FREE) --lo;
                    if (hi < n && l.kd[hi] == COOP_FREE) ++hi;
                    uint64_t tot = 0;
                    for (uint64_t j = lo + tid; j < hi; j += kResThreads) tot += l.sz[j];
                    const uint64_t total = res_sum(tot, red);
                    const uint64_t ns[1] = {total}, nc[1] = {0};
                    const uint8_t nk[1] = {COOP_FREE};
                    const uint32_t ni[1] = {0};
                    res_replace(l, n, lo, hi, 1, ns, nc, nk, ni);
                    n = n - (hi - lo) + 1;
                    k = lo;  // the only free chunk of at least S bytes
                }
            }
            if (ok && n + 1 > cap) {
                if (tid == 0) atomicOr(status, kErrCapacity);
                ok = false;
            }
            if (ok) {
                const uint64_t F = l.sz[k];
                const uint8_t fl = op_flags[o];
                const uint8_t tk = (fl & kFlagPinned) ? COOP_PINNED : COOP_EVICTABLE;
                uint64_t ns[2], nc[2];
                uint8_t nk[2];
                uint32_t ni[2];
                uint32_t m = 1;
                uint64_t at = k;
                if (F == S) {
                    ns[0] = S; nc[0] = op_cost[o]; nk[0] = tk; ni[0] = oid;
                } else if (fl & kFlagLeft) {
                    ns[0] = S; nc[0] = op_cost[o]; nk[0] = tk; ni[0] = oid;
                    ns[1] = F - S; nc[1] = 0; nk[1] = COOP_FREE; ni[1] = 0;
                    m = 2;
                } else {
                    ns[0] = F - S; nc[0] = 0; nk[0] = COOP_FREE; ni[0] = 0;
                    ns[1] = S; nc[1] = op_cost[o]; nk[1] = tk; ni[1] = oid;
                    m = 2;
                    at = k + 1;
                }
                __syncthreads();
                res_replace(l, n, k, k + 1, m, ns, nc, nk, ni);
                n = n + m - 1;
                r_block = at;
            }
        } else if (kop == kOpAlloc) {
            if (tid == 0) atomicOr(status, kErrOperation);
        }
        if (tid == 0) {
            out_block[o] = r_block;
            out_window[2 * o] = r_w0;
            out_window[2 * o + 1] = r_w1;
            out_cost[o] = r_cost;
            out_free[o] = r_free;
        }
    }
    // the pool back to its slots; unused slots empty pinned blocks
    for (uint64_t k = tid; k < cap; k += kResThreads) {
        const bool in = k < n;
        size[g + k] = in ? l.sz[k] : 0;
        cost[g + k] = in ? l.co[k] : 0;
        id[g + k] = in ? l.id[k] : 0;
        kind[g + k] = in ? l.kd[k] : static_cast<uint8_t>(COOP_PINNED);
    }
    if (tid == 0) len[b] = n;
}

constexpr size_t kLdsLimit = 160 * 1024;
constexpr size_t kStaticResLds = 1024;  // red, wred, hit (generous)

struct ReplayLayout {
    size_t seg, req_off, req_ff, req_win, ff, win, status, ff_ws, win_ws, bytes;
    size_t ff_ws_bytes, win_ws_bytes;
};

size_t align256(size_t x) { return (x + 255) & ~static_cast<size_t>(255); }

bool replay_layout(uint64_t num_pools, uint64_t cap, ReplayLayout* l) {
    if (num_pools == 0 || cap == 0 || num_pools > (1ull << 32) || cap > (1ull << 32)) return false;
    const uint64_t nb = num_pools * cap;
    size_t ffb = 0, wsb = 0;
    if (coop_first_fit_workspace_size(nb, &ffb) != COOP_OK) return false;
    if (coop_window_search_workspace_size(nb, num_pools, num_pools, &wsb) != COOP_OK) return false;
    size_t at = 0;
    l->seg = at; at = align256(at + (num_pools + 1) * 8);
    l->req_off = at; at = align256(at + (num_pools + 1) * 8);
    l->req_ff = at; at = align256(at + num_pools * 8);
    l->req_win = at; at = align256(at + num_pools * 8);
    l->ff = at; at = align256(at + num_pools * 8);
    l->win = at; at = align256(at + num_pools * sizeof(coop_window_t));
    l->status = at; at = align256(at + 8);
    l->ff_ws = at; at = align256(at + ffb);
    l->win_ws = at; at = align256(at + wsb);
    l->ff_ws_bytes = ffb;
    l->win_ws_bytes = wsb;
    l->bytes = at;
    return true;
}

}  // namespace

extern "C" {

coop_status_t coop_replay_workspace_size(uint64_t num_pools, uint64_t capacity, size_t* bytes_out) {
    if (!bytes_out) return COOP_ERR_INVALID;
    ReplayLayout l;
    if (!replay_layout(num_pools, capacity, &l)) return COOP_ERR_INVALID;
    *bytes_out = l.bytes;
    return COOP_OK;
}

coop_status_t coop_replay(uint64_t* size, uint64_t* cost, uint8_t* kind, uint32_t* id,
                          uint64_t* len, uint64_t num_pools, uint64_t capacity, const uint8_t* op,
                          const uint32_t* op_id, const uint64_t* op_size, const uint64_t* op_cost,
                          const uint8_t* op_flags, uint64_t num_ops, int32_t policy,
                          uint64_t* out_block, uint64_t* out_window, uint64_t* out_cost,
                          uint64_t* out_free, uint32_t* status_out, void* workspace,
                          size_t workspace_bytes, void* stream) {
    if (policy != COOP_POLICY_WINDOW && policy != COOP_POLICY_GREEDY) return COOP_ERR_INVALID;
    if (num_pools == 0 || num_ops == 0) return COOP_OK;
    if (!size || !cost || !kind || !id || !len || !op || !op_id || !op_size || !op_cost ||
        !op_flags || !out_block || !out_window || !out_cost || !out_free || !status_out)
        return COOP_ERR_INVALID;
    ReplayLayout l;
    if (!replay_layout(num_pools, capacity, &l)) return COOP_ERR_INVALID;
    if (!workspace || workspace_bytes < l.bytes) return COOP_ERR_WORKSPACE;
    hipStream_t s0 = static_cast<hipStream_t>(stream);
    // Pools that fit in LDS: one resident workgroup per pool, one launch.
    const size_t res_lds = resident_lds_bytes(capacity);
    if (capacity < 65536 && res_lds + kStaticResLds <= kLdsLimit) {
        hipLaunchKernelGGL(replay_status_kernel, dim3(1), dim3(1), 0, s0, status_out);
        if (hipGetLastError() != hipSuccess) return COOP_ERR_HIP;
        if (res_lds > 64 * 1024 &&
            hipFuncSetAttribute(reinterpret_cast<const void*>(replay_resident_kernel),
                                hipFuncAttributeMaxDynamicSharedMemorySize,
                                static_cast<int>(res_lds)) != hipSuccess)
            return COOP_ERR_HIP;
        hipLaunchKernelGGL(replay_resident_kernel, dim3(static_cast<uint32_t>(num_pools)),
                           dim3(kResThreads), res_lds, s0, size, cost, kind, id, len, capacity, op,
                           op_id, op_size, op_cost, op_flags, num_ops, policy, out_block,
                           out_window, out_cost, out_free, status_out);
        if (hipGetLastError() != hipSuccess) return COOP_ERR_HIP;
        return COOP_OK;
    }
    char* w = static_cast<char*>(workspace);
    uint64_t* seg = reinterpret_cast<uint64_t*>(w + l.seg);
    uint64_t* req_off = reinterpret_cast<uint64_t*>(w + l.req_off);
    uint64_t* req_ff = reinterpret_cast<uint64_t*>(w + l.req_ff);
    uint64_t* req_win = reinterpret_cast<uint64_t*>(w + l.req_win);
    uint64_t* ff = reinterpret_cast<uint64_t*>(w + l.ff);
    coop_window_t* win = reinterpret_cast<coop_window_t*>(w + l.win);
    uint32_t* status = status_out;
    hipStream_t s = static_cast<hipStream_t>(stream);
    const uint64_t nb = num_pools * capacity;
    const uint32_t small = static_cast<uint32_t>((num_pools + 1 + 255) / 256);
    hipLaunchKernelGGL(replay_init_kernel, dim3(small), dim3(256), 0, s, num_pools, capacity, seg,
                       req_off, req_ff, op, op_size, num_ops, status);
    if (hipGetLastError() != hipSuccess) return COOP_ERR_HIP;
    for (uint64_t t = 0; t < num_ops; ++t) {
        coop_status_t rc = coop_first_fit_enqueue(size, kind, nb, seg, num_pools, req_ff, req_off,
                                                  num_pools, ff, w + l.ff_ws, l.ff_ws_bytes,
                                                  stream, false);
        if (rc != COOP_OK) return rc;
        if (policy == COOP_POLICY_WINDOW) {
            hipLaunchKernelGGL(replay_gate_kernel, dim3(small), dim3(256), 0, s, num_pools, req_ff,
                               ff, req_win);
            if (hipGetLastError() != hipSuccess) return COOP_ERR_HIP;
            rc = coop_window_search_enqueue(size, cost, kind, nb, seg, num_pools, req_win,
                                            req_off, num_pools, win, w + l.win_ws,
                                            l.win_ws_bytes, stream, false);
            if (rc != COOP_OK) return rc;
        }
        hipLaunchKernelGGL(replay_update_kernel, dim3(static_cast<uint32_t>(num_pools)),
                           dim3(kThreads), 0, s, size, cost, kind, id, len, capacity, op, op_id,
                           op_size, op_cost, op_flags, num_ops, t, policy, ff, win, req_ff,
                           out_block, out_window, out_cost, out_free, status);
        if (hipGetLastError() != hipSuccess) return COOP_ERR_HIP;
    }
    return COOP_OK;
}

}  // extern "C"
