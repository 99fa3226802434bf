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

#include <hip/hip_runtime.h>

#include <stdint.h>

#include "coop.h"

namespace {

constexpr uint32_t kThreads = 256;
constexpr uint64_t kNone = ~0ull;
constexpr uint8_t kOpAlloc = 0, kOpFree = 1;
constexpr uint8_t kFlagLeft = 1, kFlagPinned = 2;
constexpr uint32_t kErrCapacity = 1, kErrOperation = 2;

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
    const uint8_t* op_flags, uint64_t num_ops, uint64_t t, const uint64_t* ff,
    const coop_window_t* win, uint64_t* req_ff, uint64_t* out_block, uint64_t* out_window,
    uint64_t* out_cost, uint64_t* out_free, uint32_t* status) {
    __shared__ uint64_t red[kThreads / 64];
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
        if (k == kNone) {
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
                          const uint8_t* op_flags, uint64_t num_ops, uint64_t* out_block,
                          uint64_t* out_window, uint64_t* out_cost, uint64_t* out_free,
                          uint32_t* status_out, void* workspace, size_t workspace_bytes,
                          void* stream) {
    if (num_pools == 0 || num_ops == 0) return COOP_OK;
    if (!size || !cost || !kind || !id || !len || !op || !op_id || !op_size || !op_cost ||
        !op_flags || !out_block || !out_window || !out_cost || !out_free || !status_out)
        return COOP_ERR_INVALID;
    ReplayLayout l;
    if (!replay_layout(num_pools, capacity, &l)) return COOP_ERR_INVALID;
    if (!workspace || workspace_bytes < l.bytes) return COOP_ERR_WORKSPACE;
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
        coop_status_t rc = coop_first_fit(size, kind, nb, seg, num_pools, req_ff, req_off, num_pools,
                                          ff, w + l.ff_ws, l.ff_ws_bytes, stream);
        if (rc != COOP_OK) return rc;
        hipLaunchKernelGGL(replay_gate_kernel, dim3(small), dim3(256), 0, s, num_pools, req_ff, ff,
                           req_win);
        if (hipGetLastError() != hipSuccess) return COOP_ERR_HIP;
        rc = coop_window_search(size, cost, kind, nb, seg, num_pools, req_win, req_off, num_pools,
                                win, w + l.win_ws, l.win_ws_bytes, stream);
        if (rc != COOP_OK) return rc;
        hipLaunchKernelGGL(replay_update_kernel, dim3(static_cast<uint32_t>(num_pools)),
                           dim3(kThreads), 0, s, size, cost, kind, id, len, capacity, op, op_id,
                           op_size, op_cost, op_flags, num_ops, t, ff, win, req_ff, out_block,
                           out_window, out_cost, out_free, status);
        if (hipGetLastError() != hipSuccess) return COOP_ERR_HIP;
    }
    return COOP_OK;
}

}  // extern "C"
