// Batched sliding-window eviction search (Coop, section 3.3) for gfx950.
//
// Problem (section 3.1 Eq. (1), window form of section 3.3): for every
// request of S bytes on a pool snapshot, find the window [start, end) of
// adjacent blocks with no pinned block, at least S bytes and the least summed
// cost of its evictable blocks; ties go to fewer bytes, then the lower start.
//
// Work decomposition
// ------------------
// Each snapshot b of N_b blocks is cut into tiles of kTile blocks
// (ceil(N_b / kTile) tiles, one for an empty snapshot).  A workgroup owns a
// tile and answers every request of the snapshot for the starts in its tile.
// Workgroups need no host planning: with f(b) = floor(seg[b] / kTile) + b,
// the tiles of snapshot b are the virtual ids [f(b), f(b) + tiles_b), and f
// is strictly increasing, so a search over seg_offsets names the snapshot.
// Ids that name no tile exit at once.  The hardware deals workgroups round
// robin to the 8 XCDs and their shader engines; the virtual id is a 5-bit
// rotation of the workgroup id, so every XCD and engine sees an even mix of
// tiles and empty ids, and consecutive tiles land on the same XCD (halo
// reads hit its L2).  A snapshot uses at most `pc` workgroups (the
// partial-key budget per request); with more tiles, each workgroup takes a
// group of consecutive tiles.
//
// Per tile
// --------
//  1. Stage: each thread loads kItems consecutive blocks (16-byte loads when
//     aligned, all issued at once) and runs a segmented exclusive scan of size
//     and of effective cost in registers (a pinned block closes its run); a
//     block-wide scan joins the threads.  LDS receives, per block k, the key
//     X[k] = (run id << 51) | (bytes of its run before k) and the matching
//     cost prefix XC[k].  Keys are monotone over the whole tile, so "first
//     end at or after S bytes in the same run" becomes a plain lower bound.
//     Both arrays are XOR-swizzled so blocked and striped accesses avoid LDS
//     bank conflicts.
//  2. Halo: when the last run continues past the tile, up to kHaloCap more
//     blocks of it (stopping at the first pinned block) are staged.
//  3. Per request: the shortest window of every start is found for all
//     starts at once by a merge path: the targets T_i = X[i] + S and the end
//     keys X[k+1] are two sorted sequences; each thread merges a fixed-length
//     slice (uniform work, no divergence) and records, for each start it
//     meets, the first end whose key reaches its target.  Each thread then
//     scores its own kItems starts (key (cost, bytes, start)) and a
//     lexicographic argmin runs across the wavefront (shuffles) and the block
//     (LDS).
//  4. Starts whose window would end past the staged region (the run outlives
//     the halo) are finished by a streaming pass over the rest of the run.
// A tile whose run byte prefix reaches 2^51 (no room left for the run id)
// keeps plain 64-bit prefixes and run ids, and bisects each start instead.
//
// Combining tiles
// ---------------
// A snapshot with one tile writes its results directly.  Otherwise every
// workgroup writes one partial key per request into the workspace and takes
// a ticket on a per-snapshot counter; the workgroup holding the last ticket
// reduces the partials and writes the results.  Counters carry a per-call
// epoch, so the workspace never needs clearing.
//
// All arithmetic is unsigned 64-bit integer; prefix differences are exact
// whenever each run's byte and cost totals fit in 64 bits.

#include <hip/hip_runtime.h>

#include <atomic>
#include <chrono>
#include <stdint.h>

#include "coop.h"

namespace {

constexpr uint32_t kThreads = 512;
constexpr uint32_t kWaves = kThreads / 64;
constexpr uint32_t kItems = 8;
constexpr uint32_t kTileLog2 = 12;
constexpr uint32_t kTile = 1u << kTileLog2;
static_assert(kTile == kThreads * kItems, "tile = threads x items");
constexpr uint32_t kHaloCap = 256;  // also the chunk length of the streaming pass
static_assert(kHaloCap <= kThreads, "one halo block per thread");
constexpr uint32_t kStage = kTile + kHaloCap;
constexpr uint32_t kSent = 24;  // +infinity keys after the staged region (>= merge slice + 2)
constexpr uint32_t kXN = kStage + 32;  // keys of blocks [0, kStage], sentinels, swizzle slack
constexpr uint32_t kValBits = 51;
constexpr uint64_t kValMask = (1ull << kValBits) - 1;
// Blocks below 2^38 bytes keep any staged byte prefix (at most kStage < 2^13
// blocks) below the 51-bit field of a key.
constexpr uint64_t kBigBlock = 1ull << 38;
static_assert(kStage < (1u << (kValBits - 38)), "staged prefixes must fit the key field");
// A key above every real key and target that stays finite after adding S'.
constexpr uint64_t kSentinel = ~0ull - kValMask;
constexpr uint64_t kNone = ~0ull;
constexpr uint64_t kPartialBudget = 1ull << 22;  // partial keys (32 B each)
constexpr uint32_t kEpochShift = 24;             // counter = epoch << 24 | tickets
constexpr uint64_t kEpochMask = (1ull << 40) - 1;

// Candidate window: ordered by (cost, bytes, start); `end` rides along.
struct Key {
    uint64_t cost, bytes, start, end;
};

__device__ __forceinline__ Key key_none() { return Key{kNone, kNone, kNone, kNone}; }

__device__ __forceinline__ bool key_less(const Key& a, const Key& b) {
    if (a.cost != b.cost) return a.cost < b.cost;
    if (a.bytes != b.bytes) return a.bytes < b.bytes;
    return a.start < b.start;
}

// Segmented-scan element over blocks where a pinned block closes its run:
// `flag` says a pinned block occurred, q/c are the size and cost sums after
// the last one, `cnt` counts pinned blocks.
struct Seg {
    uint32_t flag, cnt;
    uint64_t q, c;
};

__device__ __forceinline__ Seg seg_identity() { return Seg{0u, 0u, 0ull, 0ull}; }

// a precedes b.
__device__ __forceinline__ Seg seg_combine(const Seg& a, const Seg& b) {
    Seg r;
    r.flag = a.flag | b.flag;
    r.cnt = a.cnt + b.cnt;
    r.q = b.flag ? b.q : a.q + b.q;
    r.c = b.flag ? b.c : a.c + b.c;
    return r;
}

__device__ __forceinline__ uint64_t shfl_up_u64(uint64_t v, unsigned d) {
    const uint32_t lo = __shfl_up(static_cast<uint32_t>(v), d, 64);
    const uint32_t hi = __shfl_up(static_cast<uint32_t>(v >> 32), d, 64);
    return (static_cast<uint64_t>(hi) << 32) | lo;
}

__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t v, int m) {
    const uint32_t lo = __shfl_xor(static_cast<uint32_t>(v), m, 64);
    const uint32_t hi = __shfl_xor(static_cast<uint32_t>(v >> 32), m, 64);
    return (static_cast<uint64_t>(hi) << 32) | lo;
}

__device__ __forceinline__ uint64_t shfl_u64(uint64_t v, int src) {
    const uint32_t lo = __shfl(static_cast<uint32_t>(v), src, 64);
    const uint32_t hi = __shfl(static_cast<uint32_t>(v >> 32), src, 64);
    return (static_cast<uint64_t>(hi) << 32) | lo;
}

__device__ __forceinline__ Seg shfl_up_seg(const Seg& s, unsigned d) {
    Seg r;
    r.flag = __shfl_up(s.flag, d, 64);
    r.cnt = __shfl_up(s.cnt, d, 64);
    r.q = shfl_up_u64(s.q, d);
    r.c = shfl_up_u64(s.c, d);
    return r;
}

__device__ __forceinline__ Seg shfl_seg(const Seg& s, int src) {
    Seg r;
    r.flag = __shfl(s.flag, src, 64);
    r.cnt = __shfl(s.cnt, src, 64);
    r.q = shfl_u64(s.q, src);
    r.c = shfl_u64(s.c, src);
    return r;
}

// LDS slot of block index i: the low four bits are XORed with bits 3..6, a
// permutation inside every aligned group of 16.  Thread t stages indices
// 8t..8t+7, so for a fixed item the 16 lanes of a quarter-wave hit 16
// different 8-byte bank pairs; consecutive indices stay distinct as well.
__device__ __forceinline__ uint32_t sw(uint32_t i) { return i ^ ((i >> 3) & 15u); }

struct Params {
    const uint64_t* size;
    const uint64_t* cost;
    const uint8_t* kind;
    const uint64_t* seg;
    const uint64_t* req_size;
    const uint64_t* req_off;
    coop_window_t* out;
    Key* part;             // [num_requests][pc]
    uint64_t* counters;    // [num_segments]
    uint64_t num_blocks;
    uint64_t num_segments;
    uint64_t num_requests;
    uint64_t num_virtual;  // floor(num_blocks / kTile) + num_segments
    uint64_t pc;
    uint64_t epoch;
    uint32_t rot_bits;     // the grid is 2^rot_bits workgroups (x) by slices (y)
    uint32_t slices;       // request slices: workgroup y takes requests y, y + slices, ...
    double inv_slope;      // guess of b per virtual id, for the snapshot lookup
};

struct Smem {
    uint64_t x[kXN];    // keys (run << 51 | byte prefix), or plain byte prefixes
    uint64_t xc[kXN];   // exclusive effective-cost prefix
    uint16_t aux[kXN];  // merge output (first end per start), or run ids
    Seg wseg[kWaves];
    Key wkey[kWaves];
    uint32_t wmin[kWaves];
    uint16_t sink[kThreads];  // per-lane target of merge writes that are not taken
    uint32_t flag;
};

// Exclusive block-wide scan of one Seg per thread; `total` receives the
// aggregate of the whole block.  Each wave scans its lanes with shuffles;
// the wave totals are scanned again by the first kWaves lanes of every wave.
// Two barriers.
__device__ Seg block_exclusive_scan(Seg x, Smem& sm, Seg& total) {
    const uint32_t lane = threadIdx.x & 63u, w = threadIdx.x >> 6;
    Seg inc = x;
#pragma unroll
    for (unsigned d = 1; d < 64; d <<= 1) {
        const Seg o = shfl_up_seg(inc, d);
        if (lane >= d) inc = seg_combine(o, inc);
    }
    Seg ex = shfl_up_seg(inc, 1);
    if (lane == 0) ex = seg_identity();
    if (lane == 63) sm.wseg[w] = inc;
    __syncthreads();
    Seg t = lane < kWaves ? sm.wseg[lane] : seg_identity();
#pragma unroll
    for (unsigned d = 1; d < kWaves; d <<= 1) {
        const Seg o = shfl_up_seg(t, d);
        if (lane >= d) t = seg_combine(o, t);
    }
    Seg before = shfl_seg(t, w ? static_cast<int>(w) - 1 : 0);
    if (w == 0) before = seg_identity();
    total = shfl_seg(t, kWaves - 1);
    __syncthreads();
    return seg_combine(before, ex);
}

// Block-wide minimum of a u32; result in every thread.  Two barriers.
__device__ uint32_t block_min_u32(uint32_t x, Smem& sm) {
    const uint32_t lane = threadIdx.x & 63u, w = threadIdx.x >> 6;
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) {
        const uint32_t o = __shfl_xor(x, m, 64);
        x = o < x ? o : x;
    }
    if (lane == 0) sm.wmin[w] = x;
    __syncthreads();
    uint32_t r = sm.wmin[0];
#pragma unroll
    for (uint32_t u = 1; u < kWaves; ++u) r = sm.wmin[u] < r ? sm.wmin[u] : r;
    __syncthreads();
    return r;
}

__device__ __forceinline__ Key shfl_xor_key(const Key& k, int m) {
    Key o;
    o.cost = shfl_xor_u64(k.cost, m);
    o.bytes = shfl_xor_u64(k.bytes, m);
    o.start = shfl_xor_u64(k.start, m);
    o.end = shfl_xor_u64(k.end, m);
    return o;
}

// Block-wide lexicographic argmin; the result is valid in thread 0 only.
// Two barriers.
__device__ Key block_min_key(Key k, Smem& sm) {
    const uint32_t lane = threadIdx.x & 63u, w = threadIdx.x >> 6;
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) {
        const Key o = shfl_xor_key(k, m);
        if (key_less(o, k)) k = o;
    }
    if (lane == 0) sm.wkey[w] = k;
    __syncthreads();
    if (w == 0) {
        k = lane < kWaves ? sm.wkey[lane] : key_none();
#pragma unroll
        for (int m = kWaves / 2; m >= 1; m >>= 1) {
            const Key o = shfl_xor_key(k, m);
            if (key_less(o, k)) k = o;
        }
    }
    __syncthreads();
    return k;
}

struct Snapshot {
    uint64_t b, s0, s1, q0, q1, first;  // first = f(b), the virtual id of its first tile
};

// The snapshot b holding virtual id v: the largest b in [0, B) with
// f(b) = floor(seg[b] / kTile) + b <= v.  A guess from the average snapshot
// length is tried first, with its request offsets loaded alongside, so that
// uniform batches settle in one round of loads.  Offsets are clamped to the
// array lengths: malformed offsets give wrong answers, never an
// out-of-bounds access.
__device__ Snapshot locate_snapshot(const Params& P, uint64_t v) {
    const uint64_t B = P.num_segments;
    uint64_t g = static_cast<uint64_t>(static_cast<double>(v) * P.inv_slope);
    if (g >= B) g = B - 1;
    uint64_t sg = P.seg[g], sg1 = P.seg[g + 1];
    uint64_t rg = P.req_off[g], rg1 = P.req_off[g + 1];
    auto f = [&](uint64_t bb, uint64_t seg_b) { return (seg_b >> kTileLog2) + bb; };
    const bool hit = f(g, sg) <= v && (g + 1 == B || f(g + 1, sg1) > v);
    uint64_t b = g;
    if (!hit) {
        uint64_t lo = 0, hi = B;  // f(lo) <= v < f(hi) (f(B) taken as infinite)
        if (f(g, sg) <= v) lo = g; else hi = g;
        while (hi - lo > 1) {
            const uint64_t mid = lo + (hi - lo) / 2;
            if (f(mid, P.seg[mid]) <= v) lo = mid; else hi = mid;
        }
        b = lo;
        sg = P.seg[b];
        sg1 = P.seg[b + 1];
        rg = P.req_off[b];
        rg1 = P.req_off[b + 1];
    }
    Snapshot sn;
    sn.b = b;
    sn.first = f(b, sg);
    sn.s1 = sg1 < P.num_blocks ? sg1 : P.num_blocks;
    sn.s0 = sg < sn.s1 ? sg : sn.s1;
    sn.q1 = rg1 < P.num_requests ? rg1 : P.num_requests;
    sn.q0 = rg < sn.q1 ? rg : sn.q1;
    return sn;
}

// Loads the kItems blocks [t0 + tid*kItems, +kItems) of a tile of nt blocks.
// Blocks past nt read as pinned.  All loads are independent of each other.
__device__ __forceinline__ void load_items(const Params& P, uint64_t t0, uint32_t nt,
                                           uint64_t (&sz)[kItems], uint64_t (&ct)[kItems],
                                           uint8_t (&kd)[kItems]) {
    uint32_t i0 = threadIdx.x * kItems;
    asm volatile("" : "+v"(i0));
    const bool aligned = ((reinterpret_cast<uintptr_t>(P.size) | reinterpret_cast<uintptr_t>(P.cost)) &
                          15u) == 0 &&
                         (reinterpret_cast<uintptr_t>(P.kind) & 7u) == 0;
    if (nt == kTile && (t0 & 7u) == 0 && aligned) {
        const ulonglong2* ps = reinterpret_cast<const ulonglong2*>(P.size + t0 + i0);
        const ulonglong2* pc = reinterpret_cast<const ulonglong2*>(P.cost + t0 + i0);
        const uint2 k2 = *reinterpret_cast<const uint2*>(P.kind + t0 + i0);
#pragma unroll
        for (uint32_t j = 0; j < kItems / 2; ++j) {
            const ulonglong2 a = ps[j], b = pc[j];
            sz[2 * j] = a.x;
            sz[2 * j + 1] = a.y;
            ct[2 * j] = b.x;
            ct[2 * j + 1] = b.y;
        }
#pragma unroll
        for (uint32_t j = 0; j < 4; ++j) {
            kd[j] = static_cast<uint8_t>(k2.x >> (8 * j));
            kd[j + 4] = static_cast<uint8_t>(k2.y >> (8 * j));
        }
    } else {
#pragma unroll
        for (uint32_t j = 0; j < kItems; ++j) {
            const uint32_t i = i0 + j;
            const bool in = i < nt;
            sz[j] = in ? P.size[t0 + i] : 0;
            ct[j] = in ? P.cost[t0 + i] : 0;
            kd[j] = in ? P.kind[t0 + i] : static_cast<uint8_t>(COOP_PINNED);
        }
    }
}

__device__ __forceinline__ coop_window_t to_window(const Key& k, uint64_t S) {
    if (S == 0) return coop_window_t{0, 0, 0};
    if (k.start == kNone) return coop_window_t{kNone, kNone, kNone};
    return coop_window_t{k.start, k.end, k.cost};
}

// Stages the blocks [pos, pos + m) after the tile (halo): keys at stage
// indices [kTile, kTile + fp] (the last one is the boundary after the staged
// blocks), continuing the prefixes cq/cc of run `run`.  The halo stops at the
// first pinned block, or, in packed mode, before the first block of 2^38 bytes
// or more (its prefix might not fit the key field); `cut` reports the second
// case, in which the run goes on past the halo.  In packed mode the keys carry
// the run id; otherwise aux holds it.  Returns fp.  Five barriers.
__device__ uint32_t stage_halo(const Params& P, Smem& sm, uint64_t pos, uint32_t m, uint64_t cq,
                               uint64_t cc, uint32_t run, bool packed, bool& cut) {
    const uint32_t tid = threadIdx.x;
    uint32_t stop = 2 * m;  // 2*index for a pinned block, 2*index+1 for an oversized one
    uint64_t sz = 0, ct = 0;
    if (tid < m) {
        const uint8_t kd = P.kind[pos + tid];
        sz = P.size[pos + tid];
        ct = P.cost[pos + tid];
        ct = kd == COOP_EVICTABLE ? ct : 0;
        if (kd >= COOP_PINNED) stop = 2 * tid;
        else if (packed && sz >= kBigBlock) stop = 2 * tid + 1;
    }
    const uint32_t first = block_min_u32(stop, sm);
    const uint32_t fp = first >> 1;
    cut = fp < m && (first & 1u);
    const bool valid = tid < fp;
    Seg x = seg_identity();
    x.q = valid ? sz : 0;
    x.c = valid ? ct : 0;
    Seg tot;
    const Seg ex = block_exclusive_scan(x, sm, tot);
    const uint64_t rbits = packed ? static_cast<uint64_t>(run) << kValBits : 0;
    if (valid) {
        sm.x[sw(kTile + tid)] = rbits | (cq + ex.q);
        sm.xc[sw(kTile + tid)] = cc + ex.c;
        if (!packed) sm.aux[sw(kTile + tid)] = static_cast<uint16_t>(run);
    }
    if (tid == 0) {
        sm.x[sw(kTile + fp)] = rbits | (cq + tot.q);
        sm.xc[sw(kTile + fp)] = cc + tot.c;
        if (!packed) sm.aux[sw(kTile + fp)] = static_cast<uint16_t>(run);
    }
    __syncthreads();
    return fp;
}

// +infinity keys after the staged region [0, end]: the merge path reads past
// the end of both sequences without bounds checks.  The caller synchronises.
__device__ __forceinline__ void write_sentinels(Smem& sm, uint32_t end) {
    if (threadIdx.x < kSent) sm.x[sw(end + 1 + threadIdx.x)] = kSentinel;
}

// Finishes the pending starts [cur, nt): they all lie in the tile's last
// run and their windows end past the staged region [0, end).  The rest of
// the run is walked in chunks of kHaloCap blocks, staged (as inclusive
// prefixes) over the halo space; each chunk resolves a prefix of the pending
// starts, since their ends are monotone.  Candidates fold into `best`.
// Uniform control flow.
__device__ __forceinline__ void stream_pass(const Params& P, Smem& sm, uint32_t cur, uint32_t nt,
                                            uint32_t end, bool packed, uint64_t t0, uint64_t s0,
                                            uint64_t s1, uint64_t S, Key& best) {
    const uint32_t tid = threadIdx.x;
    const uint64_t tl = t0 - s0;
    const uint64_t vmask = packed ? kValMask : kNone;
    uint64_t cq = sm.x[sw(end)] & vmask, cc = sm.xc[sw(end)];
    uint64_t pos = t0 + end;
    __syncthreads();  // every thread has read the region end before it is reused
    while (cur < nt && pos < s1) {
        const uint64_t left = s1 - pos;
        const uint32_t m = static_cast<uint32_t>(left < kHaloCap ? left : kHaloCap);
        bool pinned = true;
        uint64_t sz = 0, ct = 0;
        if (tid < m) {
            const uint8_t kd = P.kind[pos + tid];
            pinned = kd >= COOP_PINNED;
            sz = P.size[pos + tid];
            ct = P.cost[pos + tid];
            ct = kd == COOP_EVICTABLE ? ct : 0;
        }
        const uint32_t fp = block_min_u32(pinned ? tid : m, sm);
        const bool valid = tid < fp;
        Seg x = seg_identity();
        x.q = valid ? sz : 0;
        x.c = valid ? ct : 0;
        Seg tot;
        const Seg ex = block_exclusive_scan(x, sm, tot);
        if (valid) {
            sm.x[sw(kTile + tid)] = cq + ex.q + x.q;  // inclusive prefix at the chunk block
            sm.xc[sw(kTile + tid)] = cc + ex.c + x.c;
        }
        __syncthreads();
        const uint64_t lastq = cq + tot.q;
        uint32_t still = nt;
        for (uint32_t i = cur + tid; i < nt; i += kThreads) {
            const uint64_t base = sm.x[sw(i)] & vmask;
            const uint64_t cbase = sm.xc[sw(i)];
            if (fp > 0 && lastq - base >= S) {
                uint32_t a = 0, hi = fp - 1;  // first chunk block with prefix - base >= S
                while (a < hi) {
                    const uint32_t mid = a + (hi - a) / 2;
                    if (sm.x[sw(kTile + mid)] - base >= S) hi = mid; else a = mid + 1;
                }
                const Key cand{sm.xc[sw(kTile + a)] - cbase, sm.x[sw(kTile + a)] - base, tl + i,
                               (pos - s0) + a + 1};
                if (key_less(cand, best)) best = cand;
            } else if (i < still) {
                still = i;
            }
        }
        cur = block_min_u32(still, sm);
        if (fp < m) break;  // the run ends inside this chunk
        cq = lastq;
        cc += tot.c;
        pos += m;
    }
}

__global__ __launch_bounds__(kThreads, 4) void coop_window_search_kernel(Params P) {
    __shared__ Smem sm;
    const uint32_t tid = threadIdx.x;
    // virtual id: the workgroup id rotated right by 5 bits within rot_bits bits
    const uint64_t v = (blockIdx.x >> 5) |
                       (static_cast<uint64_t>(blockIdx.x & 31u) << (P.rot_bits - 5));
    if (v >= P.num_virtual) return;

    const Snapshot sn = locate_snapshot(P, v);
    const uint64_t b = sn.b, s0 = sn.s0, s1 = sn.s1, q0 = sn.q0;
    const uint64_t R = sn.q1 - q0;
    const uint64_t nb = s1 - s0;
    const uint64_t tiles = nb ? (nb + kTile - 1) >> kTileLog2 : 1;
    const uint64_t p = v - sn.first;  // wraps (and exits) if the offsets are malformed
    // request slice: this workgroup answers requests y, y + slices, ... of the snapshot
    const uint32_t y = blockIdx.y;
    if (p >= tiles || R == 0 || y >= R) return;
    // At most pc workgroups per snapshot: each takes `stride` consecutive tiles.
    const uint64_t stride = tiles <= P.pc ? 1 : (tiles + P.pc - 1) / P.pc;
    if (stride != 1 && p % stride != 0) return;
    const uint64_t g = stride == 1 ? p : p / stride;
    const uint64_t G = stride == 1 ? tiles : (tiles + stride - 1) / stride;
    const uint64_t tau_end = p + stride < tiles ? p + stride : tiles;
    const bool direct = tiles == 1;

    for (uint64_t tau = p; tau < tau_end; ++tau) {
        const uint64_t t0 = s0 + (tau << kTileLog2);  // global index of the tile start
        const uint64_t tl = t0 - s0;                   // snapshot-local index of the tile start
        const uint32_t nt = static_cast<uint32_t>(s1 - t0 < kTile ? s1 - t0 : kTile);
        // An opaque copy of the thread's first block index: addresses derived
        // from it are recomputed in each loop instead of being kept live
        // across the whole kernel (they would not fit in registers).
        uint32_t i0 = tid * kItems;
        asm volatile("" : "+v"(i0));

        // ---- 1. stage: exclusive prefixes of this thread's kItems blocks
        uint32_t pinmask = 0;
        bool packed;
        {
            uint64_t sz[kItems], ct[kItems];
            uint8_t kd[kItems];
            load_items(P, t0, nt, sz, ct, kd);
            uint64_t acc = 0, cacc = 0;
            uint32_t runs = 0, flag = 0, lflags = 0, big = 0;
            uint32_t xr[kItems];  // run id (pinned blocks before the block) within the thread
#pragma unroll
            for (uint32_t j = 0; j < kItems; ++j) {
                const uint64_t s_j = sz[j], c_j = kd[j] == COOP_EVICTABLE ? ct[j] : 0;
                sz[j] = acc;  // from here on: byte / cost prefix of the run before block j
                ct[j] = cacc;
                xr[j] = runs;
                lflags |= flag << j;
                if (kd[j] >= COOP_PINNED) {
                    pinmask |= 1u << j;
                    acc = 0;
                    cacc = 0;
                    ++runs;
                    flag = 1;
                } else {
                    acc += s_j;
                    cacc += c_j;
                    big |= s_j >= kBigBlock ? 1u : 0u;
                }
            }
            Seg tot;
            const Seg carry = block_exclusive_scan(Seg{flag, runs, acc, cacc}, sm, tot);
#pragma unroll
            for (uint32_t j = 0; j < kItems; ++j) {
                const bool own = (lflags >> j) & 1u;
                sz[j] = own ? sz[j] : carry.q + sz[j];
                ct[j] = own ? ct[j] : carry.c + ct[j];
                xr[j] += carry.cnt;
            }
            const uint64_t lastq = flag ? acc : carry.q + acc;  // prefix after the last block
            const uint64_t lastc = flag ? cacc : carry.c + cacc;
            const uint32_t lastr = carry.cnt + runs;
            // with every block below 2^38 bytes, every prefix fits the key field
            packed = !__syncthreads_or(big);
#pragma unroll
            for (uint32_t j = 0; j < kItems; ++j) {
                const uint32_t s = sw(i0 + j);
                sm.x[s] = packed ? (static_cast<uint64_t>(xr[j]) << kValBits) | sz[j] : sz[j];
                sm.xc[s] = ct[j];
                if (!packed) sm.aux[s] = static_cast<uint16_t>(xr[j]);
            }
            if (tid == kThreads - 1) {  // boundary after the tile
                sm.x[sw(kTile)] = packed ? (static_cast<uint64_t>(lastr) << kValBits) | lastq
                                         : lastq;
                sm.xc[sw(kTile)] = lastc;
                if (!packed) sm.aux[sw(kTile)] = static_cast<uint16_t>(lastr);
            }
            __syncthreads();
        }
        const uint64_t vmask = packed ? kValMask : kNone;
        // the boundary after the tile: kept to restore it after a streaming pass
        const uint64_t xb = sm.x[sw(kTile)];
        const uint64_t xcb = sm.xc[sw(kTile)];
        const uint32_t runb = packed ? static_cast<uint32_t>(xb >> kValBits) : sm.aux[sw(kTile)];

        // ---- 2. halo: the rest of the last run, up to kHaloCap blocks
        uint32_t end = nt;
        bool open = false;
        {
            const uint32_t runl = packed ? static_cast<uint32_t>(sm.x[sw(kTile - 1)] >> kValBits)
                                         : sm.aux[sw(kTile - 1)];
            const bool last_open = nt == kTile && runb == runl;  // block kTile-1 is not pinned
            if (last_open && t0 + kTile < s1) {
                const uint64_t pos = t0 + kTile;
                const uint64_t left = s1 - pos;
                const uint32_t m = static_cast<uint32_t>(left < kHaloCap ? left : kHaloCap);
                bool cut;
                const uint32_t fp = stage_halo(P, sm, pos, m, xb & vmask, xcb, runb, packed, cut);
                end = kTile + fp;
                // open: the run goes on past the staged blocks
                open = cut || (fp == m && left > m);
            }
        }
        const uint32_t endrun = runb;  // the run reaching the end of the staged region
        write_sentinels(sm, end);
        __syncthreads();

        // ---- 3. the snapshot's requests of this slice
        for (uint64_t r = y; r < R; r += P.slices) {
            const uint64_t q = q0 + r;
            const uint64_t S = P.req_size[q];
            Key best = key_none();
            uint32_t pend = nt;
            uint32_t i0 = tid * kItems;  // opaque again, see above
            asm volatile("" : "+v"(i0));
            if (S != 0) {
                if (packed) {
                    // merge path: A = targets X[i] + S' of starts [0, nt), B = end keys
                    // X[1..end].  S' = min(S, field maximum): a target that carries
                    // into the next run id lies above every end of its own run, which
                    // is exactly the infeasible case; the scoring below re-checks.
                    const uint64_t Sc = S < kValMask ? S : kValMask;
                    const uint32_t nA = nt, nB = end, total = nA + nB;
                    const uint32_t L = (total + kThreads - 1) / kThreads;
                    const uint32_t d = tid * L < total ? tid * L : total;
                    const uint32_t dEnd = d + L < total ? d + L : total;
                    uint32_t lo = d > nB ? d - nB : 0, hi = d < nA ? d : nA;
                    while (lo < hi) {
                        const uint32_t mid = (lo + hi) >> 1;
                        // start `mid` comes before end d-1-mid iff its target <= X[d-mid]
                        const bool before = sm.x[sw(mid)] + Sc <= sm.x[sw(d - mid)];
                        lo = before ? mid + 1 : lo;
                        hi = before ? hi : mid;
                    }
                    // Past the ends the sentinels compare above every target, so all
                    // remaining starts take "no end in the region" (e = end).  Starts
                    // past nA are phantoms: their entries are never read.
                    uint32_t a = lo, bq = d - lo;
                    uint64_t ta = sm.x[sw(a)] + Sc;
                    uint64_t kb = sm.x[sw(bq + 1)];
                    for (uint32_t st = d; st < dEnd; ++st) {
                        const bool takeA = ta <= kb;
                        uint16_t* dst = takeA ? &sm.aux[sw(a)] : &sm.sink[tid];
                        *dst = static_cast<uint16_t>(bq);
                        a += takeA ? 1u : 0u;
                        bq += takeA ? 0u : 1u;
                        const uint64_t val = sm.x[sw(takeA ? a : bq + 1)];
                        ta = takeA ? val + Sc : ta;
                        kb = takeA ? kb : val;
                    }
                    __syncthreads();
#pragma unroll
                    for (uint32_t j = 0; j < kItems; ++j) {
                        const uint32_t i = i0 + j;
                        if (i >= nt || ((pinmask >> j) & 1u)) continue;
                        const uint32_t e = sm.aux[sw(i)];
                        const uint64_t xi = sm.x[sw(i)];
                        const uint32_t run = static_cast<uint32_t>(xi >> kValBits);
                        if (e < end) {
                            const uint64_t v1 = sm.x[sw(e + 1)];
                            const uint64_t bytes = (v1 & kValMask) - (xi & kValMask);
                            if (static_cast<uint32_t>(v1 >> kValBits) == run && bytes >= S) {
                                const Key cand{sm.xc[sw(e + 1)] - sm.xc[sw(i)], bytes, tl + i,
                                               tl + e + 1};
                                if (key_less(cand, best)) best = cand;
                            }
                        } else if (open && run == endrun && i < pend) {
                            pend = i;  // the window leaves the staged region
                        }
                    }
                } else {
                    // plain prefixes: find the run end, then the shortest end, by bisection
#pragma unroll 1
                    for (uint32_t j = 0; j < kItems; ++j) {
                        const uint32_t i = i0 + j;
                        if (i >= nt || ((pinmask >> j) & 1u)) continue;
                        const uint32_t run = sm.aux[sw(i)];
                        const uint64_t base = sm.x[sw(i)];
                        uint32_t lo = i, hi = end;  // first k in [i, end) that closes the run
                        while (lo < hi) {
                            const uint32_t mid = (lo + hi) >> 1;
                            if (sm.aux[sw(mid + 1)] != run) hi = mid; else lo = mid + 1;
                        }
                        const uint32_t rend = lo;  // pinned block ending the run, or end
                        lo = i;
                        hi = rend;
                        while (lo < hi) {
                            const uint32_t mid = (lo + hi) >> 1;
                            if (sm.x[sw(mid + 1)] - base >= S) hi = mid; else lo = mid + 1;
                        }
                        if (lo < rend) {
                            const Key cand{sm.xc[sw(lo + 1)] - sm.xc[sw(i)], sm.x[sw(lo + 1)] - base,
                                           tl + i, tl + lo + 1};
                            if (key_less(cand, best)) best = cand;
                        } else if (rend == end && open && i < pend) {
                            pend = i;
                        }
                    }
                }
            }
            // ---- 4. starts whose windows run past the staged region
            const uint32_t cur = open ? block_min_u32(pend, sm) : nt;
            if (cur < nt) {
                stream_pass(P, sm, cur, nt, end, packed, t0, s0, s1, S, best);
                // the streaming chunks overwrote the halo: keep only the tile
                __syncthreads();
                if (tid == 0) {
                    sm.x[sw(kTile)] = xb;
                    sm.xc[sw(kTile)] = xcb;
                    if (!packed) sm.aux[sw(kTile)] = static_cast<uint16_t>(runb);
                }
                end = kTile;  // later requests stream from the tile end
                write_sentinels(sm, end);
                __syncthreads();
            }
            best = block_min_key(best, sm);
            if (tid == 0) {
                if (direct) {
                    P.out[q] = to_window(best, S);
                } else {
                    Key* slot = P.part + q * P.pc + g;
                    if (tau != p) {
                        const Key prev = *slot;
                        if (key_less(prev, best)) best = prev;
                    }
                    *slot = best;
                }
            }
        }
        __syncthreads();  // LDS reused by the next tile
    }
    if (direct) return;

    // ---- combine the partial keys of the snapshot's workgroups
    __threadfence();
    __syncthreads();
    if (tid == 0) {
        uint32_t last = 1;
        if (G > 1 || (P.slices > 1 && R > 1)) {
            uint64_t* ctr = P.counters + b;
            uint64_t old = __hip_atomic_load(ctr, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            uint64_t want;
            do {
                want = (old >> kEpochShift) == P.epoch ? old + 1
                                                       : (P.epoch << kEpochShift) | 1ull;
            } while (!__hip_atomic_compare_exchange_strong(ctr, &old, want, __ATOMIC_ACQ_REL,
                                                           __ATOMIC_RELAXED,
                                                           __HIP_MEMORY_SCOPE_AGENT));
            // every (tile group, slice) pair of the snapshot arrives once
            const uint64_t arrivals = G * (R < P.slices ? R : P.slices);
            last = (want & ((1ull << kEpochShift) - 1)) == arrivals;
        }
        sm.flag = last;
    }
    __syncthreads();
    if (!sm.flag) return;
    __threadfence();
    for (uint64_t r = tid; r < R; r += kThreads) {
        const uint64_t q = q0 + r;
        const Key* row = P.part + q * P.pc;
        Key best = row[0];
        for (uint64_t gg = 1; gg < G; ++gg) {
            const Key o = row[gg];
            if (key_less(o, best)) best = o;
        }
        P.out[q] = to_window(best, P.req_size[q]);
    }
}

// ---------------------------------------------------------------------------
// Host side
// ---------------------------------------------------------------------------

struct Plan {
    uint64_t pc;           // partial slots per request
    uint64_t num_virtual;  // virtual workgroup ids
    uint32_t rot_bits;     // grid = 2^rot_bits workgroups
    uint32_t slices;       // request slices (grid y)
    size_t part_bytes;     // partial keys
    size_t bytes;          // total workspace
};

// grid x block must stay below 2^32 work-items: 2^23 workgroups of 512 threads
constexpr uint32_t kMaxRotBits = 23;
constexpr uint64_t kWideGrid = 2048;  // workgroups wanted before slicing requests
constexpr uint64_t kMaxSlices = 256;
static_assert(kWideGrid * kMaxSlices < (1ull << kEpochShift), "tickets fit the counter");

bool make_plan(uint64_t num_blocks, uint64_t num_segments, uint64_t num_requests, Plan* pl) {
    if (num_segments > (1ull << kMaxRotBits) || num_blocks > (1ull << 60) ||
        num_requests > (1ull << 40))
        return false;
    const uint64_t max_tiles = num_blocks ? (num_blocks + kTile - 1) >> kTileLog2 : 1;
    uint64_t pc = num_requests ? kPartialBudget / num_requests : 1;
    if (pc < 1) pc = 1;
    if (pc > max_tiles) pc = max_tiles;
    pl->pc = pc;
    pl->num_virtual = (num_blocks >> kTileLog2) + num_segments;
    uint32_t bits = 5;
    while ((1ull << bits) < pl->num_virtual) ++bits;
    if (bits > kMaxRotBits) return false;
    pl->rot_bits = bits;
    // Few tiles but many requests per snapshot (one small pool, many requests):
    // spread each snapshot's requests over up to kMaxSlices workgroups.
    pl->slices = 1;
    if (pl->num_virtual < kWideGrid && num_requests > num_segments) {
        const uint64_t per_snapshot = (num_requests + num_segments - 1) / num_segments;
        uint64_t want = (kWideGrid + pl->num_virtual - 1) / pl->num_virtual;
        if (want > per_snapshot) want = per_snapshot;
        if (want > kMaxSlices) want = kMaxSlices;
        pl->slices = static_cast<uint32_t>(want);
    }
    pl->part_bytes = (num_requests * pc * sizeof(Key) + 255) & ~static_cast<size_t>(255);
    pl->bytes = pl->part_bytes + num_segments * sizeof(uint64_t);
    return true;
}

std::atomic<uint64_t> g_calls{
    static_cast<uint64_t>(std::chrono::steady_clock::now().time_since_epoch().count())};

}  // namespace

extern "C" {

int coop_abi_version(void) { return COOP_ABI_VERSION; }

const char* coop_status_string(int status) {
    switch (status) {
        case COOP_OK: return "ok";
        case COOP_ERR_INVALID: return "invalid argument";
        case COOP_ERR_WORKSPACE: return "workspace missing or too small";
        case COOP_ERR_HIP: return "HIP launch failed";
        default: return "unknown status";
    }
}

coop_status_t coop_window_search_workspace_size(uint64_t num_blocks, uint64_t num_segments,
                                                uint64_t num_requests, size_t* bytes_out) {
    if (!bytes_out) return COOP_ERR_INVALID;
    Plan pl;
    if (!make_plan(num_blocks, num_segments, num_requests, &pl)) return COOP_ERR_INVALID;
    *bytes_out = pl.bytes;
    return COOP_OK;
}

coop_status_t coop_window_search(const uint64_t* size, const uint64_t* cost, const uint8_t* kind,
                                 uint64_t num_blocks, const uint64_t* seg_offsets,
                                 uint64_t num_segments, const uint64_t* req_sizes,
                                 const uint64_t* req_offsets, uint64_t num_requests,
                                 coop_window_t* out, void* workspace, size_t workspace_bytes,
                                 void* stream) {
    if (num_requests == 0) return COOP_OK;
    if (num_segments == 0) return COOP_ERR_INVALID;
    if (num_blocks && (!size || !cost || !kind)) return COOP_ERR_INVALID;
    if (!seg_offsets || !req_offsets || !req_sizes || !out) return COOP_ERR_INVALID;
    Plan pl;
    if (!make_plan(num_blocks, num_segments, num_requests, &pl)) return COOP_ERR_INVALID;
    if (!workspace || workspace_bytes < pl.bytes) return COOP_ERR_WORKSPACE;

    Params P;
    P.size = size;
    P.cost = cost;
    P.kind = kind;
    P.seg = seg_offsets;
    P.req_size = req_sizes;
    P.req_off = req_offsets;
    P.out = out;
    P.part = static_cast<Key*>(workspace);
    P.counters = reinterpret_cast<uint64_t*>(static_cast<char*>(workspace) + pl.part_bytes);
    P.num_blocks = num_blocks;
    P.num_segments = num_segments;
    P.num_requests = num_requests;
    P.num_virtual = pl.num_virtual;
    P.pc = pl.pc;
    P.epoch = g_calls.fetch_add(1, std::memory_order_relaxed) & kEpochMask;
    P.rot_bits = pl.rot_bits;
    P.slices = pl.slices;
    P.inv_slope = static_cast<double>(num_segments) /
                  (static_cast<double>(num_blocks) / kTile + static_cast<double>(num_segments));

    hipLaunchKernelGGL(coop_window_search_kernel, dim3(1u << pl.rot_bits, pl.slices), dim3(kThreads), 0,
                       static_cast<hipStream_t>(stream), P);
    if (hipGetLastError() != hipSuccess) return COOP_ERR_HIP;
    return COOP_OK;
}

}  // extern "C"
