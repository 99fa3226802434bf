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
//  1. Stage.  Each thread loads kItems consecutive blocks (16-byte loads when
//     aligned); the first kHaloCap threads also load one block each of the
//     halo, the blocks right after the tile, in the same round of loads.
//     Three plain prefix sums run over the tile followed by the halo: bytes
//     P, effective cost C (0 unless evictable) and the pinned count R.  A
//     window [i, k) holds no pinned block iff R[i] == R[k], and then its bytes
//     and cost are P[k] - P[i] and C[k] - C[i]; no reset at pinned blocks is
//     needed.  The sums run per thread, per wavefront (DPP row shifts and
//     broadcasts) and across the wavefronts (one barrier).  LDS receives, per
//     staged boundary k, the key X[k] = R[k] << 51 | P[k] and C[k].  Keys
//     increase with k, and for a start i the first end k with X[k] >= X[i] + S
//     is its shortest window when R[k] == R[i], while no window from i exists
//     inside the staged region otherwise.
//  2. Requests.  Wavefronts take requests: one wavefront per request when the
//     tile has at least as many requests as wavefronts, else up to kMaxWpr
//     wavefronts share one.  The targets X[i] + S of the starts and the end
//     keys X[k] are two sorted sequences; the lanes split their merge into
//     equal slices of merge steps (merge path, one bisection per lane), and
//     every step that takes a start meets that start's shortest window and
//     scores it at once.  A lexicographic argmin over the lanes (DPP) gives
//     the wavefront's answer; wavefronts sharing a request combine in LDS.
//  3. Starts whose windows end past the staged region (the region's last run
//     goes on) are a suffix of the tile, found by one search; the request's
//     wavefront finishes them by walking the rest of the run 64 blocks at a
//     time.
// A tile that holds a block of 2^38 bytes or more keeps plain 64-bit
// prefixes (P could outgrow the 51-bit field) with the run ids in a separate
// array, stages no halo, and bisects per start.
//
// Combining tiles
// ---------------
// A snapshot with one tile writes its results directly.  Otherwise every
// workgroup writes one partial key per request into the workspace and takes
// a ticket on a per-snapshot counter; the workgroup holding the last ticket
// reduces the partials and writes the results.  Counters carry a per-call
// epoch, so the workspace never needs clearing.
//
// All arithmetic is unsigned 64-bit integer.  Prefix sums wrap modulo 2^64;
// differences over a window are exact whenever each run's byte and cost
// totals fit in 64 bits.

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
constexpr uint32_t kHaloCap = 256;
static_assert(kHaloCap <= 4 * 64, "the halo is scanned by the first four wavefronts");
constexpr uint32_t kStage = kTile + kHaloCap;
// Merge steps per lane at most: all starts and ends of a staged region over
// one wavefront, rounded up to 2 mod 4 (see merge_steps).
constexpr uint32_t kMaxSteps = ((kTile + kStage + 63) / 64 + 1) / 4 * 4 + 2;
// LDS keys: boundaries [0, kStage], the sentinel after the last one, and the
// positions a lane reads past the starts once they are used up.
constexpr uint32_t kXN = ((kStage + 2 > kTile + kMaxSteps + 1 ? kStage + 2 : kTile + kMaxSteps + 1) +
                          7) / 8 * 8;
constexpr uint32_t kValBits = 51;
constexpr uint64_t kValMask = (1ull << kValBits) - 1;
constexpr uint32_t kRunShift = kValBits - 32;  // run id position in the high word of a key
// With every block below 2^38 bytes, any staged prefix (at most kStage < 2^13
// blocks) fits the 51-bit field, and no prefix wraps.
constexpr uint32_t kBigHiLog2 = 38 - 32;
static_assert(kStage < (1u << (kValBits - 38)), "staged prefixes must fit the key field");
static_assert(kStage < (1u << 16), "pinned counts fit 16 bits");
constexpr uint64_t kNone = ~0ull;
constexpr uint32_t kNone32 = ~0u;
constexpr uint32_t kMaxWpr = 4;                  // wavefronts that may share one request
constexpr uint64_t kPartialBudget = 1ull << 22;  // partial keys (32 B each)
constexpr uint32_t kEpochShift = 24;             // counter = epoch << 24 | tickets
constexpr uint64_t kEpochMask = (1ull << 40) - 1;

// DPP controls (GFX9 encoding).
constexpr int kRowShr1 = 0x111, kRowShr2 = 0x112, kRowShr4 = 0x114, kRowShr8 = 0x118;
constexpr int kRowBcast15 = 0x142, kRowBcast31 = 0x143;
constexpr int kQuadXor1 = 0xB1, kQuadXor2 = 0x4E;  // quad_perm [1,0,3,2] and [2,3,0,1]
constexpr int kRowHalfMirror = 0x141, kRowMirror = 0x140;

// Lane move within the wavefront; lanes whose source is outside the row, or
// whose row is masked off, get `old`.
template <int Ctrl, int RowMask = 0xf>
__device__ __forceinline__ uint32_t dpp32(uint32_t v, uint32_t old) {
    return static_cast<uint32_t>(__builtin_amdgcn_update_dpp(
        static_cast<int>(old), static_cast<int>(v), Ctrl, RowMask, 0xf, false));
}

template <int Ctrl, int RowMask = 0xf>
__device__ __forceinline__ uint64_t dpp64(uint64_t v, uint64_t old) {
    const uint32_t lo = dpp32<Ctrl, RowMask>(static_cast<uint32_t>(v), static_cast<uint32_t>(old));
    const uint32_t hi = dpp32<Ctrl, RowMask>(static_cast<uint32_t>(v >> 32),
                                             static_cast<uint32_t>(old >> 32));
    return (static_cast<uint64_t>(hi) << 32) | lo;
}

__device__ __forceinline__ uint32_t readlane32(uint32_t v, uint32_t lane) {
    return static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(v), static_cast<int>(lane)));
}

__device__ __forceinline__ uint64_t readlane64(uint64_t v, uint32_t lane) {
    return (static_cast<uint64_t>(readlane32(static_cast<uint32_t>(v >> 32), lane)) << 32) |
           readlane32(static_cast<uint32_t>(v), lane);
}

__device__ __forceinline__ uint64_t shfl64(uint64_t v, uint32_t src) {
    const uint32_t lo = __shfl(static_cast<uint32_t>(v), static_cast<int>(src), 64);
    const uint32_t hi = __shfl(static_cast<uint32_t>(v >> 32), static_cast<int>(src), 64);
    return (static_cast<uint64_t>(hi) << 32) | lo;
}

__device__ __forceinline__ uint32_t uniform(uint32_t v) {
    return static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(v)));
}

// Prefix-sum element: bytes, effective cost, and the pinned count in the low
// 16 bits of r (blocks of 2^38 bytes or more are counted from bit 16 up).
struct Sums {
    uint64_t q, c;
    uint32_t r;
};

template <int Ctrl, int RowMask>
__device__ __forceinline__ void sum_step(Sums& s) {
    s.q += dpp64<Ctrl, RowMask>(s.q, 0);
    s.c += dpp64<Ctrl, RowMask>(s.c, 0);
    s.r += dpp32<Ctrl, RowMask>(s.r, 0);
}

// Inclusive sums over the 16 lanes of each row.
__device__ __forceinline__ void row_inclusive_sum(Sums& s) {
    sum_step<kRowShr1, 0xf>(s);
    sum_step<kRowShr2, 0xf>(s);
    sum_step<kRowShr4, 0xf>(s);
    sum_step<kRowShr8, 0xf>(s);
}

// Inclusive sums over the wavefront: rows, then row 0 into row 1 and row 2
// into row 3, then row 1 into rows 2 and 3.
__device__ __forceinline__ void wave_inclusive_sum(Sums& s) {
    row_inclusive_sum(s);
    sum_step<kRowBcast15, 0xa>(s);
    sum_step<kRowBcast31, 0xc>(s);
}

__device__ __forceinline__ Sums readlane(const Sums& s, uint32_t lane) {
    return Sums{readlane64(s.q, lane), readlane64(s.c, lane), readlane32(s.r, lane)};
}

// A lane's best window so far.  `excess` is bytes - S (>= 0 for a window that
// meets the request), which orders like bytes and keeps every real window
// below the empty value all-ones; `start` is a staged index.
struct Cand {
    uint64_t cost, excess;
    uint32_t start;
};

__device__ __forceinline__ Cand cand_none() { return Cand{kNone, kNone, kNone32}; }

__device__ __forceinline__ bool cand_less(const Cand& a, const Cand& b) {
    if (a.cost != b.cost) return a.cost < b.cost;
    if (a.excess != b.excess) return a.excess < b.excess;
    return a.start < b.start;
}

template <int Ctrl, int RowMask>
__device__ __forceinline__ void argmin_step(Cand& k) {
    const Cand o{dpp64<Ctrl, RowMask>(k.cost, kNone), dpp64<Ctrl, RowMask>(k.excess, kNone),
                 dpp32<Ctrl, RowMask>(k.start, kNone32)};
    if (cand_less(o, k)) k = o;
}

// Lexicographic minimum over the wavefront; every lane gets it.
__device__ __forceinline__ Cand wave_argmin(Cand k) {
    argmin_step<kQuadXor1, 0xf>(k);
    argmin_step<kQuadXor2, 0xf>(k);
    argmin_step<kRowHalfMirror, 0xf>(k);
    argmin_step<kRowMirror, 0xf>(k);
    argmin_step<kRowBcast15, 0xa>(k);
    argmin_step<kRowBcast31, 0xc>(k);
    return Cand{readlane64(k.cost, 63), readlane64(k.excess, 63), readlane32(k.start, 63)};
}

// Candidate window: ordered by (cost, bytes, start); `end` rides along.
// Start and end are snapshot-local.
struct Key {
    uint64_t cost, bytes, start, end;
};

__device__ __forceinline__ Key key_none() { return Key{kNone, kNone, kNone, kNone}; }

__device__ __forceinline__ bool key_less(const Key& a, const Key& b) {
    if (a.cost != b.cost) return a.cost < b.cost;
    if (a.bytes != b.bytes) return a.bytes < b.bytes;
    return a.start < b.start;
}

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
    uint64_t x[kXN];    // keys R << 51 | P, or plain P in a tile with a huge block
    uint64_t xc[kXN];   // C
    uint16_t run[kXN];  // R, kept only in a tile with a huge block
    Sums wsum[kWaves];  // per-wavefront totals of the tile
    Sums hsum[4];       // per-wavefront totals of the halo
    Key slot[kWaves];   // answers of wavefronts that share a request
};

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
// Blocks past nt read as empty free blocks.  All loads are independent.
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
            kd[j] = in ? P.kind[t0 + i] : static_cast<uint8_t>(COOP_FREE);
        }
    }
}

__device__ __forceinline__ coop_window_t to_window(const Key& k, uint64_t S) {
    if (S == 0) return coop_window_t{0, 0, 0};
    if (k.start == kNone) return coop_window_t{kNone, kNone, kNone};
    return coop_window_t{k.start, k.end, k.cost};
}

__device__ __forceinline__ uint64_t lds_u64(const uint64_t* base, uint32_t byte_off) {
    return *reinterpret_cast<const uint64_t*>(reinterpret_cast<const char*>(base) + byte_off);
}

// Merge steps per lane for `total` merge elements over `lanes` lanes, rounded
// up to 2 mod 4: lanes then start about an odd number of keys apart, which
// spreads their first LDS reads over the banks.
__device__ __forceinline__ uint32_t merge_steps(uint32_t total, uint32_t lanes) {
    const uint32_t L = (total + lanes - 1) / lanes;
    return ((L + 1) & ~3u) + 2;
}

// Packed keys.  This lane's slice of the merge of the targets X[i] + Sc
// (starts i < nA) with the end keys X[1..nB]: merge steps [d, d + L).  Ties
// take the start first, so a start is taken when the head end key is the
// first one at or above its target: the shortest window from that start that
// reaches S bytes, valid when both ends have the same run id.  Steps past the
// lane's slice repeat work of the next lane (harmless: equal windows), and
// starts past nA are ignored.  X[nB + 1] must be all-ones, which no target
// exceeds: the end index never passes it.
__device__ __forceinline__ void merge_pass(const Smem& sm, uint32_t nA, uint32_t nB, uint32_t d,
                                           uint32_t L, uint64_t Sc, Cand& best,
                                           uint32_t& best_end) {
    // diagonal split: the number of starts among the first d merge elements
    uint32_t lo = d > nB ? d - nB : 0, hi = d < nA ? d : nA;
    while (lo < hi) {
        const uint32_t mid = (lo + hi) >> 1;
        // start `mid` precedes end key X[d - mid] iff its target is at or below it
        const bool before = sm.x[mid] + Sc <= sm.x[d - mid];
        lo = before ? mid + 1 : lo;
        hi = before ? hi : mid;
    }
    uint32_t pA = lo * 8u, pB = (d - lo + 1) * 8u;  // byte offsets of X[a] and of X[b + 1]
    const uint32_t endA = nA * 8u;
    uint64_t bc = kNone, bx = kNone;
    uint32_t bpa = kNone32, bpb = 0;
    for (uint32_t k = 0; k < L; k += 2) {
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            const uint64_t xa = lds_u64(sm.x, pA), kb = lds_u64(sm.x, pB);
            const uint64_t ca = lds_u64(sm.xc, pA), cb = lds_u64(sm.xc, pB);
            const uint64_t ta = xa + Sc;
            const bool takeA = ta <= kb;
            const bool same = (static_cast<uint32_t>(xa >> 32) ^ static_cast<uint32_t>(kb >> 32)) <
                              (1u << kRunShift);
            const bool valid = takeA & (pA < endA) & same;
            const uint64_t cost = cb - ca, ex = kb - ta;  // ex = bytes - S
            const bool better = valid & ((cost < bc) | ((cost == bc) & (ex < bx)));
            bc = better ? cost : bc;
            bx = better ? ex : bx;
            bpa = better ? pA : bpa;
            bpb = better ? pB : bpb;
            pA += takeA ? 8u : 0u;
            pB += takeA ? 0u : 8u;
        }
    }
    // Within a lane starts are met in increasing order, so strict comparison
    // kept the lowest start among equal (cost, bytes).
    const Cand c{bc, bx, bpa == kNone32 ? kNone32 : bpa / 8u};
    if (cand_less(c, best)) {
        best = c;
        best_end = bpb / 8u;
    }
}

// Plain prefixes (a tile with a huge block): starts g, g + lanes, ... below
// nA, each by two bisections: the end of its run, then its first end with
// at least S bytes.
__device__ __forceinline__ void plain_pass(const Smem& sm, uint32_t nA, uint32_t end, uint32_t g,
                                           uint32_t lanes, uint64_t S, Cand& best,
                                           uint32_t& best_end) {
    for (uint32_t i = g; i < nA; i += lanes) {
        const uint32_t run = sm.run[i];
        const uint64_t base = sm.x[i];
        uint32_t lo = i, hi = end;  // first k in [i, end) whose block closes the run
        while (lo < hi) {
            const uint32_t mid = (lo + hi) >> 1;
            if (sm.run[mid + 1] != run) hi = mid; else lo = mid + 1;
        }
        const uint32_t rend = lo;
        lo = i;
        hi = rend;
        while (lo < hi) {
            const uint32_t mid = (lo + hi) >> 1;
            if (sm.x[mid + 1] - base >= S) hi = mid; else lo = mid + 1;
        }
        if (lo < rend) {
            const Cand c{sm.xc[lo + 1] - sm.xc[i], sm.x[lo + 1] - base - S, i};
            if (cand_less(c, best)) {
                best = c;
                best_end = lo + 1;
            }
        }
    }
}

// Uniform lower bound: the first i in [lo, hi) with pred(i) (pred monotone),
// or hi.
template <typename Pred>
__device__ __forceinline__ uint32_t lower_bound(uint32_t lo, uint32_t hi, Pred pred) {
    while (lo < hi) {
        const uint32_t mid = (lo + hi) >> 1;
        if (pred(mid)) hi = mid; else lo = mid + 1;
    }
    return lo;
}

// The first start whose window cannot end inside the staged region [0, end]
// although its run reaches the region's end: starts i < nA with run id endrun
// and fewer than S bytes from i to the region end.  Such starts form a suffix.
__device__ __forceinline__ uint32_t pending_start(const Smem& sm, bool packed, uint32_t nA,
                                                  uint64_t xend, uint32_t endrun, uint64_t S,
                                                  uint64_t Sc) {
    if (packed) {
        // run id endrun and X[i] + Sc > X[end]
        const uint64_t by_run = static_cast<uint64_t>(endrun) << kValBits;
        const uint64_t by_bytes = xend >= Sc ? xend - Sc + 1 : 0;
        const uint64_t thr = by_run > by_bytes ? by_run : by_bytes;
        return lower_bound(0, nA, [&](uint32_t i) { return sm.x[i] >= thr; });
    }
    const uint32_t i0 = lower_bound(0, nA, [&](uint32_t i) { return sm.run[i] == endrun; });
    return lower_bound(i0, nA, [&](uint32_t i) { return xend - sm.x[i] < S; });
}

// Finishes the pending starts [cur, nA): all lie in the staged region's last
// run, which goes on at global block pos, where the run's prefixes are cq
// (bytes) and cc (cost).  The wavefront walks the run 64 blocks at a time
// (one per lane, wavefront prefix sums, the chunk kept in registers); each
// chunk resolves a prefix of the pending starts, 64 at a time, since their
// shortest ends are monotone.  Candidates fold into best / best_end (end
// snapshot-local).
__device__ void stream_pass(const Params& P, const Smem& sm, uint32_t cur, uint32_t nA, uint64_t pos,
                            uint64_t s0, uint64_t s1, uint64_t cq, uint64_t cc, uint64_t vmask,
                            uint64_t S, Cand& best, uint64_t& best_end) {
    const uint32_t lane = threadIdx.x & 63u;
    while (cur < nA && pos < s1) {
        const uint64_t left = s1 - pos;
        const uint32_t m = left < 64 ? static_cast<uint32_t>(left) : 64u;
        const bool in = lane < m;
        uint8_t kd = COOP_PINNED;
        uint64_t sz = 0, ct = 0;
        if (in) {
            kd = P.kind[pos + lane];
            sz = P.size[pos + lane];
            ct = P.cost[pos + lane];
        }
        const uint64_t pinned = __ballot(kd >= COOP_PINNED);
        const uint32_t fp = pinned ? static_cast<uint32_t>(__builtin_ctzll(pinned)) : 64u;  // <= m
        const bool valid = lane < fp;
        Sums s{valid ? sz : 0, valid && kd == COOP_EVICTABLE ? ct : 0, 0};
        wave_inclusive_sum(s);
        const uint64_t q = cq + s.q, c = cc + s.c;  // prefixes after this lane's block
        const uint32_t lastl = fp ? fp - 1 : 0;
        const uint64_t lastq = fp ? readlane64(q, lastl) : cq;
        const uint64_t lastc = fp ? readlane64(c, lastl) : cc;
        for (;;) {
            const uint32_t i = cur + lane;
            const bool act = i < nA;
            const uint32_t ii = act ? i : nA - 1;
            const uint64_t base = sm.x[ii] & vmask, cbase = sm.xc[ii];
            const bool ok = act && fp > 0 && lastq - base >= S;
            // the first chunk lane k < fp with q_k - base >= S
            uint32_t lo = 0, hi = lastl;
#pragma unroll
            for (int st = 0; st < 6; ++st) {
                const uint32_t mid = (lo + hi) >> 1;
                const bool ge = shfl64(q, mid) - base >= S;
                const bool more = lo < hi;
                hi = more && ge ? mid : hi;
                lo = more && !ge ? mid + 1 : lo;
            }
            const uint64_t qe = shfl64(q, lo), ce = shfl64(c, lo);
            if (ok) {
                const Cand cand{ce - cbase, qe - base - S, i};
                if (cand_less(cand, best)) {
                    best = cand;
                    best_end = (pos - s0) + lo + 1;
                }
            }
            const uint64_t res = __ballot(ok);
            const uint32_t n = ~res ? static_cast<uint32_t>(__builtin_ctzll(~res)) : 64u;
            cur += n;
            if (n < 64 || cur >= nA) break;
        }
        if (fp < m) break;  // the run closes inside this chunk
        cq = lastq;
        cc = lastc;
        pos += m;
    }
}

__device__ __forceinline__ void write_result(const Params& P, uint64_t q, uint64_t slot_index,
                                             bool direct, bool first_tile, Key k, uint64_t S) {
    if (direct) {
        P.out[q] = to_window(k, S);
    } else {
        Key* slot = P.part + q * P.pc + slot_index;
        if (!first_tile) {
            const Key prev = *slot;
            if (key_less(prev, k)) k = prev;
        }
        *slot = k;
    }
}

__global__ __launch_bounds__(kThreads, 4) void coop_window_search_kernel(Params P) {
    __shared__ Smem sm;
    const uint32_t tid = threadIdx.x;
    const uint32_t lane = tid & 63u;
    const uint32_t w = uniform(tid >> 6);
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
    // requests of this slice, and wavefronts per request
    const uint64_t K = (R - y + P.slices - 1) / P.slices;
    uint32_t wpr = 1;
    if (K < kWaves) {
        uint32_t k2 = 1;
        while (k2 < K) k2 <<= 1;
        wpr = kWaves / k2 < kMaxWpr ? kWaves / k2 : kMaxWpr;
    }

    for (uint64_t tau = p; tau < tau_end; ++tau) {
        const uint64_t t0 = s0 + (tau << kTileLog2);  // global index of the tile start
        const uint64_t tl = t0 - s0;                   // snapshot-local index of the tile start
        const uint32_t nt = static_cast<uint32_t>(s1 - t0 < kTile ? s1 - t0 : kTile);
        // halo blocks available after a full tile
        const uint64_t after = s1 - t0 - nt;
        const uint32_t hm = nt == kTile ? static_cast<uint32_t>(after < kHaloCap ? after : kHaloCap) : 0;

        // ---- 1. stage
        bool packed;
        uint32_t end;
        uint64_t xend, xcend;
        uint32_t endrun;
        {
            uint64_t sz[kItems], ct[kItems];
            uint8_t kd[kItems];
            load_items(P, t0, nt, sz, ct, kd);
            Sums h{0, 0, 0};
            if (tid < hm) {
                const uint64_t gp = t0 + kTile + tid;
                const uint8_t k = P.kind[gp];
                h.q = P.size[gp];
                const uint64_t c = P.cost[gp];
                h.c = k == COOP_EVICTABLE ? c : 0;
                h.r = (k >= COOP_PINNED ? 1u : 0u) + ((h.q >> 32) >> kBigHiLog2 ? 1u << 16 : 0u);
            }
            const Sums hown = h;
            // thread-local exclusive sums
            Sums t{0, 0, 0};
            uint32_t xr[kItems];
            uint32_t hi_or = 0;
#pragma unroll
            for (uint32_t j = 0; j < kItems; ++j) {
                const uint64_t s_j = sz[j];
                const uint64_t c_j = kd[j] == COOP_EVICTABLE ? ct[j] : 0;
                sz[j] = t.q;
                ct[j] = t.c;
                xr[j] = t.r;
                t.q += s_j;
                t.c += c_j;
                t.r += kd[j] >= COOP_PINNED ? 1u : 0u;
                hi_or |= static_cast<uint32_t>(s_j >> 32);
            }
            if (hi_or >> kBigHiLog2) t.r += 1u << 16;
            Sums wi = t;
            wave_inclusive_sum(wi);
            if (w < 4 && hm) wave_inclusive_sum(h);  // inclusive halo sums (waves 0..3)
            if (lane == 63) {
                sm.wsum[w] = wi;
                if (w < 4) sm.hsum[w] = h;
            }
            __syncthreads();
            // lanes 0..7: wavefront totals of the tile, 8..11: of the halo
            Sums bsum{0, 0, 0};
            if (lane < kWaves) bsum = sm.wsum[lane];
            else if (lane < kWaves + 4 && hm) bsum = sm.hsum[lane - kWaves];
            row_inclusive_sum(bsum);
            const Sums tile_tot = readlane(bsum, kWaves - 1);
            const Sums all_tot = readlane(bsum, kWaves + 3);
            Sums carry = readlane(bsum, w ? w - 1 : 0);
            if (w == 0) carry = Sums{0, 0, 0};
            // halo wavefront w < 4: tile total + the earlier halo wavefronts
            const Sums hcarry = readlane(bsum, kWaves - 1 + (w < 4 ? w : 0));
            // thread exclusive = block carry + wavefront inclusive - own total
            const Sums base{carry.q + wi.q - t.q, carry.c + wi.c - t.c, carry.r + wi.r - t.r};

            packed = (tile_tot.r >> 16) == 0;
            const bool use_halo = packed && hm && (all_tot.r >> 16) == 0;
            end = use_halo ? kTile + hm : nt;
            const Sums et = use_halo ? all_tot : tile_tot;
            endrun = et.r & 0xffffu;
            xend = packed ? (static_cast<uint64_t>(endrun) << kValBits) | et.q : et.q;
            xcend = et.c;

            // LDS: boundaries [0, end) by their owners, end and the sentinel by the last thread
            const uint32_t i0 = tid * kItems;
            const bool all_mine = i0 + kItems <= end;
            if (packed) {
                uint64_t xv[kItems], cv[kItems];
#pragma unroll
                for (uint32_t j = 0; j < kItems; ++j) {
                    const uint64_t pq = base.q + sz[j];
                    const uint32_t rr = base.r + xr[j];
                    xv[j] = pq | (static_cast<uint64_t>(rr) << kValBits);
                    cv[j] = base.c + ct[j];
                }
                if (all_mine) {
#pragma unroll
                    for (uint32_t j = 0; j < kItems; j += 2) {
                        *reinterpret_cast<ulonglong2*>(&sm.x[i0 + j]) = ulonglong2{xv[j], xv[j + 1]};
                        *reinterpret_cast<ulonglong2*>(&sm.xc[i0 + j]) = ulonglong2{cv[j], cv[j + 1]};
                    }
                } else {
#pragma unroll
                    for (uint32_t j = 0; j < kItems; ++j) {
                        if (i0 + j < end) {
                            sm.x[i0 + j] = xv[j];
                            sm.xc[i0 + j] = cv[j];
                        }
                    }
                }
                if (use_halo && tid < hm) {
                    // halo boundary kTile + tid: carry + wavefront inclusive - own block
                    const uint64_t pq = hcarry.q + h.q - hown.q;
                    const uint32_t rr = hcarry.r + h.r - hown.r;
                    sm.x[kTile + tid] = pq | (static_cast<uint64_t>(rr) << kValBits);
                    sm.xc[kTile + tid] = hcarry.c + h.c - hown.c;
                }
            } else {
#pragma unroll
                for (uint32_t j = 0; j < kItems; ++j) {
                    if (i0 + j < end) {
                        sm.x[i0 + j] = base.q + sz[j];
                        sm.xc[i0 + j] = base.c + ct[j];
                        sm.run[i0 + j] = static_cast<uint16_t>(base.r + xr[j]);
                    }
                }
            }
            if (tid == kThreads - 1) {
                sm.x[end] = xend;
                sm.xc[end] = xcend;
                sm.run[end] = static_cast<uint16_t>(endrun);
                sm.x[end + 1] = kNone;  // sentinel end key
            }
            __syncthreads();
        }
        const uint64_t vmask = packed ? kValMask : kNone;
        const bool open = t0 + end < s1;  // the region's last run may go on

        // ---- 2./3. requests: wavefront task vw = request (vw / wpr), slice (vw % wpr)
        const uint64_t tasks = K * wpr;
        uint64_t S_next = 0;
        if (w < tasks) S_next = P.req_size[q0 + y + (w / wpr) * P.slices];
        for (uint64_t vw = w; vw < tasks; vw += kWaves) {
            const uint64_t rl = vw / wpr;
            const uint32_t sl = static_cast<uint32_t>(vw % wpr);
            const uint64_t q = q0 + y + rl * P.slices;
            const uint64_t S = S_next;
            if (vw + kWaves < tasks) S_next = P.req_size[q0 + y + ((vw + kWaves) / wpr) * P.slices];
            Cand best = cand_none();
            uint64_t best_end = 0;
            if (S != 0 && nt != 0) {
                const uint64_t Sc = S < (1ull << kValBits) ? S : (1ull << kValBits);
                const uint32_t lanes = 64u * wpr;
                const uint32_t gl = sl * 64u + lane;
                uint32_t e32 = 0;
                if (packed) {
                    const uint32_t total = nt + end;
                    const uint32_t L = merge_steps(total, lanes);
                    const uint32_t d = gl * L < total ? gl * L : total;
                    merge_pass(sm, nt, end, d, L, Sc, best, e32);
                } else {
                    plain_pass(sm, nt, end, gl, lanes, S, best, e32);
                }
                best_end = tl + e32;
                if (open && sl == 0) {
                    const uint32_t cur = pending_start(sm, packed, nt, xend, endrun, S, Sc);
                    if (cur < nt)
                        stream_pass(P, sm, cur, nt, t0 + end, s0, s1, xend & vmask, xcend, vmask, S,
                                    best, best_end);
                }
            }
            const Cand m = wave_argmin(best);
            Key k = key_none();
            if (m.start != kNone32) {
                const uint64_t won = __ballot(best.start == m.start);
                const uint64_t e = readlane64(best_end, static_cast<uint32_t>(__builtin_ctzll(won)));
                k = Key{m.cost, m.excess + S, tl + m.start, e};
            }
            if (lane == 0) {
                if (wpr == 1) write_result(P, q, g, direct, tau == p, k, S);
                else sm.slot[vw] = k;
            }
        }
        if (wpr > 1) {
            __syncthreads();
            if (tid < K) {
                const uint64_t q = q0 + y + static_cast<uint64_t>(tid) * P.slices;
                Key k = sm.slot[tid * wpr];
                for (uint32_t u = 1; u < wpr; ++u) {
                    const Key o = sm.slot[tid * wpr + u];
                    if (key_less(o, k)) k = o;
                }
                write_result(P, q, g, direct, tau == p, k, P.req_size[q]);
            }
        }
        __syncthreads();  // LDS reused by the next tile
    }
    if (direct) return;

    // ---- combine the partial keys of the snapshot's workgroups
    __threadfence();
    __syncthreads();
    __shared__ uint32_t last_flag;
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
        last_flag = last;
    }
    __syncthreads();
    if (!last_flag) return;
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
