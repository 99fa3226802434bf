// The sliding-window search with real-valued heuristics (Coop, section 3.3:
// h(t) = c(t) / s(t), projected cost over staleness, a real number).
//
// Each evictable block carries h as a binary64 value, and a window costs the
// exact real sum of its h values: every h is rounded once to a multiple of
// 2^-64 (to nearest, ties to even; exact for h >= 2^-12) and the sums are
// taken in 128-bit fixed point (64 fraction bits).  Integer sums are
// associative, so the window that wins does not depend on how the GPU
// splits the work.  Ranking as in the integer search: least cost, then
// fewest bytes, then lowest start.
//
// Four launches:
//   1. real_tile_kernel: tiles of 2048 blocks, each writes the tile-local
//      exclusive prefix sums of bytes (u64), fixed-point cost (u128) and
//      pinned count (u16) of every block, and the tile's totals; a tile
//      holding a block with an invalid h flags its total (bit 63 of the
//      pinned count, which never exceeds 2048).  Prefix index num_blocks
//      (the end of the batch) belongs to the last tile, so there are
//      floor(num_blocks / 2048) + 1 tiles.
//   2. real_offsets_kernel: one workgroup turns the tile totals into
//      exclusive tile offsets and writes the status word (bit 0 when any
//      tile was flagged).  The global prefix at index x is then
//      offset[x >> 11] + local[x].  Prefixes run over the whole batch
//      (snapshots are not reset): window sums are differences of two
//      prefixes of one snapshot, so they come out the same.
//   3. real_search_kernel: workgroup (group, part) takes up to 16
//      consecutive requests and one of `parts` equal slices of each
//      request's snapshot.  It walks its slice in chunks of 2048 starts;
//      for each chunk it stages packed byte/pinned-count keys and cost
//      prefixes of up to 2561 indices (the chunk and the blocks after it)
//      in LDS, then runs every request of the group that shares the
//      snapshot as a merge path, each on its own wavefronts (see the
//      kernel).  A window [i, k) is valid
//      iff it holds no pinned block; its cost is C[k] - C[i].  Each
//      wavefront's minimum is kept per request in LDS; their least goes to
//      the request's partial slot.
//   4. real_reduce_kernel: one thread per request takes the least of its
//      `parts` partial slots and writes the result, the exact cost both as
//      two 64-bit words and rounded to the nearest binary64.

#include <hip/hip_runtime.h>

#include <stdint.h>

#include "coop.h"
#include "coop_host.h"

namespace {

constexpr uint32_t kThreads = 256;
constexpr uint32_t kWaves = kThreads / 64;
constexpr uint32_t kItems = 8;
constexpr uint32_t kTileLog2 = 11;
constexpr uint32_t kTile = 1u << kTileLog2;  // blocks per prefix tile
static_assert(kTile == kThreads * kItems, "tile = threads x items");
constexpr uint32_t kChunk = kThreads * kItems;  // starts per staged chunk
constexpr uint32_t kStage = kChunk + kChunk / 4;  // staged prefix indices beyond a chunk's start
// Packed staged keys: Y(x) = (pinned count since the chunk start) * 2^51 +
// (bytes since the chunk start).  With fewer than 4096 staged indices and
// staged bytes plus S below 2^51, Y(x) >= Y(i) + S holds exactly when x is
// past the run of i or [i, x) holds S bytes, and Y(x) - Y(i) < 2^51 exactly
// when [i, x) holds no pinned block (it is then the window's byte count).
constexpr uint32_t kPackBits = 51;
constexpr uint64_t kPackOne = 1ull << kPackBits;
static_assert(kStage < (1u << (63 - kPackBits)), "packed keys stay below 2^63");
constexpr uint64_t kEndKey = ~0ull;  // above every target: stops every merge
// Every lane of a request walks the same number of merge steps, at most this
// many (one wavefront's share of a chunk's merge); a lane whose slice ends
// earlier goes on into its neighbour's (the same windows again) or past the
// end keys, into this many more sentinel keys.
constexpr uint32_t kPadSteps = 80;
static_assert(kPadSteps >= ((kChunk + kStage + 63) / 64 + 1) / 4 * 4 + 2,
              "padding covers a wavefront's slice, rounded up to 2 mod 4");
constexpr uint32_t kSThreads = 512;             // threads of a search workgroup
constexpr uint32_t kSWaves = kSThreads / 64;
constexpr uint32_t kStageBatch = 5;             // staged indices per thread whose loads go together
constexpr uint32_t kMaxGroup = 16;              // requests per search workgroup
constexpr uint32_t kTargetGroups = 4096;        // search workgroups aimed for
constexpr uint64_t kResidentUnits = 512;        // search workgroups the chip holds at once
constexpr uint32_t kMaxParts = 1024;
constexpr uint32_t kOffsetThreads = 1024;
constexpr uint64_t kNone = ~0ull;
constexpr uint32_t kErrValue = 1;

struct U128 {
    uint64_t lo, hi;
};

__device__ __forceinline__ U128 add128(U128 a, U128 b) {
    U128 r;
    r.lo = a.lo + b.lo;
    r.hi = a.hi + b.hi + (r.lo < a.lo ? 1u : 0u);
    return r;
}

// a - b as one chain of subtract-with-borrow over the four 32-bit words:
// four instructions, where the compiler's form (a 64-bit difference of each
// half, the borrow taken from a compare and a select) took eight in the
// merge step.
__device__ __forceinline__ U128 sub128(U128 a, U128 b) {
    uint32_t w0 = static_cast<uint32_t>(a.lo), w1 = static_cast<uint32_t>(a.lo >> 32);
    uint32_t w2 = static_cast<uint32_t>(a.hi), w3 = static_cast<uint32_t>(a.hi >> 32);
    asm volatile("v_sub_co_u32 %0, vcc, %0, %4\n\t"
                 "v_subb_co_u32 %1, vcc, %1, %5, vcc\n\t"
                 "v_subb_co_u32 %2, vcc, %2, %6, vcc\n\t"
                 "v_subb_co_u32 %3, vcc, %3, %7, vcc"
                 : "+v"(w0), "+v"(w1), "+v"(w2), "+v"(w3)
                 : "v"(static_cast<uint32_t>(b.lo)), "v"(static_cast<uint32_t>(b.lo >> 32)),
                   "v"(static_cast<uint32_t>(b.hi)), "v"(static_cast<uint32_t>(b.hi >> 32))
                 : "vcc");
    return U128{(static_cast<uint64_t>(w1) << 32) | w0, (static_cast<uint64_t>(w3) << 32) | w2};
}

// h (binary64) in units of 2^-64, rounded to nearest, ties to even.  False
// for NaN, infinities, negative values other than -0 and values >= 2^64.
// h = m * 2^(e - 1075) for a normal number, so h * 2^64 = m * 2^(e - 1011).
__device__ __forceinline__ bool to_fixed(double h, U128& q) {
    const uint64_t bits = static_cast<uint64_t>(__double_as_longlong(h));
    const uint32_t e = static_cast<uint32_t>(bits >> 52) & 0x7ffu;
    const uint64_t frac = bits & ((1ull << 52) - 1);
    q = U128{0, 0};
    if (bits >> 63) return e == 0 && frac == 0;
    if (e >= 1023 + 64) return false;  // also infinities and NaN (e == 2047)
    if (e == 0) return true;           // subnormal: far below half a unit
    const uint64_t m = frac | (1ull << 52);
    const int s = static_cast<int>(e) - 1011;
    if (s >= 64) {
        q.hi = m << (s - 64);  // s <= 75: m << 11 < 2^64
    } else if (s > 0) {
        q.lo = m << s;
        q.hi = m >> (64 - s);
    } else if (s == 0) {
        q.lo = m;
    } else if (s > -64) {
        const int r = -s;
        uint64_t v = m >> r;
        const uint64_t rem = m & ((1ull << r) - 1), half = 1ull << (r - 1);
        if (rem > half || (rem == half && (v & 1))) ++v;
        q.lo = v;
    }  // else m < 2^53 <= half a unit times 2^-10: zero
    return true;
}

__device__ __forceinline__ uint64_t bit128(U128 v, int j) {
    return j >= 64 ? (v.hi >> (j - 64)) & 1 : (v.lo >> j) & 1;
}

// A fixed-point value to the nearest binary64, ties to even.
__device__ __forceinline__ double to_real(U128 v) {
    if (v.hi == 0 && v.lo < (1ull << 53)) return ldexp(static_cast<double>(v.lo), -64);
    const int lz = v.hi ? __clzll(v.hi) : 64 + __clzll(v.lo);
    int sh = (127 - lz) - 52;  // bits below the 53 kept, >= 1
    uint64_t m = sh >= 64 ? v.hi >> (sh - 64) : (v.lo >> sh) | (v.hi << (64 - sh));
    const bool round = bit128(v, sh - 1) != 0;
    bool sticky;
    if (sh - 1 >= 64)
        sticky = v.lo != 0 || (v.hi & ((1ull << (sh - 1 - 64)) - 1)) != 0;
    else
        sticky = (v.lo & ((1ull << (sh - 1)) - 1)) != 0;
    if (round && (sticky || (m & 1))) {
        ++m;
        if (m == (1ull << 53)) {
            m >>= 1;
            ++sh;
        }
    }
    return ldexp(static_cast<double>(m), sh - 64);
}

__device__ __forceinline__ uint64_t shfl_up64(uint64_t v, int d) {
    const uint32_t lo = __shfl_up(static_cast<uint32_t>(v), d, 64);
    const uint32_t hi = __shfl_up(static_cast<uint32_t>(v >> 32), d, 64);
    return (static_cast<uint64_t>(hi) << 32) | lo;
}

__device__ __forceinline__ uint64_t shfl_xor64(uint64_t v, int m) {
    const uint32_t lo = __shfl_xor(static_cast<uint32_t>(v), m, 64);
    const uint32_t hi = __shfl_xor(static_cast<uint32_t>(v >> 32), m, 64);
    return (static_cast<uint64_t>(hi) << 32) | lo;
}

// Prefix triple: bytes, fixed-point cost, pinned count.
struct Tri {
    uint64_t p;
    U128 c;
    uint64_t r;
};

__device__ __forceinline__ Tri add_tri(const Tri& a, const Tri& b) {
    return Tri{a.p + b.p, add128(a.c, b.c), a.r + b.r};
}

// Inclusive scan of a Tri over the wavefront.
__device__ __forceinline__ Tri wave_scan(Tri v) {
    const uint32_t lane = threadIdx.x & 63u;
    for (int d = 1; d < 64; d <<= 1) {
        const Tri x{shfl_up64(v.p, d), U128{shfl_up64(v.c.lo, d), shfl_up64(v.c.hi, d)},
                    shfl_up64(v.r, d)};
        if (lane >= static_cast<uint32_t>(d)) v = add_tri(v, x);
    }
    return v;
}

constexpr uint64_t kBadTile = 1ull << 63;  // in a tile total's pinned count

// Stage 1.  Tile t covers prefix indices [t * 2048, min((t + 1) * 2048, n + 1)).
// Each thread holds 8 consecutive blocks: 16-byte loads of sizes and h and
// an 8-byte load of kinds when the block lies wholly inside the batch and
// the inputs are aligned, single loads otherwise; the prefixes go out as
// 16-byte stores the same way.
__global__ __launch_bounds__(kThreads, 4) void real_tile_kernel(
    const uint64_t* __restrict__ size, const double* __restrict__ h,
    const uint8_t* __restrict__ kind, uint64_t n, uint64_t num_tiles, uint64_t* __restrict__ pl,
    uint64_t* __restrict__ cl_lo, uint64_t* __restrict__ cl_hi, uint16_t* __restrict__ rl,
    Tri* __restrict__ tot) {
    __shared__ Tri wtot[kWaves];
    __shared__ uint32_t wbad[kWaves];
    const uint32_t tid = threadIdx.x, lane = tid & 63u, w = tid >> 6;
    const bool aligned = ((reinterpret_cast<uintptr_t>(size) | reinterpret_cast<uintptr_t>(h)) &
                          15u) == 0 && (reinterpret_cast<uintptr_t>(kind) & 7u) == 0;
    for (uint64_t t = blockIdx.x; t < num_tiles; t += gridDim.x) {
        const uint64_t base = t * kTile + tid * kItems;
        const bool full = base + kItems <= n;
        uint64_t sz[kItems];
        double hv[kItems];
        uint8_t kd[kItems];
        if (full && aligned) {
            const ulonglong2* s2 = reinterpret_cast<const ulonglong2*>(size + base);
            const double2* h2 = reinterpret_cast<const double2*>(h + base);
#pragma unroll
            for (uint32_t v = 0; v < kItems / 2; ++v) {
                const ulonglong2 a = s2[v];
                const double2 c = h2[v];
                sz[2 * v] = a.x; sz[2 * v + 1] = a.y;
                hv[2 * v] = c.x; hv[2 * v + 1] = c.y;
            }
            const uint2 k8 = *reinterpret_cast<const uint2*>(kind + base);
#pragma unroll
            for (uint32_t u = 0; u < 4; ++u) {
                kd[u] = static_cast<uint8_t>(k8.x >> (8 * u));
                kd[u + 4] = static_cast<uint8_t>(k8.y >> (8 * u));
            }
        } else {
#pragma unroll
            for (uint32_t u = 0; u < kItems; ++u) {
                const uint64_t k = base + u;
                const bool in = k < n;
                sz[u] = in ? size[k] : 0;
                hv[u] = in ? h[k] : 0.0;
                kd[u] = in ? kind[k] : static_cast<uint8_t>(COOP_FREE);
            }
        }
        U128 cq[kItems];
        uint32_t pin = 0;  // bit u: item u pinned
        bool bad = false;
#pragma unroll
        for (uint32_t u = 0; u < kItems; ++u) {
            cq[u] = U128{0, 0};
            if (kd[u] >= COOP_PINNED) pin |= 1u << u;
            if (kd[u] == COOP_EVICTABLE && !to_fixed(hv[u], cq[u])) bad = true;
        }
        const bool wave_bad = __ballot(bad) != 0;
        Tri mine{0, U128{0, 0}, 0};
#pragma unroll
        for (uint32_t u = 0; u < kItems; ++u) {
            mine.p += sz[u];
            mine.c = add128(mine.c, cq[u]);
        }
        mine.r = __popc(pin);
        const Tri inc = wave_scan(mine);
        if (lane == 63) {
            wtot[w] = inc;
            wbad[w] = wave_bad ? 1u : 0u;
        }
        __syncthreads();
        Tri run{0, U128{0, 0}, 0};
        for (uint32_t v = 0; v < w; ++v) run = add_tri(run, wtot[v]);
        Tri all = run;
        uint32_t tile_bad = 0;
        for (uint32_t v = w; v < kWaves; ++v) all = add_tri(all, wtot[v]);
        for (uint32_t v = 0; v < kWaves; ++v) tile_bad |= wbad[v];
        if (tile_bad) all.r |= kBadTile;
        __syncthreads();
        run = add_tri(run, Tri{inc.p - mine.p, sub128(inc.c, mine.c), inc.r - mine.r});
        // each pair of prefixes goes out as soon as it is known, so that few
        // of them are held in registers at once
        if (full) {  // the workspace arrays are 256-byte aligned
            uint32_t rw[kItems / 2];
#pragma unroll
            for (uint32_t v = 0; v < kItems / 2; ++v) {
                const Tri a = run;
                run.p += sz[2 * v];
                run.c = add128(run.c, cq[2 * v]);
                run.r += (pin >> (2 * v)) & 1u;
                reinterpret_cast<ulonglong2*>(pl + base)[v] = ulonglong2{a.p, run.p};
                reinterpret_cast<ulonglong2*>(cl_lo + base)[v] = ulonglong2{a.c.lo, run.c.lo};
                reinterpret_cast<ulonglong2*>(cl_hi + base)[v] = ulonglong2{a.c.hi, run.c.hi};
                rw[v] = static_cast<uint32_t>(a.r & 0xffffu) | (static_cast<uint32_t>(run.r & 0xffffu) << 16);
                run.p += sz[2 * v + 1];
                run.c = add128(run.c, cq[2 * v + 1]);
                run.r += (pin >> (2 * v + 1)) & 1u;
            }
            *reinterpret_cast<uint4*>(rl + base) = make_uint4(rw[0], rw[1], rw[2], rw[3]);
        } else {
#pragma unroll
            for (uint32_t u = 0; u < kItems; ++u) {
                const uint64_t k = base + u;
                if (k <= n) {
                    pl[k] = run.p;
                    cl_lo[k] = run.c.lo;
                    cl_hi[k] = run.c.hi;
                    rl[k] = static_cast<uint16_t>(run.r);
                }
                run.p += sz[u];
                run.c = add128(run.c, cq[u]);
                run.r += (pin >> u) & 1u;
            }
        }
        if (tid == 0) tot[t] = all;
    }
}

// Stage 2: exclusive tile offsets, one workgroup; each thread sums a run of
// consecutive tiles, the runs are scanned, then each thread writes its
// tiles' offsets.
__global__ __launch_bounds__(kOffsetThreads) void real_offsets_kernel(const Tri* __restrict__ tot,
                                                                      uint64_t num_tiles,
                                                                      Tri* __restrict__ off,
                                                                      uint32_t* __restrict__ status) {
    __shared__ Tri wtot[kOffsetThreads / 64];
    const uint32_t tid = threadIdx.x, lane = tid & 63u, w = tid >> 6;
    const uint64_t per = (num_tiles + kOffsetThreads - 1) / kOffsetThreads;
    const uint64_t t0 = tid * per < num_tiles ? tid * per : num_tiles;
    const uint64_t t1 = t0 + per < num_tiles ? t0 + per : num_tiles;
    Tri mine{0, U128{0, 0}, 0};
    uint64_t flags = 0;
    for (uint64_t t = t0; t < t1; ++t) {
        Tri x = tot[t];
        flags |= x.r;
        x.r &= ~kBadTile;
        mine = add_tri(mine, x);
    }
    // the status word: bit 0 when any tile held an invalid h
    const int any_bad = __syncthreads_or((flags & kBadTile) != 0);
    if (tid == 0) *status = any_bad ? kErrValue : 0u;
    const Tri inc = wave_scan(mine);
    if (lane == 63) wtot[w] = inc;
    __syncthreads();
    Tri run{0, U128{0, 0}, 0};
    for (uint32_t v = 0; v < w; ++v) run = add_tri(run, wtot[v]);
    run = add_tri(run, Tri{inc.p - mine.p, sub128(inc.c, mine.c), inc.r - mine.r});
    for (uint64_t t = t0; t < t1; ++t) {
        Tri x = tot[t];
        x.r &= ~kBadTile;
        off[t] = run;
        run = add_tri(run, x);
    }
}

struct Prefix {
    const uint64_t* pl;
    const uint64_t* cl_lo;
    const uint64_t* cl_hi;
    const uint16_t* rl;
    const Tri* off;

    __device__ __forceinline__ uint64_t P(uint64_t x) const { return off[x >> kTileLog2].p + pl[x]; }
    __device__ __forceinline__ uint64_t R(uint64_t x) const { return off[x >> kTileLog2].r + rl[x]; }
    __device__ __forceinline__ U128 C(uint64_t x) const {
        return add128(off[x >> kTileLog2].c, U128{cl_lo[x], cl_hi[x]});
    }
};

// A partial result: exact cost, bytes, window [start, end) in batch indices
// (in snapshot-local indices once to_local has run; the order of candidates
// of one request is the same either way).
struct Best {
    uint64_t c_lo, c_hi, bytes, start, end;
};

__device__ __forceinline__ Best to_local(Best m, uint64_t s0) {
    if (m.start != ~0ull) {
        m.start -= s0;
        m.end -= s0;
    }
    return m;
}

__device__ __forceinline__ Best best_none() { return Best{kNone, kNone, kNone, kNone, kNone}; }

__device__ __forceinline__ bool best_less(const Best& a, const Best& b) {
    if (a.c_hi != b.c_hi) return a.c_hi < b.c_hi;
    if (a.c_lo != b.c_lo) return a.c_lo < b.c_lo;
    if (a.bytes != b.bytes) return a.bytes < b.bytes;
    return a.start < b.start;
}

// The snapshot b with req_off[b] <= r < req_off[b + 1], found by a whole
// wavefront (every lane active, same arguments): the first i in [1, B) with
// req_off[i] > r, minus one, by 64 probes a round, so a thousand snapshots take two rounds of loads instead of ten
// dependent ones.  Probes stay below B (malformed offsets give some b in
// [0, B), never an access outside req_off).
__device__ __forceinline__ uint64_t wave_owner(const uint64_t* req_off, uint64_t num_segments,
                                               uint64_t r, uint32_t lane) {
    uint64_t lo = 1, hi = num_segments;  // the first such i lies in [lo, hi] (hi: none)
    while (hi - lo > 64) {
        const uint64_t step = (hi - lo + 63) >> 6;
        const uint64_t i = lo + lane * step;
        const uint64_t m = __ballot(i >= hi || req_off[i] > r);
        const uint32_t f = m ? static_cast<uint32_t>(__builtin_ctzll(m)) : 64u;
        const uint64_t nhi = f < 64 ? lo + f * step : hi;
        lo = f ? lo + (f - 1) * step + 1 : lo;
        hi = nhi < hi ? nhi : hi;
    }
    const uint64_t m = __ballot(lo + lane >= hi || req_off[lo + lane] > r);
    return (m ? lo + static_cast<uint64_t>(__builtin_ctzll(m)) : hi) - 1;
}

struct SearchArgs {
    const uint64_t* seg;
    uint64_t num_segments;
    const uint64_t* req_sizes;
    const uint64_t* req_off;
    uint64_t num_requests;
    uint64_t group;     // requests per workgroup
    uint64_t parts;     // slices per snapshot
    uint64_t units;     // number of (group, part) work units
    Best* slots;        // num_requests * parts
};

// The least Best of the wavefront (every lane gets it).
__device__ __forceinline__ Best wave_min(Best v) {
    for (int o = 32; o >= 1; o >>= 1) {
        const Best x{shfl_xor64(v.c_lo, o), shfl_xor64(v.c_hi, o), shfl_xor64(v.bytes, o),
                     shfl_xor64(v.start, o), shfl_xor64(v.end, o)};
        if (best_less(x, v)) v = x;
    }
    return v;
}

// The same minimum over windows that the merge path found in the chunk
// starting at c0: their bytes are below 2^51 and their starts lie in
// [c0, c0 + 2^12), so (bytes, start) orders as the one word
// bytes << 12 | (start - c0), and the end need not travel: it is read from a
// lane that holds the winning start (lanes holding the same start hold the
// same window).
constexpr uint32_t kChunkBits = 12;
static_assert(kChunk <= (1u << kChunkBits), "chunk offsets fit the start field");
static_assert(kPackBits + kChunkBits < 64, "a packed key stays below the empty value");

__device__ __forceinline__ Best wave_min_chunk(const Best& v, uint64_t c0) {
    uint64_t c_lo = v.c_lo, c_hi = v.c_hi;
    uint64_t key = v.start == kNone ? kNone : (v.bytes << kChunkBits) | (v.start - c0);
    for (int o = 32; o >= 1; o >>= 1) {
        const uint64_t xl = shfl_xor64(c_lo, o), xh = shfl_xor64(c_hi, o), xk = shfl_xor64(key, o);
        const bool less = xh < c_hi || (xh == c_hi && (xl < c_lo || (xl == c_lo && xk < key)));
        c_lo = less ? xl : c_lo;
        c_hi = less ? xh : c_hi;
        key = less ? xk : key;
    }
    if (key == kNone) return best_none();
    const uint64_t start = c0 + (key & ((1ull << kChunkBits) - 1));
    const uint64_t won = __ballot(v.start == start);
    const uint32_t wl = static_cast<uint32_t>(__builtin_ctzll(won));
    const uint64_t end =
        (static_cast<uint64_t>(static_cast<uint32_t>(__builtin_amdgcn_readlane(
             static_cast<int>(v.end >> 32), static_cast<int>(wl)))) << 32) |
        static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(v.end), static_cast<int>(wl)));
    return Best{c_lo, c_hi, key >> kChunkBits, start, end};
}

// Starts [i, i_end) of one snapshot (ending at nend), walked by one thread
// from the global prefixes alone: the first start's shortest end by
// bisection, the later ones by walking on.  pred(x): x is past the run of
// the start or [start, x) holds S bytes; it is monotone in x, and its first
// x is the end of the shortest window (or of one that crosses a pinned
// block, which is then invalid).
__device__ void walk_global(const Prefix& pf, uint64_t i, uint64_t i_end, uint64_t nend,
                            uint64_t S, Best& mine) {
    uint64_t k = kNone;
    for (; i < i_end; ++i) {
        const uint64_t pi = pf.P(i), ri = pf.R(i);
        auto pred = [&](uint64_t x) { return pf.R(x) != ri || pf.P(x) - pi >= S; };
        uint64_t x;
        if (k == kNone) {
            if (!pred(nend)) return;  // no window from i, nor from any later start
            uint64_t lo = i + 1, hi = nend;
            while (lo < hi) {
                const uint64_t mid = (lo + hi) >> 1;
                if (pred(mid)) hi = mid; else lo = mid + 1;
            }
            x = lo;
        } else {
            x = k > i + 1 ? k : i + 1;
            while (x <= nend && !pred(x)) ++x;
            if (x > nend) return;
        }
        k = x;
        if (pf.R(x) == ri) {
            const U128 cost = sub128(pf.C(x), pf.C(i));
            const Best cand{cost.lo, cost.hi, pf.P(x) - pi, i, x};
            if (best_less(cand, mine)) mine = cand;
        }
    }
}

// The merge path of NR requests over one staged chunk, interleaved so that
// their chains of LDS reads overlap: targets Y[i] + S (starts i < nA) against
// end keys Y[1..nB], split over `lanes` lanes (this one is lane gl).  Each
// lane bisects its diagonal (a fixed 12 rounds: the range is at most
// nA + 1 <= 2049) and walks the same number of steps; a
// start meets, when it is merged, the first end key at or above its target,
// the end of its shortest window, and is scored on the spot (valid iff the
// keys differ by less than 2^51: no pinned block between).  nB may be the
// end key that takes in the first pinned block after the chunk, by which
// every start is merged; a lane past nA + nB only moves its end index on
// through the staged keys and the end-key padding, as no start past nA is
// taken.  mine[r] receives the lane's least window (batch indices).
template <int NR>
__device__ __forceinline__ void merge_requests(const uint64_t* Y, const U128* Cr, uint32_t nA,
                                               uint32_t nB, const uint64_t (&S)[NR], uint64_t c0,
                                               uint32_t gl, uint32_t lanes, Best (&mine)[NR]) {
    const uint32_t M = nA + nB;
    // Two interleaved merges: slices rounded up to 2 mod 4 keys, so that
    // lanes start an odd number of keys apart, spread over the LDS banks
    // (large pools 1.15 -> 1.01 ms per call; for one merge a lane it lost).
    const uint32_t L0 = (M + lanes - 1) / lanes;
    const uint32_t Ls = NR == 2 ? ((L0 + 1) & ~3u) + 2 : L0;
    const uint32_t d = gl * Ls < M ? gl * Ls : M;
    uint32_t lo[NR], hi[NR];
#pragma unroll
    for (int r = 0; r < NR; ++r) {
        lo[r] = d > nB ? d - nB : 0;
        hi[r] = d < nA ? d : nA;
    }
#pragma unroll
    for (int it = 0; it < 12; ++it) {
#pragma unroll
        for (int r = 0; r < NR; ++r) {
            if (lo[r] < hi[r]) {
                const uint32_t mid = (lo[r] + hi[r]) >> 1;
                // start mid goes before end key Y[d - mid] iff its target is at or below it
                if (Y[mid] + S[r] <= Y[d - mid]) lo[r] = mid + 1; else hi[r] = mid;
            }
        }
    }
    uint32_t pa[NR], pb[NR], bs[NR], be[NR];
    uint64_t bc_lo[NR], bc_hi[NR], bd[NR];
#pragma unroll
    for (int r = 0; r < NR; ++r) {
        pa[r] = lo[r];
        pb[r] = d - lo[r] + 1;  // next start, next end key index
        bc_lo[r] = bc_hi[r] = bd[r] = kNone;
        bs[r] = ~0u;
        be[r] = 0;
    }
    for (uint32_t t = 0; t < Ls; ++t) {  // the same count in every lane
#pragma unroll
        for (int r = 0; r < NR; ++r) {
            const uint64_t ya = Y[pa[r]], yb = Y[pb[r]];
            const U128 ca = Cr[pa[r]], cb = Cr[pb[r]];
            const bool takeA = (pa[r] < nA) & (ya + S[r] <= yb);
            const uint64_t D = yb - ya;
            const bool valid = takeA & (D < kPackOne);
            const U128 cost = sub128(cb, ca);
            const bool better =
                valid & ((cost.hi < bc_hi[r]) |
                         ((cost.hi == bc_hi[r]) &
                          ((cost.lo < bc_lo[r]) | ((cost.lo == bc_lo[r]) & (D < bd[r])))));
            bc_lo[r] = better ? cost.lo : bc_lo[r];
            bc_hi[r] = better ? cost.hi : bc_hi[r];
            bd[r] = better ? D : bd[r];
            bs[r] = better ? pa[r] : bs[r];
            be[r] = better ? pb[r] : be[r];
            pa[r] += takeA ? 1u : 0u;
            pb[r] += takeA ? 0u : 1u;
        }
    }
    // within a lane starts come in increasing order, so strict comparison kept
    // the lowest start among equal (cost, bytes)
#pragma unroll
    for (int r = 0; r < NR; ++r)
        if (bs[r] != ~0u) mine[r] = Best{bc_lo[r], bc_hi[r], bd[r], c0 + bs[r], c0 + be[r]};
}

// Stage 3.  Per chunk the workgroup stages, for the indices [c0, hi] (the
// chunk's starts and the blocks after them, at most 2561), the packed keys
// Y and the fixed-point cost prefixes relative to c0 in LDS.  Each request
// is then a merge of two sorted sequences, the targets Y(i) + S of the
// starts and the end keys Y(x): a start meets, when it is merged, the first
// end key at or above its target, which is the end of its shortest window.
// Every lane bisects its diagonal of the merge once and walks a fixed
// number of steps, scoring each start it takes on the spot.  Starts whose
// target lies above every staged end key (windows reaching past hi) are
// walked from the global prefixes, as are whole chunks whose bytes or
// request break the packed-key bounds.  A request's merge is split over
// wpr wavefronts (one when a snapshot has eight requests or more in the
// workgroup, so that each lane's bisection serves a long slice), and every
// wavefront keeps its own least window per request, so a request costs no
// barrier; the wavefronts' minima meet once per unit.
__global__ __launch_bounds__(kSThreads, 4) void real_search_kernel(Prefix pf, SearchArgs A) {
    __shared__ uint64_t Y[kStage + 1 + kPadSteps + 1];
    __shared__ U128 Cr[kStage + 1 + kPadSteps + 1];
    __shared__ Best bestw[kSWaves][kMaxGroup];
    __shared__ int big_flag;
    const uint32_t tid = threadIdx.x, lane = tid & 63u, w = tid >> 6;
    for (uint64_t L = blockIdx.x; L < A.units; L += gridDim.x) {
        const uint64_t g = L % A.parts, qg = L / A.parts;
        const uint64_t r0 = qg * A.group;
        const uint64_t r1 = r0 + A.group < A.num_requests ? r0 + A.group : A.num_requests;
        if (lane < kMaxGroup) bestw[w][lane] = best_none();
        for (uint64_t r = r0; r < r1;) {
            const uint64_t b = wave_owner(A.req_off, A.num_segments, r, lane);
            const uint64_t rend = A.req_off[b + 1] < r1 ? A.req_off[b + 1] : r1;
            const uint64_t s0 = A.seg[b], nend = A.seg[b + 1], nb = nend - s0;
            // slice g of the snapshot's starts (nb * g fits: nb < 2^40, g < 2^10)
            const uint64_t a = s0 + nb * g / A.parts, e = s0 + nb * (g + 1) / A.parts;
            // The m requests [r, rend) of snapshot b: wpr wavefronts per
            // request (a power of two, wpr * m <= kSWaves when m allows),
            // conc requests at once; wavefront w serves requests j with
            // j % conc == w / wpr, on lanes gl of `lanes`.
            const uint32_t m = static_cast<uint32_t>(rend - r);
            uint32_t wpr = 1;
            while (wpr < kSWaves && 2 * wpr * m <= kSWaves) wpr *= 2;
            const uint32_t conc = kSWaves / wpr, slot = w / wpr;
            const uint32_t gl = (w % wpr) * 64u + lane, lanes = 64u * wpr;
            for (uint64_t c0 = a; c0 < e; c0 += kChunk) {
                const uint64_t c1 = c0 + kChunk < e ? c0 + kChunk : e;
                const uint64_t hi = c0 + kStage < nend ? c0 + kStage : nend;  // staged [c0, hi]
                const uint32_t nA = static_cast<uint32_t>(c1 - c0);
                const uint32_t nB = static_cast<uint32_t>(hi - c0);
                const uint64_t pbase = pf.P(c0), rbase = pf.R(c0);
                const U128 cbase = pf.C(c0);
                __builtin_amdgcn_s_setprio(0);  // staging at the normal priority
                if (tid == 0) big_flag = 0;
                __syncthreads();  // the previous chunk's readers are done; flag cleared
                // kStageBatch indices per thread at a time, their loads issued
                // together (indices clamped to hi, so every load is in bounds;
                // only indices up to hi are staged).  A block of 2^51 bytes or
                // more could wrap the staged byte count: P(x + 1) - P(x) is
                // checked in the same pass.
                bool big = false;
                for (uint64_t xb = c0 + tid; xb <= hi; xb += kStageBatch * kSThreads) {
                    uint64_t pv[kStageBatch], pn[kStageBatch], rv[kStageBatch];
                    U128 cv[kStageBatch];
#pragma unroll
                    for (uint32_t j = 0; j < kStageBatch; ++j) {
                        const uint64_t xj = xb + j * kSThreads;
                        const uint64_t x = xj < hi ? xj : hi;
                        const uint64_t xn = x < hi ? x + 1 : x;
                        pv[j] = pf.P(x);
                        pn[j] = pf.P(xn);
                        rv[j] = pf.R(x);
                        cv[j] = pf.C(x);
                    }
#pragma unroll
                    for (uint32_t j = 0; j < kStageBatch; ++j) {
                        const uint64_t x = xb + j * kSThreads;
                        if (x <= hi) {
                            const uint64_t pr = pv[j] - pbase;
                            big |= (pr >= kPackOne) | (pn[j] - pv[j] >= kPackOne);
                            Y[x - c0] = ((rv[j] - rbase) << kPackBits) + pr;
                            Cr[x - c0] = sub128(cv[j], cbase);
                        }
                    }
                }
                if (tid <= kPadSteps) {
                    Y[nB + 1 + tid] = kEndKey;
                    Cr[nB + 1 + tid] = U128{0, 0};
                }
                if (big) big_flag = 1;
                __syncthreads();
                // the merges at a raised wave priority: the other workgroup on
                // the CU, when it stages a chunk meanwhile, yields issue slots
                __builtin_amdgcn_s_setprio(1);
                const bool packed_chunk = big_flag == 0;
                const uint64_t span = packed_chunk ? Y[nB] & (kPackOne - 1) : 0;
                // No window crosses a pinned block, so every start of the
                // chunk is merged by the end key that takes in the first
                // pinned block after it (its run field is above every
                // start's target): the merges stop there.  Found by the
                // wavefront, 64 keys a round.
                uint32_t mB = nB;
                if (packed_chunk && nB > nA + 1) {
                    const uint64_t thr = ((Y[nA] >> kPackBits) + 1) << kPackBits;
                    uint32_t lo = nA + 1, hi = nB + 1;  // first k in [lo, hi) with Y[k] >= thr, else hi
                    while (hi - lo > 64) {
                        const uint32_t step = (hi - lo + 63) >> 6;
                        const uint32_t i = lo + lane * step;
                        const uint64_t mk = __ballot(i >= hi || Y[i] >= thr);
                        const uint32_t f = mk ? static_cast<uint32_t>(__builtin_ctzll(mk)) : 64u;
                        const uint32_t nhi = f < 64 ? lo + f * step : hi;
                        lo = f ? lo + (f - 1) * step + 1 : lo;
                        hi = nhi < hi ? nhi : hi;
                    }
                    const uint64_t mk = __ballot(lo + lane >= hi || Y[lo + lane] >= thr);
                    const uint32_t k = mk ? lo + static_cast<uint32_t>(__builtin_ctzll(mk)) : hi;
                    mB = k < nB ? k : nB;
                }
                // starts whose target is above every staged end key: their windows
                // end past hi (or nowhere); a suffix of the chunk, walked globally
                // by the request's lanes (true when some start was walked)
                auto pending = [&](uint64_t S, Best& mine) -> bool {
                    if (hi >= nend) return false;
                    uint32_t plo = 0, phi = nA;
                    const uint64_t ylast = Y[nB];
                    while (plo < phi) {
                        const uint32_t mid = (plo + phi) >> 1;
                        if (Y[mid] + S > ylast) phi = mid; else plo = mid + 1;
                    }
                    const uint64_t np = nA - plo;
                    if (np) {
                        const uint64_t per = (np + lanes - 1) / lanes;
                        const uint64_t q0 = c0 + plo + gl * per;
                        walk_global(pf, q0 < c1 ? q0 : c1, q0 + per < c1 ? q0 + per : c1, nend, S,
                                    mine);
                    }
                    return np != 0;
                };
                auto fast = [&](uint64_t S) {
                    return S != 0 && packed_chunk && S <= kPackOne - span;
                };
                // this wavefront's least window of request j into its slot
                auto keep = [&](uint32_t j, const Best& best) {
                    if (lane == 0 && best_less(best, bestw[w][r + j - r0])) bestw[w][r + j - r0] = best;
                };
                // Requests j and j + conc go together: when both are packed,
                // their merges are interleaved (independent chains of LDS reads).
                for (uint32_t j = slot; j < m; j += 2 * conc) {
                    const uint64_t S0 = A.req_sizes[r + j];
                    const bool pair = j + conc < m;
                    const uint64_t S1 = pair ? A.req_sizes[r + j + conc] : 0;
                    if (pair && fast(S0) && fast(S1)) {
                        const uint64_t SS[2] = {S0, S1};
                        Best m2[2] = {best_none(), best_none()};
                        merge_requests<2>(Y, Cr, nA, mB, SS, c0, gl, lanes, m2);
#pragma unroll
                        for (uint32_t u = 0; u < 2; ++u) {
                            const bool walked = pending(SS[u], m2[u]);
                            keep(j + u * conc, to_local(walked ? wave_min(m2[u]) : wave_min_chunk(m2[u], c0), s0));
                        }
                        continue;
                    }
                    for (uint32_t u = 0; u < (pair ? 2u : 1u); ++u) {
                        const uint64_t S = u ? S1 : S0;
                        if (S == 0) continue;
                        Best mine = best_none();
                        if (fast(S)) {
                            const uint64_t SS[1] = {S};
                            Best m1[1] = {best_none()};
                            merge_requests<1>(Y, Cr, nA, mB, SS, c0, gl, lanes, m1);
                            mine = m1[0];
                            pending(S, mine);
                        } else {
                            // the packed keys would not decide correctly: global walk
                            const uint64_t per = (nA + lanes - 1) / lanes;
                            const uint64_t i0 = c0 + gl * per;
                            walk_global(pf, i0 < c1 ? i0 : c1, i0 + per < c1 ? i0 + per : c1,
                                        nend, S, mine);
                        }
                        keep(j + u * conc, to_local(wave_min(mine), s0));
                    }
                }
            }
            r = rend;
        }
        __syncthreads();
        if (tid < r1 - r0) {
            Best m = bestw[0][tid];
            for (uint32_t v = 1; v < kSWaves; ++v)
                if (best_less(bestw[v][tid], m)) m = bestw[v][tid];
            A.slots[(r0 + tid) * A.parts + g] = m;
        }
        __syncthreads();
    }
}

// Stage 4.
__global__ __launch_bounds__(kThreads) void real_reduce_kernel(SearchArgs A,
                                                               coop_window_real_t* __restrict__ out) {
    const uint64_t r = static_cast<uint64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (r >= A.num_requests) return;
    coop_window_real_t o;
    if (A.req_sizes[r] == 0) {
        o.start = o.end = o.cost_lo = o.cost_hi = 0;
        o.cost = 0.0;
        out[r] = o;
        return;
    }
    Best m = best_none();
    for (uint64_t g = 0; g < A.parts; ++g) {
        const Best x = A.slots[r * A.parts + g];
        if (best_less(x, m)) m = x;
    }
    if (m.start == kNone) {
        o.start = o.end = o.cost_lo = o.cost_hi = kNone;
        o.cost = __builtin_inf();
    } else {
        o.start = m.start;
        o.end = m.end;
        o.cost_lo = m.c_lo;
        o.cost_hi = m.c_hi;
        o.cost = to_real(U128{m.c_lo, m.c_hi});
    }
    out[r] = o;
}

struct RealLayout {
    uint64_t tiles, group, parts, units;
    size_t pl, cl_lo, cl_hi, rl, tot, off, slots, bytes;
};

size_t align256(size_t x) { return (x + 255) & ~static_cast<size_t>(255); }

bool real_layout(uint64_t num_blocks, uint64_t num_segments, uint64_t num_requests, RealLayout* l) {
    if (num_segments == 0 || num_blocks >= (1ull << 40) || num_requests >= (1ull << 40))
        return false;
    l->tiles = (num_blocks >> kTileLog2) + 1;
    uint64_t rps = num_requests / num_segments;
    l->group = rps < 1 ? 1 : (rps > kMaxGroup ? kMaxGroup : rps);
    uint64_t groups = (num_requests + l->group - 1) / l->group;
    const uint64_t avg = num_blocks / num_segments;
    uint64_t parts = groups ? (kTargetGroups + groups - 1) / groups : 1;
    const uint64_t cap = avg / kChunk > 1 ? avg / kChunk : 1;
    if (parts > cap) parts = cap;
    if (parts > kMaxParts) parts = kMaxParts;
    if (parts < 1) parts = 1;
    // Few small snapshots with many requests (parts stuck at 1): smaller
    // request groups, so that the batch still fills the chip; each
    // workgroup then stages its chunk for fewer requests.
    if (groups * parts < kResidentUnits && l->group > 1) {
        const uint64_t want = (num_requests * parts + kResidentUnits - 1) / kResidentUnits;
        if (want < l->group) {
            l->group = want < 1 ? 1 : want;
            groups = (num_requests + l->group - 1) / l->group;
        }
    }
    l->parts = parts;
    l->units = groups * parts;
    const uint64_t np = num_blocks + 1;
    size_t at = 0;
    l->pl = at; at = align256(at + np * 8);
    l->cl_lo = at; at = align256(at + np * 8);
    l->cl_hi = at; at = align256(at + np * 8);
    l->rl = at; at = align256(at + np * 2);
    l->tot = at; at = align256(at + l->tiles * sizeof(Tri));
    l->off = at; at = align256(at + l->tiles * sizeof(Tri));
    l->slots = at; at = align256(at + num_requests * parts * sizeof(Best));
    l->bytes = at;
    return true;
}

}  // namespace

extern "C" {

coop_status_t coop_window_search_real_workspace_size(uint64_t num_blocks, uint64_t num_segments,
                                                     uint64_t num_requests, size_t* bytes_out) {
    if (!bytes_out) return COOP_ERR_INVALID;
    if (num_requests == 0) {
        *bytes_out = 0;
        return COOP_OK;
    }
    RealLayout l;
    if (!real_layout(num_blocks, num_segments, num_requests, &l)) return COOP_ERR_INVALID;
    *bytes_out = l.bytes;
    return COOP_OK;
}

coop_status_t coop_window_search_real(const uint64_t* size, const double* h, const uint8_t* kind,
                                      uint64_t num_blocks, const uint64_t* seg_offsets,
                                      uint64_t num_segments, const uint64_t* req_sizes,
                                      const uint64_t* req_offsets, uint64_t num_requests,
                                      coop_window_real_t* out, uint32_t* status, void* workspace,
                                      size_t workspace_bytes, void* stream) {
    if (num_requests == 0) return COOP_OK;
    if (!seg_offsets || !req_sizes || !req_offsets || !out || !status) return COOP_ERR_INVALID;
    if (num_blocks && (!size || !h || !kind)) return COOP_ERR_INVALID;
    RealLayout l;
    if (!real_layout(num_blocks, num_segments, num_requests, &l)) return COOP_ERR_INVALID;
    if (!workspace || workspace_bytes < l.bytes) return COOP_ERR_WORKSPACE;
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (coop_host::checks_requested()) {
        // offsets and run byte totals; the exact h totals are not checked
        const coop_host::Batch b{size, nullptr, kind, num_blocks, seg_offsets, num_segments,
                                 req_offsets, num_requests, true};
        const coop_status_t rc = coop_host::check_batch(b, s);
        if (rc != COOP_OK) return rc;
    }
    char* w = static_cast<char*>(workspace);
    uint64_t* pl = reinterpret_cast<uint64_t*>(w + l.pl);
    uint64_t* cl_lo = reinterpret_cast<uint64_t*>(w + l.cl_lo);
    uint64_t* cl_hi = reinterpret_cast<uint64_t*>(w + l.cl_hi);
    uint16_t* rl = reinterpret_cast<uint16_t*>(w + l.rl);
    Tri* tot = reinterpret_cast<Tri*>(w + l.tot);
    Tri* off = reinterpret_cast<Tri*>(w + l.off);
    Best* slots = reinterpret_cast<Best*>(w + l.slots);
    const uint32_t tile_grid = static_cast<uint32_t>(l.tiles < (1u << 20) ? l.tiles : (1u << 20));
    hipLaunchKernelGGL(real_tile_kernel, dim3(tile_grid), dim3(kThreads), 0, s, size, h, kind,
                       num_blocks, l.tiles, pl, cl_lo, cl_hi, rl, tot);
    if (hipGetLastError() != hipSuccess) return COOP_ERR_HIP;
    hipLaunchKernelGGL(real_offsets_kernel, dim3(1), dim3(kOffsetThreads), 0, s, tot, l.tiles, off,
                       status);
    if (hipGetLastError() != hipSuccess) return COOP_ERR_HIP;
    const Prefix pf{pl, cl_lo, cl_hi, rl, off};
    const SearchArgs A{seg_offsets, num_segments, req_sizes, req_offsets, num_requests,
                       l.group, l.parts, l.units, slots};
    const uint32_t search_grid = static_cast<uint32_t>(l.units < (1u << 20) ? l.units : (1u << 20));
    hipLaunchKernelGGL(real_search_kernel, dim3(search_grid), dim3(kSThreads), 0, s, pf, A);
    if (hipGetLastError() != hipSuccess) return COOP_ERR_HIP;
    const uint32_t reduce_grid = static_cast<uint32_t>((num_requests + kThreads - 1) / kThreads);
    hipLaunchKernelGGL(real_reduce_kernel, dim3(reduce_grid), dim3(kThreads), 0, s, A, out);
    if (hipGetLastError() != hipSuccess) return COOP_ERR_HIP;
    return COOP_OK;
}

}  // extern "C"
