// Batched sliding-window eviction search (Coop, section 3.3) for gfx950.
//
// Problem (section 3.1 Eq. (1), window form of section 3.3): for every
// request of S bytes on a pool snapshot, find the window [start, end) of
// adjacent blocks with no pinned block, at least S bytes and the least summed
// cost of its evictable blocks; ties go to fewer bytes, then the lower start.
//
// Work decomposition
// ------------------
// Each snapshot b of N_b blocks is cut into tiles of kTile blocks (one for
// an empty snapshot).  With f(b) = floor(seg[b] / kTile) + b, the tiles of
// snapshot b are the tile ids [f(b), f(b) + tiles_b), and f is strictly
// increasing, so a search over seg_offsets names the snapshot of any id; ids
// that name no tile are skipped.  A work unit is one tile id for one slice
// of the snapshot's requests.  The grid is persistent (two workgroups per
// CU).  Units are cut into chunks of consecutive units: workgroup w first
// takes chunk w (a large one), then claims small chunks from a queue until
// it runs dry.  The queue evens out the finish times: of the two workgroups
// on a CU, the one dispatched first wins the instruction arbitration and
// runs ahead, and snapshots differ in cost.  A workgroup walks its chunk
// with a cursor over the snapshot list, and loads the next tile into
// registers while it answers the requests of the current one.
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
//     staged boundary k, the key X[k] = R[k] << 50 | P[k] and C[k].  Keys
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
//     the wavefront's answer; wavefronts sharing a request combine in LDS
//     after the barrier that ends the tile.
//  3. Starts whose windows end past the staged region (the region's last run
//     goes on) are a suffix of the tile, found by one search; the request's
//     wavefront walks on through the run 64 blocks at a time, at most
//     kWalkCap blocks past the region.  Starts still pending there are left
//     to a second kernel, coop_window_long_kernel, which finds where their
//     windows end from per-tile records (see the section before it).
// A tile that holds a block of 2^37 bytes or more keeps plain 64-bit
// prefixes (P could outgrow the 50-bit field) with the run ids in a separate
// array, stages no halo, and bisects per start.
//
// Combining tiles
// ---------------
// A snapshot held by one chunk writes its results directly.  Otherwise every
// chunk writes one partial key per request into the workspace and takes a
// ticket on a per-snapshot counter; the chunk holding the last ticket reduces
// the partials and writes the results.  A job with windows left to the
// second kernel keeps its keys in the partial slots and is finished there.  Counters and the queue carry a
// per-call tag, so the workspace never needs clearing: eager calls take it
// from a host counter; calls captured into a graph derive it from a tag word
// in the workspace, advanced by a one-thread kernel ahead of each replay.
//
// All arithmetic is unsigned 64-bit integer.  Prefix sums wrap modulo 2^64;
// differences over a window are exact whenever each run's byte and cost
// totals fit in 64 bits.

#include <hip/hip_runtime.h>

#include <atomic>
#include <chrono>
#include <mutex>
#include <stdint.h>

#include "coop.h"
#include "coop_host.h"

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
static_assert((kXN + kMaxSteps) % 2 == 0 && kXN % 2 == 0, "the LDS arrays stay 16-byte aligned");
constexpr uint32_t kValBits = 50;
constexpr uint64_t kValMask = (1ull << kValBits) - 1;
// With every block below 2^37 bytes, any staged prefix (at most kStage < 2^13
// blocks) fits the 50-bit field, and no prefix wraps.  Keys then stay below
// (kStage + 1) << 50 < 2^63, so the difference of two keys is exact as a
// signed 64-bit number (the merge relies on it).
constexpr uint32_t kBigHiLog2 = 37 - 32;
static_assert(kStage < (1u << (kValBits - 37)), "staged prefixes must fit the key field");
static_assert(kStage + 2 < (1u << (63 - kValBits)), "keys stay below 2^63");
// The end key after a staged region: above every key and target, and
// positive as a signed number.
constexpr uint64_t kEndKey = (1ull << 63) - 1;
static_assert(kStage < (1u << 16), "pinned counts fit 16 bits");
constexpr uint64_t kNone = ~0ull;
constexpr uint32_t kNone32 = ~0u;
constexpr uint32_t kMaxWpr = 8;                  // wavefronts that may share one request
constexpr uint32_t kWalkCap = 1024;              // blocks a wavefront walks past a staged region
// A walk is not started when its first pending start needs more bytes past
// the region than twice the whole region holds (a full region: kStage
// blocks, so about 8.5 x kWalkCap blocks of its average size): those windows
// go to the second kernel at once.  Only the speed depends on this guess.
static_assert(2 * (kTile + kHaloCap) >= 8 * kWalkCap, "a skipped walk is one that would almost surely fail");
// The fewest blocks of a snapshot whose windows can run past a walk: the
// walk stops before the snapshot end only if more than kTile + kHaloCap +
// kWalkCap blocks follow the tile start, which is at most 7 blocks before
// the snapshot start.
constexpr uint64_t kDeferMin = kTile + kHaloCap + kWalkCap - 6;
constexpr uint64_t kPartialBudget = 1ull << 23;  // partial keys (32 B each) before chunks grow
constexpr uint32_t kEpochShift = 24;             // counter = epoch << 24 | tickets
// Call tags (40 bits).  An eager call takes the next value of a host counter
// (bit 39 clear); a call captured into a graph takes bit 39 and 39 bits that
// an odd multiplier maps one-to-one from a word in the workspace, which a
// one-thread kernel advances ahead of every replay.  The two kinds never
// meet, and no two replays on one workspace share a tag before 2^39 calls.
constexpr uint64_t kTagMask = (1ull << 39) - 1;
constexpr uint64_t kGraphTag = 1ull << 39;
constexpr uint64_t kTagOdd = 0x9e3779b97f4a7c15ull;
// The queue word's 32-bit tag: the call tag's low 31 bits, and bit 31 set
// for graph replays (call tag bit 39), so that an eager call and a replay
// never carry the same queue tag.
__host__ __device__ constexpr uint32_t queue_tag(uint64_t call_tag) {
    return static_cast<uint32_t>(call_tag & 0x7fffffffull) | ((call_tag & kGraphTag) ? 0x80000000u : 0u);
}
static_assert(queue_tag(kGraphTag) == 0x80000000u && queue_tag(kGraphTag - 1) == 0x7fffffffu,
              "graph and eager queue tags differ in bit 31");
// Queue word: call tag << 32 | chunks claimed.  A reserve chunk slot holds a
// chunk index, kQEmpty (nothing claimed yet) or kQDone (the queue ran dry).
constexpr uint64_t kQEmpty = ~0ull, kQDone = ~0ull - 1;

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

__device__ __forceinline__ uint64_t uniform64(uint64_t v) {
    return (static_cast<uint64_t>(uniform(static_cast<uint32_t>(v >> 32))) << 32) | uniform(static_cast<uint32_t>(v));
}

// v += v of the lane Ctrl names (0 where that lane is outside the row; rows
// off in RowMask keep v), as one add and one add-with-carry whose first
// operand is the moved lane (DPP on the adds themselves).  The compiler
// moves each half with its own instruction and then adds, three times the
// instructions; these sums are most of the staging scans.  The s_nop gives
// the two wait states a DPP read needs after a VALU write of its source.
#define COOP_ADD_DPP64(lo, hi, ctrl, mask)                                                     \
    asm volatile("s_nop 1\n\t"                                                                \
                 "v_add_co_u32_dpp %0, vcc, %0, %0 " ctrl " row_mask:" mask                    \
                 " bank_mask:0xf bound_ctrl:1\n\t"                                             \
                 "v_addc_co_u32_dpp %1, vcc, %1, %1, vcc " ctrl " row_mask:" mask              \
                 " bank_mask:0xf bound_ctrl:1"                                                 \
                 : "+v"(lo), "+v"(hi)                                                          \
                 :                                                                             \
                 : "vcc")

template <int Ctrl, int RowMask>
__device__ __forceinline__ void add_dpp64(uint64_t& v) {
    uint32_t lo = static_cast<uint32_t>(v), hi = static_cast<uint32_t>(v >> 32);
    if constexpr (Ctrl == kRowShr1 && RowMask == 0xf) COOP_ADD_DPP64(lo, hi, "row_shr:1", "0xf");
    else if constexpr (Ctrl == kRowShr2 && RowMask == 0xf) COOP_ADD_DPP64(lo, hi, "row_shr:2", "0xf");
    else if constexpr (Ctrl == kRowShr4 && RowMask == 0xf) COOP_ADD_DPP64(lo, hi, "row_shr:4", "0xf");
    else if constexpr (Ctrl == kRowShr8 && RowMask == 0xf) COOP_ADD_DPP64(lo, hi, "row_shr:8", "0xf");
    else if constexpr (Ctrl == kRowBcast15 && RowMask == 0xa) COOP_ADD_DPP64(lo, hi, "row_bcast:15", "0xa");
    else if constexpr (Ctrl == kRowBcast31 && RowMask == 0xc) COOP_ADD_DPP64(lo, hi, "row_bcast:31", "0xc");
    else static_assert(Ctrl < 0, "a DPP control without an add form");
    v = (static_cast<uint64_t>(hi) << 32) | lo;
}

// Prefix-sum element: bytes (or packed key), effective cost, pinned count (or
// a flag).
struct Sums {
    uint64_t q, c;
    uint32_t r;
};

template <int Ctrl, int RowMask>
__device__ __forceinline__ void sum_step(Sums& s) {
    add_dpp64<Ctrl, RowMask>(s.q);
    add_dpp64<Ctrl, RowMask>(s.c);
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

// The same minimum for windows inside a packed staged region, whose excess
// is below 2^50 and whose start is a staged index below 2^13: (excess,
// start) then orders as the one word excess << 13 | start, and each step
// moves and compares two words instead of three.
constexpr uint32_t kStartBits = 13;
static_assert(kTile <= (1u << kStartBits), "in-region starts fit the start field");
static_assert(kValBits + kStartBits < 64, "a packed key stays below the empty value");
template <int Ctrl, int RowMask>
__device__ __forceinline__ void argmin2_step(uint64_t& cost, uint64_t& key) {
    const uint64_t oc = dpp64<Ctrl, RowMask>(cost, kNone), ok = dpp64<Ctrl, RowMask>(key, kNone);
    const bool less = oc < cost || (oc == cost && ok < key);
    cost = less ? oc : cost;
    key = less ? ok : key;
}

__device__ __forceinline__ Cand wave_argmin_packed(const Cand& k) {
    uint64_t cost = k.cost;
    uint64_t key = k.start == kNone32 ? kNone : (k.excess << kStartBits) | k.start;
    argmin2_step<kQuadXor1, 0xf>(cost, key);
    argmin2_step<kQuadXor2, 0xf>(cost, key);
    argmin2_step<kRowHalfMirror, 0xf>(cost, key);
    argmin2_step<kRowMirror, 0xf>(cost, key);
    argmin2_step<kRowBcast15, 0xa>(cost, key);
    argmin2_step<kRowBcast31, 0xc>(cost, key);
    cost = readlane64(cost, 63);
    key = readlane64(key, 63);
    if (key == kNone) return cand_none();
    return Cand{cost, key >> kStartBits, static_cast<uint32_t>(key & ((1u << kStartBits) - 1))};
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
    Key* part;             // [num_requests][pc] partial keys
    uint64_t* counters;    // [slices][num_segments] arrival tickets
    uint64_t* queue;       // chunk queue word
    uint64_t num_blocks;
    uint64_t num_segments;
    uint64_t num_requests;
    // Counts of units and chunks are below 2^32 (units < 2^32 by the plan)
    // and held in 32 bits, which keeps the kernel's uniform state within the
    // scalar registers; products of them are formed in 64 bits.
    uint32_t num_virtual;  // tile ids per slice: floor(num_blocks / kTile) + num_segments
    uint32_t units;        // work units: slices * num_virtual (below 2^32)
    uint32_t grid;         // workgroups; chunk w < grid is workgroup w's first
    uint32_t c1, c2;       // units per chunk: first chunks [0, u1), queued chunks after
                           // (c2 is a lower bound from the host, set by the kernel)
    uint32_t u1;           // units in the first chunks
    uint64_t nchunks;      // chunks in all (set by the kernel when there is a queue)
    uint64_t c1_magic;     // ceil(2^64 / c1), for division by c1
    uint64_t c2_magic;     // ceil(2^64 / c2) (set by the kernel)
    uint64_t nv_magic;     // ceil(2^64 / num_virtual)
    uint32_t qtag;         // this call's queue tag
    uint32_t queue_on;     // units past u1 go through the queue
    uint32_t pc;           // partial slots per request (at most 2^23)
    uint64_t epoch;        // this call's tag on the arrival tickets
    const uint64_t* tag_word;  // captured calls: the workspace word the tags come from
    uint32_t defer_cap;    // deferred entries, at most (the arrays: see Ext)
    uint32_t slices_log2;  // request slices (a power of two): slice y takes y, y + slices, ...
    double inv_slope;      // guess of b per tile id, for the first snapshot lookup
};

// The workspace after the queue word, laid out the same way by the host
// (make_plan): the tag word, the deferred list's word (queue tag << 32 |
// entries), the word coop_window_long_kernel claims entries by (queue tag
// << 32 | claims), the deferred entries {first unit, end unit, g, G}
// (16-byte aligned), the tile records of tile p >= 1 of every snapshot at index
// (seg[b] >> kTileLog2) + p - 1 (bytes of all its blocks, cost of its
// evictable blocks, its pinned count; written by the search kernel, read by
// coop_window_long_kernel), and one deferral bit per partial slot (bit q * pc + g: request
// q left windows to coop_window_long_kernel in its chunk part g).  Derived
// where needed rather than passed, to keep the kernels' uniform state small.
struct Ext {
    uint64_t* defer_word;
    uint64_t* claim_word;
    uint4* entries;
    uint64_t* rec_p;
    uint64_t* rec_c;
    uint64_t* rec_r;
    uint32_t* bits;
};

__device__ __forceinline__ Ext ext_of(const Params& P) {
    Ext e;
    e.defer_word = P.queue + 2;
    e.claim_word = P.queue + 3;
    e.entries = reinterpret_cast<uint4*>((reinterpret_cast<uintptr_t>(P.queue + 4) + 15) & ~uintptr_t{15});
    e.rec_p = reinterpret_cast<uint64_t*>(e.entries + P.defer_cap);
    const uint64_t nrec = P.num_blocks >> kTileLog2;
    e.rec_c = e.rec_p + nrec;
    e.rec_r = e.rec_c + nrec;
    e.bits = reinterpret_cast<uint32_t*>(e.rec_r + nrec);
    return e;
}

// A read of an array the kernel never writes (offsets, request sizes)
// through the constant address space: uniform indices then become scalar
// loads, which do not queue behind the vector loads in flight.
typedef const __attribute__((address_space(4))) uint64_t* ConstU64;
__device__ __forceinline__ uint64_t ld_const(const uint64_t* p, uint64_t i) {
    return ((ConstU64)(p))[i];
}

// floor(n / d) for n < 2^32, with magic = ceil(2^64 / d) (0 for d = 1):
// the high word of n * magic (Lemire, Kaser and Kurz, "Faster remainder by
// direct computation", 2019).
__device__ __forceinline__ uint64_t div_magic(uint64_t n, uint64_t magic) {
    return magic ? __umul64hi(n, magic) : n;
}

// The chunk holding unit u, and the units of chunk c.
__device__ __forceinline__ uint64_t chunk_of(const Params& P, uint64_t u) {
    return u < P.u1 ? div_magic(u, P.c1_magic) : P.grid + div_magic(u - P.u1, P.c2_magic);
}

__device__ __forceinline__ void chunk_range(const Params& P, uint64_t c, uint64_t& b, uint64_t& e) {
    if (c < P.grid) {
        b = c * P.c1;
        e = b + P.c1 < P.u1 ? b + P.c1 : P.u1;
    } else {
        b = P.u1 + (c - P.grid) * static_cast<uint64_t>(P.c2);
        e = b + P.c2 < P.units ? b + P.c2 : P.units;
    }
    if (b > e) b = e;
}

// Staged boundaries in LDS, as 16-byte records: boundary i's key (R << 50 |
// P, or plain P in a tile with a huge block) at kv[2i] and its cost prefix C
// at kv[2i + 1], so that one 16-byte read fetches both (a merge step takes
// two LDS reads); then the records of the end keys a merge may read past the
// sentinel.
constexpr uint32_t kKV = kXN + kMaxSteps;

struct Smem {
    __attribute__((aligned(16))) uint64_t kv[2 * kKV];
    __device__ __forceinline__ uint64_t& K(uint32_t i) { return kv[2 * i]; }
    __device__ __forceinline__ uint64_t K(uint32_t i) const { return kv[2 * i]; }
    __device__ __forceinline__ uint64_t& C(uint32_t i) { return kv[2 * i + 1]; }
    __device__ __forceinline__ uint64_t C(uint32_t i) const { return kv[2 * i + 1]; }
    uint16_t run[kXN];  // R, kept only in a tile with a huge block
    Sums wsum[kWaves];  // per-wavefront totals of the tile
    Sums hsum[4];       // per-wavefront totals of the halo
    Key slot[kWaves];   // answers of wavefronts that share a request
    uint64_t slot_s[kWaves];
    uint64_t claim;     // a chunk claimed from the queue (an entry, in the second kernel)
    uint32_t defer_mark;  // the mark (hi - 1) of the last job a wavefront deferred
};

__device__ __forceinline__ uint64_t first_id(uint64_t b, uint64_t seg_b) {
    return (seg_b >> kTileLog2) + b;
}

// Position in the snapshot list: the offsets of snapshot b and of the two
// after it.  The third pair is loaded ahead, so that stepping to the next
// snapshot needs no wait.
struct Cursor {
    uint32_t y, b;  // b < num_segments <= 2^32
    uint64_t sb, sb1, sb2;  // seg[b], seg[b + 1], seg[min(b + 2, B)]
    uint64_t rb, rb1, rb2;  // req_off likewise
};

// Places the cursor on the snapshot holding tile id v: the largest b in
// [0, B) with f(b) = floor(seg[b] / kTile) + b <= v.  A guess from the
// average snapshot length is tried first, so uniform batches settle in one
// round of loads; otherwise a bisection.
__device__ void cursor_locate(const Params& P, uint64_t v, Cursor& c) {
    const uint64_t B = P.num_segments;
    uint64_t g = static_cast<uint64_t>(static_cast<double>(v) * P.inv_slope);
    if (g >= B) g = B - 1;
    uint64_t sg = ld_const(P.seg, g), sg1 = ld_const(P.seg, g + 1);
    const bool hit = first_id(g, sg) <= v && (g + 1 == B || first_id(g + 1, sg1) > v);
    uint64_t b = g;
    if (!hit) {
        uint64_t lo = 0, hi = B;  // f(lo) <= v < f(hi) (f(B) taken as infinite)
        if (first_id(g, sg) <= v) lo = g; else hi = g;
        while (hi - lo > 1) {
            const uint64_t mid = lo + (hi - lo) / 2;
            if (first_id(mid, ld_const(P.seg, mid)) <= v) lo = mid; else hi = mid;
        }
        b = lo;
        sg = ld_const(P.seg, b);
        sg1 = ld_const(P.seg, b + 1);
    }
    const uint64_t b2 = b + 2 < B ? b + 2 : B;
    c.b = b;
    c.sb = sg;
    c.sb1 = sg1;
    c.sb2 = ld_const(P.seg, b2);
    c.rb = ld_const(P.req_off, b);
    c.rb1 = ld_const(P.req_off, b + 1);
    c.rb2 = ld_const(P.req_off, b2);
}

// Moves the cursor forward to the snapshot holding tile id v (v not below
// the cursor's first id).
__device__ __forceinline__ void cursor_advance(const Params& P, uint64_t v, Cursor& c) {
    const uint64_t B = P.num_segments;
    while (c.b + 1ull < B && v >= first_id(c.b + 1ull, c.sb1)) {
        ++c.b;
        c.sb = c.sb1;
        c.sb1 = c.sb2;
        c.rb = c.rb1;
        c.rb1 = c.rb2;
        const uint64_t b2 = c.b + 2ull < B ? c.b + 2ull : B;
        c.sb2 = ld_const(P.seg, b2);
        c.rb2 = ld_const(P.req_off, b2);
    }
}

// One tile to search: tile p of snapshot b, for the requests of slice y.
// The chunks holding the tiles of (b, y) are G consecutive ones; the
// current chunk is the g-th.  `first` / `last`: the first / last tile of
// (b, y) in the current chunk.  Offsets are clamped to the array
// lengths: malformed offsets give wrong answers, never an out-of-bounds
// access.
struct Job {
    uint32_t u, y, b;  // unit, slice, snapshot (b < num_segments <= 2^32)
    uint32_t lo, hi;   // the units of (b, y) in the current chunk; hi - 1 marks the job
    uint64_t s0, s1, q0, R, K, tiles, p;
    uint32_t g, G;     // at most pc
    bool first, last, direct;
};

// The first unit in [u, u_end) holding a tile to search (a tile of a
// snapshot with requests in the unit's slice); false if there is none.
// (y, v) is unit u as (slice, tile id) and moves along with it.
__device__ bool next_job(const Params& P, Cursor& c, bool& have_cursor, uint64_t u, uint32_t& y,
                         uint32_t& v, uint64_t u_begin, uint64_t u_end, uint64_t chunk, Job& job) {
    for (; u < u_end; ++u, ++v) {
        if (v == P.num_virtual) {
            v = 0;
            ++y;
        }
        if (!have_cursor || y != c.y) {
            cursor_locate(P, v, c);
            c.y = y;
            have_cursor = true;
        } else {
            cursor_advance(P, v, c);
        }
        const uint64_t s1 = c.sb1 < P.num_blocks ? c.sb1 : P.num_blocks;
        const uint64_t s0 = c.sb < s1 ? c.sb : s1;
        const uint64_t q1 = c.rb1 < P.num_requests ? c.rb1 : P.num_requests;
        const uint64_t q0 = c.rb < q1 ? c.rb : q1;
        const uint64_t R = q1 - q0, nb = s1 - s0;
        // tiles start at floor8(s0) + p * kTile (see tile_geom)
        const uint64_t tiles = nb ? (s1 - (s0 & ~7ull) + kTile - 1) >> kTileLog2 : 1;
        const uint64_t f = first_id(c.b, c.sb);
        const uint64_t p = v - f;  // wraps (and is skipped) if the offsets are malformed
        if (p >= tiles || y >= R) continue;  // (the loop moves v with u)
        const uint64_t ub = static_cast<uint64_t>(y) * P.num_virtual + f;  // unit of tile 0 of (b, y)
        const uint64_t lo = ub > u_begin ? ub : u_begin;
        const uint64_t hi = ub + tiles < u_end ? ub + tiles : u_end;
        job.u = u;
        job.lo = static_cast<uint32_t>(lo);
        job.hi = static_cast<uint32_t>(hi);
        job.y = y;
        job.b = c.b;
        job.s0 = s0;
        job.s1 = s1;
        job.q0 = q0;
        job.R = R;
        job.K = ((R - y - 1) >> P.slices_log2) + 1;
        job.tiles = tiles;
        job.p = p;
        const uint64_t ue = ub + tiles - 1 < P.units ? ub + tiles - 1 : P.units - 1;
        const uint64_t i_lo = chunk_of(P, ub), i_hi = chunk_of(P, ue);
        const uint64_t G = i_hi - i_lo + 1;
        job.G = static_cast<uint32_t>(G > P.pc ? P.pc : G);  // P.pc only with malformed offsets
        const uint64_t g = chunk - i_lo;
        job.g = g >= job.G ? job.G - 1 : static_cast<uint32_t>(g);  // likewise
        job.first = u == lo;
        job.last = u + 1 == hi;
        job.direct = job.G == 1;
        return true;
    }
    return false;
}

// Issues the loads of the kItems blocks [t0 + tid*kItems, +kItems) of a
// tile of nt > 0 blocks starting on a multiple of 8: 16-byte loads of size
// and cost pairs and one 8-byte load of the kinds, at indices clamped to the
// tile (blocks past nt are masked when staged), when every such load stays
// inside the arrays; else one load per block.  On the first path nothing
// uses the loaded values, so no instruction waits for them; the second
// (arrays not aligned, or the very end of the arrays) packs the kinds at once.
__device__ __forceinline__ void load_items(const Params& P, uint64_t t0, uint32_t nt, uint32_t tid,
                                           uint64_t (&sz)[kItems], uint64_t (&ct)[kItems],
                                           uint32_t (&kd)[2]) {
    const uint32_t i0 = tid * kItems;
    const bool aligned = ((reinterpret_cast<uintptr_t>(P.size) | reinterpret_cast<uintptr_t>(P.cost)) &
                          15u) == 0 &&
                         (reinterpret_cast<uintptr_t>(P.kind) & 7u) == 0;
    if (aligned && (t0 & 7u) == 0 && t0 + ((nt + 7u) & ~7u) <= P.num_blocks) {
        const uint32_t last2 = (nt - 1) & ~1u, last8 = (nt - 1) & ~7u;
#pragma unroll
        for (uint32_t j = 0; j < kItems / 2; ++j) {
            const uint32_t i = i0 + 2 * j < last2 ? i0 + 2 * j : last2;
            const ulonglong2 a = *reinterpret_cast<const ulonglong2*>(P.size + t0 + i);
            const ulonglong2 b = *reinterpret_cast<const ulonglong2*>(P.cost + t0 + i);
            sz[2 * j] = a.x;
            sz[2 * j + 1] = a.y;
            ct[2 * j] = b.x;
            ct[2 * j + 1] = b.y;
        }
        const uint2 k2 = *reinterpret_cast<const uint2*>(P.kind + t0 + (i0 < last8 ? i0 : last8));
        kd[0] = k2.x;
        kd[1] = k2.y;
    } else {
        kd[0] = 0;
        kd[1] = 0;
#pragma unroll
        for (uint32_t j = 0; j < kItems; ++j) {
            const uint32_t i = i0 + j < nt ? i0 + j : nt - 1;
            sz[j] = P.size[t0 + i];
            ct[j] = P.cost[t0 + i];
            kd[j >> 2] |= static_cast<uint32_t>(P.kind[t0 + i]) << (8 * (j & 3));
        }
    }
}

// A tile's blocks as loaded, one thread's share: kItems blocks of the tile
// and one halo block for the first kHaloCap threads.
struct TileRegs {
    uint64_t sz[kItems], ct[kItems];
    uint32_t kd[2];  // kind of block j in byte j & 3 of kd[j / 4]
    uint64_t hq, hc;
    uint32_t hk;
};

struct TileGeom {
    uint64_t t0;    // global index of the tile start (a multiple of 8)
    uint32_t nt;    // blocks in the tile, counting the lead
    uint32_t hm;    // halo blocks: the next blocks of the snapshot, up to kHaloCap
    uint32_t lead;  // blocks before the snapshot start (first tile only): pinned phantoms
};

// Tile p of a snapshot covers [a + p * kTile, +kTile) clipped to the snapshot
// end, with a = floor8(s0): every tile starts on a multiple of 8.  The
// first tile's blocks before s0 (fewer than 8) are staged as empty pinned
// blocks, so that no window starts at or crosses them.  The halo follows.
__device__ __forceinline__ TileGeom tile_geom(const Job& job) {
    TileGeom t;
    t.t0 = (job.s0 & ~7ull) + (job.p << kTileLog2);
    t.lead = job.p == 0 ? static_cast<uint32_t>(job.s0 - t.t0) : 0u;
    const uint64_t left = job.s1 - t.t0;
    t.nt = static_cast<uint32_t>(left < kTile ? left : kTile);
    const uint64_t after = left - t.nt;
    t.hm = static_cast<uint32_t>(after < kHaloCap ? after : kHaloCap);
    return t;
}

// Issues every load of a tile; nothing waits for them here.
__device__ __forceinline__ void issue_loads(const Params& P, const TileGeom& t, uint32_t tid,
                                            TileRegs& r) {
    if (t.nt) load_items(P, t.t0, t.nt, tid, r.sz, r.ct, r.kd);
    r.hq = 0;
    r.hc = 0;
    r.hk = COOP_FREE;
    if (tid < t.hm) {
        const uint64_t gp = t.t0 + t.nt + tid;
        r.hk = P.kind[gp];
        r.hq = P.size[gp];
        r.hc = P.cost[gp];
    }
}

__device__ __forceinline__ coop_window_t to_window(const Key& k, uint64_t S) {
    if (S == 0) return coop_window_t{0, 0, 0};
    if (k.start == kNone) return coop_window_t{kNone, kNone, kNone};
    return coop_window_t{k.start, k.end, k.cost};
}

__device__ __forceinline__ ulonglong2 lds_u128(const uint64_t* base, uint32_t byte_off) {
    return *reinterpret_cast<const ulonglong2*>(reinterpret_cast<const char*>(base) + byte_off);
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
// reaches S bytes.  With D = X[k] - X[i] (exact as a signed number, keys
// being below 2^63), the start is taken iff D >= Sc, and the window is valid
// iff D < 2^50, i.e. both ends have the same run id; D is then its byte
// count.  Windows are ranked by (cost, D), which orders them as (cost,
// bytes - S).  Steps past the lane's slice repeat work of the next lane
// (harmless: equal windows).  A lane may take starts past nA (boundaries of
// the halo): their windows are real windows of the snapshot, though not
// always the shortest from that start (the diagonal split counts only the
// starts below nA), so never better than the window the next tile finds
// for it; scoring them is harmless too.
// nB is the region end or an end key whose run id is above every target of
// a start below nA (the one that takes in the first pinned block after the
// tile): all nA starts are merged within the first nA + nB elements either
// way.  Past them a lane merges the staged keys that follow, which are
// real; a lane whose diagonal lies past nA + nB pairs halo starts with end
// keys past that pinned block, which never gives a valid window.  The
// region end is followed by kEndKey, above every target, and so are the
// kMaxSteps keys after it: a lane that has taken the start after the region
// end (the sentinel itself) can take nothing more, and its end index runs
// on through those keys.  Only
// the start is kept (as a byte offset, pA + pB growing by 16 a step gives the
// end pointer); the caller finds the winner's end again (merged_answer).
__device__ __forceinline__ void merge_pass(const Smem& sm, uint32_t nA, uint32_t nB, uint32_t d,
                                           uint32_t L, uint64_t Sc, Cand& best) {
    // diagonal split: the number of starts among the first d merge elements
    uint32_t lo = d > nB ? d - nB : 0, hi = d < nA ? d : nA;
    while (lo < hi) {
        const uint32_t mid = (lo + hi) >> 1;
        // start `mid` precedes end key X[d - mid] iff its target is at or below it
        const bool before = sm.K(mid) + Sc <= sm.K(d - mid);
        lo = before ? mid + 1 : lo;
        hi = before ? hi : mid;
    }
    constexpr uint32_t kStep = 16u;  // bytes per boundary record
    uint32_t pA = lo * kStep;
    const uint32_t sum0 = (d + 1) * kStep;  // pA + pB before the first step; grows by kStep a step
    const int64_t sc = static_cast<int64_t>(Sc);
    uint64_t bc = kNone, bd = kNone;
    uint32_t bpa = kNone32;
    for (uint32_t k = 0; k < L; k += 2) {
#pragma unroll
        for (uint32_t u = 0; u < 2; ++u) {
            const uint32_t pB = sum0 + (k + u) * kStep - pA;
            const ulonglong2 ra = lds_u128(sm.kv, pA), rb = lds_u128(sm.kv, pB);
            const uint64_t xa = ra.x, ca = ra.y, kb = rb.x, cb = rb.y;
            const uint64_t D = kb - xa;
            const bool takeA = static_cast<int64_t>(D) >= sc;
            const bool valid = takeA & (D < (1ull << kValBits));
            const uint64_t cost = cb - ca;
            const bool better = valid & ((cost < bc) | ((cost == bc) & (D < bd)));
            bc = better ? cost : bc;
            bd = better ? D : bd;
            bpa = better ? pA : bpa;
            pA += takeA ? kStep : 0u;
        }
    }
    // Within a lane starts are met in increasing order, so strict comparison
    // kept the lowest start among equal (cost, bytes).
    const Cand c{bc, bpa == kNone32 ? kNone : bd - Sc, bpa == kNone32 ? kNone32 : bpa / kStep};
    if (cand_less(c, best)) best = c;
}

// Plain prefixes (a tile with a huge block): starts g, g + lanes, ... below
// nA, each by two bisections: the end of its run, then its first end with
// at least S bytes.
__device__ __forceinline__ void plain_pass(const Smem& sm, uint32_t nA, uint32_t end, uint32_t g,
                                           uint32_t lanes, uint64_t S, Cand& best,
                                           uint32_t& best_end) {
    for (uint32_t i = g; i < nA; i += lanes) {
        const uint32_t run = sm.run[i];
        const uint64_t base = sm.K(i);
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
            if (sm.K(mid + 1) - base >= S) hi = mid; else lo = mid + 1;
        }
        if (lo < rend) {
            const Cand c{sm.C(lo + 1) - sm.C(i), sm.K(lo + 1) - base - S, i};
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

// The same search by a whole wavefront (every lane active, same arguments):
// 64 evenly spaced probes narrow [lo, hi) to one gap per round, so a tile
// takes two rounds of LDS reads instead of a dozen dependent ones.
template <typename Pred>
__device__ __forceinline__ uint32_t wave_lower_bound(uint32_t lo, uint32_t hi, uint32_t lane,
                                                     Pred pred) {
    while (hi - lo > 64) {
        const uint32_t step = (hi - lo + 63) >> 6;
        const uint32_t i = lo + lane * step;
        const uint64_t m = __ballot(i >= hi || pred(i));
        // pred false at every probe below lane f, true at f (or past hi)
        const uint32_t f = m ? static_cast<uint32_t>(__builtin_ctzll(m)) : 64u;
        const uint32_t nhi = f < 64 ? lo + f * step : hi;
        lo = f ? lo + (f - 1) * step + 1 : lo;
        hi = nhi < hi ? nhi : hi;
    }
    const uint64_t m = __ballot(lo + lane >= hi || pred(lo + lane));
    return m ? lo + static_cast<uint32_t>(__builtin_ctzll(m)) : hi;
}

// The first start whose window cannot end inside the staged region [0, end]
// although its run reaches the region's end: starts i < nA with run id endrun
// and fewer than S bytes from i to the region end.  Such starts form a suffix.
// Called by a whole wavefront with the same arguments.
__device__ __forceinline__ uint32_t pending_start(const Smem& sm, bool packed, uint32_t nA,
                                                  uint64_t xend, uint32_t endrun, uint64_t S,
                                                  uint64_t Sc, uint32_t lane) {
    if (packed) {
        // run id endrun and X[i] + Sc > X[end]
        const uint64_t by_run = static_cast<uint64_t>(endrun) << kValBits;
        const uint64_t by_bytes = xend >= Sc ? xend - Sc + 1 : 0;
        const uint64_t thr = by_run > by_bytes ? by_run : by_bytes;
        return wave_lower_bound(0, nA, lane, [&](uint32_t i) { return sm.K(i) >= thr; });
    }
    const uint32_t i0 =
        wave_lower_bound(0, nA, lane, [&](uint32_t i) { return sm.run[i] == endrun; });
    return wave_lower_bound(i0, nA, lane, [&](uint32_t i) { return xend - sm.K(i) < S; });
}

// Where a wavefront's walk through the run past the staged region stands:
// the next block pos, the run's prefixes before it (bytes cq, cost cc; in
// the staged region's frame), the first unresolved pending start, and
// whether the run has closed (a pinned block or the snapshot end reached).
struct WalkState {
    uint64_t pos, cq, cc;
    uint32_t cur;
    bool closed;
};

// Resolves pending starts [ws.cur, nA): all lie in the staged region's last
// run, which goes on at global block ws.pos.  The wavefront walks the run 64
// blocks at a time (one per lane, wavefront prefix sums, the chunk kept in
// registers) up to block lim; each chunk resolves a prefix of the pending
// starts, 64 at a time, since their shortest ends are monotone.  Candidates
// fold into best / best_end (end snapshot-local).  Stops when every pending
// start is resolved, at lim, or where the run closes.
__device__ void walk_pass(const Params& P, const Smem& sm, uint32_t lane, uint32_t nA, uint64_t lim,
                          uint64_t s0, uint64_t s1, uint64_t vmask, uint64_t S, WalkState& ws,
                          Cand& best, uint64_t& best_end) {
    uint32_t cur = ws.cur;
    uint64_t pos = ws.pos, cq = ws.cq, cc = ws.cc;
    // A walk that would almost surely fail is not started: where the
    // snapshot goes on past the limit (as for a walk that fails), when the
    // first pending start needs more bytes past the region than twice the
    // region holds (cq is the region's byte prefix at its end, sm.K(0) at
    // its start; a pending start has fewer than S bytes to the region end).
    if (lim == pos + kWalkCap && lim < s1) {
        const uint64_t rb = cq - (sm.K(0) & vmask);
        if (S - (cq - (sm.K(cur) & vmask)) > (rb >> 63 ? kNone : rb << 1)) lim = pos;
    }
    // the blocks of the chunk at pos; the next chunk's are loaded before
    // this one is processed
    auto load = [&](uint64_t at, uint32_t m, uint32_t& kd, uint64_t& sz, uint64_t& ct) {
        kd = COOP_PINNED;
        sz = 0;
        ct = 0;
        if (lane < m) {
            kd = P.kind[at + lane];
            sz = P.size[at + lane];
            ct = P.cost[at + lane];
        }
    };
    uint32_t m = pos < lim ? (lim - pos < 64 ? static_cast<uint32_t>(lim - pos) : 64u) : 0u;
    uint32_t kd;
    uint64_t sz, ct;
    load(pos, m, kd, sz, ct);
    while (cur < nA && pos < lim) {
        const uint64_t npos = pos + m;
        const uint32_t nm = npos < lim ? (lim - npos < 64 ? static_cast<uint32_t>(lim - npos) : 64u) : 0u;
        uint32_t nkd;
        uint64_t nsz, nct;
        load(npos, nm, nkd, nsz, nct);
        const uint64_t pinned = __ballot(kd >= COOP_PINNED);
        const uint32_t fp = pinned ? static_cast<uint32_t>(__builtin_ctzll(pinned)) : 64u;  // <= m
        const bool valid = lane < fp;
        Sums s{valid ? sz : 0, valid && kd == COOP_EVICTABLE ? ct : 0, 0};
        wave_inclusive_sum(s);
        const uint64_t q = cq + s.q, c = cc + s.c;  // prefixes after this lane's block
        const uint32_t lastl = fp ? fp - 1 : 0;
        const uint64_t lastq = fp ? readlane64(q, lastl) : cq;
        const uint64_t lastc = fp ? readlane64(c, lastl) : cc;
        // no window from the first pending start ends in this chunk: none
        // from a later one does either (ends are monotone)
        const bool none = fp == 0 || lastq - (sm.K(cur) & vmask) < S;
        for (; !none;) {
            const uint32_t i = cur + lane;
            const bool act = i < nA;
            const uint32_t ii = act ? i : nA - 1;
            const uint64_t base = sm.K(ii) & vmask, cbase = sm.C(ii);
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
        if (fp < m) {  // the run closes inside this chunk
            ws.closed = true;
            break;
        }
        cq = lastq;
        cc = lastc;
        pos = npos;
        m = nm;
        kd = nkd;
        sz = nsz;
        ct = nct;
    }
    if (pos >= s1) ws.closed = true;
    ws.cur = cur;
    ws.pos = pos;
    ws.cq = cq;
    ws.cc = cc;
}

// What staging left in LDS.
struct TileState {
    bool packed;     // keys R << 50 | P; otherwise plain P with R in sm.run
    uint32_t end;    // staged boundaries [0, end]
    uint32_t endrun; // R at the region end
    uint64_t xend;   // X at the region end
    uint64_t xcend;  // C at the region end
    uint64_t tq, tc; // the tile's totals (without the halo): X (bytes + 2^50 per
    uint32_t tr;     // pinned block, modulo 2^64), C, and the pinned count
};

template <int Ctrl, int RowMask>
__device__ __forceinline__ void sum2_step(Sums& s) {
    add_dpp64<Ctrl, RowMask>(s.q);
    add_dpp64<Ctrl, RowMask>(s.c);
}

// Inclusive sums of q and c (r untouched) over the rows, and over the wavefront.
__device__ __forceinline__ void row_inclusive_sum2(Sums& s) {
    sum2_step<kRowShr1, 0xf>(s);
    sum2_step<kRowShr2, 0xf>(s);
    sum2_step<kRowShr4, 0xf>(s);
    sum2_step<kRowShr8, 0xf>(s);
}

__device__ __forceinline__ void wave_inclusive_sum2(Sums& s) {
    row_inclusive_sum2(s);
    sum2_step<kRowBcast15, 0xa>(s);
    sum2_step<kRowBcast31, 0xc>(s);
}

// Stages a tile (and its halo) into LDS.  One pass of prefix sums: the key
// itself, X = sum of (size + 2^50 per pinned block), which is R << 50 | P
// exactly while P stays below 2^50 (every block below 2^37 bytes), C, and the
// pinned count R.  X[k], C[k] for k < end are written by their owners, the
// region end and the sentinel X[end + 1] = kEndKey by the last thread.  A
// tile holding a block of 2^37 bytes or more is staged plain instead: P =
// X - 2^50 R (exact modulo 2^64), R in sm.run, no halo.  Two barriers.
__device__ __forceinline__ TileState stage_tile(Smem& sm, const TileGeom& tg, uint32_t tid,
                                                TileRegs& r) {
    const uint32_t lane = tid & 63u;
    const uint32_t w = uniform(tid >> 6);
    const uint32_t nt = tg.nt, hm = tg.hm;
    constexpr uint64_t kRunOne = 1ull << kValBits;
    constexpr uint32_t kBigFlag = 1u << 31;  // in the R field of a wavefront total
    uint64_t hx = 0, hc = 0;
    bool hbig = false;
    if (tid < hm) {
        hx = r.hq + (r.hk >= COOP_PINNED ? kRunOne : 0);
        hc = r.hk == COOP_EVICTABLE ? r.hc : 0;
        hbig = (r.hq >> 32) >> kBigHiLog2;
    }
    const uint64_t hx_own = hx, hc_own = hc;
    const uint32_t i0 = tid * kItems;
    // thread-local exclusive sums (blocks past nt: empty free blocks; blocks
    // before the lead: empty pinned blocks)
    const uint32_t lead = tg.lead;
    Sums t{0, 0, 0};
    uint32_t hi_or = 0;
    uint32_t kinds[kItems];
    // one block: its kind k_j (masked blocks as described above) and size
    // s_j; r.sz / r.ct then hold the sums before it
    auto item = [&](uint32_t j, bool in) {
        const uint64_t s_j = in ? r.sz[j] : 0;
        const uint32_t raw = (r.kd[j >> 2] >> (8 * (j & 3))) & 0xffu;
        const uint32_t k_j = in ? raw
                                : (i0 + j < lead ? static_cast<uint32_t>(COOP_PINNED)
                                                 : static_cast<uint32_t>(COOP_FREE));
        kinds[j] = k_j;
        const uint64_t c_j = k_j == COOP_EVICTABLE ? r.ct[j] : 0;
        const uint32_t p_j = k_j >= COOP_PINNED ? 1u : 0u;
        r.sz[j] = t.q;
        r.ct[j] = t.c;
        t.q += s_j + (static_cast<uint64_t>(p_j) << kValBits);
        t.c += c_j;
        t.r += p_j;
        hi_or |= static_cast<uint32_t>(s_j >> 32);
    };
    if (nt == kTile && lead == 0) {
        // a whole tile from the snapshot's blocks (uniform): nothing masked
#pragma unroll
        for (uint32_t j = 0; j < kItems; ++j) item(j, true);
    } else {
#pragma unroll
        for (uint32_t j = 0; j < kItems; ++j)
            item(j, (nt == kTile || i0 + j < nt) && i0 + j >= lead);
    }
    Sums wi = t;
    wave_inclusive_sum(wi);
    Sums hs{hx, hc, 0};
    if (w < 4 && hm) wave_inclusive_sum2(hs);
    const bool wbig = __ballot((hi_or >> kBigHiLog2) != 0) != 0;
    const bool whbig = __ballot(hbig) != 0;
    if (lane == 63) {
        sm.wsum[w] = Sums{wi.q, wi.c, wi.r | (wbig ? kBigFlag : 0u)};
        if (w < 4) sm.hsum[w] = Sums{hs.q, hs.c, whbig ? kBigFlag : 0u};
    }
    __syncthreads();
    // lanes 0..7: wavefront totals of the tile, 8..11: of the halo
    Sums bsum{0, 0, 0};
    if (lane < kWaves) bsum = sm.wsum[lane];
    else if (lane < kWaves + 4 && hm) bsum = sm.hsum[lane - kWaves];
    const uint64_t bigs = __ballot((bsum.r & kBigFlag) != 0);
    bsum.r &= ~kBigFlag;
    row_inclusive_sum(bsum);
    const Sums tile_tot = readlane(bsum, kWaves - 1);
    Sums carry = readlane(bsum, w ? w - 1 : 0);
    if (w == 0) carry = Sums{0, 0, 0};
    const uint64_t base_x = carry.q + wi.q - t.q, base_c = carry.c + wi.c - t.c;

    TileState ts;
    ts.tq = tile_tot.q;
    ts.tc = tile_tot.c;
    ts.tr = tile_tot.r;
    ts.packed = (bigs & ((1u << kWaves) - 1)) == 0;
    if (ts.packed) {
        const bool use_halo = hm && !(bigs >> kWaves);
        const Sums all_tot = readlane(bsum, kWaves + 3);
        // halo wavefront w < 4: tile total + the earlier halo wavefronts
        const uint32_t hl = kWaves - 1 + (w < 4 ? w : 0);
        const uint64_t hcarry_x = readlane64(bsum.q, hl), hcarry_c = readlane64(bsum.c, hl);
        ts.end = use_halo ? nt + hm : nt;
        ts.xend = use_halo ? all_tot.q : tile_tot.q;
        ts.xcend = use_halo ? all_tot.c : tile_tot.c;
        ts.endrun = static_cast<uint32_t>(ts.xend >> kValBits);
        if (i0 + kItems <= nt) {
            // Lanes 128 bytes apart would put the 16-byte stores of a
            // wavefront on a few LDS banks: lane t stores its four pairs of
            // boundary records in the order (q + t) & 3, which spreads the
            // wavefront over more of them.
            ulonglong2 px[kItems / 2], pc[kItems / 2];
#pragma unroll
            for (uint32_t q = 0; q < kItems / 2; ++q) {
                px[q] = ulonglong2{base_x + r.sz[2 * q], base_x + r.sz[2 * q + 1]};
                pc[q] = ulonglong2{base_c + r.ct[2 * q], base_c + r.ct[2 * q + 1]};
            }
            const uint32_t rot = tid & 3u;
            if (rot & 1u) {
                const ulonglong2 tx = px[0], tc = pc[0];
#pragma unroll
                for (uint32_t q = 0; q < 3; ++q) { px[q] = px[q + 1]; pc[q] = pc[q + 1]; }
                px[3] = tx; pc[3] = tc;
            }
            if (rot & 2u) {
                ulonglong2 tx = px[0], tc = pc[0];
                px[0] = px[2]; pc[0] = pc[2]; px[2] = tx; pc[2] = tc;
                tx = px[1]; tc = pc[1];
                px[1] = px[3]; pc[1] = pc[3]; px[3] = tx; pc[3] = tc;
            }
#pragma unroll
            for (uint32_t q = 0; q < kItems / 2; ++q) {
                const uint32_t at = i0 + 2 * ((q + rot) & 3u);
                // the two boundaries' (key, cost) records
                *reinterpret_cast<ulonglong2*>(&sm.kv[2 * at]) = ulonglong2{px[q].x, pc[q].x};
                *reinterpret_cast<ulonglong2*>(&sm.kv[2 * at + 2]) = ulonglong2{px[q].y, pc[q].y};
            }
        } else {
#pragma unroll
            for (uint32_t j = 0; j < kItems; ++j) {
                if (i0 + j < nt) {
                    sm.K(i0 + j) = base_x + r.sz[j];
                    sm.C(i0 + j) = base_c + r.ct[j];
                }
            }
        }
        if (use_halo && tid < hm) {
            // halo boundary nt + tid: carry + wavefront inclusive - own block
            sm.K(nt + tid) = hcarry_x + hs.q - hx_own;
            sm.C(nt + tid) = hcarry_c + hs.c - hc_own;
        }
    } else {
        uint32_t rr = carry.r + wi.r - t.r;  // pinned blocks before this thread's first block
        ts.end = nt;
        ts.endrun = tile_tot.r;
        ts.xend = tile_tot.q - (static_cast<uint64_t>(tile_tot.r) << kValBits);
        ts.xcend = tile_tot.c;
#pragma unroll
        for (uint32_t j = 0; j < kItems; ++j) {
            if (i0 + j < nt) {
                sm.K(i0 + j) = base_x + r.sz[j] - (static_cast<uint64_t>(rr) << kValBits);
                sm.C(i0 + j) = base_c + r.ct[j];
                sm.run[i0 + j] = static_cast<uint16_t>(rr);
            }
            rr += kinds[j] >= COOP_PINNED ? 1u : 0u;
        }
    }
    if (tid == kThreads - 1) {
        sm.K(ts.end) = ts.xend;
        sm.C(ts.end) = ts.xcend;
        sm.run[ts.end] = static_cast<uint16_t>(ts.endrun);
        sm.K(ts.end + 1) = kEndKey;  // sentinel end key
    }
    if (tid < kMaxSteps) sm.K(ts.end + 2 + tid) = kEndKey;  // what a merge reads past the sentinel
    __syncthreads();
    return ts;
}

// A ticket on a tagged counter (tag << shift | arrivals), which an earlier
// call may have left with its own tag: the first arrival of this call swaps
// in tag | 1; every later one, once it sees this call's tag, adds 1, so
// arrivals that come together queue at the atomic unit instead of retrying
// compare-and-swaps.  The count stays below 2^shift.  Returns the ticket,
// from 1.
__device__ uint64_t take_ticket(uint64_t* ctr, uint64_t tag, uint32_t shift) {
    uint64_t old = __hip_atomic_load(ctr, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    while ((old >> shift) != tag) {
        if (__hip_atomic_compare_exchange_strong(ctr, &old, (tag << shift) | 1ull, __ATOMIC_RELAXED,
                                                 __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT))
            return 1;
    }
    const uint64_t prev = __hip_atomic_fetch_add(ctr, 1ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    return (prev & ((1ull << shift) - 1)) + 1;
}

// Partial keys are read by whichever workgroup takes a snapshot's last
// ticket, possibly on another XCD, and the XCDs' L2 caches are not coherent
// with each other.  They are written and read with device-scope relaxed
// atomics, which act at the device-coherent level (stores written through,
// loads served from there): publishing them needs only the writes to have
// completed before the ticket is taken, and no L2 write-back, which a
// release on every writer would cost on every combine.  The reader issues
// its loads only after its ticket has come back, behind an acquire.
__device__ __forceinline__ void store_key_device(Key* p, const Key& k) {
    __hip_atomic_store(&p->cost, k.cost, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(&p->bytes, k.bytes, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(&p->start, k.start, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(&p->end, k.end, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ Key load_key_device(Key* p) {
    return Key{__hip_atomic_load(&p->cost, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT),
               __hip_atomic_load(&p->bytes, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT),
               __hip_atomic_load(&p->start, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT),
               __hip_atomic_load(&p->end, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)};
}

// Deferred entries, tile records and deferral bits are handed from one
// workgroup to another (of the same kernel or of the next one on the
// stream, possibly on another XCD) the same way: device-scope atomic
// stores and loads.  A plain load can return a copy of the line that a
// cache took before the writer's store (measured: entries of one call
// read back as zeros by the long kernel).
__device__ __forceinline__ void store_entry_device(uint4* p, const uint4& v) {
    uint64_t* w = reinterpret_cast<uint64_t*>(p);
    __hip_atomic_store(w, static_cast<uint64_t>(v.x) | (static_cast<uint64_t>(v.y) << 32), __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(w + 1, static_cast<uint64_t>(v.z) | (static_cast<uint64_t>(v.w) << 32), __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ uint4 load_entry_device(uint4* p) {
    uint64_t* w = reinterpret_cast<uint64_t*>(p);
    const uint64_t a = __hip_atomic_load(w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const uint64_t b = __hip_atomic_load(w + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    // every lane reads the same entry: taking the words from the first lane
    // keeps the control flow that depends on them scalar
    return make_uint4(uniform(static_cast<uint32_t>(a)), uniform(static_cast<uint32_t>(a >> 32)),
                      uniform(static_cast<uint32_t>(b)), uniform(static_cast<uint32_t>(b >> 32)));
}

__device__ __forceinline__ Key readlane_key(const Key& k, uint32_t lane) {
    return Key{readlane64(k.cost, lane), readlane64(k.bytes, lane), readlane64(k.start, lane),
               readlane64(k.end, lane)};
}

// Stores the workgroup's key for request q: the final result once the
// workgroup has covered the whole snapshot alone (and deferred nothing),
// else its partial slot.
__device__ __forceinline__ void store_answer(const Params& P, const Job& job, uint64_t q, const Key& k,
                                             uint64_t S, bool deferred) {
    if (job.last && job.direct && !deferred) P.out[q] = to_window(k, S);
    else store_key_device(P.part + q * P.pc + job.g, k);
}

// This wavefront's answer from per-lane bests: the lexicographic minimum,
// with its end taken from a lane that holds it.
template <bool kPacked = false>
__device__ __forceinline__ Key wave_answer(const Cand& best, uint64_t best_end, uint64_t tl,
                                           uint64_t S) {
    const Cand m = kPacked ? wave_argmin_packed(best) : wave_argmin(best);
    if (m.start == kNone32) return key_none();
    const uint64_t won = __ballot(best.start == m.start);
    const uint64_t e = readlane64(best_end, static_cast<uint32_t>(__builtin_ctzll(won)));
    return Key{m.cost, m.excess + S, tl + m.start, e};
}

__device__ __forceinline__ Key min_key(const Key& a, const Key& b) { return key_less(b, a) ? b : a; }

// The wavefront's answer from the merge of a packed region: the
// lexicographic minimum of the lanes' windows; its end is the first end key
// at or above the winner's target (a wavefront search; every lane active).
__device__ __forceinline__ Key merged_answer(const Smem& sm, const Cand& best, uint64_t tl, uint64_t S,
                                             uint64_t Sc, uint32_t end, uint32_t lane) {
    const Cand m = wave_argmin_packed(best);
    if (m.start == kNone32) return key_none();
    const uint64_t target = sm.K(m.start) + Sc;
    const uint32_t e = wave_lower_bound(m.start + 1, end + 1, lane,
                                        [&](uint32_t k) { return sm.K(k) >= target; });
    return Key{m.cost, m.excess + S, tl + m.start, tl + e};
}

// Request q has windows past the walk's limit (one lane): its bit for the
// chunk part, and the job's mark.
__device__ __forceinline__ void defer_request(const Params& P, Smem& sm, const Job& job, uint64_t q) {
    const uint64_t bit = q * P.pc + job.g;
    atomicOr(ext_of(P).bits + (bit >> 5), 1u << (bit & 31u));
    sm.defer_mark = job.hi - 1;
}

// The shortest-window search of one tile for every request of the job's
// slice (see the file comment, steps 2 and 3).  Wavefront w takes tasks
// w, w + kWaves, ...; task vw is slice vw % wpr of request vw / wpr.  The
// wavefront's n-th task keeps its state in lane n: request size (s_lane),
// running key over this workgroup's tiles of the snapshot (acc, one
// wavefront per request), and first pending start.  The first loop touches
// only LDS, so it never waits for the prefetched loads; the loads of the
// rarer paths (streaming past the staged region, more than 64 tasks per
// wavefront) come after it.
__device__ __forceinline__ void tile_requests(const Params& P, Smem& sm, const Job& job,
                                              const TileGeom& tg, const TileState& ts,
                                              uint32_t wpr, uint32_t tid, Key& acc,
                                              uint64_t s_lane) {
    const uint32_t lane = tid & 63u;
    const uint32_t w = uniform(tid >> 6);
    const uint64_t tl = tg.t0 - job.s0;
    const uint32_t nt = tg.nt, end = ts.end;
    const uint64_t vmask = ts.packed ? kValMask : kNone;
    const bool open = tg.t0 + end < job.s1;  // the region's last run may go on
    // walks past the staged region stop kWalkCap blocks past its end
    const uint64_t lim = tg.t0 + end + kWalkCap < job.s1 ? tg.t0 + end + kWalkCap : job.s1;
    const uint64_t tasks = job.K * wpr;
    const uint32_t wl2 = static_cast<uint32_t>(__builtin_ctz(wpr));
    const uint32_t lanes = 64u * wpr;
    auto request = [&](uint64_t vw) { return job.q0 + job.y + ((vw >> wl2) << P.slices_log2); };
    // this wavefront's tasks held in lanes
    const uint64_t mine = tasks > w ? (tasks - w + kWaves - 1) / kWaves : 0;
    const uint32_t held = mine < 64 ? static_cast<uint32_t>(mine) : 64u;
    uint32_t pend = nt;  // lane n: first pending start of task n
    // No window of a tile start crosses a pinned block, so every tile start
    // is merged by the end key that takes in the first pinned block after
    // the tile (its run id is above every tile start's target); the end keys
    // after it matter to no tile start.  Looked for only where leaving them
    // out can shorten the lanes' slices.
    uint32_t mend = end;
    if (ts.packed && end > nt + 1 &&
        merge_steps(2 * nt + 1, lanes) < merge_steps(nt + end, lanes)) {
        const uint64_t thr = ((sm.K(nt) >> kValBits) + 1) << kValBits;
        mend = wave_lower_bound(nt + 1, end + 1, lane, [&](uint32_t i) { return sm.K(i) >= thr; });
        mend = mend < end ? mend : end;
    }

    // ---- in-region windows of every held task
    for (uint32_t n = 0; n < held; ++n) {
        const uint64_t vw = w + static_cast<uint64_t>(kWaves) * n;
        const uint32_t sl = static_cast<uint32_t>(vw & (wpr - 1));
        const uint64_t S = readlane64(s_lane, wpr == 1 ? n : static_cast<uint32_t>(vw >> wl2));
        Cand best = cand_none();
        uint64_t best_end = 0;
        if (S != 0 && nt != 0) {
            const uint64_t Sc = S < (1ull << kValBits) ? S : (1ull << kValBits);
            const uint32_t gl = sl * 64u + lane;
            uint32_t e32 = 0;
            if (ts.packed) {
                const uint32_t total = nt + mend;
                const uint32_t L = merge_steps(total, lanes);
                const uint32_t d = gl * L < total ? gl * L : total;
                merge_pass(sm, nt, mend, d, L, Sc, best);
            } else {
                plain_pass(sm, nt, end, gl, lanes, S, best, e32);
            }
            best_end = tl + e32;
            if (open && sl == 0) {
                const uint32_t cur =
                    pending_start(sm, ts.packed, nt, ts.xend, ts.endrun, S, Sc, lane);
                if (lane == n) pend = cur;
            }
        }
        // in-region windows of a packed region: excess below 2^50
        Key k = ts.packed ? merged_answer(sm, best, tl, S, S < (1ull << kValBits) ? S : (1ull << kValBits),
                                          end, lane)
                          : wave_answer(best, best_end, tl, S);
        if (wpr == 1) {
            k = min_key(readlane_key(acc, n), k);
            if (lane == n) acc = k;
        } else if (lane == 0) {
            sm.slot[vw] = k;
            sm.slot_s[vw] = S;
        }
    }
    // ---- windows that leave the staged region (the region's last run goes
    // on), walked up to the end of the next tile; windows that go further
    // are left to coop_window_long_kernel, which is told by the job's mark
    uint64_t todo = __ballot(lane < held && pend < nt);
    while (todo) {
        const uint32_t n = static_cast<uint32_t>(__builtin_ctzll(todo));
        todo &= todo - 1;
        const uint64_t vw = w + static_cast<uint64_t>(kWaves) * n;
        const uint64_t S = readlane64(s_lane, wpr == 1 ? n : static_cast<uint32_t>(vw >> wl2));
        Cand best = cand_none();
        uint64_t best_end = 0;
        WalkState ws{tg.t0 + end, ts.xend & vmask, ts.xcend, readlane32(pend, n), false};
        walk_pass(P, sm, lane, nt, lim, job.s0, job.s1, vmask, S, ws, best, best_end);
        if (ws.cur < nt && !ws.closed && lane == 0) defer_request(P, sm, job, request(vw));
        const Key k = wave_answer(best, best_end, tl, S);
        if (wpr == 1) {
            const Key a = min_key(readlane_key(acc, n), k);
            if (lane == n) acc = a;
        } else if (lane == 0) {
            sm.slot[vw] = min_key(sm.slot[vw], k);
        }
    }
    if (wpr == 1) {
        // (results of the held tasks: after the barrier that ends the tile)
        // ---- tasks past 64 per wavefront: running keys in the partial slots
        for (uint64_t vw = w + 64ull * kWaves; vw < tasks; vw += kWaves) {
            const uint64_t q = request(vw);
            const uint64_t S = ld_const(P.req_size, q);
            Cand best = cand_none();
            uint64_t best_end = 0;
            Key km = key_none();
            if (S != 0 && nt != 0) {
                const uint64_t Sc = S < (1ull << kValBits) ? S : (1ull << kValBits);
                uint32_t e32 = 0;
                if (ts.packed) {
                    const uint32_t total = nt + mend;
                    const uint32_t L = merge_steps(total, 64u);
                    const uint32_t d = lane * L < total ? lane * L : total;
                    Cand bm = cand_none();
                    merge_pass(sm, nt, mend, d, L, Sc, bm);
                    km = merged_answer(sm, bm, tl, S, Sc, end, lane);
                } else {
                    plain_pass(sm, nt, end, lane, 64u, S, best, e32);
                }
                best_end = tl + e32;
                if (open) {
                    const uint32_t cur =
                        pending_start(sm, ts.packed, nt, ts.xend, ts.endrun, S, Sc, lane);
                    if (cur < nt) {
                        WalkState ws{tg.t0 + end, ts.xend & vmask, ts.xcend, cur, false};
                        walk_pass(P, sm, lane, nt, lim, job.s0, job.s1, vmask, S, ws, best, best_end);
                        if (ws.cur < nt && !ws.closed && lane == 0) defer_request(P, sm, job, q);
                    }
                }
            }
            Key k = min_key(km, wave_answer(best, best_end, tl, S));
            if (!job.first) k = min_key(load_key_device(P.part + q * P.pc + job.g), k);
            // (a result of a snapshot covered by this workgroup alone is
            // copied to out after the barrier that ends the tile)
            if (lane == 0) store_key_device(P.part + q * P.pc + job.g, k);
        }
    }
    // (shared requests: the wavefronts' keys stay in sm.slot for
    // reduce_shared, after the barrier that ends the tile)
}

// Shared requests (wpr > 1): thread j reduces the wpr keys of request j that
// the wavefronts left in sm.slot, into its running key, and writes the
// result after the snapshot's last tile.  Called after the barrier that
// ends the tile, so every key is in place; the next tile's keys are written
// only after the next staging barriers, which wavefront 0 reaches after this.
__device__ __forceinline__ void reduce_shared(const Params& P, const Smem& sm, const Job& job,
                                              uint32_t wpr, uint32_t tid, Key& acc, bool deferred) {
    if (tid >= job.K) return;
    const uint32_t wl2 = static_cast<uint32_t>(__builtin_ctz(wpr));
    Key k = sm.slot[tid << wl2];
    for (uint32_t u = 1; u < wpr; ++u) k = min_key(k, sm.slot[(tid << wl2) + u]);
    acc = job.first ? k : min_key(acc, k);
    if (job.last)
        store_answer(P, job, job.q0 + job.y + (static_cast<uint64_t>(tid) << P.slices_log2), acc,
                     sm.slot_s[tid << wl2], deferred);
}

// After the last tile of (b, y) in the current chunk, when other chunks
// hold tiles of it too: a ticket on the (b, y) counter; the last of the G
// arrivals reduces the G partial keys of every request of the slice.  The
// partial keys are device-scope atomics (store_key_device), so the ticket
// only has to follow the completion of this workgroup's writes.
__device__ void combine_partials(const Params& P, const Job& job, uint32_t tid, uint32_t& last_flag) {
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    __builtin_amdgcn_s_waitcnt(0);  // every write of this thread has completed
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    __syncthreads();
    if (tid == 0) {
        uint64_t* ctr = P.counters + static_cast<uint64_t>(job.y) * P.num_segments + job.b;
        last_flag = take_ticket(ctr, P.epoch, kEpochShift) == job.G;
    }
    __syncthreads();
    if (!last_flag) return;
    // The last arrival reads what the others published: an agent-scope
    // acquire, so that no line its CU cached earlier is read (the partial
    // keys are read with device-scope atomics anyway).
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
    // tpr threads per request (a power of two within a wavefront), each
    // taking every tpr-th slot; then a shuffle reduction inside the group
    uint32_t tpr = 64;
    while (tpr > 1 && static_cast<uint64_t>(tpr) * job.K > kThreads) tpr >>= 1;
    const uint32_t groups = kThreads / tpr, sub = tid % tpr;
    for (uint64_t k0 = 0; k0 < job.K; k0 += groups) {
        const uint64_t k = k0 + tid / tpr;
        const bool act = k < job.K;
        const uint64_t q = job.q0 + job.y + ((act ? k : 0) << P.slices_log2);
        Key best = key_none();
        if (act) {
            for (uint64_t gg = sub; gg < job.G; gg += tpr) {
                const Key o = load_key_device(P.part + q * P.pc + gg);
                if (key_less(o, best)) best = o;
            }
        }
        for (uint32_t m = tpr >> 1; m >= 1; m >>= 1) {
            Key o;
            o.cost = __shfl_xor(best.cost, static_cast<int>(m), 64);
            o.bytes = __shfl_xor(best.bytes, static_cast<int>(m), 64);
            o.start = __shfl_xor(best.start, static_cast<int>(m), 64);
            o.end = __shfl_xor(best.end, static_cast<int>(m), 64);
            if (key_less(o, best)) best = o;
        }
        if (act && sub == 0) P.out[q] = to_window(best, P.req_size[q]);
    }
}

// The most tiles of any snapshot (as tile_geom cuts them), over the
// workgroup: queued chunks must be long enough that no snapshot spans more
// than pc - 2 of them.  Offsets are clamped as in next_job.
__device__ uint64_t max_tiles(const Params& P, Smem& sm, uint32_t tid) {
    uint64_t m = 1;
    for (uint64_t b = tid; b < P.num_segments; b += kThreads) {
        const uint64_t s1 = P.seg[b + 1] < P.num_blocks ? P.seg[b + 1] : P.num_blocks;
        const uint64_t s0 = P.seg[b] < s1 ? P.seg[b] : s1;
        const uint64_t t = (s1 - (s0 & ~7ull) + kTile - 1) >> kTileLog2;
        m = t > m ? t : m;
    }
    for (int o = 32; o >= 1; o >>= 1) {
        const uint64_t x = __shfl_xor(m, o, 64);
        m = x > m ? x : m;
    }
    if ((tid & 63u) == 0) sm.slot_s[tid >> 6] = m;
    __syncthreads();
    m = sm.slot_s[0];
    for (uint32_t i = 1; i < kWaves; ++i) m = sm.slot_s[i] > m ? sm.slot_s[i] : m;
    __syncthreads();
    return m;
}

// Claims the next queued chunk for the workgroup (every thread calls this;
// one atomic, then the result goes out through LDS).  Returns a chunk index,
// kQDone once the queue has run dry, or kQEmpty if the queue word still
// holds an earlier call's tag (this call's reset has not landed yet).
__device__ uint64_t claim_chunk(const Params& P, Smem& sm, uint32_t tid) {
    if (tid == 0) {
        const uint64_t old =
            __hip_atomic_fetch_add(P.queue, 1ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        uint64_t r = kQEmpty;
        if ((old >> 32) == P.qtag) {
            const uint64_t c = P.grid + (old & 0xffffffffull);
            r = c < P.nchunks ? c : kQDone;
        }
        sm.claim = r;
    }
    __syncthreads();
    const uint64_t r = sm.claim;
    __syncthreads();  // sm.claim is written again by the next claim
    if (r == kQEmpty) __builtin_amdgcn_s_sleep(16);
    return r;
}

// Position of the walk over the units: the current chunk and its units, and
// unit u as (slice y, tile id v).
struct Walk {
    uint64_t chunk;
    uint32_t u_begin, u_end, y, v;  // units, slice and tile id: below 2^32
};

__device__ __forceinline__ void walk_chunk(const Params& P, uint64_t c, Walk& wk) {
    wk.chunk = c;
    uint64_t b, e;
    chunk_range(P, c, b, e);
    wk.u_begin = static_cast<uint32_t>(b);
    wk.u_end = static_cast<uint32_t>(e);
    wk.y = static_cast<uint32_t>(div_magic(wk.u_begin, P.nv_magic));
    wk.v = wk.u_begin - wk.y * P.num_virtual;
}

// The first job at unit u or later: in the current chunk, else in the
// reserve chunk (claimed earlier), else in chunks claimed now, until the
// queue runs dry.  Uniform across the workgroup (claims synchronise it).
__device__ __forceinline__ bool find_job(const Params& P, Smem& sm, uint32_t tid, Cursor& cur,
                                         bool& have_cursor, Walk& wk, uint64_t& reserve, uint64_t u,
                                         Job& job) {
    for (;;) {
        if (next_job(P, cur, have_cursor, u, wk.y, wk.v, wk.u_begin, wk.u_end, wk.chunk, job))
            return true;
        u = wk.u_end;  // where next_job left (y, v)
        if (reserve == kQDone) return false;
        if (reserve == kQEmpty) {
            reserve = claim_chunk(P, sm, tid);
            continue;  // (next_job returns at once: u is the chunk end)
        }
        walk_chunk(P, reserve, wk);
        reserve = kQEmpty;
        have_cursor = false;  // a later chunk: locate from scratch
        u = wk.u_begin;
    }
}

// A call replayed from a graph: its tags come from the tag word, advanced by
// the kernel before the search on the stream, so every workgroup (of both
// search kernels) reads the same value; P.epoch holds a per-process salt.
__device__ __forceinline__ void graph_tags(Params& P) {
    if (!P.tag_word) return;
    const uint64_t t = __hip_atomic_load(P.tag_word, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    P.epoch = kGraphTag | ((t * kTagOdd + P.epoch) & kTagMask);
    P.qtag = queue_tag(P.epoch);
}

// After the last tile of a job with one wavefront per request: the held
// tasks' keys (lane n of wavefront w: request w + kWaves * n) go to out, or
// to the partial slot when other chunks hold tiles of the snapshot or a
// wavefront deferred windows; keys of tasks past 64 per wavefront, kept in
// the partial slots, are copied to out when the workgroup covered the whole
// snapshot alone and deferred nothing.
__device__ __forceinline__ void finish_held(const Params& P, const Job& job, uint32_t tid, const Key& acc,
                                            uint64_t s_lane, bool deferred) {
    const uint32_t lane = tid & 63u;
    const uint32_t w = uniform(tid >> 6);
    const uint64_t mine = job.K > w ? (job.K - w + kWaves - 1) / kWaves : 0;
    const uint32_t held = mine < 64 ? static_cast<uint32_t>(mine) : 64u;
    if (lane < held)
        store_answer(P, job, job.q0 + job.y + ((w + static_cast<uint64_t>(kWaves) * lane) << P.slices_log2),
                     acc, s_lane, deferred);
    if (job.direct && !deferred && lane == 0) {
        // the same lane stored these slots during the requests
        for (uint64_t vw = w + 64ull * kWaves; vw < job.K; vw += kWaves) {
            const uint64_t q = job.q0 + job.y + (vw << P.slices_log2);
            P.out[q] = to_window(load_key_device(P.part + q * P.pc + job.g), ld_const(P.req_size, q));
        }
    }
}

// Appends the job's part of the chunk (its units, g and G) to the deferred
// list (one thread).  The list's word carries the call's queue tag, so the
// first append of a call restarts the count.
__device__ void defer_job(const Params& P, const Job& job) {
    const Ext e = ext_of(P);
    const uint64_t idx = take_ticket(e.defer_word, P.qtag, 32) - 1;
    if (idx < P.defer_cap) store_entry_device(e.entries + idx, make_uint4(job.lo, job.hi, job.g, job.G));
}

// The record of tile p >= 1 of the job's snapshot, from what staging
// computed (one thread): bytes of all its blocks, cost of its evictable
// blocks, its pinned count.  Every unit of the tile writes the same values;
// coop_window_long_kernel, next on the stream, reads them.
__device__ __forceinline__ void publish_record(const Params& P, const Job& job, const TileState& ts) {
    const uint64_t idx = (job.s0 >> kTileLog2) + job.p - 1;
    if (job.p == 0 || idx >= (P.num_blocks >> kTileLog2)) return;
    const Ext e = ext_of(P);
    __hip_atomic_store(e.rec_p + idx, ts.tq - (static_cast<uint64_t>(ts.tr) << kValBits), __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(e.rec_c + idx, ts.tc, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(e.rec_r + idx, static_cast<uint64_t>(ts.tr), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__global__ __launch_bounds__(kThreads, 4) void coop_window_search_kernel(Params Pin) {
    __shared__ Smem sm;
    __shared__ uint32_t last_flag;
    const uint32_t tid = threadIdx.x;
    const uint32_t w = uniform(tid >> 6);
    Params P = Pin;
    graph_tags(P);
    // The queue, when there is one: workgroup 0 stamps this call's tag; claims
    // that reach the word before the stamp see an old tag and try again.
    // Queued chunks are sized from the snapshots' tile counts, the same in
    // every workgroup.
    uint64_t reserve = kQDone;
    if (P.queue_on) {
        if (blockIdx.x == 0 && tid == 0)
            __hip_atomic_store(P.queue, static_cast<uint64_t>(P.qtag) << 32, __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
        const uint64_t tmax = max_tiles(P, sm, tid);
        const uint64_t need = (tmax + P.pc - 3) / (P.pc - 2);
        P.c2 = static_cast<uint32_t>(need > P.c2 ? need : P.c2);
        P.c2_magic = P.c2 == 1 ? 0 : ~0ull / P.c2 + 1;
        P.nchunks = P.grid + (static_cast<uint64_t>(P.units) - P.u1 + P.c2 - 1) / P.c2;
        reserve = kQEmpty;
    }
    if (tid == 0) sm.defer_mark = kNone32;  // read after the barriers to come
    Walk wk;
    walk_chunk(P, blockIdx.x, wk);
    Cursor cur;
    bool have_cursor = false;
    Job job;
    if (!find_job(P, sm, tid, cur, have_cursor, wk, reserve, wk.u_begin, job)) return;
    TileGeom tg = tile_geom(job);
    TileRegs regs;
    issue_loads(P, tg, tid, regs);
    // running keys of the current (snapshot, slice) over the chunk's tiles:
    // lane j of wavefront w holds request w + kWaves * j (one wavefront per
    // request), thread j request j (shared requests)
    Key acc = key_none();
    for (;;) {
        // The thread index, opaque to the compiler: values derived from it
        // are recomputed in every iteration instead of being kept live (and
        // spilled) across the loop.
        uint32_t t = threadIdx.x;
        asm volatile("" : "+v"(t));
        uint32_t wpr = 1;
        if (job.K < kWaves) {
            uint32_t k2 = 1;
            while (k2 < job.K) k2 <<= 1;
            wpr = kWaves / k2 < kMaxWpr ? kWaves / k2 : kMaxWpr;
        }
        // The request sizes, one per lane (see tile_requests), loaded now and
        // waited for before the prefetch below: loads complete in issue
        // order, so a load waited on during the requests would wait for the
        // prefetch too.
        uint64_t s_lane = 0;
        {
            const uint64_t rl = wpr == 1 ? w + static_cast<uint64_t>(kWaves) * (t & 63u) : (t & 63u);
            if (rl < job.K) s_lane = P.req_size[job.q0 + job.y + (rl << P.slices_log2)];
        }
        // The next tile, found before staging: its scalar loads (snapshot
        // offsets) then complete during the staging barriers.  An outstanding
        // scalar load would hold up every LDS wait of the request phase (they
        // share a counter).  At the end of a chunk this enters the reserve
        // chunk, or claims one if the reserve is empty.
        Job next;
        ++wk.v;
        const bool has_next = find_job(P, sm, t, cur, have_cursor, wk, reserve, job.u + 1, next);
        // ---- 1. stage the tile whose blocks are in (or on their way to) regs
        const TileState ts = stage_tile(sm, tg, t, regs);
        if (t == 0 && job.p != 0) publish_record(P, job, ts);
        asm volatile("" : "+v"(s_lane));
        if (job.first) acc = key_none();
        // ---- keep a chunk in reserve (no vector load is in flight here, so
        // the claim waits only for itself)
        if (reserve == kQEmpty) reserve = claim_chunk(P, sm, t);
        // ---- prefetch the next tile
        const TileGeom tn = has_next ? tile_geom(next) : TileGeom{tg.t0, 0u, 0u, 0u};
        issue_loads(P, tn, t, regs);
        // ---- 2./3. the requests, at a raised wave priority up to the end of
        // the tile, so that the other workgroup on the CU, when it stages a
        // tile meanwhile, yields issue slots to them
        __builtin_amdgcn_s_setprio(1);
        tile_requests(P, sm, job, tg, ts, wpr, t, acc, s_lane);
        __syncthreads();  // LDS is restaged next
        // a job some wavefront deferred keeps its keys in the partial slots
        const bool deferred = job.last && sm.defer_mark == job.hi - 1;
        if (wpr == 1 && job.last) finish_held(P, job, t, acc, s_lane, deferred);
        if (wpr > 1) reduce_shared(P, sm, job, wpr, t, acc, deferred);
        if (job.last) {
            if (deferred) {
                if (t == 0) defer_job(P, job);
            } else if (!job.direct) {
                combine_partials(P, job, t, last_flag);
            }
        }
        __builtin_amdgcn_s_setprio(0);
        if (!has_next) break;
        job = next;
        tg = tn;
    }
}

// ---------------------------------------------------------------------------
// Windows that end more than kWalkCap blocks past the staged region
// ---------------------------------------------------------------------------
//
// coop_window_long_kernel runs after the search kernel on the stream, so it
// sees every tile record and every deferred entry of the call; no
// workgroup of it waits for another.  Each workgroup takes deferred
// entries and stages their tiles again.  For every request that deferred,
// the pending starts of a tile are resolved stretch by stretch: the
// workgroup sums the tile records forward from the region end, 512 tiles a
// round, up to the first tile that holds a pinned block or where the window
// of the first pending start ends; that tile (from the region end on, if the
// region reaches into it) is staged into a second LDS buffer as plain byte
// and cost prefixes, cut at its first pinned block, and the byte targets the
// pending starts still need past the stretch start are merged with its
// prefixes as the in-region merge does.  Starts whose windows end further go
// on to the next stretch.  Every value that decides a barrier's path (the
// tile, the stretch, the next pending start) comes from LDS, the same for
// every wavefront.

struct Sums3 {
    uint64_t q, c, r;
};

__device__ __forceinline__ Sums3 add3(const Sums3& a, const Sums3& b) {
    return Sums3{a.q + b.q, a.c + b.c, a.r + b.r};
}

template <int Ctrl, int RowMask>
__device__ __forceinline__ void sum3_step(Sums3& s) {
    add_dpp64<Ctrl, RowMask>(s.q);
    add_dpp64<Ctrl, RowMask>(s.c);
    add_dpp64<Ctrl, RowMask>(s.r);
}

__device__ __forceinline__ void wave_inclusive_sum3(Sums3& s) {
    sum3_step<kRowShr1, 0xf>(s);
    sum3_step<kRowShr2, 0xf>(s);
    sum3_step<kRowShr4, 0xf>(s);
    sum3_step<kRowShr8, 0xf>(s);
    sum3_step<kRowBcast15, 0xa>(s);
    sum3_step<kRowBcast31, 0xc>(s);
}

// Boundaries of a staged stretch past the region (a tile at most) and the
// end keys a merge may read past its last one.
constexpr uint32_t kEndPad = 64;
constexpr uint32_t kFarCache = 64;
constexpr uint32_t kEndN = kTile + 2 + kEndPad;

// The long kernel's second LDS buffer: the stretch's byte and cost
// prefixes (entry 0 is the stretch start), and scratch for workgroup
// reductions and broadcasts.
struct EndSmem {
    uint64_t pb[kEndN];
    uint64_t cb[kEndN];
    Sums3 wtot[kWaves];
    uint32_t wpin[kWaves];
    Key slot[kWaves];
    uint64_t found;     // the tile the search stopped at
    uint64_t fq, fc;    // bytes and cost from the region end to that tile's start
    // Where the first record search of request far_q's last tile stopped:
    // the region end far_ge (global), the tile far_k and the bytes and cost
    // from far_ge to its start (slot q % kFarCache).
    uint64_t far_q[kFarCache], far_ge[kFarCache], far_k[kFarCache], far_b[kFarCache], far_c[kFarCache];
};

// Where the run of a staged region's last run goes on past the region end:
// the first tile t >= kmin that holds a pinned block past the region end or
// whose end is at least `need` bytes past it (whole workgroup; every thread
// gets the same result, through LDS).  Tile records are summed forward from
// tile kmin, kThreads of them a round; `carry` holds the bytes, cost and
// pinned count from the region end to the start of tile kmin.  Returns
// tiles when no tile qualifies; else the tile, with the bytes and cost from
// the region end to its start in fq, fc.
__device__ uint64_t find_tile(const Ext& e, EndSmem& es, int64_t rb, uint64_t nrec, uint64_t tiles,
                              uint64_t kmin, Sums3 carry, uint64_t need, uint64_t& fq, uint64_t& fc) {
    const uint32_t tid = threadIdx.x;
    const uint32_t lane = tid & 63u;
    const uint32_t w = uniform(tid >> 6);
    for (uint64_t t0 = kmin;; t0 += kThreads) {
        const uint64_t t = t0 + tid;
        Sums3 v{0, 0, 1};  // past the snapshot's last tile: a wall
        if (t < tiles) {
            const int64_t i = rb + static_cast<int64_t>(t);
            v = i < 0 || static_cast<uint64_t>(i) >= nrec
                    ? Sums3{0, 0, 0}
                    : Sums3{__hip_atomic_load(e.rec_p + i, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT),
                            __hip_atomic_load(e.rec_c + i, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT),
                            __hip_atomic_load(e.rec_r + i, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)};
        }
        Sums3 s = v;
        wave_inclusive_sum3(s);
        if (lane == 63) es.wtot[w] = s;
        __syncthreads();
        Sums3 before = carry, tot = carry;
        for (uint32_t k = 0; k < kWaves; ++k) {
            const Sums3 x = es.wtot[k];
            if (k < w) before = add3(before, x);
            tot = add3(tot, x);
        }
        const Sums3 incl = add3(before, s);  // region end to the end of tile t
        const bool stop = incl.r != 0 || incl.q >= need;
        const uint64_t m = __ballot(stop);
        if (lane == 0) es.wpin[w] = m ? w * 64u + static_cast<uint32_t>(__builtin_ctzll(m)) : kNone32;
        __syncthreads();
        uint32_t first = kNone32;
        for (uint32_t k = 0; k < kWaves; ++k) first = es.wpin[k] < first ? es.wpin[k] : first;
        if (first != kNone32 && tid == first) {
            es.found = t;
            es.fq = incl.q - v.q;
            es.fc = incl.c - v.c;
        }
        __syncthreads();
        if (first != kNone32) {
            const uint64_t k = es.found;
            fq = es.fq;
            fc = es.fc;
            __syncthreads();  // es is written again by the next search
            return k < tiles ? k : tiles;
        }
        carry = tot;
    }
}

// Stages blocks [bs, be) (at most kTile) as byte and cost prefixes from the
// stretch start (whole workgroup); returns the blocks before the first
// pinned one (boundaries [0, m] are usable).  The kEndPad keys after
// boundary m are set above every target.
__device__ uint32_t stage_stretch(const Params& P, EndSmem& es, uint64_t bs, uint64_t be, uint32_t tid) {
    const uint32_t lane = tid & 63u;
    const uint32_t w = uniform(tid >> 6);
    const uint32_t n = static_cast<uint32_t>(be - bs);
    const uint32_t i0 = tid * kItems;
    uint64_t sq[kItems], sc[kItems];
    Sums3 t{0, 0, 0};
    uint32_t fp = kNone32;
    // every load is issued before any is used: the costs are loaded whatever
    // the kinds, then masked, so the stretch takes one round trip, not two
    uint32_t kd[kItems];
#pragma unroll
    for (uint32_t j = 0; j < kItems; ++j) {
        const uint32_t i = i0 + j;
        kd[j] = COOP_FREE;
        sq[j] = 0;
        sc[j] = 0;
        if (i < n) {
            kd[j] = P.kind[bs + i];
            sq[j] = P.size[bs + i];
            sc[j] = P.cost[bs + i];
        }
    }
#pragma unroll
    for (uint32_t j = 0; j < kItems; ++j) {
        const uint32_t i = i0 + j;
        const uint32_t k = kd[j];
        const uint64_t s = sq[j], c = k == COOP_EVICTABLE ? sc[j] : 0;
        if (k >= COOP_PINNED && fp == kNone32) fp = i;
        t.q += s;
        t.c += c;
        sq[j] = t.q;
        sc[j] = t.c;
    }
    Sums3 wi = t;
    wave_inclusive_sum3(wi);
    for (int o = 32; o >= 1; o >>= 1) {
        const uint32_t x = __shfl_xor(fp, o, 64);
        fp = x < fp ? x : fp;
    }
    if (lane == 63) es.wtot[w] = wi;
    if (lane == 0) es.wpin[w] = fp;
    __syncthreads();
    Sums3 carry{0, 0, 0};
    uint32_t first = n;
    for (uint32_t k = 0; k < kWaves; ++k) {
        if (k < w) carry = add3(carry, es.wtot[k]);
        first = es.wpin[k] < first ? es.wpin[k] : first;
    }
    const uint64_t bq = carry.q + wi.q - t.q, bc = carry.c + wi.c - t.c;
#pragma unroll
    for (uint32_t j = 0; j < kItems; ++j) {
        if (i0 + j < n) {
            es.pb[i0 + j + 1] = bq + sq[j];
            es.cb[i0 + j + 1] = bc + sc[j];
        }
    }
    if (tid == 0) {
        es.pb[0] = 0;
        es.cb[0] = 0;
    }
    __syncthreads();  // the prefixes past the first pinned block are overwritten next
    if (tid < kEndPad + 1) es.pb[first + 1 + tid] = kNone;
    __syncthreads();
    return first;
}

// This thread's slice of the merge of the pending starts [cur, nA) of the
// staged region with the stretch's boundaries 1..m.  Start i still needs
// T_i = S - G - (bytes from i to the region end) past the stretch start (G:
// the bytes from the region end to the stretch start); it is taken at the
// first boundary whose prefix reaches T_i, which ends its shortest window.
// Candidates fold into best / best_end (end snapshot-local).
__device__ void stretch_merge(const Smem& sm, const EndSmem& es, const TileState& ts, uint64_t vmask,
                              uint32_t cur, uint32_t nA, uint32_t m, uint64_t S, uint64_t G, uint64_t GC,
                              uint64_t bs_local, uint32_t tid, Cand& best, uint64_t& best_end) {
    const uint32_t na = nA - cur, total = na + m;
    const uint32_t L = merge_steps(total, kThreads);
    const uint32_t d = tid * L < total ? tid * L : total;
    auto target = [&](uint32_t i) -> uint64_t {
        return i < na ? S - G - ((ts.xend - sm.K(cur + i)) & vmask) : kNone;
    };
    uint32_t lo = d > m ? d - m : 0, hi = d < na ? d : na;
    while (lo < hi) {
        const uint32_t mid = (lo + hi) >> 1;
        const bool before = target(mid) <= es.pb[d - mid];
        lo = before ? mid + 1 : lo;
        hi = before ? hi : mid;
    }
    uint32_t ia = lo, ib = d - lo + 1;
    uint64_t bc = kNone, bx = kNone;
    uint32_t bi = kNone32, bk = 0;
    for (uint32_t s = 0; s < L; ++s) {
        const uint64_t T = target(ia), key = es.pb[ib];
        const bool take = key >= T;
        const bool valid = take & (ia < na) & (ib <= m);
        const uint64_t cost = (ts.xcend - sm.C(cur + (ia < na ? ia : 0))) + GC + es.cb[ib];
        const uint64_t ex = key - T;
        const bool better = valid & ((cost < bc) | ((cost == bc) & (ex < bx)));
        bc = better ? cost : bc;
        bx = better ? ex : bx;
        bi = better ? cur + ia : bi;
        bk = better ? ib : bk;
        ia += take ? 1u : 0u;
        ib += take ? 0u : 1u;
    }
    if (bi != kNone32) {
        const Cand c{bc, bx, bi};
        if (cand_less(c, best)) {
            best = c;
            best_end = bs_local + bk;
        }
    }
}

// The blocks [bs, be) whose prefixes the stretch buffer holds (bs = kNone:
// none), and m, the boundaries before the first pinned one.
struct Staged {
    uint64_t bs, be;
    uint32_t m;
};

// From the previous tile of the entry to this one: the previous region end
// (global; kNone when there is no previous tile), and, when no pinned block
// lies between the two region ends (same_run), the bytes and cost between.
struct Between {
    uint64_t prev_ge, q, c;
    bool same_run;
};

// The windows of the pending starts of a staged tile that end more than
// kWalkCap blocks past the region (whole workgroup; every thread gets the
// workgroup's key).  run_left: the bytes from the region end to the end of
// its last run, kNone until a search of this tile has reached that end; a
// request that needs more is answered at once.
__device__ Key far_windows(const Params& P, const Smem& sm, EndSmem& es, const Job& job,
                           const TileGeom& tg, const TileState& ts, uint64_t q, uint64_t S,
                           uint64_t& run_left, Staged& staged, const Between& bt) {
    const uint32_t tid = threadIdx.x;
    const uint32_t lane = tid & 63u;
    const uint32_t w = uniform(tid >> 6);
    const uint32_t nA = tg.nt;
    const uint64_t vmask = ts.packed ? kValMask : kNone;
    const uint64_t Sc = S < (1ull << kValBits) ? S : (1ull << kValBits);
    uint32_t cur = pending_start(sm, ts.packed, nA, ts.xend, ts.endrun, S, Sc, lane);
    // No pending start, or a window from the first one needs more bytes past
    // the region end than the run has left there (none from a later start
    // either): no window (the same in every thread).
    if (cur >= nA || (run_left != kNone && S - ((ts.xend - sm.K(cur)) & vmask) > run_left))
        return key_none();
    Cand best = cand_none();
    uint64_t best_end = 0;
    {
        const Ext e = ext_of(P);
        const uint64_t a = job.s0 & ~7ull;                       // tile k starts at a + k * kTile
        const int64_t rb = static_cast<int64_t>(job.s0 >> kTileLog2) - 1;  // record of tile k: rb + k
        const uint64_t nrec = P.num_blocks >> kTileLog2;
        // the staged part of tile p + 1 (the halo): bytes, cost, pinned count;
        // from the region end to the start of tile p + 1 is minus these
        uint64_t hq = 0, hc = 0, hr = 0;
        if (ts.end > nA) {
            const uint64_t dd = ts.xend - sm.K(nA);
            hq = dd & kValMask;
            hr = dd >> kValBits;
            hc = ts.xcend - sm.C(nA);
        }
        const uint64_t ge = tg.t0 + ts.end;  // global index of the region end
        uint64_t kmin = job.p + 1;
        Sums3 carry{0 - hq, 0 - hc, 0 - hr};  // region end to the start of tile kmin
        // The previous tile's first pending start lies earlier in the same
        // run, so this tile's first window ends no earlier: its search may
        // start where that one stopped (past this region), with the sums
        // from there less the bytes and cost between the two region ends
        // (no pinned block there, nor before that tile).
        const uint32_t slot = static_cast<uint32_t>(q % kFarCache);
        if (bt.same_run && es.far_q[slot] == q && es.far_ge[slot] == bt.prev_ge &&
            es.far_k[slot] >= job.p + 2) {
            kmin = es.far_k[slot];
            carry = Sums3{es.far_b[slot] - bt.q, es.far_c[slot] - bt.c, 0};
        }
        bool first_search = true;
        for (;;) {
            const uint64_t need = S - ((ts.xend - sm.K(cur)) & vmask);
            uint64_t fq, fc;
            const uint64_t k = find_tile(e, es, rb, nrec, job.tiles, kmin, carry, need, fq, fc);
            if (first_search && tid == 0) {  // read by the next tile's search (after barriers)
                es.far_q[slot] = k < job.tiles ? q : kNone;
                es.far_ge[slot] = ge;
                es.far_k[slot] = k;
                es.far_b[slot] = fq;
                es.far_c[slot] = fc;
            }
            first_search = false;
            if (k >= job.tiles) {  // the run ends with the snapshot, below `need` bytes
                run_left = fq;
                break;
            }
            const uint64_t ks = a + (k << kTileLog2), ke = ks + kTile;
            const uint64_t bs = ks > ge ? ks : ge, be = ke < job.s1 ? ke : job.s1;
            // bytes and cost from the region end to the stretch start
            const uint64_t G = k == job.p + 1 ? 0 : fq;
            const uint64_t GC = k == job.p + 1 ? 0 : fc;
            // (the buffer's content depends on [bs, be) alone: a tile's last
            // stretch is often the next tile's first)
            if (staged.bs != bs || staged.be != be) {
                staged.m = stage_stretch(P, es, bs, be, tid);
                staged.bs = bs;
                staged.be = be;
            }
            const uint32_t m = staged.m;
            const bool closed = m < be - bs || be == job.s1;
            stretch_merge(sm, es, ts, vmask, cur, nA, m, S, G, GC, bs - job.s0, tid, best, best_end);
            // the first start whose window ends past this stretch
            const uint64_t last = es.pb[m], es_last_c = es.cb[m];
            const uint32_t nxt = wave_lower_bound(cur, nA, lane, [&](uint32_t i) {
                return S - G - ((ts.xend - sm.K(i)) & vmask) > last;
            });
            __syncthreads();  // the stretch buffer is restaged next
            if (closed) run_left = G + last;  // the run ends in this stretch
            if (closed || nxt >= nA) break;
            // the stretch reached the end of tile k with no pinned block
            carry = Sums3{G + last, GC + es_last_c, 0};
            cur = nxt;
            kmin = k + 1;
        }
    }
    const Key wk = wave_answer(best, best_end, tg.t0 - job.s0, S);
    if (lane == 0) es.slot[w] = wk;
    __syncthreads();
    Key k = es.slot[0];
    for (uint32_t i = 1; i < kWaves; ++i) k = min_key(k, es.slot[i]);
    __syncthreads();  // es.slot is written again by the next call
    return k;
}

// Unit u of a deferred entry as a job (tile p of snapshot b for slice y,
// the entry's chunk part g of G); false if u names no tile.
__device__ bool entry_job(const Params& P, uint4 en, uint32_t u, Cursor& c, Job& job) {
    const uint32_t y = static_cast<uint32_t>(div_magic(u, P.nv_magic));
    const uint32_t v = u - y * P.num_virtual;
    cursor_locate(P, v, c);
    const uint64_t s1 = c.sb1 < P.num_blocks ? c.sb1 : P.num_blocks;
    const uint64_t s0 = c.sb < s1 ? c.sb : s1;
    const uint64_t q1 = c.rb1 < P.num_requests ? c.rb1 : P.num_requests;
    const uint64_t q0 = c.rb < q1 ? c.rb : q1;
    job.u = u;
    job.lo = en.x;
    job.hi = en.y;
    job.y = y;
    job.b = c.b;
    job.s0 = s0;
    job.s1 = s1;
    job.q0 = q0;
    job.R = q1 - q0;
    job.K = job.R > y ? ((job.R - y - 1) >> P.slices_log2) + 1 : 0;
    job.tiles = s1 > s0 ? (s1 - (s0 & ~7ull) + kTile - 1) >> kTileLog2 : 1;
    job.p = v - first_id(c.b, c.sb);
    job.g = en.z;
    job.G = en.w;
    job.first = u == en.x;
    job.last = u + 1 == en.y;
    job.direct = job.G == 1;
    return job.p < job.tiles;
}

// One deferred entry: the units [lo, hi) of (snapshot b, slice y) that one
// chunk held, and that chunk's partial slot g of G.  Every tile is staged
// again, and for each request whose deferral bit is set its far windows
// (far_windows) are folded into the request's partial slot, which the
// search kernel wrote.  Then, as the search kernel would have: the results,
// or the arrival ticket and the combine when the snapshot spans several
// chunks; the deferral bits are cleared.
__device__ void resolve_entry(const Params& P, Smem& sm, EndSmem& es, uint4 en, uint32_t& last_flag,
                              Staged& staged) {
    const uint32_t tid = threadIdx.x;
    Cursor c;
    Job job;
    // Bytes from the region end to the end of its last run, once a request
    // has found that end (the same for every request of the tile), and the
    // previous tile's staged halo, which carry it to the entry's next tile.
    uint64_t run_left = kNone;
    uint32_t prev_halo = 0;
    uint64_t prev_p = kNone;
    // The bytes from the start of tile prev_p + 1 to the end of the run the
    // previous region ended in, when that run reaches the tile (kNone if
    // unknown).  A tile without pinned blocks lies wholly in that run: when
    // every request that deferred there needs more bytes than this, none of
    // its starts has a window, and the tile is passed over unstaged (the
    // count then carries on by the tile's record).
    uint64_t from_start = kNone;
    for (uint32_t u = en.x; u < en.y; ++u) {
        if (!entry_job(P, en, u, c, job)) continue;  // (not reached: the entry names the job's tiles)
        if (from_start != kNone && prev_p != kNone && prev_p + 1 == job.p) {
            const Ext e = ext_of(P);
            const uint64_t idx = (job.s0 >> kTileLog2) + job.p - 1;  // the record of tile p >= 1
            bool skip = false;
            uint64_t tb = 0;
            if (idx < (P.num_blocks >> kTileLog2) &&
                uniform64(__hip_atomic_load(e.rec_r + idx, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) == 0) {
                tb = uniform64(__hip_atomic_load(e.rec_p + idx, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
                skip = true;
                for (uint64_t r = 0; r < job.K && skip; ++r) {
                    const uint64_t q = job.q0 + job.y + (r << P.slices_log2);
                    const uint64_t bit = q * P.pc + job.g;
                    const uint32_t word = uniform(__hip_atomic_load(e.bits + (bit >> 5), __ATOMIC_RELAXED,
                                                                    __HIP_MEMORY_SCOPE_AGENT));
                    const uint64_t S = ld_const(P.req_size, q);
                    if (((word >> (bit & 31u)) & 1u) && S != 0 && S <= from_start) skip = false;
                }
            }
            if (skip) {
                from_start = from_start >= tb ? from_start - tb : kNone;
                prev_p = job.p;
                prev_halo = kNone32;  // nothing staged to carry run_left by
                run_left = kNone;
                continue;
            }
        }
        const TileGeom tg = tile_geom(job);
        TileRegs regs;
        issue_loads(P, tg, tid, regs);
        const TileState ts = stage_tile(sm, tg, tid, regs);
        // The previous region ended at boundary prev_halo of this tile: with
        // no pinned block between the two region ends, the run goes on and
        // has the bytes between them fewer left.
        Between bt{kNone, 0, 0, false};
        if (prev_p != kNone && prev_p + 1 == job.p && ts.packed && prev_halo <= tg.nt) {
            const uint64_t d = ts.xend - sm.K(prev_halo);
            bt = Between{tg.t0 + prev_halo, d & kValMask, ts.xcend - sm.C(prev_halo), (d >> kValBits) == 0};
        }
        run_left = bt.same_run && run_left != kNone && run_left >= bt.q ? run_left - bt.q : kNone;
        if (run_left == kNone && from_start != kNone && prev_p != kNone && prev_p + 1 == job.p && ts.packed) {
            // after tiles passed over: from the tile start when the region
            // holds no pinned block
            const uint64_t d = ts.xend - sm.K(0);
            if ((d >> kValBits) == 0 && from_start >= d) run_left = from_start - d;
        }
        prev_p = job.p;
        prev_halo = ts.end - tg.nt;
        if (tg.t0 + ts.end < job.s1 && tg.nt != 0) {  // the region's last run may go on
            for (uint64_t r = 0; r < job.K; ++r) {
                const uint64_t q = job.q0 + job.y + (r << P.slices_log2);
                const uint64_t bit = q * P.pc + job.g;
                // (only this entry changes the bit)
                const uint32_t word = uniform(__hip_atomic_load(ext_of(P).bits + (bit >> 5), __ATOMIC_RELAXED,
                                                                __HIP_MEMORY_SCOPE_AGENT));
                const uint64_t S = ld_const(P.req_size, q);
                if (!((word >> (bit & 31u)) & 1u) || S == 0) continue;
                const Key k = far_windows(P, sm, es, job, tg, ts, q, S, run_left, staged, bt);
                // the same thread folds the request's key on every tile
                if (tid == 0 && k.start != kNone) {
                    Key* slot = P.part + q * P.pc + job.g;
                    store_key_device(slot, min_key(load_key_device(slot), k));
                }
            }
        }
        // the next tile starts at boundary nt: in the region's last run when
        // the halo holds no pinned block
        from_start = kNone;
        if (run_left != kNone && ts.packed) {
            const uint64_t d = ts.end > tg.nt ? ts.xend - sm.K(tg.nt) : 0;
            if ((d >> kValBits) == 0) from_start = run_left + d;
        }
        __syncthreads();  // LDS is restaged next
    }
    // every slot write has completed before any thread reads
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    __builtin_amdgcn_s_waitcnt(0);
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    __syncthreads();
    for (uint64_t r = tid; r < job.K; r += kThreads) {
        const uint64_t q = job.q0 + job.y + (r << P.slices_log2);
        const uint64_t bit = q * P.pc + job.g;
        atomicAnd(ext_of(P).bits + (bit >> 5), ~(1u << (bit & 31u)));
        if (job.direct)
            P.out[q] = to_window(load_key_device(P.part + q * P.pc + job.g), ld_const(P.req_size, q));
    }
    if (!job.direct) combine_partials(P, job, tid, last_flag);
    __syncthreads();  // last_flag and LDS are used by the next entry
}

// Finishes the jobs the search kernel deferred, after it on the stream.
// With nothing deferred (the list's word carries an older tag) every
// workgroup returns at once.  One workgroup per CU (the second LDS buffer);
// no workgroup waits for another: each claims entries until none is left.
__global__ __launch_bounds__(kThreads, 2) void coop_window_long_kernel(Params Pin) {
    __shared__ Smem sm;
    __shared__ EndSmem es;
    __shared__ uint32_t last_flag;
    Params P = Pin;
    graph_tags(P);
    const Ext ex = ext_of(P);
    const uint64_t word = __hip_atomic_load(ex.defer_word, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    // The loop bound and the entry words are wave-uniform values in scalar
    // registers: loop control that the compiler saw as divergent put a
    // reload of the bound under a partial execution mask and ended the loop
    // early for some workgroups.
    uint32_t n = (uniform(static_cast<uint32_t>(word >> 32)) == P.qtag) ? uniform(static_cast<uint32_t>(word)) : 0u;
    if (n > P.defer_cap) n = P.defer_cap;
    if (n == 0) return;
    Staged staged{kNone, 0, 0};
    if (threadIdx.x < kFarCache) es.far_q[threadIdx.x] = kNone;
    __syncthreads();
    // Entries are claimed one at a time (a ticket on the claim word, which
    // the call's first claim restamps with its tag): their costs differ
    // widely, and a fixed share per workgroup left some with twice the mean.
    for (;;) {
        if (threadIdx.x == 0) sm.claim = take_ticket(ex.claim_word, P.qtag, 32) - 1;
        __syncthreads();
        const uint32_t e = uniform(static_cast<uint32_t>(sm.claim));  // claims: below n + grid
        __syncthreads();  // sm.claim is written again by the next claim
        if (e >= n) break;
        const uint4 en = load_entry_device(ex.entries + e);
        // (entries are written by this call's search kernel; the checks keep
        // every access in bounds whatever the workspace holds)
        if (en.x >= en.y || en.y > P.units || en.w == 0 || en.w > P.pc || en.z >= en.w) continue;
        resolve_entry(P, sm, es, en, last_flag, staged);
    }
}

// ---------------------------------------------------------------------------
// Host side
// ---------------------------------------------------------------------------

struct Plan {
    uint64_t num_virtual;  // tile ids per slice
    uint64_t slices;       // request slices (a power of two)
    uint32_t slices_log2;
    uint64_t units;        // slices * num_virtual
    uint64_t grid;         // workgroups
    uint64_t c1, c2;       // units per first chunk, per queued chunk
    uint64_t u1;           // units in the first chunks
    uint64_t nchunks;      // first chunks (one per workgroup) and queued chunks
    uint64_t pc;           // partial slots per request
    size_t part_bytes;     // partial keys
    uint64_t defer_cap;    // deferred entries, at most
    size_t off_defer;      // the deferred list's word, the claim word, then the entries
    size_t off_entries;
    size_t off_rec;        // tile records: bytes, costs, pinned counts (u64 each)
    uint64_t num_rec;
    size_t off_bits;       // deferral bits, one per partial slot
    size_t bytes;          // total workspace
};

// Two workgroups of kThreads fit one CU (LDS); 256 CUs.  Workgroups past the
// resident ones are still correct (nothing waits on another workgroup).
constexpr uint64_t kGridWGs = 512;
constexpr uint64_t kLongGridWGs = 256;  // workgroups of coop_window_long_kernel (one per CU), at most
constexpr uint64_t kMaxSlices = 256;
constexpr uint64_t kSliceRequests = 512;  // requests per snapshot before slicing them
static_assert(kGridWGs < (1ull << kEpochShift), "tickets fit the counter");
constexpr uint64_t kQueueMinChunk = 8;         // smaller shares: no queue
constexpr uint64_t kQueueMaxSegments = 16384;  // every workgroup scans the offsets once

bool make_plan(uint64_t num_blocks, uint64_t num_segments, uint64_t num_requests, Plan* pl,
               uint64_t partial_budget = kPartialBudget) {
    if (num_segments > (1ull << 32) || num_blocks > (1ull << 60) || num_requests > (1ull << 40))
        return false;
    const uint64_t nv = (num_blocks >> kTileLog2) + num_segments;
    uint64_t slices = 1;
    if (num_requests > num_segments) {
        const uint64_t per_snapshot = (num_requests + num_segments - 1) / num_segments;
        // few tiles: spread each snapshot's requests over more workgroups
        if (nv < kGridWGs) {
            uint64_t want = (kGridWGs + nv - 1) / nv;
            if (want > per_snapshot) want = per_snapshot;
            if (want > slices) slices = want;
        }
        // many requests per snapshot: fewer per workgroup, fewer partial keys
        const uint64_t want = (per_snapshot + kSliceRequests - 1) / kSliceRequests;
        if (want > slices) slices = want;
        if (slices > kMaxSlices) slices = kMaxSlices;
    }
    uint32_t slices_log2 = 0;
    while ((1ull << slices_log2) < slices) ++slices_log2;
    slices = 1ull << slices_log2;
    if (slices * nv >= (1ull << 32)) return false;
    // deferred entries are counted in 32 bits
    if ((num_blocks / kDeferMin) * slices + slices * nv + kGridWGs >= (1ull << 32)) return false;
    pl->num_virtual = nv;
    pl->slices = slices;
    pl->slices_log2 = slices_log2;
    pl->units = slices * nv;
    const uint64_t grid = pl->units < kGridWGs ? pl->units : kGridWGs;
    uint64_t chunk = (pl->units + grid - 1) / grid;
    // A snapshot has at most T tiles, which span at most ceil(T / chunk) + 1
    // chunks: the partial slots a request needs.  Past the budget, chunks
    // grow instead (fewer workgroups).
    const uint64_t T = ((num_blocks + kTile - 1) >> kTileLog2) + 1;  // tiles of one snapshot, at most
    const uint64_t cap = partial_budget / num_requests > 2 ? partial_budget / num_requests : 2;
    if ((T + chunk - 1) / chunk + 1 > cap) {
        const uint64_t need = (T + cap - 2) / (cap - 1);
        if (need > chunk) chunk = need;
    }
    pl->grid = (pl->units + chunk - 1) / chunk;
    // An eighth of each workgroup's share goes to the queue in chunks of one
    // unit, so that the workgroups finish together; with fewer than 64
    // snapshots, whose units differ more in cost (windows cluster in parts
    // of a run), a quarter in chunks of a sixteenth of the share.  Every
    // queued chunk looks its snapshot up again; a sixteenth of the share in
    // the queue leaves the workgroups apart.  The kernel lengthens queued chunks until the largest
    // snapshot spans at most pc - 2 of them (a span of L units meets at most
    // ceil(L / c2) + 2 chunks); pc, the partial slots per request, stays
    // within the budget.
    uint64_t c1 = chunk, c2 = chunk, u1 = pl->units, nchunks = pl->grid;
    uint64_t pc = (T + chunk - 1) / chunk + 1;
    if (chunk >= kQueueMinChunk && cap >= 4 && num_segments <= kQueueMaxSegments) {
        // With a queue the first chunks need not cover the units: every
        // workgroup slot takes one (unless the partial budget grew the
        // chunks), e.g. 512 workgroups instead of 507 for 20274 units.
        const uint64_t qg = chunk == (pl->units + grid - 1) / grid ? grid : pl->grid;
        const uint64_t share = pl->units / qg;
        const uint64_t q1 = share - share / (num_segments >= 64 ? 8 : 4);
        const uint64_t q2 = num_segments >= 64 || chunk < 16 ? 1 : chunk / 16;
        const uint64_t qu1 = qg * q1;
        const uint64_t qn = qg + (pl->units - qu1 + q2 - 1) / q2;
        uint64_t qpc = (T + q2 - 1) / q2 + 2;
        if (qpc > cap) qpc = cap;
        if (qpc > qn) qpc = qn;
        if (q1 >= 1 && qu1 < pl->units && qpc >= 4) {
            pl->grid = qg;
            c1 = q1;
            c2 = q2;
            u1 = qu1;
            nchunks = qn;
            pc = qpc;
        }
    }
    if (pc > nchunks) pc = nchunks;
    pl->c1 = c1;
    pl->c2 = c2;
    pl->u1 = u1;
    pl->nchunks = nchunks;
    pl->pc = pc;
    pl->part_bytes = (num_requests * pc * sizeof(Key) + 255) & ~static_cast<size_t>(255);
    // then the arrival counters, the queue word, the tag word and the
    // deferred list's word
    pl->off_defer = pl->part_bytes + (slices * num_segments + 2) * sizeof(uint64_t);
    pl->off_entries = (pl->off_defer + 2 * sizeof(uint64_t) + 15) & ~static_cast<size_t>(15);
    // (the kernels derive these offsets from the queue word's address: see
    // Ext; the workspace is 256-byte aligned, so aligning offsets aligns
    // addresses)
    // A job defers only when a window runs more than kWalkCap blocks past
    // its staged region, so its snapshot has at least kDeferMin blocks.
    // The chunk parts of such jobs number at most the jobs plus the chunk
    // boundaries (each falls inside at most one job).
    const uint64_t big = num_blocks / kDeferMin < num_segments ? num_blocks / kDeferMin : num_segments;
    pl->defer_cap = nchunks + slices * big;
    pl->num_rec = num_blocks >> kTileLog2;
    pl->off_rec = pl->off_entries + pl->defer_cap * sizeof(uint4);
    pl->off_bits = pl->off_rec + pl->num_rec * 3 * sizeof(uint64_t);
    // (+32: the layout stays inside even if the workspace is only 8-byte aligned)
    pl->bytes = pl->off_bits + (num_requests * pc + 31) / 32 * sizeof(uint32_t) + 32;
    return true;
}

// ceil(2^64 / d) for d >= 2, and 0 for d = 1 (see div_magic).
uint64_t magic(uint64_t d) { return d == 1 ? 0 : ~0ull / d + 1; }

std::atomic<uint64_t> g_calls{
    static_cast<uint64_t>(std::chrono::steady_clock::now().time_since_epoch().count())};
const uint64_t g_salt =
    static_cast<uint64_t>(std::chrono::steady_clock::now().time_since_epoch().count()) * kTagOdd;

// Advances a workspace's tag word (one thread); recorded ahead of every
// search captured into a graph.
__global__ void window_tag_kernel(uint64_t* word) {
    const uint64_t t = __hip_atomic_load(word, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(word, t + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

}  // namespace

extern "C" {

int coop_abi_version(void) { return COOP_ABI_VERSION; }

const char* coop_status_string(int status) {
    switch (status) {
        case COOP_OK: return "ok";
        case COOP_ERR_INVALID: return "invalid argument";
        case COOP_ERR_WORKSPACE: return "workspace missing or too small";
        case COOP_ERR_HIP: return "HIP launch failed";
        case COOP_ERR_OVERFLOW: return "a run's byte or cost total exceeds 2^64 - 1";
        case COOP_ERR_TOO_LARGE: return "the batch needs more than the library's static scratch";
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

coop_status_t coop_window_search_plan(uint64_t num_blocks, uint64_t num_segments,
                                      uint64_t num_requests, coop_plan_t* plan_out) {
    if (!plan_out) return COOP_ERR_INVALID;
    Plan pl;
    if (!make_plan(num_blocks, num_segments, num_requests, &pl)) return COOP_ERR_INVALID;
    plan_out->workgroups = pl.grid;
    plan_out->slices = pl.slices;
    plan_out->units = pl.units;
    plan_out->first_chunk_units = pl.c1;
    plan_out->first_units = pl.u1;
    plan_out->queued_chunk_units = pl.c2;
    plan_out->chunks_max = pl.nchunks;
    plan_out->partial_slots = pl.pc;
    return COOP_OK;
}

coop_status_t coop_window_search(const uint64_t* size, const uint64_t* cost, const uint8_t* kind,
                                 uint64_t num_blocks, const uint64_t* seg_offsets,
                                 uint64_t num_segments, const uint64_t* req_sizes,
                                 const uint64_t* req_offsets, uint64_t num_requests,
                                 coop_window_t* out, void* workspace, size_t workspace_bytes,
                                 void* stream) {
    return coop_window_search_enqueue(size, cost, kind, num_blocks, seg_offsets, num_segments,
                                      req_sizes, req_offsets, num_requests, out, workspace,
                                      workspace_bytes, stream, coop_host::checks_requested());
}

}  // extern "C"

namespace {

// Validates the host-visible arguments, runs the debug checks when asked,
// and enqueues the search of a batch under plan pl.  The workspace holds
// the plan's partial keys, arrival counters and queue word; tag_word is
// the word a captured call's tags come from (inside the workspace, or at a
// fixed place of the static scratch).
coop_status_t launch_search(const Plan& pl, const uint64_t* size, const uint64_t* cost,
                            const uint8_t* kind, uint64_t num_blocks, const uint64_t* seg_offsets,
                            uint64_t num_segments, const uint64_t* req_sizes,
                            const uint64_t* req_offsets, uint64_t num_requests, coop_window_t* out,
                            void* workspace, uint64_t* tag_word, hipStream_t s, bool check) {
    if (check) {
        const coop_host::Batch b{size, cost, kind, num_blocks, seg_offsets, num_segments,
                                 req_offsets, num_requests, true};
        const coop_status_t rc = coop_host::check_batch(b, s);
        if (rc != COOP_OK) return rc;
    }

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
    P.queue = P.counters + pl.slices * num_segments;
    P.num_blocks = num_blocks;
    P.num_segments = num_segments;
    P.num_requests = num_requests;
    P.num_virtual = static_cast<uint32_t>(pl.num_virtual);
    P.units = static_cast<uint32_t>(pl.units);
    P.grid = static_cast<uint32_t>(pl.grid);
    P.c1 = static_cast<uint32_t>(pl.c1);
    P.c2 = static_cast<uint32_t>(pl.c2);
    P.u1 = static_cast<uint32_t>(pl.u1);
    P.nchunks = pl.nchunks;
    P.c1_magic = magic(pl.c1);
    P.c2_magic = magic(pl.c2);
    P.nv_magic = magic(pl.num_virtual);
    P.pc = static_cast<uint32_t>(pl.pc);
    P.queue_on = pl.nchunks > pl.grid ? 1u : 0u;
    P.slices_log2 = pl.slices_log2;
    P.inv_slope = static_cast<double>(num_segments) /
                  (static_cast<double>(num_blocks) / kTile + static_cast<double>(num_segments));
    P.defer_cap = static_cast<uint32_t>(pl.defer_cap);

    // A captured launch replays with the arguments it was recorded with, so
    // its tag cannot come from the host: it comes from the tag word,
    // advanced by a kernel recorded just before.
    hipStreamCaptureStatus capture = hipStreamCaptureStatusNone;
    if (hipStreamIsCapturing(s, &capture) != hipSuccess) return COOP_ERR_HIP;
    if (capture == hipStreamCaptureStatusNone) {
        const uint64_t call = g_calls.fetch_add(1, std::memory_order_relaxed);
        P.epoch = call & kTagMask;
        P.qtag = queue_tag(P.epoch);
        P.tag_word = nullptr;
    } else {
        hipLaunchKernelGGL(window_tag_kernel, dim3(1), dim3(1), 0, s, tag_word);
        if (hipGetLastError() != hipSuccess) return COOP_ERR_HIP;
        P.epoch = g_salt;
        P.qtag = 0;
        P.tag_word = tag_word;
    }

    hipLaunchKernelGGL(coop_window_search_kernel, dim3(static_cast<uint32_t>(pl.grid)),
                       dim3(kThreads), 0, s, P);
    if (hipGetLastError() != hipSuccess) return COOP_ERR_HIP;
    const uint64_t long_grid = pl.defer_cap < kLongGridWGs ? (pl.defer_cap ? pl.defer_cap : 1)
                                                           : kLongGridWGs;
    hipLaunchKernelGGL(coop_window_long_kernel, dim3(static_cast<uint32_t>(long_grid)),
                       dim3(kThreads), 0, s, P);
    if (hipGetLastError() != hipSuccess) return COOP_ERR_HIP;
    return COOP_OK;
}

// Host arguments every entry point checks before planning.
coop_status_t check_args(const uint64_t* size, const uint64_t* cost, const uint8_t* kind,
                         uint64_t num_blocks, const uint64_t* seg_offsets, uint64_t num_segments,
                         const uint64_t* req_sizes, const uint64_t* req_offsets,
                         coop_window_t* out) {
    if (num_segments == 0) return COOP_ERR_INVALID;
    if (num_blocks && (!size || !cost || !kind)) return COOP_ERR_INVALID;
    if (!seg_offsets || !req_offsets || !req_sizes || !out) return COOP_ERR_INVALID;
    return COOP_OK;
}

// ---------------------------------------------------------------------------
// The search without a workspace argument: its cross-workgroup state lives
// in a fixed device array of the library, one per GPU.
// ---------------------------------------------------------------------------

constexpr size_t kScratchBytes = size_t{32} << 20;
// The first 256 bytes hold the tag word of captured calls (at the same place
// whatever the plan); the plan's workspace follows.
constexpr size_t kScratchTagBytes = 256;
static __device__ __align__(256) uint64_t scratch[kScratchBytes / sizeof(uint64_t)];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
void* g_scratch_ptr[kMaxDevices] = {};

// The device address of `scratch` on the stream's device.  Host code may
// never use the array's name as an address (it names a host-side stand-in);
// the address is looked up once per device, with that device current, and
// kept.
coop_status_t scratch_address(hipStream_t s, void** ptr) {
    int dev = 0, cur = 0;
    if (hipGetDevice(&cur) != hipSuccess) return COOP_ERR_HIP;
    if (hipStreamGetDevice(s, &dev) != hipSuccess) return COOP_ERR_HIP;
    if (dev < 0 || dev >= kMaxDevices) return COOP_ERR_HIP;
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (!g_scratch_ptr[dev]) {
        if (dev != cur && hipSetDevice(dev) != hipSuccess) return COOP_ERR_HIP;
        void* p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (dev != cur) (void)hipSetDevice(cur);
        if (e != hipSuccess || p == nullptr) {
            (void)hipGetLastError();
            return COOP_ERR_HIP;
        }
        g_scratch_ptr[dev] = p;
    }
    *ptr = g_scratch_ptr[dev];
    return COOP_OK;
}

// The plan for the static scratch: the largest partial-key budget (a power
// of two) whose workspace fits; false when none does.
bool static_plan(uint64_t num_blocks, uint64_t num_segments, uint64_t num_requests, Plan* pl) {
    for (uint64_t budget = kPartialBudget; budget >= 2; budget >>= 1) {
        if (!make_plan(num_blocks, num_segments, num_requests, pl, budget)) return false;
        if (pl->bytes <= kScratchBytes - kScratchTagBytes) return true;
    }
    return false;
}

}  // namespace

extern "C" {

size_t coop_window_search_static_capacity(void) { return kScratchBytes - kScratchTagBytes; }

coop_status_t coop_window_search_static(const uint64_t* size, const uint64_t* cost,
                                        const uint8_t* kind, uint64_t num_blocks,
                                        const uint64_t* seg_offsets, uint64_t num_segments,
                                        const uint64_t* req_sizes, const uint64_t* req_offsets,
                                        uint64_t num_requests, coop_window_t* out,
                                        void* stream) {
    if (num_requests == 0) return COOP_OK;
    coop_status_t rc = check_args(size, cost, kind, num_blocks, seg_offsets, num_segments,
                                  req_sizes, req_offsets, out);
    if (rc != COOP_OK) return rc;
    Plan pl;
    if (!make_plan(num_blocks, num_segments, num_requests, &pl)) return COOP_ERR_INVALID;
    if (!static_plan(num_blocks, num_segments, num_requests, &pl)) return COOP_ERR_TOO_LARGE;
    hipStream_t s = static_cast<hipStream_t>(stream);
    void* base = nullptr;
    rc = scratch_address(s, &base);
    if (rc != COOP_OK) return rc;
    uint64_t* tag_word = static_cast<uint64_t*>(base);
    void* workspace = static_cast<char*>(base) + kScratchTagBytes;
    return launch_search(pl, size, cost, kind, num_blocks, seg_offsets, num_segments, req_sizes,
                         req_offsets, num_requests, out, workspace, tag_word, s, false);
}

}  // extern "C"

coop_status_t coop_window_search_enqueue(const uint64_t* size, const uint64_t* cost,
                                         const uint8_t* kind, uint64_t num_blocks,
                                         const uint64_t* seg_offsets, uint64_t num_segments,
                                         const uint64_t* req_sizes, const uint64_t* req_offsets,
                                         uint64_t num_requests, coop_window_t* out,
                                         void* workspace, size_t workspace_bytes, void* stream,
                                         bool check) {
    if (num_requests == 0) return COOP_OK;
    const coop_status_t rc = check_args(size, cost, kind, num_blocks, seg_offsets, num_segments,
                                        req_sizes, req_offsets, out);
    if (rc != COOP_OK) return rc;
    Plan pl;
    if (!make_plan(num_blocks, num_segments, num_requests, &pl)) return COOP_ERR_INVALID;
    if (!workspace || workspace_bytes < pl.bytes) return COOP_ERR_WORKSPACE;
    uint64_t* tag_word = reinterpret_cast<uint64_t*>(static_cast<char*>(workspace) + pl.part_bytes) +
                         pl.slices * num_segments + 1;
    return launch_search(pl, size, cost, kind, num_blocks, seg_offsets, num_segments, req_sizes,
                         req_offsets, num_requests, out, workspace, tag_word,
                         static_cast<hipStream_t>(stream), check);
}
