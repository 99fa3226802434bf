// Batched first fit (Coop, section 2.1 and Algorithm 1) for gfx950.
//
// For every request of S bytes on a pool snapshot: the leftmost free chunk
// (kind 0) holding at least S bytes -- where a first-fit allocator places the
// tensor, and what Algorithm 1's find_free_block_not_less_than returns before
// any eviction is tried.  The answer is the chunk's index in its snapshot, or
// ~0 when the snapshot has none.
//
// Two launches on the caller's stream:
//  1. Summary: one pass over the blocks (size and kind, 9 bytes each, read
//     once for every request) writes, for every 64-block group and every
//     4096-block tile of the concatenated block array, the largest key of a
//     free chunk in it, key(s) = s + 1 saturated at 2^64 - 1 (0: no free
//     chunk).  Groups and tiles are aligned to the array, not to snapshots.
//  2. Search: one wavefront per request walks its snapshot from the left.
//     Where whole tiles (then whole groups) fit inside what is left of the
//     snapshot, 512 tile keys (64 group keys) are tested at once against
//     key(S); the first one that passes is entered one level down, and
//     inside a group the 64 blocks are tested exactly.  A key passes
//     whenever its entry holds a fit; the saturation lets it pass without a
//     fit only for S = 2^64 - 1 and a chunk of 2^64 - 2 bytes, and then the
//     walk simply continues after that entry.  Everything left of the walk's
//     position is known to hold no fit, so the first exact hit is the
//     answer.

#include <hip/hip_runtime.h>

#include <stdint.h>

#include "coop.h"
#include "coop_host.h"

namespace {

constexpr uint32_t kThreads = 512;
constexpr uint32_t kItems = 8;
constexpr uint32_t kGroupLog2 = 6;  // 64 blocks per group: 8 threads of 8 blocks
constexpr uint32_t kTileLog2 = 12;  // 4096 blocks per tile: one workgroup
constexpr uint64_t kGroup = 1ull << kGroupLog2;
constexpr uint64_t kTile = 1ull << kTileLog2;
static_assert(kTile == kThreads * kItems, "a tile is one workgroup's blocks");
static_assert(kGroup == 8 * kItems, "a group is eight threads' blocks");
constexpr uint32_t kSearchWaves = 4;      // requests per search workgroup
constexpr uint32_t kTilesPerLane = 8;     // tile summaries one lane tests per step
constexpr uint64_t kMaxSummaryWGs = 1ull << 20;
constexpr uint64_t kMaxSearchWGs = 1ull << 18;
constexpr uint64_t kNone = ~0ull;

// Summary key of a chunk size (or of a request size): s + 1, saturated.
__device__ __forceinline__ uint64_t fit_key(uint64_t s) { return s == kNone ? kNone : s + 1; }

__device__ __forceinline__ uint64_t max64(uint64_t a, uint64_t b) { return a > b ? a : b; }

__device__ __forceinline__ uint64_t shfl_xor64(uint64_t v, int m) {
    const uint32_t lo = __shfl_xor(static_cast<uint32_t>(v), m, 64);
    const uint32_t hi = __shfl_xor(static_cast<uint32_t>(v >> 32), m, 64);
    return (static_cast<uint64_t>(hi) << 32) | lo;
}

// Pass 1.  Workgroup w takes tiles w, w + grid, ...; thread t of a tile
// holds blocks [8t, 8t + 8), eight consecutive threads one group.
__global__ __launch_bounds__(kThreads) void first_fit_summary_kernel(
    const uint64_t* __restrict__ size, const uint8_t* __restrict__ kind, uint64_t n,
    uint64_t* __restrict__ g1, uint64_t* __restrict__ g2) {
    __shared__ uint64_t wave_max[kThreads / 64];
    const uint32_t tid = threadIdx.x, lane = tid & 63u, w = tid >> 6;
    const uint64_t tiles = (n + kTile - 1) >> kTileLog2;
    const bool aligned =
        ((reinterpret_cast<uintptr_t>(size) & 15u) | (reinterpret_cast<uintptr_t>(kind) & 7u)) == 0;
    for (uint64_t tile = blockIdx.x; tile < tiles; tile += gridDim.x) {
        const uint64_t k0 = (tile << kTileLog2) + tid * kItems;
        uint64_t m = 0;
        if (aligned && k0 + kItems <= n) {
            const uint2 kk = *reinterpret_cast<const uint2*>(kind + k0);
#pragma unroll
            for (uint32_t j = 0; j < kItems / 2; ++j) {
                const ulonglong2 s = *reinterpret_cast<const ulonglong2*>(size + k0 + 2 * j);
                const uint32_t kw = j < 2 ? kk.x : kk.y;
                const uint32_t ka = (kw >> (16 * (j & 1))) & 0xffu;
                const uint32_t kb = (kw >> (16 * (j & 1) + 8)) & 0xffu;
                m = max64(m, ka == COOP_FREE ? fit_key(s.x) : 0);
                m = max64(m, kb == COOP_FREE ? fit_key(s.y) : 0);
            }
        } else {
            for (uint32_t j = 0; j < kItems; ++j) {
                const uint64_t k = k0 + j;
                if (k < n && kind[k] == COOP_FREE) m = max64(m, fit_key(size[k]));
            }
        }
        // groups: eight consecutive lanes
        m = max64(m, shfl_xor64(m, 1));
        m = max64(m, shfl_xor64(m, 2));
        m = max64(m, shfl_xor64(m, 4));
        const uint64_t group = (tile << (kTileLog2 - kGroupLog2)) + (tid >> 3);
        if ((lane & 7u) == 0 && (group << kGroupLog2) < n) g1[group] = m;
        // the tile
        m = max64(m, shfl_xor64(m, 8));
        m = max64(m, shfl_xor64(m, 16));
        m = max64(m, shfl_xor64(m, 32));
        if (lane == 0) wave_max[w] = m;
        __syncthreads();
        if (tid == 0) {
            uint64_t t = wave_max[0];
            for (uint32_t i = 1; i < kThreads / 64; ++i) t = max64(t, wave_max[i]);
            g2[tile] = t;
        }
        __syncthreads();  // wave_max is rewritten for the next tile
    }
}

// Pass 2.  Wavefront w of workgroup g takes requests g * 4 + w, then onward
// by the grid's stride.
__global__ __launch_bounds__(64 * kSearchWaves) void first_fit_search_kernel(
    const uint64_t* __restrict__ size, const uint8_t* __restrict__ kind, uint64_t n,
    const uint64_t* __restrict__ seg, uint64_t num_segments, const uint64_t* __restrict__ req_size,
    const uint64_t* __restrict__ req_off, uint64_t num_requests, const uint64_t* __restrict__ g1,
    const uint64_t* __restrict__ g2, uint64_t* __restrict__ out) {
    const uint32_t lane = threadIdx.x & 63u;
    const uint32_t w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    for (uint64_t q = static_cast<uint64_t>(blockIdx.x) * kSearchWaves + w; q < num_requests;
         q += static_cast<uint64_t>(gridDim.x) * kSearchWaves) {
        // The snapshot: the first i in [0, B] with req_off[i] > q, minus one,
        // found 64 probes at a time.
        uint64_t lo = 0, hi = num_segments + 1;
        while (hi - lo > 64) {
            const uint64_t step = (hi - lo + 63) >> 6;
            const uint64_t i = lo + lane * step;
            const uint64_t m = __ballot(i >= hi || req_off[i] > q);
            const uint32_t f = m ? static_cast<uint32_t>(__builtin_ctzll(m)) : 64u;
            const uint64_t nhi = f < 64 ? lo + f * step : hi;
            lo = f ? lo + (f - 1) * step + 1 : lo;
            hi = nhi < hi ? nhi : hi;
        }
        const uint64_t mb = __ballot(lo + lane >= hi || req_off[lo + lane] > q);
        const uint64_t first = mb ? lo + __builtin_ctzll(mb) : hi;
        const uint64_t b = first ? (first - 1 < num_segments ? first - 1 : num_segments - 1) : 0;
        // snapshot bounds, clamped to the array (malformed offsets give wrong
        // answers, never an access outside it)
        uint64_t s1 = seg[b + 1], s0 = seg[b];
        s1 = s1 < n ? s1 : n;
        s0 = s0 < s1 ? s0 : s1;
        const uint64_t S = req_size[q], T = fit_key(S);

        uint64_t pos = s0, lim = s1, found = kNone;
        uint32_t top = 2;  // coarsest level allowed: 2 tiles, 1 groups, 0 blocks
        while (pos < s1) {
            if (pos >= lim) {
                lim = s1;
                top = 2;
            }
            if (top == 2 && (pos & (kTile - 1)) == 0 && pos + kTile <= lim) {
                // kTilesPerLane consecutive tiles per lane: a long run of
                // tiles without a fit goes by 512 tiles a step
                const uint64_t t0 = pos >> kTileLog2;
                const uint64_t span = 64 * kTilesPerLane;
                const uint64_t tl = lim >> kTileLog2, tn = tl < t0 + span ? tl : t0 + span;
                const uint64_t tb = t0 + lane * kTilesPerLane;
                uint32_t jf = kTilesPerLane;
#pragma unroll
                for (uint32_t j = kTilesPerLane; j-- > 0;)
                    if (tb + j < tn && g2[tb + j] >= T) jf = j;
                const uint64_t m = __ballot(jf < kTilesPerLane);
                if (m) {
                    const uint32_t f = static_cast<uint32_t>(__builtin_ctzll(m));
                    const uint32_t j = __builtin_amdgcn_readlane(jf, f);
                    pos = (t0 + f * kTilesPerLane + j) << kTileLog2;
                    lim = pos + kTile;
                    top = 1;
                } else {
                    pos = tn << kTileLog2;
                }
                continue;
            }
            if (top >= 1 && (pos & (kGroup - 1)) == 0 && pos + kGroup <= lim) {
                const uint64_t a0 = pos >> kGroupLog2;
                const uint64_t al = lim >> kGroupLog2;
                const uint64_t edge = ((pos >> kTileLog2) + 1) << (kTileLog2 - kGroupLog2);
                const uint64_t an = al < edge ? al : edge;  // up to the next tile boundary
                const uint64_t g = a0 + lane;
                const uint64_t m = __ballot(g < an && g1[g] >= T);
                if (m) {
                    pos = (a0 + __builtin_ctzll(m)) << kGroupLog2;
                    lim = pos + kGroup;
                    top = 0;
                } else {
                    pos = an << kGroupLog2;
                }
                continue;
            }
            const uint64_t edge = (pos | (kGroup - 1)) + 1;
            const uint64_t bn = lim < edge ? lim : edge;
            const uint64_t k = pos + lane;
            const uint64_t m = __ballot(k < bn && kind[k] == COOP_FREE && size[k] >= S);
            if (m) {
                found = pos + __builtin_ctzll(m) - s0;
                break;
            }
            pos = bn;
        }
        if (lane == 0) out[q] = found;
    }
}

struct FitLayout {
    uint64_t groups, tiles;
    size_t g2_offset, bytes;
};

FitLayout fit_layout(uint64_t num_blocks) {
    FitLayout l;
    l.groups = (num_blocks + kGroup - 1) >> kGroupLog2;
    l.tiles = (num_blocks + kTile - 1) >> kTileLog2;
    l.g2_offset = (l.groups * sizeof(uint64_t) + 255) & ~static_cast<size_t>(255);
    l.bytes = l.g2_offset + l.tiles * sizeof(uint64_t);
    return l;
}

}  // namespace

extern "C" {

coop_status_t coop_first_fit_workspace_size(uint64_t num_blocks, size_t* bytes_out) {
    if (!bytes_out || num_blocks > (1ull << 60)) return COOP_ERR_INVALID;
    *bytes_out = fit_layout(num_blocks).bytes;
    return COOP_OK;
}

coop_status_t coop_first_fit(const uint64_t* size, const uint8_t* kind, uint64_t num_blocks,
                             const uint64_t* seg_offsets, uint64_t num_segments,
                             const uint64_t* req_sizes, const uint64_t* req_offsets,
                             uint64_t num_requests, uint64_t* out, void* workspace,
                             size_t workspace_bytes, void* stream) {
    return coop_first_fit_enqueue(size, kind, num_blocks, seg_offsets, num_segments, req_sizes,
                                  req_offsets, num_requests, out, workspace, workspace_bytes,
                                  stream, coop_host::checks_requested());
}

}  // extern "C"

coop_status_t coop_first_fit_enqueue(const uint64_t* size, const uint8_t* kind,
                                     uint64_t num_blocks, const uint64_t* seg_offsets,
                                     uint64_t num_segments, const uint64_t* req_sizes,
                                     const uint64_t* req_offsets, uint64_t num_requests,
                                     uint64_t* out, void* workspace, size_t workspace_bytes,
                                     void* stream, bool check) {
    if (num_requests == 0) return COOP_OK;
    if (num_segments == 0 || num_blocks > (1ull << 60)) return COOP_ERR_INVALID;
    if (num_blocks && (!size || !kind)) return COOP_ERR_INVALID;
    if (!seg_offsets || !req_offsets || !req_sizes || !out) return COOP_ERR_INVALID;
    const FitLayout l = fit_layout(num_blocks);
    if (l.bytes && (!workspace || workspace_bytes < l.bytes)) return COOP_ERR_WORKSPACE;
    uint64_t* g1 = static_cast<uint64_t*>(workspace);
    uint64_t* g2 = reinterpret_cast<uint64_t*>(static_cast<char*>(workspace) + l.g2_offset);
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (check) {
        // first fit sums nothing: only the offset rules
        const coop_host::Batch b{size, nullptr, kind, num_blocks, seg_offsets, num_segments,
                                 req_offsets, num_requests, false};
        const coop_status_t rc = coop_host::check_batch(b, s);
        if (rc != COOP_OK) return rc;
    }
    if (l.tiles) {
        const uint64_t grid = l.tiles < kMaxSummaryWGs ? l.tiles : kMaxSummaryWGs;
        hipLaunchKernelGGL(first_fit_summary_kernel, dim3(static_cast<uint32_t>(grid)), dim3(kThreads),
                           0, s, size, kind, num_blocks, g1, g2);
        if (hipGetLastError() != hipSuccess) return COOP_ERR_HIP;
    }
    const uint64_t want = (num_requests + kSearchWaves - 1) / kSearchWaves;
    const uint64_t grid = want < kMaxSearchWGs ? want : kMaxSearchWGs;
    hipLaunchKernelGGL(first_fit_search_kernel, dim3(static_cast<uint32_t>(grid)),
                       dim3(64 * kSearchWaves), 0, s, size, kind, num_blocks, seg_offsets,
                       num_segments, req_sizes, req_offsets, num_requests, g1, g2, out);
    if (hipGetLastError() != hipSuccess) return COOP_ERR_HIP;
    return COOP_OK;
}
