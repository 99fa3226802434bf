// Host-side pieces shared by the library's sources (no device code here).
//
// 1. The debug checks.  The batch rules that live in device memory (the
//    offset arrays, and that a run's byte and cost totals fit in 64 bits)
//    are not checked by the kernels: a launch that breaks them gives
//    unspecified results, while every access stays inside the arrays.  When
//    the environment sets COOP_DEBUG=1, the public entry points first copy
//    those arrays back on the call's stream, synchronise it, and check them
//    on the host; a batch that breaks a rule is rejected before any launch.
//    A stream that is capturing a graph cannot be synchronised, so calls
//    made during a capture skip the checks.
//
// 2. The enqueue functions behind coop_window_search and coop_first_fit,
//    with the checks as a parameter: the replay's stepwise path calls them on
//    arrays it builds itself, once per operation, without checks.
#pragma once

#include <hip/hip_runtime.h>

#include <stdint.h>

#include <cstdlib>
#include <cstring>
#include <vector>

#include "coop.h"

#define COOP_HIDDEN __attribute__((visibility("hidden")))

// Nothing below is part of the exported ABI.
#pragma GCC visibility push(hidden)

namespace coop_host {

// COOP_DEBUG=1 in the environment, read on every call.
inline bool checks_requested() {
    const char* e = std::getenv("COOP_DEBUG");
    return e != nullptr && std::strcmp(e, "1") == 0;
}

struct Batch {
    const uint64_t* size;
    const uint64_t* cost;  // may be null: costs are then not summed
    const uint8_t* kind;
    uint64_t num_blocks;
    const uint64_t* seg_offsets;
    uint64_t num_segments;
    const uint64_t* req_offsets;
    uint64_t num_requests;
    bool run_sums;  // check the per-run byte (and cost) totals
};

template <typename T>
inline bool copy_back(std::vector<T>& host, const T* dev, uint64_t n, hipStream_t s) {
    host.resize(n);
    if (n == 0) return true;
    return hipMemcpyAsync(host.data(), dev, n * sizeof(T), hipMemcpyDeviceToHost, s) == hipSuccess;
}

// offsets[0] == 0, never decreasing, offsets[n] == total.
inline bool offsets_valid(const std::vector<uint64_t>& o, uint64_t total) {
    if (o.empty() || o.front() != 0 || o.back() != total) return false;
    for (size_t i = 1; i < o.size(); ++i)
        if (o[i] < o[i - 1]) return false;
    return true;
}

// COOP_OK, COOP_ERR_INVALID (an offset rule broken), COOP_ERR_OVERFLOW (a
// run's byte total, or the cost total of its evictable blocks, above
// 2^64 - 1) or COOP_ERR_HIP (a copy or the synchronisation failed).
inline coop_status_t check_batch(const Batch& b, hipStream_t s) {
    hipStreamCaptureStatus capture = hipStreamCaptureStatusNone;
    if (hipStreamIsCapturing(s, &capture) != hipSuccess) return COOP_ERR_HIP;
    if (capture != hipStreamCaptureStatusNone) return COOP_OK;
    std::vector<uint64_t> seg, roff, size, cost;
    std::vector<uint8_t> kind;
    bool ok = copy_back(seg, b.seg_offsets, b.num_segments + 1, s) &&
              copy_back(roff, b.req_offsets, b.num_segments + 1, s);
    if (b.run_sums) {
        ok = ok && copy_back(size, b.size, b.num_blocks, s) && copy_back(kind, b.kind, b.num_blocks, s);
        if (b.cost) ok = ok && copy_back(cost, b.cost, b.num_blocks, s);
    }
    if (!ok || hipStreamSynchronize(s) != hipSuccess) return COOP_ERR_HIP;
    if (!offsets_valid(seg, b.num_blocks) || !offsets_valid(roff, b.num_requests))
        return COOP_ERR_INVALID;
    if (!b.run_sums) return COOP_OK;
    for (uint64_t g = 0; g < b.num_segments; ++g) {
        uint64_t bytes = 0, total = 0;  // of the current run
        for (uint64_t k = seg[g]; k < seg[g + 1]; ++k) {
            if (kind[k] >= COOP_PINNED) {
                bytes = total = 0;
                continue;
            }
            if (__builtin_add_overflow(bytes, size[k], &bytes)) return COOP_ERR_OVERFLOW;
            if (b.cost && kind[k] == COOP_EVICTABLE && __builtin_add_overflow(total, cost[k], &total))
                return COOP_ERR_OVERFLOW;
        }
    }
    return COOP_OK;
}

}  // namespace coop_host

COOP_HIDDEN coop_status_t coop_window_search_enqueue(
    const uint64_t* size, const uint64_t* cost, const uint8_t* kind, uint64_t num_blocks,
    const uint64_t* seg_offsets, uint64_t num_segments, const uint64_t* req_sizes,
    const uint64_t* req_offsets, uint64_t num_requests, coop_window_t* out, void* workspace,
    size_t workspace_bytes, void* stream, bool check);

COOP_HIDDEN coop_status_t coop_first_fit_enqueue(
    const uint64_t* size, const uint8_t* kind, uint64_t num_blocks, const uint64_t* seg_offsets,
    uint64_t num_segments, const uint64_t* req_sizes, const uint64_t* req_offsets,
    uint64_t num_requests, uint64_t* out, void* workspace, size_t workspace_bytes, void* stream,
    bool check);

#pragma GCC visibility pop
