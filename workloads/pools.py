"""Seeded synthetic pool snapshots shaped like DNN tensor pools.

This module only draws inputs.  It holds none of the search arithmetic, and
both the GPU path and the CPU oracle are fed from it.

A batch is a set of address-sorted pool snapshots (the memory layout of
section 3.1), concatenated as a structure of arrays:
  size  uint64[N]   bytes of each block (multiple of 512, the allocator grain)
  cost  uint64[N]   eviction cost of evictable blocks; written as 0 for
                    free and pinned blocks
  kind  uint8[N]    0 free chunk, 1 evictable tensor, 2 pinned tensor
  seg_offsets uint64[B+1]   snapshot b is blocks [seg[b], seg[b+1])
  req_sizes   uint64[Q]     requested bytes S
  req_offsets uint64[B+1]   requests of snapshot b are [req[b], req[b+1])

The five standard workloads (index 0..4) follow the recipe written down in
the design notes: tiny single pool, batched mid pools, large pools with
request reuse, a ragged heavy-tailed batch with clustered pinned blocks, and
one huge pool.  Every draw comes from numpy's PCG64 seeded with
[workload index, seed], so a (workload, seed) pair always yields the same
arrays.
"""
from __future__ import annotations

import dataclasses
import hashlib
from typing import Optional

import numpy as np

FREE, EVICTABLE, PINNED = 0, 1, 2
GRAIN = 512  # allocation granularity in bytes
KiB, MiB, GiB = 1 << 10, 1 << 20, 1 << 30


@dataclasses.dataclass(frozen=True)
class PoolSpec:
    """Distribution parameters of one workload."""
    name: str
    num_segments: int
    blocks: tuple            # (lo, hi): N_b uniform on [lo, hi]; lo == hi for fixed N
    requests_per_segment: int
    size_dist: str           # "loguniform" or "pareto"
    size_lo: int
    size_hi: int
    pareto_alpha: float = 0.0
    kinds: str = "iid"       # "iid" or "clustered"
    p_free: float = 0.0
    p_pinned: float = 0.0
    cost_dist: str = "uniform"   # "uniform" (integers) or "loguniform"
    cost_lo: int = 1
    cost_hi: int = 1
    req_dist: str = "loguniform"  # "loguniform" or "run_percentile"
    req_lo: int = 0
    req_hi: int = 0
    # clustered kinds (workload 3)
    pinned_run_p: float = 0.0     # pinned run length ~ Geometric(p) on {1, 2, ...}
    open_run_p: float = 0.0       # unpinned run length ~ Geometric(p)
    first_run_pinned_p: float = 0.0
    free_in_open_run_p: float = 0.0
    infeasible_p: float = 0.0


CONFIGS = (
    PoolSpec("tiny single pool", 1, (1000, 1000), 1000, "loguniform", 512, 64 * MiB,
             p_free=0.10, p_pinned=0.05, cost_dist="uniform", cost_lo=1, cost_hi=10**6,
             req_lo=1 * MiB, req_hi=256 * MiB),
    PoolSpec("batched mid pools", 1024, (4096, 4096), 1, "loguniform", 512, 64 * MiB,
             p_free=0.10, p_pinned=0.05, cost_dist="uniform", cost_lo=1, cost_hi=10**6,
             req_lo=4 * MiB, req_hi=1 * GiB),
    PoolSpec("large pools, multi-request reuse", 256, (65536, 65536), 16, "loguniform",
             512, 256 * MiB, p_free=0.15, p_pinned=0.03, cost_dist="loguniform",
             cost_lo=1, cost_hi=10**9, req_lo=16 * MiB, req_hi=4 * GiB),
    PoolSpec("ragged heavy-tailed batch", 4096, (64, 32768), 4, "pareto", 512, 1 * GiB,
             pareto_alpha=1.2, kinds="clustered", cost_dist="uniform", cost_lo=0,
             cost_hi=2**40, req_dist="run_percentile", pinned_run_p=0.3,
             open_run_p=9 / 70, first_run_pinned_p=0.3, free_in_open_run_p=1 / 7,
             infeasible_p=0.10),
    PoolSpec("single huge pool", 1, (1 << 24, 1 << 24), 4096, "loguniform", 512, 64 * MiB,
             p_free=0.20, p_pinned=0.01, cost_dist="loguniform", cost_lo=1,
             cost_hi=10**12, req_lo=64 * MiB, req_hi=16 * GiB),
)


@dataclasses.dataclass
class Pools:
    """One generated batch (numpy arrays on the host)."""
    size: np.ndarray
    cost: np.ndarray
    kind: np.ndarray
    seg_offsets: np.ndarray
    req_sizes: np.ndarray
    req_offsets: np.ndarray
    spec: Optional[PoolSpec] = None
    seed: int = 0

    @property
    def num_blocks(self) -> int:
        return int(self.size.shape[0])

    @property
    def num_segments(self) -> int:
        return int(self.seg_offsets.shape[0]) - 1

    @property
    def num_requests(self) -> int:
        return int(self.req_sizes.shape[0])

    def arrays(self):
        return (self.size, self.cost, self.kind, self.seg_offsets, self.req_sizes,
                self.req_offsets)

    def digest(self) -> str:
        """SHA-256 over all arrays, for reports."""
        h = hashlib.sha256()
        for a in self.arrays():
            h.update(np.ascontiguousarray(a).tobytes())
        return h.hexdigest()


def _loguniform(rng, lo, hi, n):
    x = rng.random(n)
    x *= np.log(hi) - np.log(lo)
    x += np.log(lo)
    return np.exp(x, out=x)


def _round_up_grain(x):
    """Rounds byte counts up to a whole number of 512-byte grains (at least one)."""
    x = np.asarray(x, dtype=np.float64)
    x /= GRAIN
    np.ceil(x, out=x)
    np.maximum(x, 1.0, out=x)
    return x.astype(np.uint64) * np.uint64(GRAIN)


def _sizes(spec: PoolSpec, rng, n):
    if spec.size_dist == "loguniform":
        return _round_up_grain(_loguniform(rng, spec.size_lo, spec.size_hi, n))
    if spec.size_dist == "pareto":
        # x = x_m * U^(-1/alpha) with U uniform on (0, 1]
        x = rng.random(n)
        np.subtract(1.0, x, out=x)
        np.log(x, out=x)
        x *= -1.0 / spec.pareto_alpha
        np.exp(x, out=x)
        x *= spec.size_lo
        np.minimum(x, spec.size_hi, out=x)
        return _round_up_grain(x)
    raise ValueError(spec.size_dist)


def _costs(spec: PoolSpec, rng, n):
    if spec.cost_dist == "uniform":
        return rng.integers(spec.cost_lo, spec.cost_hi, size=n, endpoint=True,
                            dtype=np.uint64)
    if spec.cost_dist == "loguniform":
        c = np.floor(_loguniform(rng, spec.cost_lo, spec.cost_hi, n))
        return np.clip(c, spec.cost_lo, spec.cost_hi).astype(np.uint64)
    raise ValueError(spec.cost_dist)


def _iid_kinds(spec: PoolSpec, rng, n):
    u = rng.random(n)
    kind = np.full(n, EVICTABLE, dtype=np.uint8)
    kind[u < spec.p_free] = FREE
    kind[(u >= spec.p_free) & (u < spec.p_free + spec.p_pinned)] = PINNED
    return kind


def _clustered_kinds(spec: PoolSpec, rng, n):
    """Alternating pinned / unpinned runs with geometric lengths; inside an
    unpinned run each block is free with probability free_in_open_run_p."""
    first_pinned = rng.random() < spec.first_run_pinned_p
    mean_pair = 1.0 / spec.pinned_run_p + 1.0 / spec.open_run_p
    pieces, total = [], 0
    while total < n:
        m = int((n - total) / mean_pair * 1.2) + 8
        lp = rng.geometric(spec.pinned_run_p, size=m)
        lo = rng.geometric(spec.open_run_p, size=m)
        pair = np.empty(2 * m, dtype=np.int64)
        if first_pinned:
            pair[0::2], pair[1::2] = lp, lo
        else:
            pair[0::2], pair[1::2] = lo, lp
        pieces.append(pair)
        total += int(pair.sum())
    lens = np.concatenate(pieces)
    labels = np.zeros(len(lens), dtype=bool)
    labels[0 if first_pinned else 1::2] = True
    pinned = np.repeat(labels, lens)[:n]
    free = rng.random(n) < spec.free_in_open_run_p
    return np.where(pinned, PINNED, np.where(free, FREE, EVICTABLE)).astype(np.uint8)


def _run_totals(size, kind):
    """Byte totals of the maximal unpinned stretches of one snapshot."""
    open_ = kind != PINNED
    if not open_.any():
        return np.zeros(0, dtype=np.uint64)
    starts = np.flatnonzero(open_ & ~np.concatenate(([False], open_[:-1])))
    ends = np.flatnonzero(open_ & ~np.concatenate((open_[1:], [False]))) + 1
    csum = np.concatenate(([0], np.cumsum(size, dtype=np.uint64)))
    return csum[ends] - csum[starts]


def _nearest_rank(sorted_vals, pct):
    k = max(1, int(np.ceil(pct / 100.0 * len(sorted_vals))))
    return sorted_vals[k - 1]


def generate(spec: PoolSpec, seed: int = 0, stream: int = 0) -> Pools:
    """Draws one batch for `spec`.  `stream` is the first seed word (the
    workload index for the standard workloads)."""
    rng = np.random.default_rng([stream, seed])
    B = spec.num_segments
    lo, hi = spec.blocks
    if lo == hi:
        nb = np.full(B, lo, dtype=np.int64)
    else:
        nb = rng.integers(lo, hi, size=B, endpoint=True)
    seg = np.zeros(B + 1, dtype=np.uint64)
    seg[1:] = np.cumsum(nb)
    n = int(seg[-1])

    size = _sizes(spec, rng, n)
    if spec.kinds == "iid":
        kind = _iid_kinds(spec, rng, n)
    else:
        kind = np.empty(n, dtype=np.uint8)
        for b in range(B):
            kind[seg[b]:seg[b + 1]] = _clustered_kinds(spec, rng, int(nb[b]))
    cost = _costs(spec, rng, n)
    cost[kind != EVICTABLE] = 0

    R = spec.requests_per_segment
    req_off = np.arange(B + 1, dtype=np.uint64) * np.uint64(R)
    if spec.req_dist == "loguniform":
        req = np.ceil(_loguniform(rng, spec.req_lo, spec.req_hi, B * R)).astype(np.uint64)
    elif spec.req_dist == "run_percentile":
        req = np.empty(B * R, dtype=np.uint64)
        for b in range(B):
            s0, s1 = int(seg[b]), int(seg[b + 1])
            totals = np.sort(_run_totals(size[s0:s1], kind[s0:s1]))
            for r in range(R):
                if len(totals) == 0:
                    S = GRAIN
                else:
                    S = int(_nearest_rank(totals, 50 if r % 2 == 0 else 95))
                    if rng.random() < spec.infeasible_p:
                        S = int(totals[-1]) + GRAIN
                req[b * R + r] = S
    else:
        raise ValueError(spec.req_dist)
    return Pools(size, cost, kind, seg, req, req_off, spec, seed)


def make_config(k: int, seed: int = 0, **overrides) -> Pools:
    """Standard workload k (0..4), optionally with spec fields replaced
    (e.g. num_segments=8 for a smaller batch of the same shape)."""
    spec = CONFIGS[k]
    if overrides:
        spec = dataclasses.replace(spec, **overrides)
    return generate(spec, seed, stream=k)


def from_lists(snapshots, requests) -> Pools:
    """Builds a batch from python lists: snapshots is a list of
    (size, cost, kind) triples of equal-length sequences, requests a list of
    request-size lists (one per snapshot)."""
    sizes, costs, kinds, seg, req, roff = [], [], [], [0], [], [0]
    for (s, c, k), rq in zip(snapshots, requests):
        sizes += list(s); costs += list(c); kinds += list(k)
        seg.append(len(sizes))
        req += list(rq)
        roff.append(len(req))
    return Pools(np.array(sizes, dtype=np.uint64), np.array(costs, dtype=np.uint64),
                 np.array(kinds, dtype=np.uint8), np.array(seg, dtype=np.uint64),
                 np.array(req, dtype=np.uint64), np.array(roff, dtype=np.uint64))


def real_costs(pools: Pools, seed: int = 0, max_staleness: int = 4096) -> np.ndarray:
    """Real-valued heuristics for a batch (float64, one per block): each
    evictable block's integer cost divided by a staleness drawn uniform on
    {1..max_staleness}, rounded to the nearest binary64; 0 for free and
    pinned blocks.  Seeded by (seed, number of blocks), independent of the
    draws that made the batch."""
    rng = np.random.default_rng([0x5EA1, seed, pools.num_blocks])
    s = rng.integers(1, max_staleness + 1, pools.num_blocks).astype(np.float64)
    h = pools.cost.astype(np.float64) / s
    h[pools.kind != EVICTABLE] = 0.0
    return h


# One pool laid out as section 3.5 describes: unevictable parameters at both
# ends, everything between them one pinned-free run of activations.
LONG_RUN_SETS = ("spread", "small", "half", "whole")


def long_run(seed: int = 16, n: int = 1 << 24, request_set: str = "spread") -> Pools:
    """One snapshot of n blocks: sizes log-uniform on [512 B, 64 MiB] (rounded
    up to 512 B), a fifth of the blocks free, the first 37 and last 53 pinned
    (the parameters), costs log-uniform on [1, 1e12).  Request sets, in bytes
    of the run between the parameters: "spread" (16: one block, the mean
    block, 100 and 5000 mean blocks, k/12 of the run for k = 1..11, the whole
    run), "small" (16, geometric from 512 B to 5000 mean blocks), "half" (one
    request, half the run), "whole" (one request, the whole run)."""
    rng = np.random.default_rng(seed)
    lo, hi = np.log(512.0), np.log(64.0 * (1 << 20))
    size = ((np.exp(lo + rng.random(n) * (hi - lo)) + 511) // 512 * 512).astype(np.uint64)
    kind = np.where(rng.random(n) < 0.2, FREE, EVICTABLE).astype(np.uint8)
    kind[:37] = PINNED
    kind[-53:] = PINNED
    cost = np.floor(np.exp(rng.random(n) * np.log(1e12))).astype(np.uint64)
    run = int(size[37:-53].sum())
    mean = int(size.mean())
    sets = {
        "spread": [512, mean, 100 * mean, 5000 * mean] + [run * k // 12 for k in range(1, 12)] + [run],
        "small": [int(x) for x in np.geomspace(512, 5000 * mean, 16)],
        "half": [run // 2],
        "whole": [run],
    }
    req = np.array(sets[request_set], dtype=np.uint64)
    return Pools(size, cost, kind, np.array([0, n], dtype=np.uint64), req,
                 np.array([0, len(req)], dtype=np.uint64))
