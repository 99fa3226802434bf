"""The seeded generator draws what the input recipe says, deterministically."""
import numpy as np
import pytest

import workloads
from workloads import EVICTABLE, FREE, GRAIN, PINNED


def _common(p):
    assert p.size.dtype == np.uint64 and p.cost.dtype == np.uint64
    assert p.kind.dtype == np.uint8
    assert p.seg_offsets[0] == 0 and p.seg_offsets[-1] == p.num_blocks
    assert p.req_offsets[0] == 0 and p.req_offsets[-1] == p.num_requests
    assert np.all(np.diff(p.seg_offsets.astype(np.int64)) >= 0)
    assert np.all(p.size % GRAIN == 0) and np.all(p.size >= GRAIN)
    assert np.all(p.cost[p.kind != EVICTABLE] == 0)
    assert set(np.unique(p.kind).tolist()) <= {FREE, EVICTABLE, PINNED}


def test_deterministic():
    a = workloads.make_config(1, 7, num_segments=16)
    b = workloads.make_config(1, 7, num_segments=16)
    c = workloads.make_config(1, 8, num_segments=16)
    assert a.digest() == b.digest() != c.digest()


@pytest.mark.parametrize("k", [0, 1, 2])
def test_iid_workloads(k):
    spec = workloads.CONFIGS[k]
    p = workloads.make_config(k, 0, num_segments=min(spec.num_segments, 64))
    _common(p)
    assert np.all(np.diff(p.seg_offsets.astype(np.int64)) == spec.blocks[0])
    assert np.all(np.diff(p.req_offsets.astype(np.int64)) == spec.requests_per_segment)
    frac = np.bincount(p.kind, minlength=3) / p.num_blocks
    tol = 4 * np.sqrt(0.25 / p.num_blocks)      # four binomial standard deviations
    assert abs(frac[FREE] - spec.p_free) < tol and abs(frac[PINNED] - spec.p_pinned) < tol
    assert p.size.max() <= spec.size_hi
    ev = p.cost[p.kind == EVICTABLE]
    assert ev.min() >= spec.cost_lo and ev.max() <= spec.cost_hi
    assert p.req_sizes.min() >= spec.req_lo and p.req_sizes.max() <= spec.req_hi
    # log-uniform sizes: the median of log(size) sits at the middle of the
    # log range (tolerance: four standard errors of a sample median)
    mid = 0.5 * (np.log(spec.size_lo) + np.log(spec.size_hi))
    se = 0.5 * (np.log(spec.size_hi) - np.log(spec.size_lo)) / np.sqrt(p.num_blocks)
    assert abs(np.median(np.log(p.size.astype(np.float64))) - mid) < 4 * se + 0.01


def test_ragged_clustered_workload():
    spec = workloads.CONFIGS[3]
    p = workloads.make_config(3, 0, num_segments=256)
    _common(p)
    nb = np.diff(p.seg_offsets.astype(np.int64))
    assert nb.min() >= spec.blocks[0] and nb.max() <= spec.blocks[1]
    frac_pinned = (p.kind == PINNED).mean()
    assert 0.25 < frac_pinned < 0.35
    assert p.size.max() <= spec.size_hi
    # pinned blocks come in clusters: mean pinned-run length near 1/0.3
    pin = (p.kind == PINNED).astype(np.int8)
    starts = np.sum((pin[1:] == 1) & (pin[:-1] == 0))
    assert 2.8 < pin.sum() / max(starts, 1) < 3.9


def test_huge_pool_shape():
    p = workloads.make_config(4, 0, blocks=(1 << 16, 1 << 16), requests_per_segment=32)
    _common(p)
    assert p.num_segments == 1 and p.num_requests == 32


def test_from_lists():
    p = workloads.from_lists([([512, 1024], [0, 5], [0, 1]), ([], [], [])], [[1, 2], [3]])
    assert p.seg_offsets.tolist() == [0, 2, 2]
    assert p.req_offsets.tolist() == [0, 2, 3]


def test_real_costs():
    """h = cost / staleness with staleness on 1..4096: deterministic, zero off
    evictable blocks, within [cost / 4096, cost], and not mostly integers."""
    p = workloads.make_config(1, 0, num_segments=16)
    h = workloads.real_costs(p, 3)
    assert h.dtype == np.float64 and len(h) == p.num_blocks
    assert np.array_equal(h, workloads.real_costs(p, 3))
    assert not np.array_equal(h, workloads.real_costs(p, 4))
    ev = p.kind == EVICTABLE
    assert (h[~ev] == 0).all()
    c = p.cost[ev].astype(np.float64)
    assert (h[ev] <= c).all() and (h[ev] >= c / 4096 * (1 - 1e-15)).all()
    assert np.mean(h[ev] != np.floor(h[ev])) > 0.9


def test_long_run_pool_layout():
    """workloads.long_run: one snapshot, parameters pinned at both ends and
    one pinned-free run between them; the spread set ends with the whole run
    and the half set asks for half of it; the same seed gives the same pool."""
    for name in workloads.LONG_RUN_SETS:
        p = workloads.long_run(n=1 << 14, request_set=name)
        assert p.num_segments == 1 and p.num_blocks == 1 << 14
        k = p.kind
        assert (k[:37] == workloads.PINNED).all() and (k[-53:] == workloads.PINNED).all()
        assert (k[37:-53] < workloads.PINNED).all()
        run = int(p.size[37:-53].sum())
        req = [int(x) for x in p.req_sizes]
        if name == "spread":
            assert len(req) == 16 and req[-1] == run and req[0] == 512
        if name == "half":
            assert req == [run // 2]
        if name == "whole":
            assert req == [run]
        assert (p.size % 512 == 0).all() and (p.size >= 512).all()
    a, b = workloads.long_run(n=1 << 12), workloads.long_run(n=1 << 12)
    assert a.digest() == b.digest()
