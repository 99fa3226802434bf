"""Pins the CPU oracle to things other than itself.

* hand-derived worked examples (tests/golden/window_examples.txt);
* brute force over every window, and Eq. (1) over every subset of
  evictable blocks (section 3.1), on tiny random pools;
* an independent pure-python enumeration of Eq. (1);
* special cases that reduce to textbook problems solved with numpy
  routines: all-free pools (shortest subarray with sum >= S) and equal sizes
  (minimum-sum window of fixed length);
* symmetries (mirror, scaling), monotonicity in S, and the invariants of
  tests/checks.py on every standard workload.
"""
import itertools

import numpy as np
import pytest

import oracle
import workloads
from checks import INF, check_results, run_totals

U64MAX = (1 << 64) - 1


def _single(ex):
    return (np.array(ex["size"], dtype=np.uint64), np.array(ex["cost"], dtype=np.uint64),
            np.array(ex["kind"], dtype=np.uint8))


def _expected_row(exp):
    return (U64MAX, U64MAX, U64MAX) if exp is None else exp


def test_golden_examples_sweep(golden_examples):
    assert len(golden_examples) >= 10
    for ex in golden_examples:
        size, cost, kind = _single(ex)
        reqs = [s for s, _ in ex["req"]]
        out = oracle.search_single(size, cost, kind, reqs)
        for (S, exp), row in zip(ex["req"], out.tolist()):
            assert tuple(row) == _expected_row(exp), (ex["name"], S, row, exp)


def test_golden_examples_brute_windows(golden_examples):
    for ex in golden_examples:
        size, cost, kind = _single(ex)
        reqs = np.array([s for s, _ in ex["req"]], dtype=np.uint64)
        out = oracle.brute_windows(size, cost, kind, [0, len(size)], reqs, [0, len(reqs)])
        for (S, exp), row in zip(ex["req"], out.tolist()):
            assert tuple(row) == _expected_row(exp), (ex["name"], S, row, exp)


def test_golden_examples_eq1(golden_examples):
    for ex in golden_examples:
        size, cost, kind = _single(ex)
        reqs = np.array([s for s, _ in ex["req"]], dtype=np.uint64)
        out = oracle.brute_eq1(size, cost, kind, [0, len(size)], reqs, [0, len(reqs)])
        for (S, exp), c in zip(ex["req"], out.tolist()):
            assert c == _expected_row(exp)[2], (ex["name"], S, c, exp)


def _random_tiny_batch(rng, nseg, max_n, max_evictable=12):
    """Several tiny snapshots with awkward features: zero sizes, pinned kinds
    other than 2, stored costs on free and pinned blocks, and requests at the
    exact run totals."""
    snaps, reqs = [], []
    for _ in range(nseg):
        n = int(rng.integers(0, max_n + 1))
        kind = rng.choice([0, 1, 1, 1, 2, 3, 255], size=n).astype(np.uint8)
        ev = np.flatnonzero(kind == 1)
        if len(ev) > max_evictable:
            kind[ev[max_evictable:]] = 0
        size = rng.choice([0, 1, 2, 3, 5, 8, 512, 4096], size=n).astype(np.uint64)
        cost = rng.integers(0, 20, size=n).astype(np.uint64)
        totals = run_totals(size, kind)
        cand = [0, 1, 2, 7, 100, 4096, 10000, U64MAX] + totals + [t + 1 for t in totals]
        cand += [t - 1 for t in totals if t > 0]
        pick = rng.choice(len(cand), size=min(len(cand), 12), replace=False)
        r = sorted(set(int(cand[i]) for i in pick))
        snaps.append((size, cost, kind))
        reqs.append(r)
    return workloads.from_lists(snaps, reqs)


@pytest.mark.parametrize("seed", range(40))
def test_sweep_matches_brute_windows(seed):
    rng = np.random.default_rng(1000 + seed)
    p = _random_tiny_batch(rng, nseg=8, max_n=14)
    a = oracle.window_search(*p.arrays())
    b = oracle.brute_windows(*p.arrays())
    assert np.array_equal(a, b)


@pytest.mark.parametrize("seed", range(40))
def test_sweep_cost_matches_eq1(seed):
    rng = np.random.default_rng(2000 + seed)
    p = _random_tiny_batch(rng, nseg=6, max_n=13)
    a = oracle.window_search(*p.arrays())
    c = oracle.brute_eq1(*p.arrays())
    assert np.array_equal(a[:, 2], c)
    # Infeasible exactly when Eq. (1) has no qualifying subset.
    assert np.array_equal(a[:, 0] == INF, c == INF)


def _eq1_python(size, cost, kind, S):
    """Eq. (1) by itertools, independent of the C code: the cheapest set of
    evictable blocks whose eviction leaves a contiguous available stretch of
    at least S bytes (free chunks are available from the start)."""
    ev = [k for k in range(len(size)) if kind[k] == 1]
    best = None
    for r in range(len(ev) + 1):
        for subset in itertools.combinations(ev, r):
            chosen = set(subset)
            largest = run = 0
            for k in range(len(size)):
                avail = kind[k] == 0 or k in chosen
                run = run + size[k] if avail else 0
                largest = max(largest, run)
            if largest >= S:
                c = sum(cost[k] for k in subset)
                best = c if best is None or c < best else best
    return best


@pytest.mark.parametrize("seed", range(12))
def test_sweep_cost_matches_python_eq1(seed):
    rng = np.random.default_rng(3000 + seed)
    n = int(rng.integers(1, 10))
    kind = [int(x) for x in rng.choice([0, 1, 1, 2], size=n)]
    size = [int(x) for x in rng.integers(1, 6, size=n)]
    cost = [int(x) for x in rng.integers(0, 9, size=n)]
    reqs = list(range(0, sum(size) + 2))
    out = oracle.search_single(size, cost, kind, reqs)
    for S, row in zip(reqs, out.tolist()):
        ref = _eq1_python(size, cost, kind, S)
        if ref is None:
            assert row == [U64MAX] * 3, (S, row)
        else:
            assert row[2] == ref, (S, row, ref)


@pytest.mark.parametrize("seed", range(10))
def test_all_free_is_shortest_subarray(seed):
    """All blocks free: every window costs 0, so the answer is the shortest
    (in bytes) window reaching S, lowest start on ties.  Reference: numpy
    prefix sums and searchsorted."""
    rng = np.random.default_rng(4000 + seed)
    n = 300
    size = rng.integers(1, 1000, size=n).astype(np.uint64)
    cost = rng.integers(0, 100, size=n).astype(np.uint64)   # stored, must be ignored
    kind = np.zeros(n, dtype=np.uint8)
    P = np.concatenate(([0], np.cumsum(size.astype(np.int64))))
    reqs = [1, 500, 1000, 5000, 20000, int(P[-1]), int(P[-1]) + 1]
    out = oracle.search_single(size, cost, kind, reqs)
    for S, row in zip(reqs, out.tolist()):
        e = np.searchsorted(P, P[:-1] + S, side="left")
        ok = e <= n
        if not ok.any():
            assert row == [U64MAX] * 3
            continue
        starts = np.flatnonzero(ok)
        bytes_ = P[e[starts]] - P[starts]
        i = starts[np.argmin(bytes_)]
        assert row == [int(i), int(e[i]), 0], (S, row)


@pytest.mark.parametrize("seed", range(10))
def test_equal_sizes_is_fixed_length_min_sum(seed):
    """All blocks evictable with equal size u: the window has exactly
    ceil(S/u) blocks, and the answer is the minimum-sum window of that
    length (first on ties).  Reference: numpy convolution and argmin."""
    rng = np.random.default_rng(5000 + seed)
    n, u = 200, 4096
    size = np.full(n, u, dtype=np.uint64)
    cost = rng.integers(0, 50, size=n).astype(np.uint64)
    kind = np.ones(n, dtype=np.uint8)
    reqs = [1, u, u + 1, 7 * u, 33 * u - 5, n * u, n * u + 1]
    out = oracle.search_single(size, cost, kind, reqs)
    for S, row in zip(reqs, out.tolist()):
        L = -(-S // u)
        if L > n:
            assert row == [U64MAX] * 3
            continue
        sums = np.convolve(cost.astype(np.int64), np.ones(L, dtype=np.int64), mode="valid")
        i = int(np.argmin(sums))
        assert row == [i, i + L, int(sums[i])], (S, row)


@pytest.mark.parametrize("seed", range(8))
def test_mirror_and_scale(seed):
    rng = np.random.default_rng(6000 + seed)
    p = _random_tiny_batch(rng, nseg=1, max_n=60, max_evictable=60)
    size, cost, kind, seg, req, roff = p.arrays()
    a = oracle.window_search(*p.arrays())
    # Mirroring the address order keeps the optimal cost and feasibility.
    m = oracle.window_search(size[::-1], cost[::-1], kind[::-1], seg, req, roff)
    assert np.array_equal(a[:, 2], m[:, 2])
    # Scaling every size and request by k keeps (start, end, cost).
    k = np.uint64(3)
    big = req < np.uint64(1 << 60)
    s = oracle.window_search(size * k, cost, kind, seg, np.where(big, req * k, req), roff)
    assert np.array_equal(a[big], s[big])


def test_cost_monotone_in_request():
    p = workloads.make_config(0, 0)
    size, cost, kind = p.size, p.cost, p.kind
    reqs = np.unique(np.concatenate([p.req_sizes, np.arange(1, 60) * (1 << 22)]))
    out = oracle.search_single(size, cost, kind, reqs)
    c = out[:, 2]
    assert np.all(c[1:] >= c[:-1])


@pytest.mark.parametrize("k,overrides", [
    (0, {}),
    (1, {"num_segments": 64}),
    (2, {"num_segments": 2, "blocks": (20000, 20000)}),
    (3, {"num_segments": 48}),
    (4, {"blocks": (200000, 200000), "requests_per_segment": 64}),
])
def test_invariants_on_workloads(k, overrides):
    p = workloads.make_config(k, 0, **overrides)
    out = oracle.window_search(*p.arrays(), threads=4)
    check_results(p, out)


def test_threads_do_not_change_results():
    p = workloads.make_config(3, 1, num_segments=64)
    a = oracle.window_search(*p.arrays(), threads=1)
    b = oracle.window_search(*p.arrays(), threads=7)
    assert np.array_equal(a, b)


def test_run_overflow_is_reported():
    big = np.array([1 << 63, 1 << 63], dtype=np.uint64)
    with pytest.raises(oracle.OracleError) as e:
        oracle.search_single(big, [0, 0], [0, 0], [1])
    assert e.value.code == -4
    # Two halves separated by a pinned block are fine.
    out = oracle.search_single(np.array([1 << 63, 1, 1 << 63], dtype=np.uint64),
                               [0, 0, 0], [0, 2, 0], [1 << 63])
    assert out.tolist() == [[0, 1, 0]]
    with pytest.raises(oracle.OracleError) as e:
        oracle.search_single([1, 1], [U64MAX, 1], [1, 1], [2])
    assert e.value.code == -4


def test_invalid_offsets_are_rejected():
    size = np.ones(4, dtype=np.uint64)
    with pytest.raises(oracle.OracleError) as e:
        oracle.window_search(size, size, np.zeros(4, np.uint8), [0, 3], [1], [0, 1])
    assert e.value.code == -1
    with pytest.raises(oracle.OracleError):
        oracle.window_search(size, size, np.zeros(4, np.uint8), [0, 3, 2], [1, 1], [0, 1, 2])
    with pytest.raises(oracle.OracleError):
        oracle.window_search(size, size, np.zeros(4, np.uint8), [0, 4], [1], [0, 2])


def test_empty_batches():
    z = np.zeros(0, dtype=np.uint64)
    out = oracle.window_search(z, z, np.zeros(0, np.uint8), [0, 0, 0], [0, 5, 1], [0, 2, 3])
    assert out.tolist() == [[0, 0, 0], [U64MAX] * 3, [U64MAX] * 3]
