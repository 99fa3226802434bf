"""Pins the oracle's search with real-valued heuristics (section 3.3 defines
h = c / s, a real number; a window costs the exact sum of its h values) to
things other than itself:

* hand-derived examples (tests/golden/real_examples.txt): section 3.4's
  x0..x4 with h = c / s, a case that real values decide and integer ones
  would not, the rounding of values below 2^-12 to multiples of 2^-64, and a
  case that binary64 addition in address order would get wrong;
* brute force over every window with exact rational sums
  (fractions.Fraction) on tiny random pools, the returned binary64 cost
  checked against Python's correctly rounded conversion;
* integer-valued h reproduces the separately pinned integer search;
* scaling every h by a power of two scales the costs and keeps the windows;
* invalid values and overflowing runs are refused.
"""
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle
from conftest import parse_real_golden

MiB = 1 << 20
U64MAX = (1 << 64) - 1
GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden",
                      "real_examples.txt")


def _one(blocks, reqs):
    kind = np.array([k for k, _, _ in blocks], np.uint8)
    size = np.array([s for _, s, _ in blocks], np.uint64)
    h = np.array([x for _, _, x in blocks], np.float64)
    return oracle.window_search_real(size, h, kind, [0, len(blocks)], reqs, [0, len(reqs)])


def test_golden_real():
    ex = parse_real_golden(GOLDEN)
    assert len(ex) >= 7
    for e in ex:
        res, cost = _one(e["blocks"], [s for s, _ in e["reqs"]])
        for q, (S, want) in enumerate(e["reqs"]):
            got = res[q].tolist()
            if want is None:
                assert got == [U64MAX] * 4 and cost[q] == np.inf, (e["name"], S)
                continue
            start, end, hi, lo = want
            assert got == [start, end, lo, hi], (e["name"], S, got)
            assert cost[q] == float(Fraction((hi << 64) + lo, 1 << 64)), (e["name"], S)


def _units(x):
    """h in units of 2^-64, rounded to nearest with ties to even (Python's
    round of a Fraction)."""
    return round(Fraction(float(x)) * (1 << 64))


def _brute(size, h, kind, S):
    """Every window, exact integer sums of the rounded units; (cost, bytes,
    start, end) minimal."""
    n = len(size)
    if S == 0:
        return (0, 0, 0, 0)
    best = None
    for i in range(n):
        c, b = 0, 0
        for j in range(i, n):
            if kind[j] >= 2:
                break
            b += int(size[j])
            if kind[j] == 1:
                c += _units(h[j])
            if b >= S:
                key = (c, b, i, j + 1)
                if best is None or key[:3] < best[:3]:
                    best = key
                break  # longer windows from i cost no less
    return best


def _random_h(rng, n):
    """Binary64 values of several kinds: quotients c / s (mostly not dyadic),
    small integers (ties), fractions of 2^-20, large values, zeros, values
    whose last bit is worth 2^-64 (in [2^-12, 2^-11)) and values below 2^-12
    that round."""
    pick = rng.integers(0, 7, n)
    c = rng.integers(1, 10**6, n).astype(np.float64)
    s = rng.integers(1, 4096, n).astype(np.float64)
    odd = np.ldexp((rng.integers(1 << 51, 1 << 52, n) * 2 + 1).astype(np.float64), -64)
    tiny = np.ldexp(rng.integers(1, 64, n).astype(np.float64), -int(rng.integers(64, 72)))
    h = np.select([pick == 0, pick == 1, pick == 2, pick == 3, pick == 4, pick == 5],
                  [c / s, np.floor(c / 64), np.ldexp(c, -20), c * 2.0**20, odd, tiny], 0.0)
    return h


@pytest.mark.parametrize("seed", range(8))
def test_brute_force_exact_rationals(seed):
    rng = np.random.default_rng([7, seed])
    for trial in range(40):
        n = int(rng.integers(0, 14))
        size = (rng.integers(1, 9, n) * MiB).astype(np.uint64)
        kind = rng.choice([0, 1, 1, 1, 2], n).astype(np.uint8)
        h = _random_h(rng, n)
        h[kind != 1] = rng.choice([np.nan, -1.0, 5.0])   # ignored off evictable blocks
        reqs = [0, 1, int(rng.integers(1, 40)) * MiB, int(rng.integers(1, 12)) * MiB]
        res, cost = oracle.window_search_real(size, h, kind, [0, n], reqs, [0, len(reqs)])
        for q, S in enumerate(reqs):
            want = _brute(size, h, kind, S)
            if want is None:
                assert res[q].tolist() == [U64MAX] * 4 and cost[q] == np.inf
                continue
            units, _, i, j = want
            assert res[q].tolist() == [i, j, units & U64MAX, units >> 64], (seed, trial, S)
            assert cost[q] == float(Fraction(units, 1 << 64)), (seed, trial, S)


def test_integer_values_match_the_integer_search():
    import workloads
    for k in (0, 1):
        p = workloads.make_config(k, 0)
        if k == 1:
            p = workloads.from_lists(
                [(p.size[:4096], p.cost[:4096], p.kind[:4096])], [[int(p.req_sizes[0]), 1 << 22]])
        h = p.cost.astype(np.float64)
        assert (h.astype(np.uint64) == p.cost).all()   # exact below 2^53
        want = oracle.window_search(p.size, p.cost, p.kind, p.seg_offsets, p.req_sizes,
                                    p.req_offsets, threads=4)
        res, cost = oracle.window_search_real(p.size, h, p.kind, p.seg_offsets, p.req_sizes,
                                              p.req_offsets, threads=4)
        ok = want[:, 0] != np.uint64(U64MAX)
        assert (res[:, :2] == want[:, :2]).all()
        assert (res[ok, 3] == want[ok, 2]).all() and (res[ok, 2] == 0).all()
        assert (cost[ok] == want[ok, 2].astype(np.float64)).all()


@pytest.mark.parametrize("e", [-3, 5, 20])
def test_power_of_two_scaling(e):
    rng = np.random.default_rng(11)
    n = 3000
    size = (rng.integers(1, 64, n) * MiB).astype(np.uint64)
    kind = rng.choice([0, 1, 1, 1, 1, 2], n).astype(np.uint8)
    h = np.floor(rng.uniform(1, 1e6, n))
    reqs = (rng.integers(1, 400, 50) * MiB).astype(np.uint64)
    a, ca = oracle.window_search_real(size, h, kind, [0, n], reqs, [0, len(reqs)])
    b, cb = oracle.window_search_real(size, np.ldexp(h, e), kind, [0, n], reqs, [0, len(reqs)])
    assert (a[:, :2] == b[:, :2]).all()
    ok = a[:, 0] != np.uint64(U64MAX)
    for q in np.flatnonzero(ok):
        ua = (int(a[q, 3]) << 64) | int(a[q, 2])
        ub = (int(b[q, 3]) << 64) | int(b[q, 2])
        assert ub == (ua << e if e >= 0 else ua >> -e)
    assert (cb[ok] == np.ldexp(ca[ok], e)).all()


def test_invalid_values_and_overflow():
    size = np.array([MiB, MiB], np.uint64)
    kind = np.array([1, 1], np.uint8)
    for bad in (np.nan, -1.0, np.inf, 2.0**64):
        with pytest.raises(oracle.OracleError) as ei:
            oracle.window_search_real(size, [1.0, bad], kind, [0, 2], [MiB], [0, 1])
        assert ei.value.code == -6
    # -0.0 and values just below 2^64 are valid
    oracle.window_search_real(size, [-0.0, np.nextafter(2.0**64, 0)], kind, [0, 2], [MiB], [0, 1])
    # two halves of 2^64 in one run: the run's total reaches 2^64
    with pytest.raises(oracle.OracleError) as ei:
        oracle.window_search_real(size, [2.0**63, 2.0**63], kind, [0, 2], [MiB], [0, 1])
    assert ei.value.code == -4
    # separated by a pinned block they are fine
    res, cost = oracle.window_search_real(np.array([MiB] * 3, np.uint64), [2.0**63, 0, 2.0**63],
                                          np.array([1, 2, 1], np.uint8), [0, 3], [MiB], [0, 1])
    assert res[0].tolist() == [0, 1, 0, 1 << 63] and cost[0] == 2.0**63
