"""Pins the first-fit oracle (section 2.1; find_free_block_not_less_than in
Algorithm 1) to things other than itself:

* hand-derived worked examples (tests/golden/first_fit_examples.txt);
* an independent formulation: the running maximum of free-chunk sizes is
  non-decreasing, so the first fit is numpy.searchsorted of S in it;
* invariants: the answer is a free chunk of at least S bytes and no earlier
  free chunk fits; no answer exactly when the largest free chunk is smaller
  than S; answers move right as S grows;
* agreement with the window search: a fitting free chunk is a zero-cost
  window of at least S bytes (section 3.3 treats free chunks as zero-cost
  entries), so first fit succeeds only where the window search finds cost 0.
"""
import os

import numpy as np
import pytest

import oracle
import workloads

U64MAX = (1 << 64) - 1
GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden",
                      "first_fit_examples.txt")
KINDS = {"F": 0, "E": 1, "P": 2}


def _value(tok, unit):
    return int(tok[:-1]) * unit if tok.endswith("u") else int(tok)


def load_examples(path=GOLDEN):
    examples, cur, unit = [], None, 1
    for raw in open(path):
        line = raw.split("#", 1)[0].strip()
        if not line:
            continue
        tok = line.split()
        if tok[0] == "example":
            cur = {"name": tok[1], "size": [], "kind": [], "req": []}
            examples.append(cur)
            unit = 1
        elif tok[0] == "unit":
            unit = int(tok[1])
        elif tok[0] == "block":
            cur["kind"].append(KINDS[tok[1]] if tok[1] in KINDS else int(tok[1]))
            cur["size"].append(_value(tok[2], unit))
        elif tok[0] == "S":
            assert tok[2] == "->", line
            cur["req"].append((_value(tok[1], unit), None if tok[3] == "none" else int(tok[3])))
        else:
            raise ValueError(f"bad line: {line}")
    return examples


def _ff_single(size, kind, reqs):
    return oracle.first_fit(np.array(size, np.uint64), np.array(kind, np.uint8),
                            [0, len(size)], np.array(reqs, np.uint64), [0, len(reqs)])


def test_golden_examples():
    examples = load_examples()
    assert len(examples) >= 6
    for ex in examples:
        got = _ff_single(ex["size"], ex["kind"], [s for s, _ in ex["req"]])
        for (S, want), g in zip(ex["req"], got.tolist()):
            assert g == (U64MAX if want is None else want), (ex["name"], S, g, want)


def _searchsorted_first_fit(size, kind, S):
    """Independent formulation: the running maximum of free sizes is
    non-decreasing; the first index where it reaches S is the first fit."""
    free = np.where(kind == 0, size, np.uint64(0))
    if len(size) == 0:
        return U64MAX
    run_max = np.maximum.accumulate(free)
    if S == 0:
        idx = np.flatnonzero(kind == 0)
        return int(idx[0]) if len(idx) else U64MAX
    k = int(np.searchsorted(run_max, np.uint64(S), side="left"))
    return k if k < len(size) else U64MAX


@pytest.mark.parametrize("seed", range(6))
def test_matches_running_maximum_search(seed):
    rng = np.random.default_rng(300 + seed)
    for _ in range(40):
        n = int(rng.integers(0, 60))
        size = (rng.integers(0, 32, size=n) * 512).astype(np.uint64)
        kind = rng.choice([0, 1, 1, 2, 7], size=n).astype(np.uint8)
        reqs = [0, 1, 512, 4096, 8192, 16384] + [int(x) for x in rng.integers(0, 20000, 6)]
        got = _ff_single(size, kind, reqs)
        for S, g in zip(reqs, got.tolist()):
            assert g == _searchsorted_first_fit(size, kind, S), (seed, n, S)


def _check_invariants(pools, got):
    seg, roff = pools.seg_offsets, pools.req_offsets
    for b in range(pools.num_segments):
        s0, s1 = int(seg[b]), int(seg[b + 1])
        size, kind = pools.size[s0:s1], pools.kind[s0:s1]
        free = np.where(kind == 0, size, np.uint64(0))
        biggest = int(free.max()) if s1 > s0 and (kind == 0).any() else -1
        for q in range(int(roff[b]), int(roff[b + 1])):
            S, k = int(pools.req_sizes[q]), int(got[q])
            if k == U64MAX:
                assert biggest < S, (b, q, S, biggest)
                continue
            assert k < s1 - s0 and kind[k] == 0 and int(size[k]) >= S, (b, q)
            # no free chunk before k fits
            assert k == 0 or int(free[:k].max()) < S or (S == 0 and not (kind[:k] == 0).any())


@pytest.mark.parametrize("k,overrides", [
    (0, {}), (1, {"num_segments": 64}), (2, {"num_segments": 4}), (3, {"num_segments": 48}),
])
def test_invariants_on_standard_workloads(k, overrides):
    pools = workloads.make_config(k, 0, **overrides)
    got = oracle.first_fit(pools.size, pools.kind, pools.seg_offsets, pools.req_sizes,
                           pools.req_offsets, threads=4)
    _check_invariants(pools, got)


def test_monotone_in_request_size():
    rng = np.random.default_rng(17)
    n = 3000
    size = (rng.integers(1, 4096, size=n) * 512).astype(np.uint64)
    kind = rng.choice([0, 1, 1, 1, 2], size=n).astype(np.uint8)
    reqs = np.sort(rng.integers(0, 4096 * 512, size=200)).astype(np.uint64)
    got = _ff_single(size, kind, reqs)
    hits = got[got != U64MAX]
    assert (np.diff(hits.astype(np.int64)) >= 0).all()
    # once a request misses, every larger one misses too
    miss = np.flatnonzero(got == U64MAX)
    if len(miss):
        assert (got[miss[0]:] == U64MAX).all()


def test_first_fit_implies_zero_cost_window():
    pools = workloads.make_config(3, 1, num_segments=32)
    ff = oracle.first_fit(pools.size, pools.kind, pools.seg_offsets, pools.req_sizes,
                          pools.req_offsets)
    win = oracle.window_search(pools.size, pools.cost, pools.kind, pools.seg_offsets,
                               pools.req_sizes, pools.req_offsets)
    for q in range(pools.num_requests):
        if ff[q] != U64MAX and pools.req_sizes[q] > 0:
            assert win[q, 2] == 0, q


def test_rejects_bad_offsets():
    with pytest.raises(oracle.OracleError):
        oracle.first_fit(np.zeros(4, np.uint64), np.zeros(4, np.uint8), [0, 3],
                         np.zeros(1, np.uint64), [0, 1])
