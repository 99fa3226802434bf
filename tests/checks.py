"""Properties every correct search result has, whoever computed it.

Used on oracle outputs (pinning the oracle at full size, where nothing can
be enumerated) and on GPU outputs.  Definitions follow section 3.1 Eq. (1)
and section 3.3: a window is a stretch of adjacent blocks with no pinned
block whose byte total reaches S; its cost is the summed cost of its
evictable blocks.
"""
import numpy as np

INF = np.uint64(0xFFFFFFFFFFFFFFFF)


def run_totals(size, kind):
    """Byte totals (python ints) of the maximal unpinned stretches."""
    totals, cur, inrun = [], 0, False
    for s, k in zip(size.tolist(), kind.tolist()):
        if k >= 2:
            if inrun:
                totals.append(cur)
            cur, inrun = 0, False
        else:
            cur += s
            inrun = True
    if inrun:
        totals.append(cur)
    return totals


def check_results(pools, out, sample=None):
    """Asserts the invariants for the rows of `out` (uint64 (Q, 3)).
    `sample` optionally restricts the check to those request indices."""
    size, cost, kind, seg, req, roff = pools.arrays()
    out = np.asarray(out, dtype=np.uint64)
    B = len(seg) - 1
    qs = range(len(req)) if sample is None else sample
    owner = np.searchsorted(roff, np.asarray(list(qs), dtype=np.uint64), side="right") - 1
    largest_cache = {}
    for q, b in zip(qs, owner.tolist()):
        assert 0 <= b < B
        s0, s1 = int(seg[b]), int(seg[b + 1])
        n = s1 - s0
        S = int(req[q])
        st, en, c = (int(x) for x in out[q])
        if S == 0:
            assert (st, en, c) == (0, 0, 0), (q, S, out[q])
            continue
        if b not in largest_cache:
            t = run_totals(size[s0:s1], kind[s0:s1])
            largest_cache[b] = max(t) if t else 0
        if st == int(INF):
            assert en == int(INF) and c == int(INF), (q, out[q])
            assert largest_cache[b] < S, f"request {q}: reported infeasible but a run holds {largest_cache[b]} >= {S}"
            continue
        assert 0 <= st < en <= n, (q, out[q], n)
        k = kind[s0 + st:s0 + en]
        assert (k < 2).all(), f"request {q}: window contains a pinned block"
        sz = [int(x) for x in size[s0 + st:s0 + en]]
        cs = [int(x) if kk == 1 else 0 for x, kk in zip(cost[s0 + st:s0 + en], k.tolist())]
        assert sum(sz) >= S, (q, sum(sz), S)
        assert sum(cs) == c, (q, sum(cs), c)
        # Tight on both sides when sizes are positive: dropping the first or
        # the last block must leave fewer than S bytes.
        if all(x > 0 for x in sz):
            assert sum(sz[1:]) < S, (q, "start not tight")
            assert sum(sz[:-1]) < S, (q, "end not tight")
