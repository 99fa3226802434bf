"""Pins the oracle's DTR-style greedy eviction policy (the baseline Coop is
compared against; section 3.3 restates DTR's heuristic h = c / (m * s)) to
things other than itself:

* hand-derived worked replays (tests/golden/greedy_examples.txt), among
  them a tie, a failure after evictions, and costs whose ratios double
  precision cannot tell apart;
* a brute-force replay written here in plain Python, with h compared as
  exact fractions, on every step of generated training traces;
* with a budget large enough for every tensor nothing is evicted, and the
  greedy and window policies then give the same replay.
"""
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle
from conftest import parse_greedy_golden
from workloads import traces

U64MAX = (1 << 64) - 1
MiB = 1 << 20
GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden",
                      "greedy_examples.txt")
GREEDY = 1


def _state(blocks, cap):
    size = np.zeros(cap, np.uint64)
    kind = np.full(cap, 2, np.uint8)
    cost = np.zeros(cap, np.uint64)
    ids = np.zeros(cap, np.uint32)
    for j, (k, s, i, c) in enumerate(blocks):
        size[j], kind[j], ids[j], cost[j] = s, k, i, c
    return {"size": size, "cost": cost, "kind": kind, "id": ids,
            "len": np.array([len(blocks)], np.uint64), "capacity": cap}


def _blocks(st):
    n = int(st["len"][0])
    return [(int(st["kind"][j]), int(st["size"][j]), int(st["id"][j]), int(st["cost"][j]))
            for j in range(n)]


def test_golden_greedy():
    cases = parse_greedy_golden(GOLDEN)
    assert len(cases) >= 6
    for case in cases:
        st = _state(case["pool"], 16)
        for stp in case["steps"]:
            o = stp["op"]
            assert o[0] == "alloc"
            tr = {"op": [0], "op_id": [int(o[1])], "op_size": [int(o[2]) * MiB],
                  "op_cost": [int(o[3])], "op_flags": [1 if o[4] == "left" else 0]}
            st, out = oracle.replay(st, tr, policy=GREEDY)
            e = stp["expect"]
            where = (case["name"], o)
            assert int(out["block"][0, 0]) == (U64MAX if e[0] == "none" else int(e[0])), where
            assert e[1] == "evict"
            assert out["window"][0, 0].tolist() == [int(e[2]), U64MAX], where
            assert int(out["cost"][0, 0]) == int(e[3]), where
            assert int(out["free"][0, 0]) == int(e[4]) * MiB, where
            assert [b[:3] for b in _blocks(st)] == stp["after"], (where, _blocks(st))


# --- brute force ----------------------------------------------------------

def _h(blk, op_id):
    """h = c / (m * s) as an exact fraction (zero size or staleness as 1)."""
    k, m, i, c = blk
    s = (op_id - i) % (1 << 32)
    return Fraction(c, max(m, 1) * max(s, 1))


def _free_and_merge(pool, j):
    lo, hi = j, j + 1
    if lo > 0 and pool[lo - 1][0] == 0:
        lo -= 1
    if hi < len(pool) and pool[hi][0] == 0:
        hi += 1
    total = sum(b[1] for b in pool[lo:hi])
    return pool[:lo] + [(0, total, 0, 0)] + pool[hi:], lo


def _first_fit(pool, S):
    return next((j for j, b in enumerate(pool) if b[0] == 0 and b[1] >= S), None)


def _brute_step(pool, op, oid, S, c, flags):
    """One operation on a list of (kind, size, id, cost); returns the new list
    and (block, evicted count, evicted cost, free bytes before)."""
    if op == 1:
        j = next((j for j, b in enumerate(pool) if b[0] != 0 and b[2] == oid), None)
        if j is None:
            return pool, (U64MAX, 0, 0, U64MAX)
        pool, lo = _free_and_merge(pool, j)
        return pool, (lo, 0, 0, U64MAX)
    k = _first_fit(pool, S)
    count, evc, free0 = 0, 0, U64MAX
    if k is None:
        free0 = sum(b[1] for b in pool if b[0] == 0)
        while k is None:
            cand = [j for j, b in enumerate(pool) if b[0] == 1]
            if not cand:
                break
            v = min(cand, key=lambda j: (_h(pool[j], oid), j))
            count += 1
            evc += pool[v][3]
            pool, _ = _free_and_merge(pool, v)
            k = _first_fit(pool, S)
        if count == 0:
            free0 = U64MAX
        if k is None:
            return pool, (U64MAX, count, evc % (1 << 64), free0)
    F = pool[k][1]
    t = (2 if flags & 2 else 1, S, oid, c)
    if F == S:
        new, at = [t], k
    elif flags & 1:
        new, at = [t, (0, F - S, 0, 0)], k
    else:
        new, at = [(0, F - S, 0, 0), t], k + 1
    return pool[:k] + new + pool[k + 1:], (at, count, evc % (1 << 64), free0)


def _pool0(st, tr):
    cap, T = st["capacity"], tr["num_ops"]
    s0 = {k: np.array(st[k][:cap]) for k in ("size", "cost", "kind", "id")}
    s0["len"] = np.array(st["len"][:1], np.uint64)
    s0["capacity"] = cap
    return s0, {k: np.array(tr[k][:T]) for k in ("op", "op_id", "op_size", "op_cost",
                                                  "op_flags")}


@pytest.mark.parametrize("k,seed", [(0, 0), (0, 1), (1, 2), (1, 5)])
def test_whole_trace_against_brute_force(k, seed):
    st, tr = traces.make_replay(k, seed)
    st, tr = _pool0(st, tr)
    pool = _blocks(st)
    post, out = oracle.replay(st, tr, policy=GREEDY)
    evictions = 0
    for t in range(len(tr["op"])):
        pool, (blk, cnt, evc, free0) = _brute_step(
            pool, int(tr["op"][t]), int(tr["op_id"][t]), int(tr["op_size"][t]),
            int(tr["op_cost"][t]), int(tr["op_flags"][t]))
        got_w = out["window"][0, t].tolist()
        assert int(out["block"][0, t]) == blk, t
        assert got_w == ([cnt, U64MAX] if cnt else [U64MAX, U64MAX]), t
        assert int(out["cost"][0, t]) == evc, t
        assert int(out["free"][0, t]) == free0, t
        evictions += cnt
    assert evictions > 0
    assert _blocks(post) == pool


def test_ample_budget_policies_agree():
    cap = 64
    st = _state([(2, 4 * MiB, 1, 0), (0, 1000 * MiB, 0, 0), (2, 4 * MiB, 2, 0)], cap)
    sizes = [3, 5, 2, 7, 1, 4]
    n = len(sizes)
    tr = {"op": [0] * n + [1, 1], "op_id": list(range(10, 10 + n)) + [12, 10],
          "op_size": [s * MiB for s in sizes] + [0, 0], "op_cost": [1] * n + [0, 0],
          "op_flags": [1, 0] * (n // 2) + [0, 0]}
    a_state, a = oracle.replay(st, tr, policy=0)
    b_state, b = oracle.replay(st, tr, policy=GREEDY)
    for key in a:
        assert np.array_equal(a[key], b[key]), key
    assert (a["free"] == U64MAX).all()
    assert _blocks(a_state) == _blocks(b_state)


def test_policies_differ_on_training_traces():
    """Same trace, two policies: both replay it, and they choose differently."""
    st, tr = traces.make_replay(1, 7)
    _, a = oracle.replay(st, tr, threads=4, policy=0)
    _, b = oracle.replay(st, tr, threads=4, policy=GREEDY)
    ev_a, ev_b = a["free"] != U64MAX, b["free"] != U64MAX
    assert ev_a.any() and ev_b.any()
    assert (b["window"][..., 1][ev_b] == U64MAX).all()
    assert not np.array_equal(a["block"], b["block"])


def test_rejects_unknown_policy():
    st = _state([(0, 8 * MiB, 0, 0)], 4)
    tr = {"op": [0], "op_id": [5], "op_size": [MiB], "op_cost": [1], "op_flags": [0]}
    with pytest.raises(oracle.OracleError):
        oracle.replay(st, tr, policy=2)
