"""Pins the replay oracle (Algorithm 1 with section 3.4's placement, and
releases) to things other than itself:

* a hand-derived worked replay (tests/golden/replay_examples.txt);
* every step of generated training traces, taken one operation at a time,
  checked against the separately pinned first-fit and window-search oracles
  on the state before the step (which chunk, which window, which cost, the
  free bytes sampled), and against allocator invariants after it: the pool
  keeps its bytes, no two free chunks touch, tensor ids stay unique, a
  placed tensor has its size, kind and id at the reported block, at the
  chunk's left end for an expensive operation and its right end otherwise;
* a budget large enough for every tensor: no eviction ever, and a forward
  pass of only expensive (or only cheap) tensors lays them out from the
  chunk's left end in allocation order (or from its right end, the latest
  leftmost) -- the textbook first-fit layout.
"""
import os

import numpy as np
import pytest

import oracle
from workloads import traces

U64MAX = (1 << 64) - 1
MiB = 1 << 20
GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden",
                      "replay_examples.txt")
KIND = {"F": 0, "E": 1, "P": 2}


def _state(blocks, cap):
    size = np.zeros(cap, np.uint64)
    kind = np.full(cap, 2, np.uint8)
    cost = np.zeros(cap, np.uint64)
    ids = np.zeros(cap, np.uint32)
    for j, (k, s, i) in enumerate(blocks):
        size[j], kind[j], ids[j] = s, k, i
    return {"size": size, "cost": cost, "kind": kind, "id": ids,
            "len": np.array([len(blocks)], np.uint64), "capacity": cap}


def _one_op(op, oid, size=0, cost=0, flags=0):
    return {"op": [op], "op_id": [oid], "op_size": [size], "op_cost": [cost],
            "op_flags": [flags]}


def _blocks(st, b=0):
    cap = st["capacity"]
    n = int(st["len"][b])
    base = b * cap
    return [(int(st["kind"][base + j]), int(st["size"][base + j]), int(st["id"][base + j]))
            for j in range(n)]


def _parse_blocks(text):
    out = []
    for part in text.split("|"):
        k, s, i = part.split()
        out.append((KIND[k], int(s) * MiB, int(i)))
    return out


def test_golden_replay():
    pool, steps, cur = [], [], None
    for raw in open(GOLDEN):
        line = raw.split("#", 1)[0].strip()
        if not line:
            continue
        tok = line.split()
        if tok[0] == "pool":
            pool.append((KIND[tok[1]], int(tok[2]) * MiB, int(tok[3])))
        elif tok[0] == "op":
            cur = {"op": tok[1:]}
            steps.append(cur)
        elif tok[0] == "expect":
            cur["expect"] = tok[1:]
        elif tok[0] == "after":
            cur["after"] = _parse_blocks(line[len("after"):])
    assert len(steps) >= 8
    st = _state(pool, 16)
    costs = {}
    for stp in steps:
        o = stp["op"]
        if o[0] == "alloc":
            oid, s, c = int(o[1]), int(o[2]) * MiB, int(o[3])
            costs[oid] = c
            tr = _one_op(0, oid, s, c, 1 if o[4] == "left" else 0)
        else:
            tr = _one_op(1, int(o[1]))
        st, out = oracle.replay(st, tr)
        e = stp["expect"]
        want_block = U64MAX if e[0] == "none" else int(e[0])
        assert int(out["block"][0, 0]) == want_block, (o, out["block"])
        if len(e) > 1:
            assert e[1] == "window"
            assert out["window"][0, 0].tolist() == [int(e[2]), int(e[3])], o
            assert int(out["cost"][0, 0]) == int(e[4]), o
            assert int(out["free"][0, 0]) == int(e[5]) * MiB, o
        else:
            assert out["window"][0, 0].tolist() == [U64MAX, U64MAX], o
            assert int(out["free"][0, 0]) == U64MAX, o
        assert _blocks(st) == stp["after"], (o, _blocks(st))


def _check_step(pre, post, tr, out, t):
    """One operation of pool 0, against the first-fit and window oracles."""
    before, after = _blocks(pre), _blocks(post)
    assert sum(s for _, s, _ in after) == sum(s for _, s, _ in before)
    for (k1, _, _), (k2, _, _) in zip(after, after[1:]):
        assert not (k1 == 0 and k2 == 0), "two free chunks touch"
    live = [i for k, _, i in after if k != 0]
    assert len(live) == len(set(live))
    blk = int(out["block"][0, 0])
    if tr["op"][0] == 1:
        ids = [i for k, _, i in before if k != 0]
        if tr["op_id"][0] in ids:
            assert after[blk][0] == 0 and tr["op_id"][0] not in live
        else:
            assert blk == U64MAX and after == before
        return
    S, flags = int(tr["op_size"][0]), int(tr["op_flags"][0])
    size = np.array([s for _, s, _ in before], np.uint64)
    kind = np.array([k for k, _, _ in before], np.uint8)
    cost = np.array([int(pre["cost"][j]) for j in range(len(before))], np.uint64)
    n = len(before)
    ff = int(oracle.first_fit(size, kind, [0, n], [S], [0, 1])[0])
    win = oracle.window_search(size, cost, kind, [0, n], [S], [0, 1])[0].tolist()
    if ff != U64MAX:
        assert out["window"][0, 0].tolist() == [U64MAX, U64MAX]
        F = int(size[ff])
        want = ff if (F == S or flags & 1) else ff + 1
        assert blk == want
    elif win[0] == U64MAX:
        assert blk == U64MAX and after == before
        return
    else:
        assert out["window"][0, 0].tolist() == win[:2] and int(out["cost"][0, 0]) == win[2]
        assert int(out["free"][0, 0]) == int(size[kind == 0].sum())
    k, s, i = after[blk]
    assert (k, s, i) == ((2 if flags & 2 else 1), S, int(tr["op_id"][0]))
    assert int(post["cost"][blk]) == int(tr["op_cost"][0])
    # the chunk's leftover, if any, lies on the side away from the chosen end
    # (the chunk had no free neighbour, so the other side is occupied)
    wrong = blk - 1 if flags & 1 else blk + 1
    assert not (0 <= wrong < len(after) and after[wrong][0] == 0)


def _pool0(st, tr):
    """Pool 0 of a generated replay, as a one-pool state and its trace."""
    cap, T = st["capacity"], tr["num_ops"]
    s0 = {k: np.array(st[k][:cap]) for k in ("size", "cost", "kind", "id")}
    s0["len"] = np.array(st["len"][:1], np.uint64)
    s0["capacity"] = cap
    return s0, {k: np.array(tr[k][:T]) for k in ("op", "op_id", "op_size", "op_cost",
                                                  "op_flags")}


@pytest.mark.parametrize("k,seed", [(0, 0), (0, 1), (1, 2)])
def test_every_step_against_first_fit_and_window_oracles(k, seed):
    st, tr = traces.make_replay(k, seed)
    st, tr = _pool0(st, tr)
    T = len(tr["op"])
    evictions = 0
    for t in range(T):
        one = {key: tr[key][t:t + 1] for key in tr}
        post, out = oracle.replay(st, one)
        _check_step(st, post, one, out, t)
        evictions += int(out["free"][0, 0] != U64MAX)
        st = post
    assert evictions > 0


def test_whole_trace_equals_stepwise():
    st, tr = traces.make_replay(1, 3)
    whole_state, whole = oracle.replay(st, tr, threads=4)
    s0, t0 = _pool0(st, tr)
    blocks = []
    for t in range(len(t0["op"])):
        s0, out = oracle.replay(s0, {key: t0[key][t:t + 1] for key in t0})
        blocks.append(int(out["block"][0, 0]))
    assert blocks == whole["block"][0].tolist()
    assert _blocks(s0) == _blocks(whole_state)


@pytest.mark.parametrize("flags", [1, 0])
def test_ample_budget_is_textbook_first_fit(flags):
    cap = 64
    st = _state([(2, 4 * MiB, 1), (0, 1000 * MiB, 0), (2, 4 * MiB, 2)], cap)
    sizes = [3, 5, 2, 7, 1, 4]
    tr = {"op": [0] * len(sizes), "op_id": list(range(10, 10 + len(sizes))),
          "op_size": [s * MiB for s in sizes], "op_cost": [1] * len(sizes),
          "op_flags": [flags] * len(sizes)}
    post, out = oracle.replay(st, tr)
    assert (out["free"] == U64MAX).all()
    got = [(s // MiB, i) for k, s, i in _blocks(post) if k == 1]
    if flags:  # from the left end, in allocation order
        assert got == [(s, 10 + j) for j, s in enumerate(sizes)]
    else:      # from the right end: the latest allocation is leftmost
        assert got == [(s, 10 + j) for j, s in reversed(list(enumerate(sizes)))]
    assert _blocks(post)[0][1] == 4 * MiB and _blocks(post)[-1][1] == 4 * MiB


def test_rejects_invalid_operations_and_overflowing_pools():
    st = _state([(0, 8 * MiB, 0)], 2)
    with pytest.raises(oracle.OracleError):
        oracle.replay(st, _one_op(0, 5, 0, 1, 1))       # zero-byte allocation
    with pytest.raises(oracle.OracleError):
        oracle.replay(st, {"op": [0, 0], "op_id": [5, 6], "op_size": [MiB, MiB],
                           "op_cost": [1, 1], "op_flags": [0, 0]})  # third block: no slot
