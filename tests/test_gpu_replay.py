"""GPU replay of Algorithm 1 (coop_replay) equals the CPU oracle's replay:
every operation's outcome (block, evicted window, its cost, the free-bytes
sample) and the final pools, slot for slot, through the C ABI -- under
Coop's sliding-window eviction and under the DTR-style greedy baseline."""
import sys

import numpy as np
import pytest

import oracle
from conftest import GOLDEN, parse_greedy_golden
from workloads import traces

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

U64MAX = (1 << 64) - 1
MiB = 1 << 20
WINDOW, GREEDY = 0, 1


def _announce(label):
    print(f"[gpu case] replay: {label}", flush=True)
    sys.stdout.flush()


def gpu_replay(state, trace, policy=WINDOW):
    import paper_2311_00591_amd as coop
    st, tr = coop.replay_to_device(state, trace)
    r = coop.Replay(st, tr, policy=policy)
    r.launch()
    torch.cuda.synchronize()
    P, T = r.num_pools, r.num_ops
    host = lambda t, dt: t.cpu().numpy().view(dt)
    state_after = {"size": host(st["size"], np.uint64), "cost": host(st["cost"], np.uint64),
                   "kind": st["kind"].cpu().numpy(), "id": host(st["id"], np.uint32),
                   "len": host(st["len"], np.uint64), "capacity": st["capacity"]}
    outs = {"block": host(r.block, np.uint64).reshape(P, T),
            "window": host(r.window, np.uint64).reshape(P, T, 2),
            "cost": host(r.cost, np.uint64).reshape(P, T),
            "free": host(r.free, np.uint64).reshape(P, T)}
    return state_after, outs, int(r.status.item())


def assert_same(state, trace, label, policy=WINDOW):
    want_state, want = oracle.replay(state, trace, threads=8, policy=policy)
    got_state, got, status = gpu_replay(state, trace, policy)
    assert status == 0, f"{label}: status {status}"
    for k in ("block", "window", "cost", "free"):
        bad = np.argwhere(got[k] != want[k])
        if len(bad):
            p, t = bad[0][:2]
            raise AssertionError(f"{label}: {k} differs at pool {p} op {t}: gpu "
                                 f"{got[k][p, t].tolist()} oracle {want[k][p, t].tolist()}")
    assert np.array_equal(got_state["len"], want_state["len"]), label
    cap = state["capacity"]
    for b in range(len(want_state["len"])):
        n = int(want_state["len"][b])
        used, rest = slice(b * cap, b * cap + n), slice(b * cap + n, (b + 1) * cap)
        for k in ("size", "cost", "kind", "id"):
            assert np.array_equal(got_state[k][used], want_state[k][used]), \
                f"{label}: pool {b}: final {k} differs"
        # unused slots stay empty pinned blocks for the search kernels
        assert (got_state["size"][rest] == 0).all() and (got_state["kind"][rest] == 2).all()


@pytest.mark.parametrize("policy", [WINDOW, GREEDY])
@pytest.mark.parametrize("k,seed", [(0, 0), (0, 1), (1, 0), (1, 2)])
def test_generated_traces(k, seed, policy):
    _announce(f"config {k} seed {seed} policy {policy}")
    state, trace = traces.make_replay(k, seed)
    assert_same(state, trace, f"config {k} seed {seed} policy {policy}", policy)


@pytest.mark.parametrize("policy", [WINDOW, GREEDY])
def test_training_replay_full_size(policy):
    """The training-replay workload the benchmark times (512 pools of 1024
    operations), whole."""
    _announce(f"training replay, policy {policy}")
    state, trace = traces.make_replay(2, 0)
    assert_same(state, trace, f"training policy {policy}", policy)


def test_greedy_worked_replays():
    """The hand-derived cases of tests/golden/greedy_examples.txt, each pool
    replayed on the GPU."""
    import os
    cases = parse_greedy_golden(os.path.join(GOLDEN, "greedy_examples.txt"))
    for case in cases:
        _announce(f"greedy worked case {case['name']}")
        cap = 16
        state = {"size": np.zeros(cap, np.uint64), "cost": np.zeros(cap, np.uint64),
                 "kind": np.full(cap, 2, np.uint8), "id": np.zeros(cap, np.uint32),
                 "len": np.array([len(case["pool"])], np.uint64), "capacity": cap}
        for j, (kd, sz, i, c) in enumerate(case["pool"]):
            state["kind"][j], state["size"][j], state["id"][j], state["cost"][j] = kd, sz, i, c
        for stp in case["steps"]:
            o = stp["op"]
            trace = {"op": np.zeros(1, np.uint8), "op_id": np.array([int(o[1])]),
                     "op_size": np.array([int(o[2]) * MiB], np.uint64),
                     "op_cost": np.array([int(o[3])], np.uint64),
                     "op_flags": np.array([1 if o[4] == "left" else 0], np.uint8)}
            new_state, got, status = gpu_replay(state, trace, GREEDY)
            assert status == 0
            e = stp["expect"]
            assert int(got["block"][0, 0]) == (U64MAX if e[0] == "none" else int(e[0])), o
            assert got["window"][0, 0].tolist() == [int(e[2]), U64MAX], o
            assert int(got["cost"][0, 0]) == int(e[3]), o
            assert int(got["free"][0, 0]) == int(e[4]) * MiB, o
            n = int(new_state["len"][0])
            blocks = [(int(new_state["kind"][j]), int(new_state["size"][j]),
                       int(new_state["id"][j])) for j in range(n)]
            assert blocks == stp["after"], (case["name"], o, blocks)
            state = new_state


def test_unknown_policy_is_rejected():
    import paper_2311_00591_amd as coop
    state, trace = traces.make_replay(0, 0)
    st, tr = coop.replay_to_device(state, trace)
    with pytest.raises(ValueError):
        coop.Replay(st, tr, policy=2)


def test_resnet_pattern_tight_budget():
    _announce("resnet pattern, tight budget")
    state, trace = traces.make_replay(1, 5, pattern="resnet", budget_frac=0.5, num_pools=32)
    assert_same(state, trace, "resnet")


def test_worked_replay():
    """The hand-derived replay of tests/golden/replay_examples.txt."""
    _announce("worked replay")
    cap = 16
    size = np.zeros(cap, np.uint64)
    kind = np.full(cap, 2, np.uint8)
    ids = np.zeros(cap, np.uint32)
    size[:3] = [4 * MiB, 10 * MiB, 2 * MiB]
    kind[:3] = [2, 0, 2]
    ids[:3] = [1, 0, 2]
    state = {"size": size, "cost": np.zeros(cap, np.uint64), "kind": kind, "id": ids,
             "len": np.array([3], np.uint64), "capacity": cap}
    trace = {"op": [0, 0, 0, 1, 0, 1, 1, 0, 0], "op_id": [10, 11, 12, 11, 13, 12, 10, 14, 15],
             "op_size": [3 * MiB, 4 * MiB, 4 * MiB, 0, 2 * MiB, 0, 0, 9 * MiB, 12 * MiB],
             "op_cost": [30, 5, 40, 0, 7, 0, 0, 1, 1], "op_flags": [1, 0, 1, 0, 0, 0, 0, 0, 1]}
    trace = {k: np.array(v) for k, v in trace.items()}
    _, got, status = gpu_replay(state, trace)
    assert status == 0
    assert got["block"][0].tolist() == [1, 3, 2, U64MAX, 4, 2, 1, 2, U64MAX]
    assert got["window"][0, 2].tolist() == [3, 4] and got["cost"][0, 2] == 5
    assert got["window"][0, 7].tolist() == [1, 3] and got["free"][0, 7] == 8 * MiB
    assert_same(state, trace, "worked replay")


def test_out_of_slots_is_reported():
    """A pool whose capacity cannot hold the next block: the allocation is
    skipped and status bit 0 is set (the oracle refuses such a replay)."""
    _announce("out of slots")
    cap = 3
    state = {"size": np.array([8 * MiB, 0, 0], np.uint64), "cost": np.zeros(3, np.uint64),
             "kind": np.array([0, 2, 2], np.uint8), "id": np.zeros(3, np.uint32),
             "len": np.array([1], np.uint64), "capacity": cap}
    trace = {"op": np.zeros(3, np.uint8), "op_id": np.array([5, 6, 7]),
             "op_size": np.array([MiB, MiB, MiB]), "op_cost": np.ones(3),
             "op_flags": np.zeros(3, np.uint8)}
    got_state, got, status = gpu_replay(state, trace)
    assert status & 1
    assert got["block"][0].tolist()[:2] == [1, 1] and got["block"][0, 2] == U64MAX
    assert int(got_state["len"][0]) == 3


@pytest.mark.parametrize("policy", [WINDOW, GREEDY])
def test_pools_too_large_for_lds_take_the_stepwise_path(policy):
    """Capacity beyond what one workgroup's LDS holds: the replay runs one
    step per operation with the batched first-fit and window kernels."""
    _announce(f"stepwise path, policy {policy}")
    state, trace = traces.make_replay(1, 7, layers=2700, num_pools=6, iterations=1,
                                      budget_frac=0.9)
    # 31 bytes of LDS per slot (sizes or byte prefixes, costs, cost
    # prefixes, ids, pinned counts, kinds): above 160 KiB
    assert state["capacity"] * 31 > 160 * 1024
    assert_same(state, trace, f"stepwise policy {policy}", policy)


@pytest.mark.parametrize("policy", [WINDOW, GREEDY])
def test_large_pools_held_in_lds(policy):
    """A capacity that still fits one workgroup's LDS but needs more than
    64 KiB of it (one pool per CU)."""
    _announce(f"large resident pools, policy {policy}")
    state, trace = traces.make_replay(1, 7, layers=2200, num_pools=6, iterations=1,
                                      budget_frac=0.9)
    assert 64 * 1024 < state["capacity"] * 31 < 150 * 1024
    assert_same(state, trace, f"large resident policy {policy}", policy)
