"""Every entry point captured into a HIP graph (through torch.cuda.graph) and
replayed several times, with eager calls and host synchronisations between
the replays and the inputs rewritten in place between them: every replay
must match the oracle (or, where the inputs do not change, the eager call)
bit for bit.  The window search carries tags across workgroups; a replay
reuses the recorded arguments, so these tests check that its tags still
change from one replay to the next and never meet an eager call's.
"""
import os
import sys

import numpy as np
import pytest

import oracle
import workloads
from workloads import traces

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

WINDOW, GREEDY = 0, 1


def _threads():
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def _announce(label):
    print(f"[gpu case] graph: {label}", flush=True)
    sys.stdout.flush()


def _u64(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.uint64).view(np.int64))


def _variant(pools, seed):
    """Same shapes and offsets, other costs, kinds and request sizes."""
    rng = np.random.default_rng(seed)
    return workloads.Pools(pools.size.copy(), rng.permutation(pools.cost),
                           np.roll(pools.kind, 1 + int(rng.integers(0, 7))).copy(),
                           pools.seg_offsets.copy(), rng.permutation(pools.req_sizes),
                           pools.req_offsets.copy())


def _load(dev, pools):
    """Writes a batch's contents into the static device tensors in place."""
    size, cost, kind, seg, req, roff = dev
    size.copy_(_u64(pools.size))
    cost.copy_(_u64(pools.cost))
    kind.copy_(torch.from_numpy(np.ascontiguousarray(pools.kind, dtype=np.uint8)))
    seg.copy_(_u64(pools.seg_offsets))
    req.copy_(_u64(pools.req_sizes))
    roff.copy_(_u64(pools.req_offsets))


def _same(got, want, label):
    got = got.cpu().numpy().view(np.uint64)
    bad = np.flatnonzero((got != want).reshape(len(want), -1).any(axis=1))
    assert len(bad) == 0, f"{label}: {len(bad)} of {len(want)} differ, first {int(bad[0])}"


def _capture(fn):
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        fn()
    torch.cuda.synchronize()
    return g


def _long_run_batch():
    """Two snapshots, each one pinned-free run of 24 tiles between pinned
    ends, with requests up to the whole run: windows far past the staged
    regions, left to the second kernel, whose workgroups claim deferred
    entries through a tagged word that each replay must restart."""
    rng = np.random.default_rng(31)
    snaps, reqs = [], []
    for _ in range(2):
        n = 24 * 4096 + int(rng.integers(0, 4096))
        size = (rng.integers(1, 64, size=n) * 512).astype(np.uint64)
        kind = np.where(rng.random(n) < 0.2, 0, 1).astype(np.uint8)
        kind[0] = kind[-1] = 2
        cost = rng.integers(0, 10**6, size=n).astype(np.uint64)
        run = int(size[1:-1].sum())
        snaps.append((size, cost, kind))
        reqs.append([run, run // 2, run // 5, run // 50, 1 << 20, run + 1])
    return workloads.from_lists(snaps, reqs)


@pytest.mark.parametrize("case", ["tickets", "queue", "long"])
def test_window_search_replays(case):
    import paper_2311_00591_amd as coop
    if case == "tickets":
        a = workloads.make_config(0, 3)
    elif case == "long":
        a = _long_run_batch()
    else:
        a = workloads.make_config(3, 5, num_segments=1200)
    info = coop.plan_info(a.num_blocks, a.num_segments, a.num_requests)
    if case == "queue":
        assert info["chunks_max"] > info["workgroups"], info
    else:
        assert info["workgroups"] > 1, info
    b = _variant(a, 11)
    _announce(f"window search, {case}, {a.num_blocks} blocks {a.num_requests} requests")
    want_a = oracle.window_search(*a.arrays(), threads=_threads())
    want_b = oracle.window_search(*b.arrays(), threads=_threads())
    dev_a = coop.to_device(a, "cuda")
    dev_b = coop.to_device(b, "cuda")
    ws_bytes = coop.workspace_size(a.num_blocks, a.num_segments, a.num_requests)
    workspace = torch.full((ws_bytes,), 0x5a, dtype=torch.uint8, device="cuda")
    # two prepared calls on one workspace: one to capture, one run eagerly
    cap_a = coop.WindowSearch(*dev_a, workspace=workspace)
    cap_b = coop.WindowSearch(*dev_b, workspace=workspace)
    eager = coop.WindowSearch(*coop.to_device(b, "cuda"), workspace=workspace)
    _same(cap_a().clone(), want_a, "eager before capture")
    g_a = _capture(cap_a.launch)
    g_b = _capture(cap_b.launch)
    for r in range(3):
        cap_a.out.fill_(-1)
        g_a.replay()
        torch.cuda.synchronize()
        _same(cap_a.out, want_a, f"replay {r} of graph a")
        _same(eager().clone(), want_b, f"eager call after replay {r}")
        g_b.replay()
        g_a.replay()
        torch.cuda.synchronize()
        _same(cap_b.out, want_b, f"replay {r} of graph b")
        _same(cap_a.out, want_a, f"second replay {r} of graph a")
    # inputs rewritten in place: the replay reads what the buffers hold now
    _load(dev_a, b)
    g_a.replay()
    torch.cuda.synchronize()
    _same(cap_a.out, want_b, "graph a replayed on the other batch")
    _load(dev_a, a)
    g_a.replay()
    torch.cuda.synchronize()
    _same(cap_a.out, want_a, "graph a replayed on its own batch again")


def test_first_fit_replays():
    import paper_2311_00591_amd as coop
    a = workloads.make_config(1, 4, num_segments=256)
    b = _variant(a, 12)
    _announce(f"first fit, {a.num_blocks} blocks {a.num_requests} requests")
    want = [oracle.first_fit(p.size, p.kind, p.seg_offsets, p.req_sizes, p.req_offsets,
                             threads=_threads()) for p in (a, b)]
    dev = coop.to_device(a, "cuda")
    size, _, kind, seg, req, roff = dev
    ff = coop.FirstFit(size, kind, seg, req, roff)
    ff.launch()
    torch.cuda.synchronize()
    _same(ff.out, want[0], "eager first fit")
    g = _capture(ff.launch)
    for r in range(4):
        _load(dev, (a, b)[r % 2])
        ff.out.fill_(-1)
        g.replay()
        torch.cuda.synchronize()
        _same(ff.out, want[r % 2], f"first fit replay {r}")


def test_real_search_replays():
    import paper_2311_00591_amd as coop
    a = workloads.make_config(1, 6, num_segments=256)
    b = _variant(a, 13)
    _announce(f"real search, {a.num_blocks} blocks {a.num_requests} requests")
    h = [workloads.real_costs(p, seed=s) for p, s in ((a, 1), (b, 2))]
    want = [oracle.window_search_real(p.size, hh, p.kind, p.seg_offsets, p.req_sizes,
                                      p.req_offsets, threads=_threads())
            for p, hh in zip((a, b), h)]
    dev = coop.to_device(a, "cuda")
    size, _, kind, seg, req, roff = dev
    ht = torch.from_numpy(np.ascontiguousarray(h[0], dtype=np.float64)).to("cuda")
    rs = coop.WindowSearchReal(size, ht, kind, seg, req, roff)
    g = None
    for r in range(5):
        k = r % 2
        _load(dev, (a, b)[k])
        ht.copy_(torch.from_numpy(np.ascontiguousarray(h[k], dtype=np.float64)))
        rs.out.fill_(-1)
        if r == 0:
            rs.launch()     # eager first, then captured
        else:
            if g is None:
                g = _capture(rs.launch)
            g.replay()
        torch.cuda.synchronize()
        out = rs.out.cpu().numpy()
        wk, wc = want[k]
        assert int(rs.status.item()) == 0, f"real replay {r}: status"
        assert np.array_equal(out[:, :4].view(np.uint64), wk), f"real replay {r}: windows"
        assert np.array_equal(out[:, 4].copy().view(np.uint64), wc.view(np.uint64)), \
            f"real replay {r}: costs"


def _replay_case(k, seed, ops, **overrides):
    state, trace = traces.make_replay(k, seed, **overrides)
    T = trace["num_ops"]
    if ops < T:
        P = len(state["len"])
        trace = {key: (v.reshape(P, T)[:, :ops].copy().reshape(-1) if key != "num_ops" else ops)
                 for key, v in trace.items()}
    return state, trace


@pytest.mark.parametrize("path", ["resident", "stepwise"])
@pytest.mark.parametrize("policy", [WINDOW, GREEDY])
def test_replay_replays(path, policy):
    """The replay updates its pools in place: the state is restored eagerly
    before each graph replay, and every replay must redo the same steps."""
    import paper_2311_00591_amd as coop
    if path == "resident":
        state, trace = _replay_case(1, 3, 10 ** 9, num_pools=8)
    else:
        # pools too large for LDS, a short prefix of the trace
        state, trace = _replay_case(1, 7, 48, layers=2700, num_pools=3, budget_frac=0.3)
        assert state["capacity"] * 31 > 160 * 1024
    _announce(f"replay {path}, policy {policy}, {len(state['len'])} pools "
              f"{trace['num_ops']} ops capacity {state['capacity']}")
    want_state, want = oracle.replay(state, trace, threads=_threads(), policy=policy)
    st, tr = coop.replay_to_device(state, trace)
    initial = {key: v.clone() for key, v in st.items() if key != "capacity"}
    rp = coop.Replay(st, tr, policy=policy)
    P, T = rp.num_pools, rp.num_ops

    def restore():
        for key, v in initial.items():
            st[key].copy_(v)
        for t in (rp.block, rp.window, rp.cost, rp.free):
            t.fill_(-1)

    def check(label):
        torch.cuda.synchronize()
        assert int(rp.status.item()) == 0, f"{label}: status {int(rp.status.item())}"
        got = {"block": rp.block.cpu().numpy().view(np.uint64).reshape(P, T),
               "window": rp.window.cpu().numpy().view(np.uint64).reshape(P, T, 2),
               "cost": rp.cost.cpu().numpy().view(np.uint64).reshape(P, T),
               "free": rp.free.cpu().numpy().view(np.uint64).reshape(P, T)}
        for key in got:
            assert np.array_equal(got[key], want[key]), f"{label}: {key} differs"
        assert np.array_equal(st["len"].cpu().numpy().view(np.uint64), want_state["len"]), label

    restore()
    rp.launch()
    check("eager replay")
    restore()
    torch.cuda.synchronize()
    g = _capture(rp.launch)
    for r in range(3):
        restore()
        g.replay()
        check(f"graph replay {r}")
        restore()
        rp.launch()
        check(f"eager call after graph replay {r}")
