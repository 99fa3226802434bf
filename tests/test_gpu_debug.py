"""The debug checks (COOP_DEBUG=1 in the environment): a batch that breaks a
rule living in device memory is rejected on the host before anything is
launched, and valid batches give the same results as without the checks.

Broken batches are only ever passed with the checks on: without them such a
batch would reach the kernels.
"""
import os
import sys

import numpy as np
import pytest

import oracle
import workloads

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

INVALID, OVERFLOW = -1, -4


def _threads():
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def _announce(label):
    print(f"[gpu case] debug checks: {label}", flush=True)
    sys.stdout.flush()


@pytest.fixture
def checks(monkeypatch):
    monkeypatch.setenv("COOP_DEBUG", "1")


def _calls(pools):
    """The three checked entry points on one batch, each returning its
    output tensor (already launched); h = the real-valued costs."""
    import paper_2311_00591_amd as coop
    size, cost, kind, seg, req, roff = coop.to_device(pools, "cuda")
    h = torch.from_numpy(workloads.real_costs(pools, seed=3)).to("cuda")
    ws = coop.WindowSearch(size, cost, kind, seg, req, roff)
    ff = coop.FirstFit(size, kind, seg, req, roff)
    rs = coop.WindowSearchReal(size, h, kind, seg, req, roff)
    for o in (ws.out, ff.out, rs.out):
        o.fill_(7)
    return {"window": ws, "first_fit": ff, "real": rs}


def test_valid_batches_give_the_same_results(checks):
    for k, over in ((0, {}), (3, {"num_segments": 64})):
        pools = workloads.make_config(k, 2, **over)
        _announce(f"valid batch, workload {k}")
        c = _calls(pools)
        c["window"].launch()
        c["first_fit"].launch()
        c["real"].launch()
        torch.cuda.synchronize()
        a = pools.arrays()
        want = oracle.window_search(*a, threads=_threads())
        assert np.array_equal(c["window"].out.cpu().numpy().view(np.uint64), want)
        want = oracle.first_fit(pools.size, pools.kind, pools.seg_offsets, pools.req_sizes,
                                pools.req_offsets, threads=_threads())
        assert np.array_equal(c["first_fit"].out.cpu().numpy().view(np.uint64), want)
        want, want_cost = oracle.window_search_real(
            pools.size, workloads.real_costs(pools, seed=3), pools.kind, pools.seg_offsets,
            pools.req_sizes, pools.req_offsets, threads=_threads())
        out = c["real"].out.cpu().numpy()
        assert int(c["real"].status.item()) == 0
        assert np.array_equal(out[:, :4].view(np.uint64), want)
        assert np.array_equal(out[:, 4].copy().view(np.uint64), want_cost.view(np.uint64))


def _broken(pools, which):
    seg, roff = pools.seg_offsets.copy(), pools.req_offsets.copy()
    if which == "segment offsets decrease":
        seg[2], seg[3] = seg[3], seg[2]
    elif which == "first segment offset not zero":
        seg[0] = 1
    elif which == "last segment offset not the block count":
        seg[-1] -= 1
    elif which == "request offsets decrease":
        roff[1], roff[2] = roff[2], roff[1]
    elif which == "last request offset not the request count":
        roff[-1] += 1
    return workloads.Pools(pools.size, pools.cost, pools.kind, seg, pools.req_sizes, roff)


@pytest.mark.parametrize("which", ["segment offsets decrease", "first segment offset not zero",
                                   "last segment offset not the block count",
                                   "request offsets decrease",
                                   "last request offset not the request count"])
def test_broken_offsets_are_rejected_before_launch(checks, which):
    import paper_2311_00591_amd as coop
    base = workloads.make_config(3, 4, num_segments=16)
    pools = _broken(base, which)
    assert pools.seg_offsets[3] != pools.seg_offsets[2] or "request" in which
    if which == "request offsets decrease":
        assert pools.req_offsets[1] > pools.req_offsets[2]
    _announce(which)
    c = _calls(pools)
    for name, call in c.items():
        with pytest.raises(coop.CoopError) as e:
            call.launch()
        assert e.value.status == INVALID, (name, e.value.status)
    torch.cuda.synchronize()
    for name, call in c.items():
        assert bool((call.out == 7).all()), f"{name}: output written"


def test_run_totals_past_64_bits_are_rejected(checks):
    import paper_2311_00591_amd as coop
    E, P = workloads.EVICTABLE, workloads.PINNED
    big = 1 << 63
    # bytes of one run overflow: every summing entry point rejects it
    bytes_over = workloads.from_lists([([8, big, big], [1, 1, 1], [E, E, E])], [[16]])
    _announce("run byte total past 2^64")
    c = _calls(bytes_over)
    for name in ("window", "real"):
        with pytest.raises(coop.CoopError) as e:
            c[name].launch()
        assert e.value.status == OVERFLOW, name
    # first fit sums nothing
    c["first_fit"].launch()
    torch.cuda.synchronize()
    assert c["first_fit"].out.cpu().numpy().view(np.uint64).tolist() == [2**64 - 1]
    # evictable costs of one run overflow: the integer search rejects it
    cost_over = workloads.from_lists([([512, 512, 512], [big, 5, big], [E, E, E])], [[1024]])
    _announce("run cost total past 2^64")
    c = _calls(cost_over)
    with pytest.raises(coop.CoopError) as e:
        c["window"].launch()
    assert e.value.status == OVERFLOW
    torch.cuda.synchronize()
    assert bool((c["window"].out == 7).all())
    # the same totals split by a pinned block fit: accepted, and exact
    split = workloads.from_lists([([8, big, 512, big, 512], [1, big, 0, big, 3],
                                   [E, E, P, E, E])], [[big + 8, 4, 2**64 - 1]])
    _announce("large totals split by a pinned block")
    c = _calls(split)
    c["window"].launch()
    torch.cuda.synchronize()
    want = oracle.window_search(*split.arrays())
    assert np.array_equal(c["window"].out.cpu().numpy().view(np.uint64), want)


def test_captured_calls_skip_the_checks(checks):
    """A stream that is capturing cannot be synchronised: the captured call
    records the search only, and its replays still match the oracle."""
    import paper_2311_00591_amd as coop
    pools = workloads.make_config(0, 5)
    _announce("capture with the checks requested")
    c = _calls(pools)
    ws = c["window"]
    ws.launch()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        ws.launch()
    want = oracle.window_search(*pools.arrays(), threads=_threads())
    for _ in range(2):
        ws.out.fill_(7)
        g.replay()
        torch.cuda.synchronize()
        assert np.array_equal(ws.out.cpu().numpy().view(np.uint64), want)
    assert coop.load_library() is not None
