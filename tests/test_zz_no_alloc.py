"""coop_window_search_static (the search whose cross-workgroup state lives
in the library's static device array) gives the same results as
coop_window_search, call after call, and allocates no device memory."""
import sys

import numpy as np
import pytest

import oracle
import workloads

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def _announce(label):
    print(f"[gpu case] {label}", flush=True)
    sys.stdout.flush()


def test_static_matches_the_workspace_entry_point_twice_in_a_row():
    import paper_2311_00591_amd as coop
    big = workloads.make_config(3, 7, num_segments=600)
    small = workloads.make_config(2, 8, num_segments=3, blocks=(20000, 20000),
                                  requests_per_segment=5)
    assert small.num_blocks < big.num_blocks and small.num_requests < big.num_requests
    _announce(f"static scratch: {big.num_requests} then {small.num_requests} requests")
    batches = []
    for pools in (big, small):
        dev = coop.to_device(pools, "cuda")
        ref = coop.window_search(*dev)  # workspace entry point (loads the library's code)
        out = torch.empty((pools.num_requests, 3), dtype=torch.int64, device="cuda")
        batches.append((pools, dev, ref, out))
    torch.cuda.synchronize()
    free0 = torch.cuda.mem_get_info()[0]
    for pools, dev, _, out in batches:
        coop.window_search_static(*dev, out=out)
    torch.cuda.synchronize()
    assert torch.cuda.mem_get_info()[0] == free0, "the static entry point allocated device memory"
    for pools, dev, ref, out in batches:
        got = out.cpu().numpy().view(np.uint64)
        assert np.array_equal(got, ref.cpu().numpy().view(np.uint64))
        assert np.array_equal(got, oracle.window_search(*pools.arrays(), threads=8))


def test_static_scratch_plan_with_a_reduced_partial_budget():
    """A batch whose usual workspace exceeds the static array: the static
    entry point plans with fewer partial slots and still matches."""
    import paper_2311_00591_amd as coop
    pools = workloads.make_config(3, 9)
    assert coop.workspace_size(pools.num_blocks, pools.num_segments,
                               pools.num_requests) > coop.static_capacity()
    _announce(f"static scratch, reduced budget: {pools.num_requests} requests")
    dev = coop.to_device(pools, "cuda")
    got = coop.window_search_static(*dev)
    torch.cuda.synchronize()
    want = oracle.window_search(*pools.arrays(), threads=16)
    assert np.array_equal(got.cpu().numpy().view(np.uint64), want)


def _long_runs(seed, tiles):
    """One pinned-free run of about `tiles` tiles between pinned ends, with
    requests up to the whole run: windows go to the second kernel."""
    rng = np.random.default_rng(seed)
    n = tiles * 4096 + int(rng.integers(0, 4096))
    size = (rng.integers(1, 64, size=n) * 512).astype(np.uint64)
    kind = np.where(rng.random(n) < 0.2, 0, 1).astype(np.uint8)
    kind[0] = kind[-1] = 2
    cost = rng.integers(0, 10**6, size=n).astype(np.uint64)
    run = int(size[1:-1].sum())
    return workloads.from_lists([(size, cost, kind)], [[run, run // 3, run // 40, run + 1]])


def test_static_long_windows_twice_in_a_row():
    """Windows left to the second kernel, whose deferred list and entry
    claims live in the static array too: two calls in a row, the second
    smaller, each equal to the workspace entry point's results."""
    import paper_2311_00591_amd as coop
    batches = []
    for seed, tiles in ((41, 30), (42, 12)):
        pools = _long_runs(seed, tiles)
        dev = coop.to_device(pools, "cuda")
        ref = coop.window_search(*dev)
        out = torch.empty((pools.num_requests, 3), dtype=torch.int64, device="cuda")
        batches.append((pools, dev, ref, out))
    _announce(f"static scratch, long windows: {batches[0][0].num_blocks} then "
              f"{batches[1][0].num_blocks} blocks")
    torch.cuda.synchronize()
    for pools, dev, _, out in batches:
        coop.window_search_static(*dev, out=out)
    torch.cuda.synchronize()
    for pools, dev, ref, out in batches:
        got = out.cpu().numpy().view(np.uint64)
        assert np.array_equal(got, ref.cpu().numpy().view(np.uint64))
        assert np.array_equal(got, oracle.window_search(*pools.arrays(), threads=8))
