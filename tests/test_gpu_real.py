"""GPU search with real-valued heuristics (coop_window_search_real) equals
the CPU oracle's, bit for bit, through the C ABI: start, end, the exact
fixed-point cost (two 64-bit words) and the binary64 cost, for the five
standard workloads at full size (heuristics h = cost / staleness), the
hand-derived examples, windows longer than the staged prefixes, the
rounding of exact sums to binary64, degenerate snapshots and invalid
values."""
import os
import sys

import numpy as np
import pytest

import oracle
import workloads
from conftest import GOLDEN, parse_real_golden

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

U64MAX = (1 << 64) - 1
MiB = 1 << 20


def _threads():
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def _announce(label):
    print(f"[gpu case] real: {label}", flush=True)
    sys.stdout.flush()


def gpu_real(pools, h, workspace_fill=None):
    import paper_2311_00591_amd as coop
    size, _, kind, seg, req, roff = coop.to_device(pools, "cuda")
    ht = torch.from_numpy(np.ascontiguousarray(h, dtype=np.float64)).to("cuda")
    ws = None
    if workspace_fill is not None:
        need = coop.real_workspace_size(pools.num_blocks, pools.num_segments, pools.num_requests)
        ws = torch.full((max(need, 1),), workspace_fill, dtype=torch.uint8, device="cuda")
    r = coop.WindowSearchReal(size, ht, kind, seg, req, roff, workspace=ws)
    r.launch()
    torch.cuda.synchronize()
    out = r.out.cpu().numpy()
    return out[:, :4].view(np.uint64), out[:, 4].copy().view(np.float64), int(r.status.item())


def assert_parity(pools, h, label, workspace_fill=None):
    want, want_cost = oracle.window_search_real(pools.size, h, pools.kind, pools.seg_offsets,
                                                pools.req_sizes, pools.req_offsets,
                                                threads=_threads())
    got, got_cost, status = gpu_real(pools, h, workspace_fill)
    assert status == 0, f"{label}: status {status}"
    bad = np.flatnonzero((got != want).any(axis=1) |
                         (got_cost.view(np.uint64) != want_cost.view(np.uint64)))
    if len(bad):
        q = int(bad[0])
        raise AssertionError(f"{label}: {len(bad)} of {len(want)} requests differ; first q={q} "
                             f"S={int(pools.req_sizes[q])} gpu={got[q].tolist()} "
                             f"{got_cost[q]!r} oracle={want[q].tolist()} {want_cost[q]!r}")
    return got


@pytest.mark.parametrize("k", [0, 1, 2, 3, 4])
def test_standard_workload_full_size(k):
    _announce(f"workload {k} full size")
    pools = workloads.make_config(k, 0)
    got = assert_parity(pools, workloads.real_costs(pools), f"workload {k}")
    assert (got[:, 0] != np.uint64(U64MAX)).any()


@pytest.mark.parametrize("k,seed,overrides", [
    (0, 3, {}),
    (1, 3, {"num_segments": 100}),
    (2, 3, {"num_segments": 5}),
    (3, 3, {"num_segments": 300}),
    (4, 3, {"blocks": (1 << 20, 1 << 20), "requests_per_segment": 64}),
])
def test_other_seeds(k, seed, overrides):
    _announce(f"workload {k} seed {seed} {overrides}")
    pools = workloads.make_config(k, seed, **overrides)
    assert_parity(pools, workloads.real_costs(pools, seed), f"workload {k} seed {seed}",
                  workspace_fill=0xA5)


def test_worked_examples():
    exs = parse_real_golden(os.path.join(GOLDEN, "real_examples.txt"))
    snaps, reqs, hs = [], [], []
    for e in exs:
        snaps.append(([s for _, s, _ in e["blocks"]], [0] * len(e["blocks"]),
                      [k for k, _, _ in e["blocks"]]))
        reqs.append([S for S, _ in e["reqs"]])
        hs += [x for _, _, x in e["blocks"]]
    pools = workloads.from_lists(snaps, reqs)
    _announce("worked examples")
    got, cost, status = gpu_real(pools, np.array(hs))
    assert status == 0
    q = 0
    for e in exs:
        for S, want in e["reqs"]:
            if want is None:
                assert got[q].tolist() == [U64MAX] * 4 and cost[q] == np.inf, (e["name"], S)
            else:
                start, end, hi, lo = want
                assert got[q].tolist() == [start, end, lo, hi], (e["name"], S, got[q])
            q += 1
    assert_parity(pools, np.array(hs), "worked examples")


def test_windows_longer_than_the_staged_prefixes():
    """Runs of tens of thousands of small blocks and requests needing
    thousands of them: the ends lie past the 4096 staged prefixes, so the
    bisection and the walk continue in global memory."""
    rng = np.random.default_rng(5)
    snaps, reqs, hs = [], [], []
    for n in (30000, 9000, 4097, 4095, 2049):
        size = rng.integers(1, 4, n) * 512
        kind = np.where(rng.random(n) < 0.0004, 2, 1)
        snaps.append((size, rng.integers(1, 100, n), kind))
        tot = int(size.sum())
        reqs.append([tot // 3, tot // 7, 512 * 5000, 512 * 2100, 512 * 4000, 1, tot])
        hs.append(rng.integers(1, 10**6, n) / rng.integers(1, 3000, n))
    pools = workloads.from_lists(snaps, reqs)
    _announce("long windows")
    h = np.concatenate(hs)
    h[pools.kind != 1] = 0.0
    assert_parity(pools, h, "long windows")


def test_merges_stop_at_the_first_pinned_block_after_the_chunk():
    """Pinned blocks from none to dense, so that the first one after a
    chunk's 2048 starts lies anywhere in the 512 staged blocks that follow
    (the merges stop at the end key that takes it in), with 1, 4 and 16
    requests per snapshot (one or two merges a lane)."""
    rng = np.random.default_rng(29)
    snaps, reqs, hs = [], [], []
    for p_pin in (0.0, 0.002, 0.02, 0.2):
        for nreq in (1, 4, 16):
            n = 3 * 2048 + 600
            size = rng.integers(1, 64, n) * 512
            kind = np.where(rng.random(n) < p_pin, 2, 1)
            kind[rng.random(n) < 0.1] = 0
            snaps.append((size, rng.integers(0, 1000, n), kind))
            base = [1, 4096, 3 * 4096 + 1, 40 * 4096, 300 * 4096, 5000 * 4096, 1 << 40]
            reqs.append([int(base[i % len(base)] + rng.integers(0, 4096)) for i in range(nreq)])
            hs.append(rng.integers(1, 10**6, n) / rng.integers(1, 3000, n))
    # pinned blocks right at and after the first chunk's end
    n = 2 * 2048 + 600
    size = np.full(n, 4096)
    kind = np.ones(n, dtype=np.int64)
    kind[[2047, 2048, 2049, 2300]] = 2
    snaps.append((size, np.full(n, 7), kind))
    reqs.append([1, 4096, 8192, 3 * 4096, 100 * 4096])
    hs.append(np.full(n, 0.5))
    pools = workloads.from_lists(snaps, reqs)
    _announce("merges stop at the first pinned block after the chunk")
    h = np.concatenate(hs).astype(np.float64)
    h[pools.kind != 1] = 0.0
    assert_parity(pools, h, "first pinned block after the chunk")


def test_exact_sums_round_to_binary64():
    """Exact sums with more than 53 significant bits: ties to even, both
    ways, and plain rounding, each in a snapshot of its own."""
    cases = [[2.0**53, 1.0], [2.0**53, 3.0], [2.0**53, 1.0, 2.0**-64 * 0 + 2.0**-60],
             [2.0**60, 2.0**-3, 2.0**-12], [2.0**-12 + 2.0**-64, 2.0**40],
             [1.0 / 3, 1.0 / 7, 1.0 / 11], [2.0**63, 2.0**62, 2.0**61]]
    snaps, reqs, hs = [], [], []
    for c in cases:
        snaps.append(([MiB] * len(c), [0] * len(c), [1] * len(c)))
        reqs.append([len(c) * MiB])
        hs += c
    pools = workloads.from_lists(snaps, reqs)
    _announce("rounding of exact sums")
    got = assert_parity(pools, np.array(hs), "rounding")
    assert (got[:, 0] == 0).all()


def test_degenerate_snapshots():
    snaps = [([], [], []), ([MiB], [0], [2]), ([MiB, MiB], [0, 0], [2, 2]),
             ([MiB], [0], [0]), ([MiB, 2 * MiB], [0, 0], [1, 1])]
    reqs = [[1, 0], [1], [MiB, 0], [MiB, MiB + 1], [0, 1, 3 * MiB, 3 * MiB + 1]]
    pools = workloads.from_lists(snaps, reqs)
    h = np.array([np.nan, np.nan, -1.0, 5.0, 0.25, 0.5])  # off evictable blocks: ignored
    _announce("degenerate snapshots")
    got, cost, status = gpu_real(pools, h)
    assert status == 0
    assert_parity(pools, h, "degenerate")
    assert got[0].tolist() == [U64MAX] * 4 and got[1].tolist() == [0] * 4


@pytest.mark.parametrize("bad", [np.nan, -1.0, np.inf, 2.0**64])
def test_invalid_values_set_the_status_bit(bad):
    pools = workloads.from_lists([([MiB, MiB], [0, 0], [1, 1])], [[MiB]])
    _announce(f"invalid h {bad}")
    _, _, status = gpu_real(pools, np.array([1.0, bad]))
    assert status & 1
    # -0.0 is a valid zero, and the status word is cleared by every call
    _, _, status = gpu_real(pools, np.array([1.0, -0.0]))
    assert status == 0


def test_unaligned_inputs():
    """Inputs that start 8 bytes (sizes, h) and 1 byte (kinds) past an
    aligned address take the single-load path of the prefix kernel."""
    import paper_2311_00591_amd as coop
    pools = workloads.make_config(1, 4, num_segments=8)
    h = workloads.real_costs(pools, 4)
    _announce("unaligned inputs")

    def shifted(a, dt):
        t = torch.zeros(len(a) + 1, dtype=dt, device="cuda")
        t[1:] = torch.from_numpy(np.ascontiguousarray(a)).to("cuda")
        return t[1:]

    size = shifted(pools.size.view(np.int64), torch.int64)
    ht = shifted(h, torch.float64)
    kind = shifted(pools.kind, torch.uint8)
    assert size.data_ptr() % 16 == 8 and kind.data_ptr() % 8 == 1
    _, _, _, seg, req, roff = coop.to_device(pools, "cuda")
    r = coop.WindowSearchReal(size, ht, kind, seg, req, roff)
    r.launch()
    torch.cuda.synchronize()
    want, want_cost = oracle.window_search_real(pools.size, h, pools.kind, pools.seg_offsets,
                                                pools.req_sizes, pools.req_offsets, threads=4)
    out = r.out.cpu().numpy()
    assert int(r.status.item()) == 0
    assert np.array_equal(out[:, :4].view(np.uint64), want)
    assert np.array_equal(out[:, 4].copy().view(np.uint64), want_cost.view(np.uint64))
