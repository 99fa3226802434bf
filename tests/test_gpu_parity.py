"""GPU results equal the CPU oracle's, bit for bit, through the C ABI.

Every comparison is element by element on (start, end, cost); costs are
integers, so there is no tolerance.  The standard workloads run at their
full sizes in the same launch configuration the benchmark times, plus
adversarial pools aimed at the tile edges, the halo, the streaming pass for
runs longer than the staged region, the cross-workgroup combine and the
strided tile assignment.
"""
import os
import sys

import numpy as np
import pytest

import oracle
import workloads
from checks import check_results

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

TILE = 4096
U64MAX = (1 << 64) - 1


def _threads():
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def gpu_search(pools, workspace_fill=None):
    import paper_2311_00591_amd as coop
    dev = coop.to_device(pools, "cuda")
    ws = None
    if workspace_fill is not None:
        need = coop.workspace_size(pools.num_blocks, pools.num_segments, pools.num_requests)
        ws = torch.full((max(need, 1),), workspace_fill, dtype=torch.uint8, device="cuda")
    out = coop.window_search(*dev, workspace=ws)
    torch.cuda.synchronize()
    return out.cpu().numpy().view(np.uint64)


def assert_parity(pools, got, label):
    want = oracle.window_search(*pools.arrays(), threads=_threads())
    bad = np.flatnonzero((got != want).any(axis=1))
    if len(bad):
        q = int(bad[0])
        raise AssertionError(f"{label}: {len(bad)} of {len(want)} requests differ; first q={q} "
                             f"S={int(pools.req_sizes[q])} gpu={got[q].tolist()} "
                             f"oracle={want[q].tolist()}")


def _announce(label):
    print(f"[gpu case] {label}", flush=True)
    sys.stdout.flush()


@pytest.mark.parametrize("seed", [0, 1, 2])
@pytest.mark.parametrize("k", [0, 1, 2, 3, 4])
def test_standard_workload_full_size(k, seed):
    """Every request of each standard workload, at its full size, for three
    seeds, in the launch configuration the benchmark times."""
    _announce(f"workload {k} full size seed {seed}")
    pools = workloads.make_config(k, seed)
    got = gpu_search(pools)
    assert_parity(pools, got, f"workload {k} seed {seed}")
    if k != 4:
        check_results(pools, got)
    else:
        check_results(pools, got, sample=range(0, pools.num_requests, 37))


def _pools(snaps, reqs):
    return workloads.from_lists(snaps, reqs)


def test_tile_edges_and_ragged_tails():
    """Snapshots of lengths around multiples of the tile, pinned blocks at
    and around every tile edge, requests from tiny to whole-run."""
    _announce("tile edges")
    rng = np.random.default_rng(11)
    snaps, reqs = [], []
    for n in [1, 2, 63, 64, 65, TILE - 1, TILE, TILE + 1, 2 * TILE - 1, 2 * TILE,
              2 * TILE + 3, 3 * TILE + 777]:
        size = (rng.integers(1, 64, size=n) * 512).astype(np.uint64)
        kind = rng.choice([0, 1, 1, 1, 1, 1, 1, 2], size=n).astype(np.uint8)
        for e in range(TILE, n + 2, TILE):
            for d in (-2, -1, 0, 1):
                if 0 <= e + d < n and rng.random() < 0.5:
                    kind[e + d] = 2
        cost = rng.integers(0, 1000, size=n).astype(np.uint64)
        snaps.append((size, cost, kind))
        reqs.append([0, 1, 512, 4096, 65536, 1 << 20, 1 << 22, 1 << 24, U64MAX])
    pools = _pools(snaps, reqs)
    assert_parity(pools, gpu_search(pools), "tile edges")


def test_merge_stops_at_the_halos_first_pinned_block():
    """Tiles whose halo holds its first pinned block at offsets 0, 1, 5,
    128, 255 or nowhere; 16 requests per snapshot (one wavefront per
    request: the merge leaves out the end keys past that block), 4 and 1
    (wider slices: it keeps them); equal sizes and costs give many equal
    windows across the tile ends."""
    _announce("merge end at the halo's first pinned block")
    rng = np.random.default_rng(23)
    snaps, reqs = [], []
    for off in (0, 1, 5, 128, 255, None):
        for nreq, equal in ((16, False), (16, True), (4, False), (1, False)):
            n = 2 * TILE + 300
            if equal:
                size = np.full(n, 4096, dtype=np.uint64)
                cost = np.full(n, 7, dtype=np.uint64)
                kind = np.ones(n, dtype=np.uint8)
            else:
                size = (rng.integers(1, 64, size=n) * 512).astype(np.uint64)
                cost = rng.integers(0, 1000, size=n).astype(np.uint64)
                kind = rng.choice([0, 1, 1, 1, 1, 1, 1, 1], size=n).astype(np.uint8)
                kind[rng.random(n) < 0.01] = 2
            for e in (TILE, 2 * TILE):  # each tile's halo: pinned only from off on
                kind[e:e + 256][kind[e:e + 256] >= 2] = 1
                if off is not None and e + off < n:
                    kind[e + off] = 3
            snaps.append((size, cost, kind))
            base = [1, 4096, 3 * 4096 + 1, 40 * 4096, 300 * 4096, 5000 * 4096, 1 << 40]
            reqs.append([int(base[i % len(base)] + rng.integers(0, 4096)) for i in range(nreq)])
    pools = _pools(snaps, reqs)
    assert_parity(pools, gpu_search(pools), "halo's first pinned block")


def _clustered_kinds(rng, n, pinned_mean, open_mean):
    """Alternating pinned and open stretches of geometric lengths; inside an
    open stretch a fifth of the blocks are free."""
    kind = np.empty(n, dtype=np.uint8)
    i, pinned = 0, bool(rng.random() < 0.5)
    while i < n:
        m = int(rng.geometric(1.0 / (pinned_mean if pinned else open_mean)))
        kind[i:i + m] = 2 if pinned else np.where(rng.random(min(m, n - i)) < 0.2, 0, 1)
        i += m
        pinned = not pinned
    return kind


def test_clustered_pinned_stretches():
    """Clustered pinned stretches of mean length 1.2 to 40 between open runs
    of mean length 2 to 30, stretches across tile edges and the start of the
    halo, snapshots almost all pinned, long open runs between dense pinned
    clusters (windows that leave the staged region), and costs from a tiny
    range so that ties decide by the start."""
    _announce("clustered pinned stretches")
    rng = np.random.default_rng(19)
    snaps, reqs = [], []
    for s in range(36):
        n = int(rng.integers(1, 5 * TILE + 300))
        pm, om = [(2, 6), (3.3, 7.8), (8, 4), (40, 10), (1.2, 30), (2, 2)][s % 6]
        kind = _clustered_kinds(rng, n, pm, om)
        if s % 4 == 0:  # pinned across tile edges and the start of the halo
            for e in range(TILE, n, TILE):
                kind[max(0, e - 5):min(n, e + 7)] = 2
        if s % 9 == 4:  # almost all pinned
            kind[:] = 2
            kind[rng.integers(0, n, size=max(1, n // 50))] = 1
        if s % 7 == 3 and n > 3 * TILE:  # a long open run between dense clusters
            a = int(rng.integers(0, n - 2 * TILE))
            kind[a:a + 2 * TILE] = np.where(rng.random(2 * TILE) < 0.2, 0, 1)
        size = (rng.integers(1, 64, size=n) * 512).astype(np.uint64)
        hi = 4 if s % 2 else 10**6
        cost = rng.integers(0, hi, size=n).astype(np.uint64)
        snaps.append((size, cost, kind))
        tot = int(size[kind < 2].sum())
        mean = int(size.mean())
        reqs.append([1, 512, mean, 4 * mean, 50 * mean, 3000 * mean, tot // 3, tot,
                     int(rng.integers(1, max(2, tot)))])
    pools = _pools(snaps, reqs)
    got = gpu_search(pools)
    assert_parity(pools, got, "clustered pinned stretches")
    check_results(pools, got)


def test_runs_longer_than_the_staged_region():
    """One pin-free run far longer than tile + halo: windows of thousands of
    blocks cross many tiles and are finished by the streaming pass."""
    _announce("long runs")
    rng = np.random.default_rng(12)
    n = 40 * TILE + 123
    size = (rng.integers(1, 16, size=n) * 512).astype(np.uint64)
    kind = np.where(rng.random(n) < 0.2, 0, 1).astype(np.uint8)
    cost = rng.integers(1, 10**6, size=n).astype(np.uint64)
    mean = int(size.mean())
    reqs = [mean * w for w in (1, 100, 1500, 5000, 20000, 39 * TILE)] + [int(size.sum())]
    # a second snapshot: the same run cut by one pinned block in the middle
    kind2 = kind.copy()
    kind2[n // 2] = 2
    pools = _pools([(size, cost, kind), (size, cost, kind2)], [reqs, reqs])
    assert_parity(pools, gpu_search(pools), "long runs")


def test_one_run_of_2_24_blocks_with_parameters_at_both_ends():
    """The pool layout of section 3.5: unevictable parameters at the two ends
    of the pool, everything between them one pinned-free run of about 2^24
    blocks.  Requests from one block to the whole run: most tiles' windows
    run far past the tile after theirs and are finished by the jumps over
    tile records."""
    _announce("one run of 2^24 blocks")
    rng = np.random.default_rng(16)
    n = 1 << 24
    lo, hi = np.log(512.0), np.log(64.0 * (1 << 20))
    size = ((np.exp(lo + rng.random(n) * (hi - lo)) + 511) // 512 * 512).astype(np.uint64)
    kind = np.where(rng.random(n) < 0.2, 0, 1).astype(np.uint8)
    kind[:37] = 2
    kind[-53:] = 2
    cost = np.floor(np.exp(rng.random(n) * np.log(1e12))).astype(np.uint64)
    run = int(size[37:-53].sum())
    mean = int(size.mean())
    reqs = [512, mean, 100 * mean, 5000 * mean, 1 << 40, run // 16, run // 4, run // 2,
            run - (1 << 30), run - 512, run, run + 1]
    pools = _pools([(size, cost, kind)], [reqs])
    got = gpu_search(pools)
    assert_parity(pools, got, "one run of 2^24 blocks")
    check_results(pools, got, sample=range(5))  # (whole-run windows take minutes in Python)


def test_long_runs_mixed_batch():
    """Snapshots of 1 to 30 tiles with few pinned blocks, one to nine
    requests each (shared requests and one wavefront per request), windows
    from one block to whole runs: jobs deferred whole, in part, split over
    chunks and held by one workgroup."""
    _announce("long runs, mixed batch")
    rng = np.random.default_rng(17)
    snaps, reqs = [], []
    for s in range(40):
        n = int(rng.integers(1, 30 * TILE))
        size = (rng.integers(1, 64, size=n) * 512).astype(np.uint64)
        kind = np.where(rng.random(n) < 0.2, 0, 1).astype(np.uint8)
        if s % 3 == 0:
            kind[:3] = 2
            kind[-2:] = 2
        elif s % 3 == 1:
            kind[rng.integers(0, n, size=int(rng.integers(1, 5)))] = 2
        if s % 5 == 0:  # large blocks first, small ones after
            size[: n // 2] *= np.uint64(997)
        cost = rng.integers(0, 10**6, size=n).astype(np.uint64)
        snaps.append((size, cost, kind))
        tot = int(size[kind < 2].sum())
        r = [int(x) for x in rng.integers(1, max(2, tot), size=int(rng.integers(0, 5)))]
        r += [tot // 2, tot, tot + 1, 1, 0][: int(rng.integers(1, 6))]
        reqs.append(r)
    pools = _pools(snaps, reqs)
    got = gpu_search(pools)
    assert_parity(pools, got, "long runs, mixed batch")
    check_results(pools, got)


def test_long_runs_cut_by_pinned_blocks():
    """Runs of 2 to 12 tiles separated by single pinned blocks placed at tile
    edges, inside the 256-block halo and mid-tile, with requests at each
    run's exact byte total, one byte more, and between: a tile whose windows
    cannot close in its run learns where the run ends, and what it learned
    must not carry past a pinned block into the next run."""
    _announce("long runs cut by pinned blocks")
    rng = np.random.default_rng(21)
    snaps, reqs = [], []
    for s in range(12):
        cuts, pos = [], 0
        for _ in range(int(rng.integers(2, 5))):
            pos += int(rng.integers(2, 13)) * TILE + [0, 1, 100, 255, 256, 2048][int(rng.integers(0, 6))]
            cuts.append(pos)
        n = pos + int(rng.integers(1, 3 * TILE))
        size = (rng.integers(1, 64, size=n) * 512).astype(np.uint64)
        kind = np.where(rng.random(n) < 0.2, 0, 1).astype(np.uint8)
        kind[np.array(cuts)] = 2
        cost = rng.integers(0, 10**6, size=n).astype(np.uint64)
        snaps.append((size, cost, kind))
        bounds = [0] + cuts + [n]
        runs = [int(size[a + (a > 0):b].sum()) for a, b in zip(bounds[:-1], bounds[1:])]
        r = []
        for t in runs:
            r += [t, t + 1, t // 2, t - 512]
        r += [max(runs) + 1, int(rng.integers(1, max(runs)))]
        reqs.append(r)
    pools = _pools(snaps, reqs)
    got = gpu_search(pools)
    assert_parity(pools, got, "long runs cut by pinned blocks")
    check_results(pools, got)


def test_long_runs_measured_from_tile_starts():
    """Requests of exactly the bytes from a tile's first block to the end of
    its run, one byte fewer and one more, on runs of 10 to 30 tiles whose
    ends (pinned blocks) sit mid-tile, at a tile's first block and inside a
    halo: the second kernel passes over a tile only when every request that
    deferred there needs more than that count, and a pinned block inside a
    tile must stop the count.  Half- and whole-run requests make the search
    kernel leave its walks past the staged region unstarted."""
    _announce("long runs measured from tile starts")
    rng = np.random.default_rng(23)
    snaps, reqs = [], []
    base = 0  # global index of the snapshot's first block
    for s in range(6):
        n = int(rng.integers(10, 31)) * TILE + int(rng.integers(0, TILE))
        size = (rng.integers(1, 64, size=n) * 512).astype(np.uint64)
        kind = np.where(rng.random(n) < 0.2, 0, 1).astype(np.uint8)
        # the snapshot's tiles start at local indices p * TILE - (base & 7)
        cuts = sorted({int(rng.integers(TILE, n - TILE)) for _ in range(int(rng.integers(1, 3)))})
        if s % 3 == 0:  # at a tile's first block
            cuts = [c - (c + (base & 7)) % TILE for c in cuts]
        elif s % 3 == 1:  # inside a halo (the first 256 blocks of a tile)
            cuts = [c - (c + (base & 7)) % TILE + 100 for c in cuts]
        kind[np.array(cuts)] = 2
        cost = rng.integers(0, 10**6, size=n).astype(np.uint64)
        ends = cuts + [n]
        r = []
        for _ in range(8):
            # a tile start (batch tiles begin at multiples of 8 before the
            # snapshot, then every TILE blocks), the end of its run
            a = TILE * int(rng.integers(1, n // TILE)) - (base & 7)
            e = min(x for x in ends if x > a)
            t = int(size[a:e].sum())
            r += [t - 1, t, t + 1]
        run0 = int(size[:cuts[0]].sum())
        r += [run0 // 2, run0, int(size.sum())]
        snaps.append((size, cost, kind))
        reqs.append(r)
        base += n
    pools = _pools(snaps, reqs)
    got = gpu_search(pools)
    assert_parity(pools, got, "long runs measured from tile starts")
    check_results(pools, got)


def test_long_runs_with_more_than_64_requests_per_wavefront():
    """A three-tile run with 20,000 requests among 40 one-request snapshots:
    each wavefront holds more than 64 of the big snapshot's requests, whose
    running keys live in the partial slots, and their long windows are
    deferred."""
    _announce("long runs, > 64 requests per wavefront")
    rng = np.random.default_rng(18)
    n = 3 * TILE + 1000
    size = (rng.integers(1, 64, size=n) * 512).astype(np.uint64)
    kind = np.where(rng.random(n) < 0.2, 0, 1).astype(np.uint8)
    kind[0] = kind[-1] = 2
    cost = rng.integers(0, 10**6, size=n).astype(np.uint64)
    tot = int(size[1:-1].sum())
    snaps = [(size, cost, kind)]
    reqs = [[int(x) for x in rng.integers(1, tot + 2, size=20000)]]
    for _ in range(40):
        m = int(rng.integers(1, 100))
        snaps.append(((rng.integers(1, 64, size=m) * 512).astype(np.uint64),
                      rng.integers(0, 100, size=m).astype(np.uint64),
                      rng.choice([0, 1, 1, 2], size=m).astype(np.uint8)))
        reqs.append([int(rng.integers(1, 1 << 16))])
    pools = _pools(snaps, reqs)
    import paper_2311_00591_amd as coop
    info = coop.plan_info(pools.num_blocks, pools.num_segments, pools.num_requests)
    assert 20000 / info["slices"] > 512, info
    got = gpu_search(pools)
    assert_parity(pools, got, "long runs, > 64 requests per wavefront")


def test_degenerate_snapshots():
    _announce("degenerate snapshots")
    z = np.zeros(0, dtype=np.uint64)
    pinned = (np.full(5000, 512, np.uint64), np.zeros(5000, np.uint64),
              np.full(5000, 2, np.uint8))
    zero_size = (np.array([0, 0, 512, 0, 1024], np.uint64), np.array([3, 0, 5, 1, 2], np.uint64),
                 np.array([1, 1, 1, 0, 1], np.uint8))
    stored = (np.array([512, 512, 512], np.uint64), np.array([99, 98, 97], np.uint64),
              np.array([0, 3, 255], np.uint8))
    extreme = (np.array([1, 1], np.uint64), np.array([1 << 63, (1 << 63) - 1], np.uint64),
               np.array([1, 1], np.uint8))
    snaps = [(z, z, np.zeros(0, np.uint8)), pinned, zero_size, stored, extreme,
             (z, z, np.zeros(0, np.uint8))]
    reqs = [[0, 1, U64MAX], [0, 1, 512], [0, 1, 512, 1024, 1536, 2048], [1, 512, 513],
            [1, 2, 3, U64MAX], []]
    pools = _pools(snaps, reqs)
    got = gpu_search(pools)
    assert_parity(pools, got, "degenerate")
    assert got[3 + 3 + 6 + 3 + 1].tolist() == [0, 2, U64MAX]  # extreme snapshot, S = 2


def test_ties_across_tiles():
    """Identical blocks everywhere: every window of the same length ties on
    cost and bytes, so the lowest start must win across workgroups."""
    _announce("ties")
    n = 9 * TILE + 5
    size = np.full(n, 1024, np.uint64)
    cost = np.full(n, 7, np.uint64)
    kind = np.ones(n, np.uint8)
    kind[::997] = 2
    pools = _pools([(size, cost, kind)], [[1, 1024, 5000, 1024 * 500, 1024 * 996, 1024 * 997]])
    assert_parity(pools, gpu_search(pools), "ties")


def test_many_requests_cap_workgroups_per_snapshot():
    """With ~1M requests the partial budget allows only 4 workgroups per
    snapshot, so a 20-tile snapshot is swept by workgroups striding over
    tiles."""
    _announce("strided tiles")
    rng = np.random.default_rng(13)
    n_big = 20 * TILE
    size = (rng.integers(1, 64, size=n_big) * 512).astype(np.uint64)
    kind = rng.choice([0, 1, 1, 1, 1, 2], size=n_big).astype(np.uint8)
    cost = rng.integers(0, 10**9, size=n_big).astype(np.uint64)
    snaps = [(size, cost, kind)]
    reqs = [[int(x) for x in rng.integers(1, 1 << 26, size=6)]]
    one = (np.array([512], np.uint64), np.array([1], np.uint64), np.array([1], np.uint8))
    nsmall = (1 << 20) // 8
    for _ in range(nsmall):
        snaps.append(one)
        reqs.append([1, 512, 513, 0, 7, 100, 600, 1])
    pools = _pools(snaps, reqs)
    import paper_2311_00591_amd as coop
    assert coop.workspace_size(pools.num_blocks, pools.num_segments,
                               pools.num_requests) <= (1 << 22) * 32 + 8 * (nsmall + 1) + 256
    assert_parity(pools, gpu_search(pools), "strided tiles")


def test_millions_of_tiny_snapshots():
    """2^22 snapshots of 0..3 blocks (a quarter empty), one request each:
    snapshot indices and tile ids in the millions, most tile ids naming an
    empty remainder, and the cursor stepping over many snapshots per tile."""
    _announce("2^22 tiny snapshots")
    rng = np.random.default_rng(21)
    B = 1 << 22
    nb = rng.integers(0, 4, size=B)
    seg = np.zeros(B + 1, np.uint64)
    seg[1:] = np.cumsum(nb)
    n = int(seg[-1])
    size = (rng.integers(1, 1 << 12, size=n) * 512).astype(np.uint64)
    kind = rng.choice(np.array([0, 1, 1, 1, 2], np.uint8), size=n)
    cost = rng.integers(0, 1 << 40, size=n).astype(np.uint64)
    req = rng.integers(0, 1 << 22, size=B).astype(np.uint64)
    roff = np.arange(B + 1, dtype=np.uint64)
    pools = workloads.Pools(size, cost, kind, seg, req, roff)
    got = gpu_search(pools)
    assert_parity(pools, got, "2^22 tiny snapshots")
    check_results(pools, got, sample=range(0, B, 4099))


def test_workspace_contents_do_not_matter_and_calls_repeat():
    _announce("workspace garbage / repeat")
    pools = workloads.make_config(2, 3, num_segments=6, blocks=(30000, 30000),
                                  requests_per_segment=7)
    a = gpu_search(pools, workspace_fill=0xFF)
    b = gpu_search(pools, workspace_fill=0x00)
    c = gpu_search(pools, workspace_fill=0x5A)
    assert np.array_equal(a, b) and np.array_equal(b, c)
    assert_parity(pools, a, "workspace garbage")


def test_same_workspace_back_to_back():
    """Repeated launches sharing one workspace on one stream (the per-call
    counters must not leak between calls)."""
    _announce("back to back")
    import paper_2311_00591_amd as coop
    pools = workloads.make_config(2, 4, num_segments=4, blocks=(20000, 20000),
                                  requests_per_segment=3)
    ws = coop.WindowSearch(*coop.to_device(pools, "cuda"))
    outs = []
    for _ in range(5):
        outs.append(ws().clone())
    torch.cuda.synchronize()
    want = oracle.window_search(*pools.arrays())
    for o in outs:
        assert np.array_equal(o.cpu().numpy().view(np.uint64), want)


def test_huge_sizes_take_the_plain_prefix_path():
    """Tiles whose byte total reaches 2^51 cannot pack the run id into the
    key; they keep plain 64-bit prefixes and bisect each start."""
    _announce("huge sizes (plain prefixes)")
    rng = np.random.default_rng(14)
    n = 3 * TILE + 500
    size = (rng.integers(1, 1 << 12, size=n).astype(np.uint64) << np.uint64(38))
    kind = rng.choice([0, 1, 1, 1], size=n).astype(np.uint8)
    kind[::400] = 2  # runs of < 400 blocks keep run totals below 2^64
    cost = rng.integers(0, 1 << 40, size=n).astype(np.uint64)
    reqs = [1, 1 << 40, 1 << 50, 1 << 52, 1 << 55, 1 << 58, U64MAX]
    pools = _pools([(size, cost, kind)], [reqs])
    assert int(size[kind < 2].astype(object).sum()) >= 1 << 51
    assert_parity(pools, gpu_search(pools), "huge sizes")


def test_halo_that_would_overflow_the_key_field():
    """A small tile whose last run continues into blocks so large that the
    halo's byte prefix would reach 2^51: the halo is dropped and those windows
    go through the streaming pass."""
    _announce("halo overflow")
    n = TILE + 300
    size = np.full(n, 512, np.uint64)
    size[TILE:] = np.uint64(1) << np.uint64(46)  # 64 of them reach 2^52
    cost = np.arange(n, dtype=np.uint64) % np.uint64(97)
    kind = np.ones(n, np.uint8)
    kind[:TILE - 40:37] = 2
    reqs = [1, 512 * 30, 1 << 46, (1 << 46) + 1, 1 << 50, 1 << 52, 1 << 55]
    pools = _pools([(size, cost, kind)], [reqs])
    assert_parity(pools, gpu_search(pools), "halo overflow")


def _queue_plan(pools):
    import paper_2311_00591_amd as coop
    return coop.plan_info(pools.num_blocks, pools.num_segments, pools.num_requests)


def test_queued_chunks_back_to_back():
    """Enough tiles that a quarter of the units go through the chunk queue;
    three launches share one workspace, so each must stamp the queue with
    its own tag before any claim counts."""
    _announce("queued chunks, back to back")
    import paper_2311_00591_amd as coop
    pools = workloads.make_config(3, 5, num_segments=1200)
    info = _queue_plan(pools)
    assert info["chunks_max"] > info["workgroups"], info
    ws = coop.WindowSearch(*coop.to_device(pools, "cuda"))
    outs = [ws().clone() for _ in range(3)]
    torch.cuda.synchronize()
    want = oracle.window_search(*pools.arrays(), threads=_threads())
    for o in outs:
        got = o.cpu().numpy().view(np.uint64)
        bad = np.flatnonzero((got != want).any(axis=1))
        assert len(bad) == 0, f"{len(bad)} requests differ, first q={int(bad[0])}"


def test_queued_chunks_sized_by_the_largest_snapshot():
    """Many requests leave few partial slots per request, and one snapshot
    of 100 tiles among thousands of tiny ones: the kernel must lengthen the
    queued chunks so that the big snapshot spans no more chunks than slots."""
    _announce("queued chunks sized on the device")
    rng = np.random.default_rng(15)
    n_big = 100 * TILE
    size = (rng.integers(1, 64, size=n_big) * 512).astype(np.uint64)
    kind = rng.choice([0, 1, 1, 1, 1, 1, 1, 2], size=n_big).astype(np.uint8)
    cost = rng.integers(0, 10**9, size=n_big).astype(np.uint64)
    snaps = [(size, cost, kind)]
    reqs = [[int(x) for x in rng.integers(1, 1 << 28, size=105)]]
    for _ in range(5000):
        s = (rng.integers(1, 64, size=64) * 512).astype(np.uint64)
        k = rng.choice([0, 1, 1, 1, 2], size=64).astype(np.uint8)
        c = rng.integers(0, 10**6, size=64).astype(np.uint64)
        snaps.append((s, c, k))
        reqs.append([int(x) for x in rng.integers(1, 1 << 22, size=105)])
    pools = _pools(snaps, reqs)
    info = _queue_plan(pools)
    assert info["chunks_max"] > info["workgroups"], info
    # the host's minimum chunk would let the 101-tile snapshot span more
    # chunks than there are partial slots
    assert -(-101 // info["queued_chunk_units"]) + 2 > info["partial_slots"], info
    assert_parity(pools, gpu_search(pools), "queued chunks sized on the device")
