"""GPU first fit (coop_first_fit) equals the CPU oracle's, index for index,
through the C ABI: the standard workloads at full size, and pools aimed at
the summary levels (64-block groups, 4096-block tiles) and their edges."""
import os
import sys

import numpy as np
import pytest

import oracle
import workloads

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

U64MAX = (1 << 64) - 1
TILE, GROUP = 4096, 64


def _threads():
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def _announce(label):
    print(f"[gpu case] first fit: {label}", flush=True)
    sys.stdout.flush()


def _dev(a, dtype=np.uint64):
    a = np.ascontiguousarray(a, dtype=dtype)
    if dtype == np.uint64:
        a = a.view(np.int64)
    return torch.from_numpy(a).to("cuda")


def gpu_first_fit(size, kind, seg, req, roff, workspace_fill=None, size_offset=0):
    import paper_2311_00591_amd as coop
    size_d = _dev(np.concatenate([np.zeros(size_offset, np.uint64), size]))[size_offset:]
    ws = None
    if workspace_fill is not None:
        need = coop.first_fit_workspace_size(len(size))
        ws = torch.full((max(need, 1),), workspace_fill, dtype=torch.uint8, device="cuda")
    out = coop.first_fit(size_d, _dev(kind, np.uint8), _dev(seg), _dev(req), _dev(roff),
                         workspace=ws)
    torch.cuda.synchronize()
    return out.cpu().numpy().view(np.uint64)


def assert_parity(size, kind, seg, req, roff, got, label):
    want = oracle.first_fit(size, kind, seg, req, roff, threads=_threads())
    bad = np.flatnonzero(got != want)
    if len(bad):
        q = int(bad[0])
        raise AssertionError(f"{label}: {len(bad)} of {len(want)} differ; first q={q} "
                             f"S={int(req[q])} gpu={int(got[q])} oracle={int(want[q])}")


@pytest.mark.parametrize("k", [0, 1, 2, 3])
def test_standard_workload_full_size(k):
    _announce(f"workload {k}")
    p = workloads.make_config(k, 0)
    got = gpu_first_fit(p.size, p.kind, p.seg_offsets, p.req_sizes, p.req_offsets)
    assert_parity(p.size, p.kind, p.seg_offsets, p.req_sizes, p.req_offsets, got, f"workload {k}")


def test_single_huge_pool_sampled():
    """Workload 4's pool (2^24 blocks) with every 37th request plus requests
    small enough to fit; the oracle walks the whole pool for every miss."""
    _announce("workload 4, sampled requests")
    p = workloads.make_config(4, 0)
    req = np.concatenate([p.req_sizes[::37], np.array([0, 1, 512, 1 << 20, 1 << 25, 1 << 26],
                                                      np.uint64)])
    roff = np.array([0, len(req)], np.uint64)
    got = gpu_first_fit(p.size, p.kind, p.seg_offsets, req, roff)
    assert_parity(p.size, p.kind, p.seg_offsets, req, roff, got, "workload 4 sampled")


def _batch(snaps, reqs):
    size = np.concatenate([s for s, _ in snaps]) if snaps else np.zeros(0, np.uint64)
    kind = np.concatenate([k for _, k in snaps]) if snaps else np.zeros(0, np.uint8)
    seg = np.cumsum([0] + [len(s) for s, _ in snaps]).astype(np.uint64)
    req = np.array([x for r in reqs for x in r], dtype=np.uint64)
    roff = np.cumsum([0] + [len(r) for r in reqs]).astype(np.uint64)
    return size.astype(np.uint64), kind.astype(np.uint8), seg, req, roff


def test_summary_level_edges():
    """Snapshots starting and ending inside groups and tiles, each with a
    single fitting chunk placed at a level edge, next to neighbours whose big
    free chunks share a group or tile with them."""
    _announce("summary level edges")
    rng = np.random.default_rng(21)
    snaps, reqs = [], []
    for n in [1, 5, 63, 64, 65, 127, 4095, 4096, 4097, 8191, 3 * TILE + 77, 70 * TILE + 5]:
        for where in ["first", "last", "group", "tile", "none"]:
            size = (rng.integers(1, 8, size=n) * 512).astype(np.uint64)
            kind = rng.choice([0, 1, 1, 2], size=n).astype(np.uint8)
            big = np.uint64(1 << 30)
            pos = {"first": 0, "last": n - 1, "group": min(n - 1, GROUP),
                   "tile": min(n - 1, TILE), "none": None}[where]
            if pos is not None:
                size[pos], kind[pos] = big, 0
            snaps.append((size, kind))
            reqs.append([0, 1, 512, 4096, 1 << 29, 1 << 30, (1 << 30) + 1])
            # a neighbour snapshot of 3 blocks with a huge free chunk in the middle
            snaps.append((np.array([512, 1 << 40, 512], np.uint64), np.array([1, 0, 1], np.uint8)))
            reqs.append([1 << 35, 1 << 41])
    size, kind, seg, req, roff = _batch(snaps, reqs)
    got = gpu_first_fit(size, kind, seg, req, roff)
    assert_parity(size, kind, seg, req, roff, got, "level edges")


def test_degenerate_and_saturated_sizes():
    _announce("degenerate / saturated")
    z = (np.zeros(0, np.uint64), np.zeros(0, np.uint8))
    sat = (np.array([U64MAX - 1, 7, U64MAX, U64MAX - 1], np.uint64),
           np.array([0, 0, 0, 0], np.uint8))
    zero = (np.array([0, 0, 512], np.uint64), np.array([1, 0, 0], np.uint8))
    occupied = (np.full(9000, 1 << 30, np.uint64), np.full(9000, 1, np.uint8))
    snaps = [z, sat, zero, z, occupied]
    reqs = [[0, 1, U64MAX], [0, 1, 8, U64MAX - 1, U64MAX], [0, 1, 512, 513], [], [0, 1]]
    size, kind, seg, req, roff = _batch(snaps, reqs)
    got = gpu_first_fit(size, kind, seg, req, roff)
    assert_parity(size, kind, seg, req, roff, got, "degenerate")
    assert got.tolist()[3:8] == [0, 0, 0, 0, 2]  # S = ~0 skips the 2^64-2 chunks


def test_unaligned_arrays_and_garbage_workspace():
    _announce("unaligned size array, garbage workspace")
    p = workloads.make_config(3, 2, num_segments=64)
    a = gpu_first_fit(p.size, p.kind, p.seg_offsets, p.req_sizes, p.req_offsets,
                      workspace_fill=0xFF, size_offset=1)
    b = gpu_first_fit(p.size, p.kind, p.seg_offsets, p.req_sizes, p.req_offsets,
                      workspace_fill=0x00)
    assert np.array_equal(a, b)
    assert_parity(p.size, p.kind, p.seg_offsets, p.req_sizes, p.req_offsets, a, "unaligned")


def test_many_snapshots_and_requests():
    """2^15 tiny snapshots (the request-to-snapshot search takes several
    rounds) with requests that mostly fit."""
    _announce("many snapshots")
    rng = np.random.default_rng(22)
    B = 1 << 15
    lens = rng.integers(0, 40, size=B)
    size = (rng.integers(1, 64, size=int(lens.sum())) * 512).astype(np.uint64)
    kind = rng.choice([0, 0, 1, 2], size=len(size)).astype(np.uint8)
    seg = np.concatenate([[0], np.cumsum(lens)]).astype(np.uint64)
    per = rng.integers(0, 5, size=B)
    req = (rng.integers(0, 70, size=int(per.sum())) * 512).astype(np.uint64)
    roff = np.concatenate([[0], np.cumsum(per)]).astype(np.uint64)
    got = gpu_first_fit(size, kind, seg, req, roff)
    assert_parity(size, kind, seg, req, roff, got, "many snapshots")
