"""The C ABI library loads, exports what include/coop.h declares, and
validates host-visible arguments without touching a GPU."""
import ctypes
import os
import re

import pytest

import paper_2311_00591_amd as coop
from conftest import ROOT

HEADER = os.path.join(ROOT, "include", "coop.h")


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(coop_[a-z_0-9]+)\s*\(", text)))


def test_exports_every_declared_symbol():
    names = _declared_functions()
    assert {"coop_window_search", "coop_window_search_workspace_size",
            "coop_status_string", "coop_abi_version"} <= set(names)
    lib = coop.load_library()
    for n in names:
        assert hasattr(lib, n), n


def test_abi_version_matches_header():
    m = re.search(r"#define COOP_ABI_VERSION (\d+)", open(HEADER).read())
    assert coop.load_library().coop_abi_version() == int(m.group(1))


def test_status_strings():
    lib = coop.load_library()
    for s in (0, -1, -2, -3, -4, 7):
        assert lib.coop_status_string(s)
    # the binding's table agrees with the library for every named status
    for s, text in coop._STATUS.items():
        assert lib.coop_status_string(s).decode() == text
    assert b"unknown" in lib.coop_status_string(7)


def test_only_the_declared_functions_are_exported():
    """The unchecked enqueue functions and the debug-check helpers are
    internal: the dynamic symbol table holds the header's functions only."""
    import subprocess
    nm = subprocess.run(["nm", "-D", "--defined-only", coop.LIBRARY], capture_output=True,
                        text=True, check=True).stdout
    exported = {line.split()[-1] for line in nm.splitlines() if " T " in line or " W " in line}
    ours = {n for n in exported if "coop" in n}
    assert ours == set(_declared_functions()), sorted(ours ^ set(_declared_functions()))


def test_workspace_size_depends_on_counts_only():
    a = coop.workspace_size(4096 * 1024, 1024, 1024)
    assert a == coop.workspace_size(4096 * 1024, 1024, 1024) > 0
    assert coop.workspace_size(1 << 24, 1, 4096) >= coop.workspace_size(1 << 20, 1, 4096)
    # partial storage is bounded: 2^23 keys of 32 bytes, one counter per
    # (request slice, snapshot) -- at most 256 slices -- the queue, tag and
    # deferred-list words, a deferred entry (16 bytes) per chunk and per
    # (slice, snapshot that can defer), a 24-byte record per tile and a
    # deferral bit per partial key
    p = coop.plan_info(1 << 30, 1, 1 << 20)
    keys = (1 << 20) * p["partial_slots"]
    assert keys <= 1 << 23
    nrec = (1 << 30) >> 12
    assert coop.workspace_size(1 << 30, 1, 1 << 20) <= (
        keys * 32 + 256 * 8 + 24 + 256 + 16 * (p["chunks_max"] + 256) + 16
        + 24 * nrec + keys // 8 + 64)
    lib = coop.load_library()
    assert lib.coop_window_search_workspace_size(1, 1, 1, None) == -1
    out = ctypes.c_size_t()
    assert lib.coop_window_search_workspace_size(1, 1 << 40, 1, ctypes.byref(out)) == -1


def _call(**kw):
    args = dict(size=8, cost=8, kind=8, n=4, seg=8, B=1, req=8, roff=8, Q=1, out=8,
                ws=8, wsb=1 << 30, stream=None)
    args.update(kw)
    return coop.load_library().coop_window_search(
        args["size"], args["cost"], args["kind"], args["n"], args["seg"], args["B"],
        args["req"], args["roff"], args["Q"], args["out"], args["ws"], args["wsb"],
        args["stream"])


def test_validation_rejects_bad_host_arguments():
    # Non-null but never dereferenced: validation fails before any launch.
    assert _call(Q=0) == 0
    assert _call(Q=0, size=None, seg=None) == 0
    assert _call(B=0) == -1
    assert _call(size=None) == -1
    assert _call(kind=None) == -1
    assert _call(seg=None) == -1
    assert _call(req=None) == -1
    assert _call(roff=None) == -1
    assert _call(out=None) == -1
    assert _call(ws=None) == -2
    assert _call(wsb=1) == -2
    assert _call(B=1 << 40) == -1


def test_no_cpu_fallback():
    import torch
    t = torch.zeros(4, dtype=torch.int64)
    with pytest.raises(ValueError, match="GPU"):
        coop.window_search(t, t, torch.zeros(4, dtype=torch.uint8), torch.tensor([0, 4]),
                           torch.tensor([1]), torch.tensor([0, 1]))


def test_gpu_path_shares_nothing_with_the_oracle():
    gpu_src = open(os.path.join(ROOT, "paper_2311_00591_amd", "csrc",
                                "coop_window_search.hip")).read()
    oracle_src = open(os.path.join(ROOT, "oracle", "coop_oracle.c")).read()
    assert "coop_oracle" not in gpu_src and "oracle" not in gpu_src.lower()
    assert '#include "coop.h"' not in oracle_src
    pkg = open(os.path.join(ROOT, "paper_2311_00591_amd", "__init__.py")).read()
    assert "import oracle" not in pkg and "from oracle" not in pkg


def test_plan_queue_and_partial_slots():
    # an eighth of the units (a quarter with fewer than 64 snapshots) go
    # through the queue once each workgroup has at least 8; the first chunks
    # tile [0, first_units) exactly
    p = coop.plan_info(66_267_909, 4096, 16384)
    assert p["chunks_max"] > p["workgroups"] and 256 < p["workgroups"] <= 512
    assert p["first_units"] == p["workgroups"] * p["first_chunk_units"] < p["units"]
    assert p["queued_chunk_units"] >= 1 and p["partial_slots"] >= 4
    assert p["partial_slots"] * 16384 <= 1 << 23
    # two units per workgroup: no queue
    p = coop.plan_info(4096 * 1024, 1024, 1024)
    assert p["chunks_max"] == p["workgroups"] and p["first_units"] == p["units"]
    # too many snapshots for every workgroup to scan their offsets: no queue
    p = coop.plan_info(1 << 26, 1 << 15, 1 << 15)
    assert p["chunks_max"] == p["workgroups"]
    lib = coop.load_library()
    assert lib.coop_window_search_plan(1, 1, 1, None) == -1


@pytest.mark.parametrize("n", [1, 4097, 1_000_003, 66_267_909, 1 << 24, 1 << 30])
@pytest.mark.parametrize("b", [1, 7, 1024, 4096, 1 << 15])
@pytest.mark.parametrize("per", [1, 4, 16, 600])
def test_plan_chunks_cover_every_unit(n, b, per):
    if b > n:
        pytest.skip("more snapshots than blocks")
    q = b * per
    p = coop.plan_info(n, b, q)
    units, grid = p["units"], p["workgroups"]
    assert 1 <= grid <= 512 and grid <= units
    c1, u1, c2 = p["first_chunk_units"], p["first_units"], p["queued_chunk_units"]
    if p["chunks_max"] > grid:
        # with a queue: the first chunks tile [0, u1), the queued ones the rest
        assert u1 == grid * c1 < units and c1 >= 1 and c2 >= 1
        assert u1 + (p["chunks_max"] - grid) * c2 >= units
        # every workgroup slot takes a first chunk unless the partial
        # budget grew the chunks (a snapshot of T tiles must meet at most
        # cap chunks, cap = the budget's keys per request)
        g0 = min(units, 512)
        chunk0 = -(-units // g0)
        tiles = -(-n // 4096) + 1
        cap = max((1 << 23) // q, 2)
        if -(-tiles // chunk0) + 1 <= cap:
            assert grid == g0
    else:
        assert u1 == units and grid * c1 >= units > (grid - 1) * c1
    assert p["partial_slots"] >= 1 and p["partial_slots"] <= p["chunks_max"]
    if q <= 1 << 21:
        assert p["partial_slots"] * q <= 1 << 23


def test_plan_queues_a_quarter_with_few_snapshots():
    # one snapshot of 2^24 blocks, 16 requests: 4097 units, a share of 8, 6 first units each
    p = coop.plan_info(1 << 24, 1, 16)
    assert p["workgroups"] == 512 and p["first_chunk_units"] == 8 - 8 // 4
    assert p["first_units"] == 512 * p["first_chunk_units"] < p["units"]


def test_plan_takes_every_workgroup_slot_on_the_ragged_batch():
    # 20274 units over 512 workgroups: 35 first units each, the rest queued
    p = coop.plan_info(66_267_909, 4096, 16384)
    assert p["units"] == 20274 and p["workgroups"] == 512
    assert p["first_units"] == 512 * 35


def test_replay_rejects_unknown_policy_and_null_buffers():
    # validation happens before any launch, so no GPU is touched
    lib = coop.load_library()
    nz = 16  # non-null, never dereferenced
    bufs = [nz] * 5

    def call(policy, P=1, T=1, ptr=nz):
        return lib.coop_replay(*bufs, P, 8, ptr, nz, nz, nz, nz, T, policy, nz, nz, nz, nz, nz,
                               nz, 1 << 20, None)

    assert call(2) == -1
    assert call(-1) == -1
    assert call(2, P=0) == -1          # the policy is checked even for an empty batch
    assert call(coop.POLICY_GREEDY, P=0) == 0
    assert call(coop.POLICY_WINDOW, T=0) == 0
    assert call(coop.POLICY_GREEDY, ptr=None) == -1
    assert lib.coop_replay(*bufs, 1, 8, nz, nz, nz, nz, nz, 1, 1, nz, nz, nz, nz, nz, nz, 1,
                           None) == -2  # workspace too small


def test_real_search_validates_host_arguments():
    lib = coop.load_library()
    nz = 16

    def call(B=1, Q=1, ws=nz, wsb=1 << 30, **null):
        a = dict(size=nz, h=nz, kind=nz, seg=nz, req=nz, roff=nz, out=nz, status=nz)
        a.update(null)
        return lib.coop_window_search_real(a["size"], a["h"], a["kind"], 8, a["seg"], B, a["req"],
                                           a["roff"], Q, a["out"], a["status"], ws, wsb, None)

    assert call(Q=0, seg=None) == 0
    for name in ("size", "h", "kind", "seg", "req", "roff", "out", "status"):
        assert call(**{name: None}) == -1, name
    assert call(B=0) == -1
    assert call(ws=None) == -2
    assert call(wsb=1) == -2
    assert coop.real_workspace_size(8, 1, 1) > 0
    assert coop.real_workspace_size(8, 1, 0) == 0


def test_static_entry_validates_and_bounds_its_scratch():
    """coop_window_search_static: the host checks and the size limit come
    before the scratch lookup or any launch, so no GPU is touched."""
    lib = coop.load_library()
    nz = 16

    def call(n=4, B=1, Q=1, **null):
        a = dict(size=nz, cost=nz, kind=nz, seg=nz, req=nz, roff=nz, out=nz)
        a.update(null)
        return lib.coop_window_search_static(a["size"], a["cost"], a["kind"], n, a["seg"], B,
                                             a["req"], a["roff"], Q, a["out"], None)

    assert coop.static_capacity() == (32 << 20) - 256
    assert call(Q=0, seg=None) == 0
    for name in ("size", "cost", "kind", "seg", "req", "roff", "out"):
        assert call(**{name: None}) == -1, name
    assert call(B=0) == -1
    assert call(B=1 << 40) == -1
    # two partial keys of 32 bytes per request no longer fit
    assert call(Q=1 << 20) == -5
    assert call(n=1 << 24, B=1 << 23, Q=1 << 23) == -5
    assert lib.coop_status_string(-5) == coop._STATUS[-5].encode()
    # a batch that fits with the full partial-key budget is planned as usual
    assert coop.workspace_size(66_267_909, 4096, 16384) > coop.static_capacity()
