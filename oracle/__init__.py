"""CPU oracle for the Coop sliding-window eviction search.

TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the
benchmark's CPU-baseline leg import this package; the GPU library never
does, and the two share no code.  See coop_oracle.h for what is computed
(section 3.1 Eq. (1) and section 3.3 of the Coop paper).

All arrays are numpy: size/cost/seg_offsets/req_sizes/req_offsets uint64,
kind uint8.  Results are uint64 arrays of shape (Q, 3) holding
(start, end, cost); an infeasible request reads (2**64-1, 2**64-1, 2**64-1).
"""
import ctypes
import os

import numpy as np

from . import build as _build

INFEASIBLE = np.uint64(0xFFFFFFFFFFFFFFFF)

_ERRORS = {-1: "invalid arguments", -4: "a run total overflows 64 bits",
           -5: "input too large for brute force",
           -6: "a heuristic value is NaN, negative or at least 2^64"}

_lib = None


class OracleError(RuntimeError):
    def __init__(self, code: int):
        super().__init__(f"oracle returned {code}: {_ERRORS.get(code, 'unknown error')}")
        self.code = code


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_build.LIBRARY):
            _build.build()
        lib = ctypes.CDLL(_build.LIBRARY)
        p64 = ctypes.POINTER(ctypes.c_uint64)
        p8 = ctypes.POINTER(ctypes.c_uint8)
        common = [p64, p64, p8, ctypes.c_uint64, p64, ctypes.c_uint64, p64, p64,
                  ctypes.c_uint64, p64]
        lib.coop_oracle_window_search.argtypes = common + [ctypes.c_int]
        lib.coop_oracle_brute_windows.argtypes = common
        lib.coop_oracle_brute_eq1.argtypes = common
        lib.coop_oracle_first_fit.argtypes = [p64, p8, ctypes.c_uint64, p64, ctypes.c_uint64,
                                              p64, p64, ctypes.c_uint64, p64, ctypes.c_int]
        pd = ctypes.POINTER(ctypes.c_double)
        lib.coop_oracle_window_search_real.argtypes = [p64, pd, p8, ctypes.c_uint64, p64,
                                                       ctypes.c_uint64, p64, p64,
                                                       ctypes.c_uint64, p64, pd, ctypes.c_int]
        for f in (lib.coop_oracle_window_search, lib.coop_oracle_brute_windows,
                  lib.coop_oracle_brute_eq1, lib.coop_oracle_first_fit,
                  lib.coop_oracle_window_search_real):
            f.restype = ctypes.c_int
        _lib = lib
    return _lib


def _u64(a):
    return np.ascontiguousarray(a, dtype=np.uint64)


def _ptr(a, ctype):
    return a.ctypes.data_as(ctypes.POINTER(ctype))


def _args(size, cost, kind, seg_offsets, req_sizes, req_offsets):
    size, cost, seg_offsets = _u64(size), _u64(cost), _u64(seg_offsets)
    req_sizes, req_offsets = _u64(req_sizes), _u64(req_offsets)
    kind = np.ascontiguousarray(kind, dtype=np.uint8)
    if not (len(size) == len(cost) == len(kind)):
        raise ValueError("size, cost and kind must have the same length")
    if len(seg_offsets) != len(req_offsets) or len(seg_offsets) < 1:
        raise ValueError("seg_offsets and req_offsets must both have num_segments + 1 entries")
    keep = (size, cost, kind, seg_offsets, req_sizes, req_offsets)
    cargs = [_ptr(size, ctypes.c_uint64), _ptr(cost, ctypes.c_uint64),
             _ptr(kind, ctypes.c_uint8), len(size), _ptr(seg_offsets, ctypes.c_uint64),
             len(seg_offsets) - 1, _ptr(req_sizes, ctypes.c_uint64),
             _ptr(req_offsets, ctypes.c_uint64), len(req_sizes)]
    return keep, cargs


def window_search(size, cost, kind, seg_offsets, req_sizes, req_offsets, threads=1):
    """Linear two-pointer sweep; returns uint64 (Q, 3) = (start, end, cost)."""
    keep, cargs = _args(size, cost, kind, seg_offsets, req_sizes, req_offsets)
    out = np.empty((len(keep[4]), 3), dtype=np.uint64)
    rc = _load().coop_oracle_window_search(*cargs, _ptr(out, ctypes.c_uint64), int(threads))
    if rc != 0:
        raise OracleError(rc)
    return out


def window_search_real(size, h, kind, seg_offsets, req_sizes, req_offsets, threads=1):
    """The search with real-valued heuristics h (float64, see coop_oracle.h).
    Returns (uint64 (Q, 4) = (start, end, exact cost low, high words in units
    of 2^-64), float64 (Q,) = the exact cost rounded to nearest)."""
    h = np.ascontiguousarray(h, dtype=np.float64)
    keep, cargs = _args(size, np.zeros(len(h), np.uint64), kind, seg_offsets, req_sizes,
                        req_offsets)
    cargs[1] = _ptr(h, ctypes.c_double)
    out = np.empty((len(keep[4]), 4), dtype=np.uint64)
    cost = np.empty(len(keep[4]), dtype=np.float64)
    rc = _load().coop_oracle_window_search_real(*cargs, _ptr(out, ctypes.c_uint64),
                                                _ptr(cost, ctypes.c_double), int(threads))
    if rc != 0:
        raise OracleError(rc)
    return out, cost


def brute_windows(size, cost, kind, seg_offsets, req_sizes, req_offsets):
    """Every window enumerated; returns uint64 (Q, 3).  Snapshots <= 512 blocks."""
    keep, cargs = _args(size, cost, kind, seg_offsets, req_sizes, req_offsets)
    out = np.empty((len(keep[4]), 3), dtype=np.uint64)
    rc = _load().coop_oracle_brute_windows(*cargs, _ptr(out, ctypes.c_uint64))
    if rc != 0:
        raise OracleError(rc)
    return out


def brute_eq1(size, cost, kind, seg_offsets, req_sizes, req_offsets):
    """Eq. (1) over every evictable subset; returns uint64 (Q,) minimal cost."""
    keep, cargs = _args(size, cost, kind, seg_offsets, req_sizes, req_offsets)
    out = np.empty(len(keep[4]), dtype=np.uint64)
    rc = _load().coop_oracle_brute_eq1(*cargs, _ptr(out, ctypes.c_uint64))
    if rc != 0:
        raise OracleError(rc)
    return out


def search_single(size, cost, kind, requests, threads=1):
    """Convenience wrapper: one snapshot, a list of request sizes."""
    requests = _u64(requests)
    return window_search(size, cost, kind, [0, len(size)], requests, [0, len(requests)],
                         threads=threads)


def first_fit(size, kind, seg_offsets, req_sizes, req_offsets, threads=1):
    """Leftmost free chunk of at least S bytes (section 2.1, Algorithm 1's
    find_free_block_not_less_than); returns uint64 (Q,) snapshot-local block
    indices, 2**64-1 where the snapshot has no such chunk."""
    size, seg_offsets = _u64(size), _u64(seg_offsets)
    req_sizes, req_offsets = _u64(req_sizes), _u64(req_offsets)
    kind = np.ascontiguousarray(kind, dtype=np.uint8)
    if len(size) != len(kind):
        raise ValueError("size and kind must have the same length")
    if len(seg_offsets) != len(req_offsets) or len(seg_offsets) < 1:
        raise ValueError("seg_offsets and req_offsets must both have num_segments + 1 entries")
    out = np.empty(len(req_sizes), dtype=np.uint64)
    rc = _load().coop_oracle_first_fit(
        _ptr(size, ctypes.c_uint64), _ptr(kind, ctypes.c_uint8), len(size),
        _ptr(seg_offsets, ctypes.c_uint64), len(seg_offsets) - 1,
        _ptr(req_sizes, ctypes.c_uint64), _ptr(req_offsets, ctypes.c_uint64), len(req_sizes),
        _ptr(out, ctypes.c_uint64), int(threads))
    if rc != 0:
        raise OracleError(rc)
    return out


def replay(state, trace, threads=1, policy=0):
    """Algorithm 1 replayed on independent pools (see coop_oracle.h);
    policy 0 evicts the sliding window, policy 1 the DTR-style greedy choice.

    state: dict of numpy arrays size/cost (uint64, num_pools * capacity),
    kind (uint8), id (uint32), len (uint64, num_pools), and 'capacity';
    trace: dict op (uint8), op_id (uint32), op_size/op_cost (uint64),
    op_flags (uint8), each num_pools * num_ops.  Returns (new_state,
    outputs) with outputs block (uint64, P x T), window (P x T x 2), cost,
    free (P x T)."""
    cap = int(state["capacity"])
    P = len(state["len"])
    T = len(trace["op"]) // max(P, 1)
    st = {k: np.array(state[k], copy=True) for k in ("size", "cost", "kind", "id", "len")}
    st["size"] = _u64(st["size"]); st["cost"] = _u64(st["cost"]); st["len"] = _u64(st["len"])
    st["kind"] = np.ascontiguousarray(st["kind"], dtype=np.uint8)
    st["id"] = np.ascontiguousarray(st["id"], dtype=np.uint32)
    st["capacity"] = cap
    tr = {"op": np.ascontiguousarray(trace["op"], dtype=np.uint8),
          "op_id": np.ascontiguousarray(trace["op_id"], dtype=np.uint32),
          "op_size": _u64(trace["op_size"]), "op_cost": _u64(trace["op_cost"]),
          "op_flags": np.ascontiguousarray(trace["op_flags"], dtype=np.uint8)}
    if any(len(v) != P * T for v in tr.values()) or len(st["size"]) != P * cap:
        raise ValueError("inconsistent replay array lengths")
    out_block = np.empty(P * T, dtype=np.uint64)
    out_window = np.empty(2 * P * T, dtype=np.uint64)
    out_cost = np.empty(P * T, dtype=np.uint64)
    out_free = np.empty(P * T, dtype=np.uint64)
    lib = _load()
    p64, p8, p32 = (ctypes.POINTER(ctypes.c_uint64), ctypes.POINTER(ctypes.c_uint8),
                    ctypes.POINTER(ctypes.c_uint32))
    lib.coop_oracle_replay.argtypes = [p64, p64, p8, p32, p64, ctypes.c_uint64, ctypes.c_uint64,
                                       p8, p32, p64, p64, p8, ctypes.c_uint64, p64, p64, p64, p64,
                                       ctypes.c_int, ctypes.c_int]
    lib.coop_oracle_replay.restype = ctypes.c_int
    rc = lib.coop_oracle_replay(
        _ptr(st["size"], ctypes.c_uint64), _ptr(st["cost"], ctypes.c_uint64),
        _ptr(st["kind"], ctypes.c_uint8), _ptr(st["id"], ctypes.c_uint32),
        _ptr(st["len"], ctypes.c_uint64), P, cap, _ptr(tr["op"], ctypes.c_uint8),
        _ptr(tr["op_id"], ctypes.c_uint32), _ptr(tr["op_size"], ctypes.c_uint64),
        _ptr(tr["op_cost"], ctypes.c_uint64), _ptr(tr["op_flags"], ctypes.c_uint8), T,
        _ptr(out_block, ctypes.c_uint64), _ptr(out_window, ctypes.c_uint64),
        _ptr(out_cost, ctypes.c_uint64), _ptr(out_free, ctypes.c_uint64), int(policy),
        int(threads))
    if rc != 0:
        raise OracleError(rc)
    outs = {"block": out_block.reshape(P, T), "window": out_window.reshape(P, T, 2),
            "cost": out_cost.reshape(P, T), "free": out_free.reshape(P, T)}
    return st, outs
