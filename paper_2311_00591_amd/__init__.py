"""MI355X (gfx950) batched sliding-window eviction search of Coop.

Thin ctypes binding over libcoop.so (include/coop.h): argument marshalling
only; every step of the search runs in the HIP kernels.  PyTorch supplies the
device memory and the stream.  There is no CPU fallback: without the built
library or a GPU the calls raise.

Unsigned 64-bit arrays travel in torch.int64 (or torch.uint64) storage; the
bit patterns are what the library reads.  Results come back as int64 (Q, 3)
tensors holding (start, end, cost); an infeasible request reads (-1, -1, -1),
the two's-complement view of the all-ones sentinel.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIBRARY = os.path.join(_PKG, "libcoop.so")

COOP_FREE, COOP_EVICTABLE, COOP_PINNED = 0, 1, 2
INFEASIBLE = -1  # int64 view of the all-ones sentinel
POLICY_WINDOW, POLICY_GREEDY = 0, 1  # coop_replay's eviction policies

_STATUS = {0: "ok", -1: "invalid argument", -2: "workspace missing or too small",
           -3: "HIP launch failed", -4: "a run's byte or cost total exceeds 2^64 - 1",
           -5: "the batch needs more than the library's static scratch"}

_lib = None


class CoopError(RuntimeError):
    def __init__(self, status: int, text: str):
        super().__init__(f"coop status {status}: {text}")
        self.status = status


class CoopPlan(ctypes.Structure):
    """coop_plan_t."""
    _fields_ = [(name, ctypes.c_uint64) for name in (
        "workgroups", "slices", "units", "first_chunk_units", "first_units",
        "queued_chunk_units", "chunks_max", "partial_slots")]


def load_library():
    """Loads libcoop.so; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIBRARY):
        raise ImportError(f"{LIBRARY} is missing: build it with __graft_entry__.build() "
                          "(or python -m paper_2311_00591_amd._build)")
    lib = ctypes.CDLL(LIBRARY)
    u64, vp, sz = ctypes.c_uint64, ctypes.c_void_p, ctypes.c_size_t
    lib.coop_abi_version.argtypes = []
    lib.coop_abi_version.restype = ctypes.c_int
    lib.coop_status_string.argtypes = [ctypes.c_int]
    lib.coop_status_string.restype = ctypes.c_char_p
    lib.coop_window_search_workspace_size.argtypes = [u64, u64, u64, ctypes.POINTER(sz)]
    lib.coop_window_search_workspace_size.restype = ctypes.c_int
    lib.coop_window_search_plan.argtypes = [u64, u64, u64, ctypes.POINTER(CoopPlan)]
    lib.coop_window_search_plan.restype = ctypes.c_int
    lib.coop_window_search.argtypes = [vp, vp, vp, u64, vp, u64, vp, vp, u64, vp, vp, sz, vp]
    lib.coop_first_fit_workspace_size.argtypes = [u64, ctypes.POINTER(sz)]
    lib.coop_first_fit_workspace_size.restype = ctypes.c_int
    lib.coop_first_fit.argtypes = [vp, vp, u64, vp, u64, vp, vp, u64, vp, vp, sz, vp]
    lib.coop_first_fit.restype = ctypes.c_int
    lib.coop_replay_workspace_size.argtypes = [u64, u64, ctypes.POINTER(sz)]
    lib.coop_replay_workspace_size.restype = ctypes.c_int
    lib.coop_replay.argtypes = [vp, vp, vp, vp, vp, u64, u64, vp, vp, vp, vp, vp, u64,
                                ctypes.c_int32, vp, vp, vp, vp, vp, vp, sz, vp]
    lib.coop_replay.restype = ctypes.c_int
    lib.coop_window_search.restype = ctypes.c_int
    lib.coop_window_search_static.argtypes = [vp, vp, vp, u64, vp, u64, vp, vp, u64, vp, vp]
    lib.coop_window_search_static.restype = ctypes.c_int
    lib.coop_window_search_static_capacity.argtypes = []
    lib.coop_window_search_static_capacity.restype = sz
    lib.coop_window_search_real_workspace_size.argtypes = [u64, u64, u64, ctypes.POINTER(sz)]
    lib.coop_window_search_real_workspace_size.restype = ctypes.c_int
    lib.coop_window_search_real.argtypes = [vp, vp, vp, u64, vp, u64, vp, vp, u64, vp, vp, vp,
                                            sz, vp]
    lib.coop_window_search_real.restype = ctypes.c_int
    _lib = lib
    return lib


def _check(status: int):
    if status != 0:
        text = load_library().coop_status_string(status).decode()
        raise CoopError(status, text)


def workspace_size(num_blocks: int, num_segments: int, num_requests: int) -> int:
    """Device workspace bytes coop_window_search needs for these counts."""
    out = ctypes.c_size_t(0)
    _check(load_library().coop_window_search_workspace_size(
        int(num_blocks), int(num_segments), int(num_requests), ctypes.byref(out)))
    return out.value


def plan_info(num_blocks: int, num_segments: int, num_requests: int) -> dict:
    """How the library splits a batch of these counts (coop_plan_t as a dict)."""
    plan = CoopPlan()
    _check(load_library().coop_window_search_plan(
        int(num_blocks), int(num_segments), int(num_requests), ctypes.byref(plan)))
    return {name: int(getattr(plan, name)) for name, _ in CoopPlan._fields_}


def _u64_tensor(t: torch.Tensor, name: str, device) -> torch.Tensor:
    if t.dtype not in (torch.int64, torch.uint64):
        raise TypeError(f"{name} must be int64/uint64 storage, got {t.dtype}")
    if t.device != device:
        raise ValueError(f"{name} is on {t.device}, expected {device}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    return t.data_ptr() if t is not None and t.numel() > 0 else None


class WindowSearch:
    """A prepared call for fixed device tensors: validates and marshals once,
    so that repeated launches (benchmarks, serving loops) cost one ctypes
    call each.  The tensors must stay alive and unchanged in shape."""

    def __init__(self, size, cost, kind, seg_offsets, req_sizes, req_offsets,
                 out: Optional[torch.Tensor] = None,
                 workspace: Optional[torch.Tensor] = None):
        device = size.device
        if device.type != "cuda":
            raise ValueError("coop window search runs on the GPU; tensors are on "
                             f"{device} (there is no CPU fallback)")
        lib = load_library()
        self.size = _u64_tensor(size, "size", device)
        self.cost = _u64_tensor(cost, "cost", device)
        if kind.dtype != torch.uint8 or kind.device != device or not kind.is_contiguous():
            raise TypeError("kind must be a contiguous uint8 tensor on the same device")
        self.kind = kind
        self.seg_offsets = _u64_tensor(seg_offsets, "seg_offsets", device)
        self.req_sizes = _u64_tensor(req_sizes, "req_sizes", device)
        self.req_offsets = _u64_tensor(req_offsets, "req_offsets", device)
        n, b1, q = size.numel(), seg_offsets.numel(), req_sizes.numel()
        if cost.numel() != n or kind.numel() != n:
            raise ValueError("size, cost and kind must have the same length")
        if b1 < 1 or req_offsets.numel() != b1:
            raise ValueError("seg_offsets and req_offsets need num_segments + 1 entries")
        self.num_blocks, self.num_segments, self.num_requests = n, b1 - 1, q
        if out is None:
            out = torch.empty((q, 3), dtype=torch.int64, device=device)
        if out.shape != (q, 3) or out.dtype != torch.int64 or not out.is_contiguous():
            raise ValueError("out must be a contiguous int64 (Q, 3) tensor")
        self.out = out
        need = workspace_size(n, b1 - 1, q)
        if workspace is None:
            workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=device)
        if workspace.numel() * workspace.element_size() < need:
            raise ValueError(f"workspace holds {workspace.numel()} bytes, needs {need}")
        self.workspace = workspace
        self.workspace_bytes = workspace.numel() * workspace.element_size()
        self._fn = lib.coop_window_search
        self._args = (_ptr(self.size), _ptr(self.cost), _ptr(self.kind), n,
                      _ptr(self.seg_offsets), b1 - 1, _ptr(self.req_sizes),
                      _ptr(self.req_offsets), q, _ptr(self.out), _ptr(self.workspace),
                      self.workspace_bytes)

    def launch(self, stream: Optional[int] = None) -> None:
        """Enqueues the search on `stream` (default: torch's current stream)."""
        if stream is None:
            stream = torch.cuda.current_stream(self.size.device).cuda_stream
        _check(self._fn(*self._args, stream))

    def __call__(self, stream: Optional[int] = None) -> torch.Tensor:
        self.launch(stream)
        return self.out


def window_search(size, cost, kind, seg_offsets, req_sizes, req_offsets, *,
                  out: Optional[torch.Tensor] = None,
                  workspace: Optional[torch.Tensor] = None,
                  stream: Optional[int] = None) -> torch.Tensor:
    """One batched search on device tensors; returns int64 (Q, 3)
    (start, end, cost).  Asynchronous on `stream` like any torch op."""
    ws = WindowSearch(size, cost, kind, seg_offsets, req_sizes, req_offsets, out, workspace)
    return ws(stream)


def window_search_static(size, cost, kind, seg_offsets, req_sizes, req_offsets, *,
                         out: Optional[torch.Tensor] = None,
                         stream: Optional[int] = None) -> torch.Tensor:
    """coop_window_search_static: the batched search without a workspace
    (its state lives in the library's static device array, shared by every
    call on the GPU).  Returns int64 (Q, 3); with `out` given, nothing is
    allocated on the device."""
    device = size.device
    if device.type != "cuda":
        raise ValueError("coop window search runs on the GPU; tensors are on "
                         f"{device} (there is no CPU fallback)")
    size = _u64_tensor(size, "size", device)
    cost = _u64_tensor(cost, "cost", device)
    if kind.dtype != torch.uint8 or kind.device != device or not kind.is_contiguous():
        raise TypeError("kind must be a contiguous uint8 tensor on the same device")
    seg_offsets = _u64_tensor(seg_offsets, "seg_offsets", device)
    req_sizes = _u64_tensor(req_sizes, "req_sizes", device)
    req_offsets = _u64_tensor(req_offsets, "req_offsets", device)
    n, b1, q = size.numel(), seg_offsets.numel(), req_sizes.numel()
    if cost.numel() != n or kind.numel() != n:
        raise ValueError("size, cost and kind must have the same length")
    if b1 < 1 or req_offsets.numel() != b1:
        raise ValueError("seg_offsets and req_offsets need num_segments + 1 entries")
    if out is None:
        out = torch.empty((q, 3), dtype=torch.int64, device=device)
    if out.shape != (q, 3) or out.dtype != torch.int64 or not out.is_contiguous():
        raise ValueError("out must be a contiguous int64 (Q, 3) tensor")
    if stream is None:
        stream = torch.cuda.current_stream(device).cuda_stream
    _check(load_library().coop_window_search_static(
        _ptr(size), _ptr(cost), _ptr(kind), n, _ptr(seg_offsets), b1 - 1, _ptr(req_sizes),
        _ptr(req_offsets), q, _ptr(out), stream))
    return out


def static_capacity() -> int:
    """Workspace bytes coop_window_search_static's static array holds."""
    return int(load_library().coop_window_search_static_capacity())


def real_workspace_size(num_blocks: int, num_segments: int, num_requests: int) -> int:
    """Device workspace bytes coop_window_search_real needs."""
    out = ctypes.c_size_t(0)
    _check(load_library().coop_window_search_real_workspace_size(
        int(num_blocks), int(num_segments), int(num_requests), ctypes.byref(out)))
    return out.value


class WindowSearchReal:
    """A prepared coop_window_search_real call: the search with real-valued
    heuristics h (float64 device tensor in place of cost).  Results: `out`,
    int64 (Q, 5) = (start, end, exact cost low word, high word, binary64 cost
    bits) -- `cost` is its last column viewed as float64 -- and `status`
    (int32, bit 0: an invalid h)."""

    def __init__(self, size, h, kind, seg_offsets, req_sizes, req_offsets,
                 workspace: Optional[torch.Tensor] = None):
        device = size.device
        if device.type != "cuda":
            raise ValueError("coop window search runs on the GPU; tensors are on "
                             f"{device} (there is no CPU fallback)")
        lib = load_library()
        self.size = _u64_tensor(size, "size", device)
        if h.dtype != torch.float64 or h.device != device or not h.is_contiguous():
            raise TypeError("h must be a contiguous float64 tensor on the same device")
        self.h = h
        if kind.dtype != torch.uint8 or kind.device != device or not kind.is_contiguous():
            raise TypeError("kind must be a contiguous uint8 tensor on the same device")
        self.kind = kind
        self.seg_offsets = _u64_tensor(seg_offsets, "seg_offsets", device)
        self.req_sizes = _u64_tensor(req_sizes, "req_sizes", device)
        self.req_offsets = _u64_tensor(req_offsets, "req_offsets", device)
        n, b1, q = size.numel(), seg_offsets.numel(), req_sizes.numel()
        if h.numel() != n or kind.numel() != n:
            raise ValueError("size, h and kind must have the same length")
        if b1 < 1 or req_offsets.numel() != b1:
            raise ValueError("seg_offsets and req_offsets need num_segments + 1 entries")
        self.num_blocks, self.num_segments, self.num_requests = n, b1 - 1, q
        self.out = torch.empty((q, 5), dtype=torch.int64, device=device)
        self.cost = self.out[:, 4].view(torch.float64)
        self.status = torch.zeros(1, dtype=torch.int32, device=device)
        need = real_workspace_size(n, b1 - 1, q)
        if workspace is None:
            workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=device)
        if workspace.numel() * workspace.element_size() < need:
            raise ValueError(f"workspace holds {workspace.numel()} bytes, needs {need}")
        self.workspace = workspace
        self._fn = lib.coop_window_search_real
        self._args = (_ptr(self.size), _ptr(self.h), _ptr(self.kind), n,
                      _ptr(self.seg_offsets), b1 - 1, _ptr(self.req_sizes),
                      _ptr(self.req_offsets), q, _ptr(self.out), _ptr(self.status),
                      _ptr(self.workspace), workspace.numel() * workspace.element_size())

    def launch(self, stream: Optional[int] = None) -> None:
        if stream is None:
            stream = torch.cuda.current_stream(self.size.device).cuda_stream
        _check(self._fn(*self._args, stream))

    def __call__(self, stream: Optional[int] = None) -> torch.Tensor:
        self.launch(stream)
        return self.out


def first_fit_workspace_size(num_blocks: int) -> int:
    """Device workspace bytes coop_first_fit needs for num_blocks blocks."""
    out = ctypes.c_size_t(0)
    _check(load_library().coop_first_fit_workspace_size(int(num_blocks), ctypes.byref(out)))
    return out.value


class FirstFit:
    """A prepared first-fit call (coop_first_fit) for fixed device tensors:
    for every request, the snapshot-local index of the leftmost free chunk of
    at least S bytes, -1 (2**64-1 as uint64) where there is none."""

    def __init__(self, size, kind, seg_offsets, req_sizes, req_offsets,
                 out: Optional[torch.Tensor] = None,
                 workspace: Optional[torch.Tensor] = None):
        device = size.device
        if device.type != "cuda":
            raise ValueError("coop first fit runs on the GPU; tensors are on "
                             f"{device} (there is no CPU fallback)")
        lib = load_library()
        self.size = _u64_tensor(size, "size", device)
        if kind.dtype != torch.uint8 or kind.device != device or not kind.is_contiguous():
            raise TypeError("kind must be a contiguous uint8 tensor on the same device")
        self.kind = kind
        self.seg_offsets = _u64_tensor(seg_offsets, "seg_offsets", device)
        self.req_sizes = _u64_tensor(req_sizes, "req_sizes", device)
        self.req_offsets = _u64_tensor(req_offsets, "req_offsets", device)
        n, b1, q = size.numel(), seg_offsets.numel(), req_sizes.numel()
        if kind.numel() != n:
            raise ValueError("size and kind must have the same length")
        if b1 < 1 or req_offsets.numel() != b1:
            raise ValueError("seg_offsets and req_offsets need num_segments + 1 entries")
        if out is None:
            out = torch.empty(q, dtype=torch.int64, device=device)
        if out.shape != (q,) or out.dtype != torch.int64 or not out.is_contiguous():
            raise ValueError("out must be a contiguous int64 (Q,) tensor")
        self.out = out
        need = first_fit_workspace_size(n)
        if workspace is None:
            workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=device)
        if workspace.numel() * workspace.element_size() < need:
            raise ValueError(f"workspace holds {workspace.numel()} bytes, needs {need}")
        self.workspace = workspace
        self._fn = lib.coop_first_fit
        self._args = (_ptr(self.size), _ptr(self.kind), n, _ptr(self.seg_offsets), b1 - 1,
                      _ptr(self.req_sizes), _ptr(self.req_offsets), q, _ptr(self.out),
                      _ptr(self.workspace), workspace.numel() * workspace.element_size())

    def launch(self, stream: Optional[int] = None) -> None:
        if stream is None:
            stream = torch.cuda.current_stream(self.size.device).cuda_stream
        _check(self._fn(*self._args, stream))

    def __call__(self, stream: Optional[int] = None) -> torch.Tensor:
        self.launch(stream)
        return self.out


def first_fit(size, kind, seg_offsets, req_sizes, req_offsets, *,
              out: Optional[torch.Tensor] = None,
              workspace: Optional[torch.Tensor] = None,
              stream: Optional[int] = None) -> torch.Tensor:
    """One batched first fit on device tensors; returns int64 (Q,)."""
    return FirstFit(size, kind, seg_offsets, req_sizes, req_offsets, out, workspace)(stream)


def replay_workspace_size(num_pools: int, capacity: int) -> int:
    """Device workspace bytes coop_replay needs."""
    out = ctypes.c_size_t(0)
    _check(load_library().coop_replay_workspace_size(int(num_pools), int(capacity),
                                                     ctypes.byref(out)))
    return out.value


class Replay:
    """A prepared coop_replay call: Algorithm 1 replayed on independent pools
    held in device tensors (updated in place by every launch).

    state: dict of device tensors size/cost (int64 holding u64, P*cap),
    kind (uint8), id (int32 holding u32), len (int64, P) and int capacity;
    trace: dict of device tensors op (uint8), op_id (int32), op_size/op_cost
    (int64), op_flags (uint8), each P*T.  Outputs: block, cost, free (int64,
    P*T), window (int64, P*T*2), status (int32, 1).  policy: POLICY_WINDOW
    (Coop's sliding window) or POLICY_GREEDY (DTR's heuristic, one tensor at
    a time)."""

    def __init__(self, state, trace, workspace: Optional[torch.Tensor] = None,
                 policy: int = 0):
        dev = state["size"].device
        if dev.type != "cuda":
            raise ValueError("coop replay runs on the GPU (there is no CPU fallback)")
        lib = load_library()
        self.state, self.trace = state, trace
        P = state["len"].numel()
        cap = int(state["capacity"])
        T = trace["op"].numel() // max(P, 1)
        for k, dt in (("size", torch.int64), ("cost", torch.int64), ("kind", torch.uint8),
                      ("id", torch.int32)):
            t = state[k]
            if t.dtype != dt or t.numel() != P * cap or not t.is_contiguous() or t.device != dev:
                raise ValueError(f"state[{k!r}] must be a contiguous {dt} tensor of {P * cap}")
        for k, dt in (("op", torch.uint8), ("op_id", torch.int32), ("op_size", torch.int64),
                      ("op_cost", torch.int64), ("op_flags", torch.uint8)):
            t = trace[k]
            if t.dtype != dt or t.numel() != P * T or not t.is_contiguous() or t.device != dev:
                raise ValueError(f"trace[{k!r}] must be a contiguous {dt} tensor of {P * T}")
        if policy not in (POLICY_WINDOW, POLICY_GREEDY):
            raise ValueError(f"unknown policy {policy}")
        self.num_pools, self.capacity, self.num_ops, self.policy = P, cap, T, policy
        self.block = torch.empty(P * T, dtype=torch.int64, device=dev)
        self.window = torch.empty(P * T * 2, dtype=torch.int64, device=dev)
        self.cost = torch.empty(P * T, dtype=torch.int64, device=dev)
        self.free = torch.empty(P * T, dtype=torch.int64, device=dev)
        self.status = torch.zeros(1, dtype=torch.int32, device=dev)
        need = replay_workspace_size(P, cap)
        if workspace is None:
            workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
        if workspace.numel() * workspace.element_size() < need:
            raise ValueError(f"workspace holds {workspace.numel()} bytes, needs {need}")
        self.workspace = workspace
        self._fn = lib.coop_replay
        self._args = (state["size"].data_ptr(), state["cost"].data_ptr(), state["kind"].data_ptr(),
                      state["id"].data_ptr(), state["len"].data_ptr(), P, cap,
                      trace["op"].data_ptr(), trace["op_id"].data_ptr(),
                      trace["op_size"].data_ptr(), trace["op_cost"].data_ptr(),
                      trace["op_flags"].data_ptr(), T, policy, self.block.data_ptr(),
                      self.window.data_ptr(), self.cost.data_ptr(), self.free.data_ptr(),
                      self.status.data_ptr(), workspace.data_ptr(),
                      workspace.numel() * workspace.element_size())

    def launch(self, stream: Optional[int] = None) -> None:
        if stream is None:
            stream = torch.cuda.current_stream(self.status.device).cuda_stream
        _check(self._fn(*self._args, stream))


def replay_to_device(state, trace, device="cuda"):
    """Moves a host replay (numpy, as workloads.traces.generate returns) to the GPU."""
    import numpy as np

    def t(a, dt, view=None):
        a = np.ascontiguousarray(a, dtype=dt)
        return torch.from_numpy(a.view(view) if view else a).to(device)

    st = {"size": t(state["size"], np.uint64, np.int64), "cost": t(state["cost"], np.uint64, np.int64),
          "kind": t(state["kind"], np.uint8), "id": t(state["id"], np.uint32, np.int32),
          "len": t(state["len"], np.uint64, np.int64), "capacity": int(state["capacity"])}
    tr = {"op": t(trace["op"], np.uint8), "op_id": t(trace["op_id"], np.uint32, np.int32),
          "op_size": t(trace["op_size"], np.uint64, np.int64),
          "op_cost": t(trace["op_cost"], np.uint64, np.int64),
          "op_flags": t(trace["op_flags"], np.uint8)}
    return st, tr


def to_device(pools, device="cuda"):
    """Moves a host batch (numpy arrays, e.g. workloads.Pools) to the GPU as
    the tensors window_search takes."""
    import numpy as np

    def u64(a):
        return torch.from_numpy(np.ascontiguousarray(a, dtype=np.uint64).view(np.int64)).to(device)

    return (u64(pools.size), u64(pools.cost),
            torch.from_numpy(np.ascontiguousarray(pools.kind, dtype=np.uint8)).to(device),
            u64(pools.seg_offsets), u64(pools.req_sizes), u64(pools.req_offsets))


__all__ = ["COOP_EVICTABLE", "COOP_FREE", "COOP_PINNED", "CoopError", "FirstFit",
           "INFEASIBLE", "LIBRARY", "POLICY_GREEDY", "POLICY_WINDOW", "Replay", "WindowSearch",
           "first_fit", "first_fit_workspace_size", "load_library", "plan_info",
           "real_workspace_size", "replay_to_device", "replay_workspace_size", "static_capacity",
           "to_device", "window_search", "window_search_static", "WindowSearchReal",
           "workspace_size"]
