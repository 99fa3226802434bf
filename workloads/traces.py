"""Seeded synthetic allocation traces for the Algorithm 1 replay.

This module only draws inputs (pools and operation sequences); it holds none
of the replay or search arithmetic.  Shapes follow the paper's setting:

* a pool holds a fixed budget of bytes; the parameters are unevictable
  tensors allocated at its two ends (section 3.4), the rest starts as one
  free chunk;
* a training iteration runs a forward pass that allocates one activation
  per layer, then a backward pass that, layer by layer from the last,
  allocates a gradient of the same size, releases the layer's activation and
  then the gradient;
* layers repeat a GPT-2-like pattern (matmul, layer norm, GELU) or a
  ResNet-like one (conv, ReLU); matmul and conv are super-linear (class C1,
  expensive: placed at the left end of a chunk), the others linear (C2,
  cheap: right end);
* eviction costs are the operation's cost density times the tensor size,
  with Table 1's densities (us per MB), stored as integer nanoseconds.

Operation encoding (one row per operation): op 0 allocate, 1 release;
op_flags bit 0 expensive, bit 1 unevictable.
"""
from __future__ import annotations

import dataclasses

import numpy as np

MiB = 1 << 20
GRAIN = 512

# Table 1 cost densities, us per MB: (GPT-2 column, ResNet-50 column)
DENSITY = {"matmul": 33.5, "layernorm": 4.2, "gelu": 3.8, "conv": 35.6, "relu": 3.9}
EXPENSIVE = {"matmul", "conv"}
PATTERNS = {"gpt": ("matmul", "layernorm", "gelu"), "resnet": ("conv", "relu")}


@dataclasses.dataclass(frozen=True)
class TraceSpec:
    name: str
    num_pools: int
    layers: int
    iterations: int
    pattern: str = "gpt"
    act_lo: int = 1 * MiB          # activation sizes: log-uniform, rounded up to 512 B
    act_hi: int = 64 * MiB
    budget_frac: float = 0.6       # free bytes / one forward pass's activation bytes
    params: int = 4                # unevictable blocks at each end
    param_lo: int = 4 * MiB
    param_hi: int = 256 * MiB


REPLAY_CONFIGS = (
    TraceSpec("tiny replay", 4, 12, 2),
    TraceSpec("mid replay", 64, 96, 2, budget_frac=0.85),
    TraceSpec("training replay", 512, 1024, 1, budget_frac=0.85),
)


def _round_up(x):
    return ((x + GRAIN - 1) // GRAIN) * GRAIN


def generate(spec: TraceSpec, seed: int = 0):
    """Returns (state, trace) as numpy arrays in the layout oracle.replay
    and the GPU replay take."""
    rng = np.random.default_rng([0x7e, spec.layers, seed])
    P, L, it = spec.num_pools, spec.layers, spec.iterations
    pattern = PATTERNS[spec.pattern]
    T = it * 4 * L
    cap = 2 * spec.params + 2 * L + 16
    size = np.zeros(P * cap, np.uint64)
    cost = np.zeros(P * cap, np.uint64)
    kind = np.full(P * cap, 2, np.uint8)   # unused slots: empty unevictable blocks
    ids = np.zeros(P * cap, np.uint32)
    lens = np.zeros(P, np.uint64)
    op = np.zeros(P * T, np.uint8)
    op_id = np.zeros(P * T, np.uint32)
    op_size = np.zeros(P * T, np.uint64)
    op_cost = np.zeros(P * T, np.uint64)
    op_flags = np.zeros(P * T, np.uint8)
    ln_lo, ln_hi = np.log(spec.act_lo), np.log(spec.act_hi)
    for b in range(P):
        acts = np.array([_round_up(int(np.exp(ln_lo + rng.random() * (ln_hi - ln_lo))))
                         for _ in range(L)], dtype=np.uint64)
        params = [_round_up(int(np.exp(np.log(spec.param_lo) + rng.random() *
                                       (np.log(spec.param_hi) - np.log(spec.param_lo)))))
                  for _ in range(2 * spec.params)]
        free = _round_up(int(spec.budget_frac * int(acts.sum())))
        blocks = params[:spec.params] + [free] + params[spec.params:]
        n = len(blocks)
        base = b * cap
        size[base:base + n] = blocks
        kind[base:base + n] = 2
        kind[base + spec.params] = 0
        ids[base:base + n] = list(range(1, spec.params + 1)) + [0] + \
            list(range(spec.params + 1, 2 * spec.params + 1))
        lens[b] = n
        t = b * T
        nid = 2 * spec.params + 1
        for _ in range(it):
            act_ids = []
            for l in range(L):
                kind_op = pattern[l % len(pattern)]
                s = int(acts[l])
                op[t], op_id[t], op_size[t] = 0, nid, s
                op_cost[t] = int(round(DENSITY[kind_op] * s / MiB * 1000))
                op_flags[t] = 1 if kind_op in EXPENSIVE else 0
                act_ids.append(nid)
                nid += 1
                t += 1
            for l in reversed(range(L)):
                kind_op = pattern[l % len(pattern)]
                s = int(acts[l])
                op[t], op_id[t], op_size[t] = 0, nid, s
                op_cost[t] = int(round(DENSITY[kind_op] * s / MiB * 1000))
                op_flags[t] = 1 if kind_op in EXPENSIVE else 0
                t += 1
                op[t], op_id[t] = 1, act_ids[l]
                t += 1
                op[t], op_id[t] = 1, nid
                nid += 1
                t += 1
        assert t == (b + 1) * T
    state = {"size": size, "cost": cost, "kind": kind, "id": ids, "len": lens, "capacity": cap}
    trace = {"op": op, "op_id": op_id, "op_size": op_size, "op_cost": op_cost,
             "op_flags": op_flags, "num_ops": T}
    return state, trace


def make_replay(k: int, seed: int = 0, **overrides):
    spec = REPLAY_CONFIGS[k]
    if overrides:
        spec = dataclasses.replace(spec, **overrides)
    return generate(spec, seed)
