"""Benchmark of the batched sliding-window eviction search on one MI355X.

A step is one coop_window_search call: every request of one batch of
synthetic pool snapshots, inputs already resident in HBM (--op first_fit:
one coop_first_fit call on the same batch instead).  The headline workload
is the ragged heavy-tailed batch (4096 snapshots of 64..32768 blocks, four
requests each, about 66 M blocks), the largest batch; the batched mid pools,
the large pools with 16 requests each and the single huge pool are timed in
the same run and reported under per_config.  To measure HBM rather than the
256 MB Infinity Cache, the
batch is replicated into enough distinct device buffers that consecutive
steps never find their inputs cached (each copy is revisited only after
more than twice the cache size has been streamed); --copies 1 gives the
warm-cache number.

Prints one JSON line (rank 0): queries/s as `value`, blocks scanned/s, the
HBM roofline of the search kernel (algorithmic bytes per launch, counted per
request, / average launch time, timed with HIP events on the launch stream),
the fraction of compulsory bytes (every block once), an integer-arithmetic
roofline, and the CPU oracle timed on this host as a reported baseline.
"""
import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "eviction-window queries/sec and blocks scanned/sec; % of HBM roofline"
FIT_METRIC = "first-fit queries/sec; % of HBM roofline"
REPLAY_METRIC = "Algorithm 1 replay: allocator operations/sec over independent pools"
PEAK_HBM_GBS = 8000.0          # MI355X HBM3E, published
INFINITY_CACHE_BYTES = 256 << 20
KERNEL = "coop_window_search_kernel"
HEADLINE_CONFIG = 3   # the ragged heavy-tailed batch: the largest batch
KERNEL_SOURCE = os.path.join(ROOT, "paper_2311_00591_amd", "csrc", "coop_window_search.hip")


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", type=int, default=None,
                    help="standard workload index 0..4 (default: the ragged batch, 3, as the "
                         "headline, with --extra-configs timed in the same run)")
    ap.add_argument("--extra-configs", default="1,2,4",
                    help="window search without --config: further workloads timed after the "
                         "headline and reported under per_config")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--copies", type=int, default=0,
                    help="distinct device copies of the batch (0: enough to defeat the cache)")
    ap.add_argument("--cpu-seconds", type=float, default=8.0,
                    help="CPU-oracle budget for the headline workload, half of it for each "
                         "further one (0: no CPU baseline)")
    ap.add_argument("--no-parity", action="store_true")
    ap.add_argument("--medians", action="store_true",
                    help="window search: after the timed region, also time single launches "
                         "(medians, cold and warm cache)")
    ap.add_argument("--policy", choices=["window", "greedy"], default="window",
                    help="replay eviction policy timed by --op replay: Coop's sliding window "
                         "or the DTR-style greedy baseline")
    ap.add_argument("--op", choices=["window", "first_fit", "replay", "real", "long"], default="window",
                    help="window: the eviction-window search; first_fit: the free-chunk "
                         "lookup that precedes it; replay: Algorithm 1 over training traces "
                         "(--config picks the trace set)")
    return ap.parse_args()


def workload_bytes(pools):
    """Algorithmic bytes of one pass: every request reads its snapshot's
    size (8 B), cost (8 B) and kind (1 B) per block, its S (8 B), and writes
    its 24-byte result."""
    nb = np.diff(pools.seg_offsets.astype(np.int64))
    R = np.diff(pools.req_offsets.astype(np.int64))
    block_queries = int((nb * R).sum())
    return block_queries, 17 * block_queries + 32 * pools.num_requests, \
        17 * pools.num_blocks + 32 * pools.num_requests


FIT_SOURCE = os.path.join(ROOT, "paper_2311_00591_amd", "csrc", "coop_first_fit.hip")


def fit_bytes(pools):
    """Algorithmic bytes of one batched first fit: size (8 B) and kind (1 B)
    of every block once, whatever the number of requests, plus S (8 B) and
    the 8-byte result per request."""
    return 9 * pools.num_blocks + 16 * pools.num_requests


def per_launch_ms(launch, count, stream):
    """Milliseconds of each of `count` launches, timed one by one with events
    on `stream` (outside the timed region; for medians)."""
    import torch
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(count)]
    for i, (a, b) in enumerate(evs):
        a.record(stream)
        launch(i)
        b.record(stream)
    torch.cuda.synchronize()
    return [a.elapsed_time(b) for a, b in evs]


def copy_ceiling(dev, nbytes=1 << 30, reps=10):
    """Measured HBM ceiling: GB/s (bytes read + bytes written) of a plain
    device-to-device copy of `nbytes`, timed with events over `reps` copies
    after one warm-up; the buffers are 4x the Infinity Cache, so every copy
    streams from HBM."""
    import torch
    a = torch.empty(nbytes, dtype=torch.uint8, device=dev)
    b = torch.empty(nbytes, dtype=torch.uint8, device=dev)
    a.fill_(1)
    b.copy_(a)
    torch.cuda.synchronize()
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(reps):
        b.copy_(a)
    stop.record()
    torch.cuda.synchronize()
    gbs = 2 * nbytes * reps / (start.elapsed_time(stop) / 1e3) / 1e9
    del a, b
    torch.cuda.empty_cache()
    return gbs


def source_digest(source=None):
    """First 16 hex digits of the sha256 of a kernel's source file."""
    with open(source or KERNEL_SOURCE, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def _profile_record(workload_name):
    """This workload's entry of the committed rocprofv3 counter summary
    (profiles/pmc_traffic.json), if it was taken on the current kernel source."""
    path = os.path.join(ROOT, "profiles", "pmc_traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        data = json.load(f)
    rec = data.get(workload_name)
    if not rec or rec.get("source_digest") != source_digest():
        return None
    return rec


def measured_traffic(workload_name):
    """HBM bytes per launch (FETCH_SIZE + WRITE_SIZE, calibrated) from the
    committed counter summary, if it was taken on the current kernel source."""
    rec = _profile_record(workload_name)
    return rec.get("bytes_per_launch") if rec else None


# Issue peak of the vector ALU: 256 CUs x 4 SIMDs x 2.4 GHz, a wave64
# instruction occupying a 16-lane SIMD for 4 cycles.
PEAK_VALU_ISSUE = 256 * 4 * 2.4e9 / 4


def valu_issue(workload_name, block_queries, t):
    """The search kernel's VALU roofline: its wavefront instructions per
    launch (SQ_INSTS_VALU from the committed counter summary, current kernel
    source only) over this run's time per call, against the issue peak."""
    rec = _profile_record(workload_name)
    if not rec or not rec.get("valu_insts_per_launch"):
        return None
    n = rec["valu_insts_per_launch"]
    return {"bound": "valu_issue", "achieved": n / t, "peak": PEAK_VALU_ISSUE,
            "unit": "wavefront instructions/s", "frac": n / t / PEAK_VALU_ISSUE,
            "insts_per_launch": n, "insts_per_block_query": n / block_queries,
            "source": rec.get("profile")}


def cpu_baseline(pools, target_s, op="window", h=None):
    import oracle
    try:
        threads = len(os.sched_getaffinity(0))
    except AttributeError:
        threads = os.cpu_count() or 1
    threads = max(1, min(threads, 64))
    if op == "window":
        args = pools.arrays()
        fn, what = oracle.window_search, "two-pointer sweep"
    elif op == "real":
        args = (pools.size, h, pools.kind, pools.seg_offsets, pools.req_sizes, pools.req_offsets)
        fn, what = oracle.window_search_real, "two-pointer sweep, 128-bit fixed-point costs"
    else:
        args = (pools.size, pools.kind, pools.seg_offsets, pools.req_sizes, pools.req_offsets)
        fn, what = oracle.first_fit, "left-to-right walk per request"
    t0 = time.perf_counter()
    fn(*args, threads=threads)
    one = time.perf_counter() - t0
    reps = max(1, min(1000, int(target_s / max(one, 1e-6))))
    t0 = time.perf_counter()
    for _ in range(reps):
        fn(*args, threads=threads)
    dt = time.perf_counter() - t0
    # one thread, on the whole workload when that takes under a quarter of
    # the budget, else not measured
    single = None
    if one * threads < target_s / 4:
        t0 = time.perf_counter()
        fn(*args, threads=1)
        single = pools.num_requests / (time.perf_counter() - t0)
    return {"value": reps * pools.num_requests / dt, "unit": "queries/s", "cores": threads,
            "kind": "oracle", "single_thread_value": single, "cpu_model": _cpu_model(),
            "sample": f"whole workload ({pools.num_requests} requests) x {reps} passes, "
                      f"{dt:.1f} s, {what}, {threads} threads"}


def _cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def sub_requests(pools, idx):
    """The batch with only requests idx (sorted indices into req_sizes): same
    blocks and snapshots, req_offsets recounted."""
    import workloads
    idx = np.asarray(idx, dtype=np.int64)
    roff = np.searchsorted(idx, pools.req_offsets.astype(np.int64), side="left").astype(np.uint64)
    return workloads.Pools(pools.size, pools.cost, pools.kind, pools.seg_offsets,
                           pools.req_sizes[idx], roff)


def _threads():
    try:
        threads = len(os.sched_getaffinity(0))
    except AttributeError:
        threads = os.cpu_count() or 1
    return max(1, min(threads, 64))


def _even_sample(n, m):
    """m evenly spaced indices of range(n) (all of them when m >= n)."""
    if m >= n:
        return np.arange(n, dtype=np.int64)
    return np.unique((np.arange(m, dtype=np.float64) * n / m).astype(np.int64))


def oracle_window_timed(pools, budget_s, threads):
    """The oracle's answers and its rate on this host: whole passes over the
    batch when one pass fits the budget, else an evenly spaced sample of
    requests sized to it.  Returns (request indices answered, their oracle
    results, CPU-baseline record)."""
    import oracle
    Q = pools.num_requests
    # two probes separate the per-call cost (a pass over the blocks) from
    # the per-request cost
    times = []
    for m0 in (max(1, min(Q, 8 * threads)), max(1, min(Q, 32 * threads))):
        probe = _even_sample(Q, m0)
        t0 = time.perf_counter()
        oracle.window_search(*sub_requests(pools, probe).arrays(), threads=threads)
        times.append((len(probe), time.perf_counter() - t0))
    (m1_, t1_), (m2_, t2_) = times
    per_req = max((t2_ - t1_) / (m2_ - m1_) if m2_ > m1_ else t2_ / m2_, t2_ / m2_ / 8, 1e-9)
    fixed = max(0.0, t2_ - per_req * m2_)
    m = Q if fixed + per_req * Q <= budget_s else max(m2_, int((budget_s - fixed) / per_req))
    idx = _even_sample(Q, m)
    batch = pools if len(idx) == Q else sub_requests(pools, idx)
    t0 = time.perf_counter()
    want = oracle.window_search(*batch.arrays(), threads=threads)
    dt = time.perf_counter() - t0
    passes = 1
    if len(idx) == Q and dt < budget_s / 2:
        passes += max(0, min(1000, int((budget_s - dt) / max(dt, 1e-6))))
        t0 = time.perf_counter()
        for _ in range(passes - 1):
            oracle.window_search(*batch.arrays(), threads=threads)
        dt += time.perf_counter() - t0
    # one thread, on an evenly spaced sample taking about a quarter of the budget
    m1 = max(1, min(Q, int(budget_s / 4 / max(per_req * threads, 1e-9))))
    s1 = sub_requests(pools, _even_sample(Q, m1))
    t0 = time.perf_counter()
    oracle.window_search(*s1.arrays(), threads=1)
    d1 = time.perf_counter() - t0
    what = (f"whole workload ({Q} requests) x {passes} passes" if len(idx) == Q else
            f"{len(idx)} of {Q} requests, evenly spaced")
    cpu = {"value": passes * len(idx) / dt, "unit": "queries/s", "cores": threads,
           "kind": "oracle", "single_thread_value": s1.num_requests / d1,
           "cpu_model": _cpu_model(),
           "sample": f"{what}, {dt:.1f} s, two-pointer sweep, {threads} threads; one thread: "
                     f"{s1.num_requests} requests evenly spaced, {d1:.1f} s"}
    return idx, want, cpu


# Peak of the u64 lane operations the search needs (see alu_ops): 256 CUs x
# 4 SIMDs x 16 lanes x 2.4 GHz, one 32-bit or single-instruction 64-bit
# lane operation per lane and cycle (no packed forms).
PEAK_ALU_TOPS = 256 * 4 * 16 * 2.4e9 / 1e12
ALU_OPS_PER_BLOCK_QUERY = 8


def alu_ops(block_queries):
    """Algorithmic integer operations of one pass: per block and request the
    start's target (an add) and its end search (two compares: every start
    and every end key is met once by a two-pointer sweep), the window's cost
    and bytes (two subtractions), and its place in the ranking (two compares
    on cost and bytes, one on the run): 8 u64 operations.  The prefix sums
    (two adds per block) are shared by the snapshot's requests and left out."""
    return ALU_OPS_PER_BLOCK_QUERY * block_queries


def bench_window_config(k, args, dev, cpu_budget, steps, warmup):
    """One workload: parity with the oracle, warm-up, `steps` timed calls,
    rooflines and the oracle's rate.  Returns the record (without the
    top-level contract keys)."""
    import torch

    import paper_2311_00591_amd as coop
    import workloads

    spec = workloads.CONFIGS[k]
    pools = workloads.make_config(k, args.seed)
    block_queries, alg_bytes, unique_bytes = workload_bytes(pools)
    batch_dev_bytes = 17 * pools.num_blocks + 16 * pools.num_segments + 8 * pools.num_requests
    copies = args.copies or max(1, -(-2 * INFINITY_CACHE_BYTES // batch_dev_bytes) + 1)

    base = coop.to_device(pools, dev)
    out = torch.empty((pools.num_requests, 3), dtype=torch.int64, device=dev)
    ws_bytes = coop.workspace_size(pools.num_blocks, pools.num_segments, pools.num_requests)
    workspace = torch.empty(max(ws_bytes, 1), dtype=torch.uint8, device=dev)
    calls = []
    for c in range(copies):
        t = base if c == 0 else tuple(x.clone() for x in base)
        calls.append(coop.WindowSearch(*t, out=out, workspace=workspace))
    torch.cuda.synchronize()

    stream = torch.cuda.current_stream(dev)
    sh = stream.cuda_stream
    parity = parity_sample = cpu = None
    threads = _threads()
    if not args.no_parity or cpu_budget > 0:
        calls[0].launch(sh)
        torch.cuda.synchronize()
        got = out.cpu().numpy().view(np.uint64)
        idx, want, cpu = oracle_window_timed(pools, max(cpu_budget, 1.0), threads)
        parity = bool(np.array_equal(got[idx], want))
        parity_sample = ("every request" if len(idx) == pools.num_requests else
                         f"{len(idx)} of {pools.num_requests} requests, evenly spaced")
        if cpu_budget <= 0:
            cpu = None
        if args.no_parity:
            parity = parity_sample = None

    for i in range(warmup):
        calls[i % copies].launch(sh)
    torch.cuda.synchronize()

    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    w0 = time.perf_counter()
    start.record(stream)
    for i in range(steps):
        calls[i % copies].launch(sh)
    stop.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    ms = start.elapsed_time(stop) / steps
    t = ms / 1e3

    achieved = alg_bytes / t / 1e9
    ops = alu_ops(block_queries)
    alu = {"bound": "alu", "achieved": ops / t / 1e12, "peak": PEAK_ALU_TOPS, "unit": "TOP/s",
           "frac": ops / t / 1e12 / PEAK_ALU_TOPS, "ops_per_launch": ops,
           "ops_per_block_query": ALU_OPS_PER_BLOCK_QUERY}
    hbm = {"bound": "hbm", "achieved": achieved, "peak": PEAK_HBM_GBS, "unit": "GB/s",
           "frac": achieved / PEAK_HBM_GBS, "traffic": measured_traffic(spec.name),
           "algorithmic_bytes_per_launch": alg_bytes,
           "bytes_counted": "per request: 17 B per block of its snapshot + 32 B",
           "compulsory_frac": unique_bytes / t / 1e9 / PEAK_HBM_GBS,
           "compulsory_bytes_per_launch": unique_bytes}
    # Where the staged tiles serve so many requests that the per-request
    # count passes the HBM peak, the bound is the integer arithmetic.
    if achieved > PEAK_HBM_GBS:
        roofline = dict(alu, per_request_hbm=hbm)
    else:
        roofline = dict(hbm, alu=alu)
    roofline["kernel"] = KERNEL
    roofline["valu_issue"] = valu_issue(spec.name, block_queries, t)
    single = None
    if args.medians:
        n_each = max(20, steps)
        cold_each = per_launch_ms(lambda i: calls[i % copies].launch(sh), n_each, stream)
        warm_each = per_launch_ms(lambda i: calls[0].launch(sh), n_each, stream)
        single = {"count": n_each, "median_cold": float(np.median(cold_each)),
                  "median_warm": float(np.median(warm_each)), "min_cold": float(np.min(cold_each))}
    nb = np.diff(pools.seg_offsets.astype(np.int64))
    rec = {
        "workload": f"{spec.name}: B={pools.num_segments} snapshots, "
                    f"N_b={int(nb.min())}..{int(nb.max())} blocks, "
                    f"{pools.num_requests} requests (standard workload {k})",
        "config_index": k,
        "value": pools.num_requests / t,
        "unit": "queries/s",
        "ms_per_step": ms,
        "steps": steps,
        "warmup": warmup,
        "num_segments": pools.num_segments,
        "num_blocks": pools.num_blocks,
        "num_requests": pools.num_requests,
        "seed": args.seed,
        "input_sha256": pools.digest()[:16],
        "resident_copies": copies,
        "cache": "cold" if copies > 1 else "warm",
        "blocks_scanned_per_s": block_queries / t,
        "hbm_roofline_pct": 100.0 * achieved / PEAK_HBM_GBS,
        "compulsory_hbm_pct": 100.0 * unique_bytes / t / 1e9 / PEAK_HBM_GBS,
        "roofline": roofline,
        "cpu_baseline": cpu,
        "parity_vs_oracle": parity,
        "parity_sample": parity_sample,
        "wall_s_timed_region": wall,
        "single_launch_ms": single,
    }
    del calls, base, out, workspace
    torch.cuda.empty_cache()
    return rec


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py: the search runs on one GPU only (asked for {args.gpus}); "
              "sharding across GPUs is not implemented", file=sys.stderr)
        sys.exit(2)

    import torch

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    if args.op == "replay":
        return bench_replay(args, dev)
    if args.op == "long":
        return bench_long(args, dev)
    import workloads
    if args.op in ("first_fit", "real"):
        k = HEADLINE_CONFIG if args.config is None else args.config
        pools = workloads.make_config(k, args.seed)
        spec = workloads.CONFIGS[k]
        if args.op == "first_fit":
            return bench_first_fit(args, pools, spec, dev, k)
        return bench_real(args, pools, spec, dev, k)

    # The window search: the headline workload, then (by default) the other
    # batched workloads in the same run, each timed the same way.
    head_k = HEADLINE_CONFIG if args.config is None else args.config
    extra = [] if args.config is not None else [int(x) for x in args.extra_configs.split(",") if x]
    head = bench_window_config(head_k, args, dev, args.cpu_seconds, args.steps, args.warmup)
    per_config = {}
    for k in extra:
        if k == head_k:
            continue
        steps = args.steps if k != 4 else max(1, min(args.steps, 10))
        warmup = args.warmup if k != 4 else max(1, min(args.warmup, 2))
        per_config[f"config{k}"] = bench_window_config(k, args, dev, args.cpu_seconds / 2,
                                                       steps, warmup)
    ceiling = copy_ceiling(dev)
    for r in [head, *per_config.values()]:
        rf = r["roofline"]
        hb = rf if rf["bound"] == "hbm" else rf["per_request_hbm"]
        hb["copy_ceiling"] = ceiling
        hb["frac_of_copy_ceiling"] = hb["achieved"] / ceiling
    rec = {
        "metric": METRIC,
        "value": head["value"],
        "unit": "queries/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": head["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u64",
        "data": "synthetic",
        "config": {k2: head[k2] for k2 in ("workload", "num_segments", "num_blocks",
                                             "num_requests", "seed", "input_sha256",
                                             "resident_copies", "cache")},
        "blocks_scanned_per_s": head["blocks_scanned_per_s"],
        "hbm_roofline_pct": head["hbm_roofline_pct"],
        "compulsory_hbm_pct": head["compulsory_hbm_pct"],
        "roofline": head["roofline"],
        "cpu_baseline": head["cpu_baseline"],
        "parity_vs_oracle": head["parity_vs_oracle"],
        "parity_sample": head["parity_sample"],
        "wall_s_timed_region": head["wall_s_timed_region"],
        "single_launch_ms": head["single_launch_ms"],
        "per_config": per_config,
        "kernel_source": source_digest(),
    }
    print(json.dumps(rec), flush=True)


LONG_METRIC = "long-window search on one 2^24-block pinned-free run: microseconds per request"


def bench_long(args, dev):
    """Windows far longer than a tile: one pool of 2^24 blocks laid out as
    section 3.5 describes (parameters pinned at both ends, one pinned-free
    run between them), four request sets (workloads.long_run), each timed as
    `steps` calls after `warmup`, with parity against the oracle on every
    request.  Prints one JSON line; `value` is the spread set's microseconds
    per request."""
    import torch

    import oracle
    import paper_2311_00591_amd as coop
    import workloads

    sets = {}
    digest = None
    for name in workloads.LONG_RUN_SETS:
        pools = workloads.long_run(request_set=name)
        batch_dev_bytes = 17 * pools.num_blocks + 16 * pools.num_segments + 8 * pools.num_requests
        copies = args.copies or max(1, -(-2 * INFINITY_CACHE_BYTES // batch_dev_bytes) + 1)
        base = coop.to_device(pools, dev)
        out = torch.empty((pools.num_requests, 3), dtype=torch.int64, device=dev)
        ws = torch.empty(max(coop.workspace_size(pools.num_blocks, pools.num_segments,
                                                 pools.num_requests), 1), dtype=torch.uint8, device=dev)
        calls = [coop.WindowSearch(*(base if c == 0 else tuple(x.clone() for x in base)),
                                   out=out, workspace=ws) for c in range(copies)]
        torch.cuda.synchronize()
        stream = torch.cuda.current_stream(dev)
        sh = stream.cuda_stream
        parity = None
        if not args.no_parity:
            calls[0].launch(sh)
            torch.cuda.synchronize()
            got = out.cpu().numpy().view(np.uint64)
            want = oracle.window_search(*pools.arrays(), threads=_threads())
            parity = bool(np.array_equal(got, want))
        for i in range(args.warmup):
            calls[i % copies].launch(sh)
        torch.cuda.synchronize()
        start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        start.record(stream)
        for i in range(args.steps):
            calls[i % copies].launch(sh)
        stop.record(stream)
        torch.cuda.synchronize()
        ms = start.elapsed_time(stop) / args.steps
        sets[name] = {"requests": pools.num_requests, "ms_per_call": ms,
                      "us_per_request": ms * 1e3 / pools.num_requests,
                      "request_bytes": [int(x) for x in pools.req_sizes],
                      "parity_vs_oracle": parity, "resident_copies": copies,
                      "input_sha256": pools.digest()[:16]}
        digest = digest or pools.digest()[:16]
        del calls, base, out, ws
        torch.cuda.empty_cache()
    head = sets["spread"]
    print(json.dumps({
        "metric": LONG_METRIC, "value": head["us_per_request"], "unit": "us/request",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": head["ms_per_call"],
        "higher_is_better": False, "scaling": "weak", "vs_baseline": None, "dtype": "u64",
        "data": "synthetic",
        "config": {"workload": "one snapshot of 2^24 blocks, parameters pinned at both ends, "
                               "16 requests from one block to the whole run (workloads.long_run)"},
        "sets": sets, "parity_vs_oracle": all(v["parity_vs_oracle"] is not False for v in sets.values()),
        "kernel_source": source_digest()}), flush=True)


def bench_first_fit(args, pools, spec, dev, k):
    import torch

    import paper_2311_00591_amd as coop

    alg_bytes = fit_bytes(pools)
    batch_dev_bytes = 9 * pools.num_blocks + 16 * pools.num_segments + 8 * pools.num_requests
    copies = args.copies or max(1, -(-2 * INFINITY_CACHE_BYTES // batch_dev_bytes) + 1)
    size, _, kind, seg, req, roff = coop.to_device(pools, dev)
    out = torch.empty(pools.num_requests, dtype=torch.int64, device=dev)
    workspace = torch.empty(max(coop.first_fit_workspace_size(pools.num_blocks), 1),
                            dtype=torch.uint8, device=dev)
    calls = []
    for c in range(copies):
        t = (size, kind) if c == 0 else (size.clone(), kind.clone())
        calls.append(coop.FirstFit(*t, seg, req, roff, out=out, workspace=workspace))
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream(dev)
    sh = stream.cuda_stream
    parity = None
    if not args.no_parity:
        import oracle
        calls[0].launch(sh)
        torch.cuda.synchronize()
        got = out.cpu().numpy().view(np.uint64)
        want = oracle.first_fit(pools.size, pools.kind, pools.seg_offsets, pools.req_sizes,
                                pools.req_offsets, threads=16)
        parity = bool(np.array_equal(got, want))
    for i in range(args.warmup):
        calls[i % copies].launch(sh)
    torch.cuda.synchronize()
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    w0 = time.perf_counter()
    start.record(stream)
    for i in range(args.steps):
        calls[i % copies].launch(sh)
    stop.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    ms = start.elapsed_time(stop) / args.steps
    t = ms / 1e3
    achieved = alg_bytes / t / 1e9
    cpu = cpu_baseline(pools, args.cpu_seconds, "first_fit") if args.cpu_seconds > 0 else None
    nb = np.diff(pools.seg_offsets.astype(np.int64))
    rec = {
        "metric": FIT_METRIC,
        "value": pools.num_requests / t,
        "unit": "queries/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u64",
        "data": "synthetic",
        "config": {
            "workload": f"first fit on {spec.name}: B={pools.num_segments} snapshots, "
                        f"N_b={int(nb.min())}..{int(nb.max())} blocks, "
                        f"{pools.num_requests} requests (standard workload {k})",
            "num_segments": pools.num_segments,
            "num_blocks": pools.num_blocks,
            "num_requests": pools.num_requests,
            "seed": args.seed,
            "input_sha256": pools.digest()[:16],
            "resident_copies": copies,
            "cache": "cold" if copies > 1 else "warm",
        },
        "hbm_roofline_pct": 100.0 * achieved / PEAK_HBM_GBS,
        "roofline": {
            "kernel": "first_fit_summary_kernel + first_fit_search_kernel (one call)",
            "bound": "hbm",
            "achieved": achieved,
            "peak": PEAK_HBM_GBS,
            "unit": "GB/s",
            "frac": achieved / PEAK_HBM_GBS,
            "traffic": None,
            "algorithmic_bytes_per_launch": alg_bytes,
        },
        "cpu_baseline": cpu,
        "parity_vs_oracle": parity,
        "wall_s_timed_region": wall,
        "kernel_source": source_digest(FIT_SOURCE),
    }
    print(json.dumps(rec), flush=True)


REAL_SOURCE = os.path.join(ROOT, "paper_2311_00591_amd", "csrc", "coop_window_search_real.hip")


def bench_real(args, pools, spec, dev, k):
    """The search with real-valued heuristics h = cost / staleness on a
    standard workload: same metric and byte accounting as the integer
    search (17 B per block and request: size, h, kind), timed per call."""
    import torch

    import paper_2311_00591_amd as coop
    import workloads

    h = workloads.real_costs(pools, args.seed)
    block_queries, alg_bytes, unique_bytes = workload_bytes(pools)
    alg_bytes += 8 * pools.num_requests  # the 40-byte result instead of 24 (plus 8 B of S)
    batch_dev_bytes = 17 * pools.num_blocks + 16 * pools.num_segments + 8 * pools.num_requests
    copies = args.copies or max(1, -(-2 * INFINITY_CACHE_BYTES // batch_dev_bytes) + 1)
    size, _, kind, seg, req, roff = coop.to_device(pools, dev)
    ht = torch.from_numpy(h).to(dev)
    ws = torch.empty(max(coop.real_workspace_size(pools.num_blocks, pools.num_segments,
                                                  pools.num_requests), 1),
                     dtype=torch.uint8, device=dev)
    calls = []
    for c in range(copies):
        t = (size, ht, kind) if c == 0 else (size.clone(), ht.clone(), kind.clone())
        calls.append(coop.WindowSearchReal(*t, seg, req, roff, workspace=ws))
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream(dev)
    sh = stream.cuda_stream
    parity = None
    status = None
    if not args.no_parity:
        import oracle
        calls[0].launch(sh)
        torch.cuda.synchronize()
        out = calls[0].out.cpu().numpy()
        status = int(calls[0].status.item())
        want, want_cost = oracle.window_search_real(pools.size, h, pools.kind, pools.seg_offsets,
                                                    pools.req_sizes, pools.req_offsets,
                                                    threads=16)
        parity = bool(np.array_equal(out[:, :4].view(np.uint64), want) and
                      np.array_equal(out[:, 4].copy().view(np.uint64), want_cost.view(np.uint64))
                      and status == 0)
    for i in range(args.warmup):
        calls[i % copies].launch(sh)
    torch.cuda.synchronize()
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    w0 = time.perf_counter()
    start.record(stream)
    for i in range(args.steps):
        calls[i % copies].launch(sh)
    stop.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    ms = start.elapsed_time(stop) / args.steps
    t = ms / 1e3
    achieved = alg_bytes / t / 1e9
    cpu = cpu_baseline(pools, args.cpu_seconds, "real", h) if args.cpu_seconds > 0 else None
    nb = np.diff(pools.seg_offsets.astype(np.int64))
    rec = {
        "metric": METRIC,
        "value": pools.num_requests / t,
        "unit": "queries/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f64 heuristics, u128 fixed-point sums",
        "data": "synthetic",
        "config": {
            "workload": f"real-valued heuristics on {spec.name}: B={pools.num_segments} "
                        f"snapshots, N_b={int(nb.min())}..{int(nb.max())} blocks, "
                        f"{pools.num_requests} requests, h = cost / staleness U{{1..4096}} "
                        f"(standard workload {k})",
            "num_segments": pools.num_segments,
            "num_blocks": pools.num_blocks,
            "num_requests": pools.num_requests,
            "seed": args.seed,
            "input_sha256": pools.digest()[:16],
            "resident_copies": copies,
            "cache": "cold" if copies > 1 else "warm",
        },
        "blocks_scanned_per_s": block_queries / t,
        "hbm_roofline_pct": 100.0 * achieved / PEAK_HBM_GBS,
        "roofline": {
            "kernel": "real_tile_kernel + real_offsets_kernel + real_search_kernel + "
                      "real_reduce_kernel (one call)",
            "bound": "hbm",
            "achieved": achieved,
            "peak": PEAK_HBM_GBS,
            "unit": "GB/s",
            "frac": achieved / PEAK_HBM_GBS,
            "traffic": None,
            "algorithmic_bytes_per_launch": alg_bytes,
        },
        "cpu_baseline": cpu,
        "parity_vs_oracle": parity,
        "status": status,
        "wall_s_timed_region": wall,
        "kernel_source": source_digest(REAL_SOURCE),
    }
    print(json.dumps(rec), flush=True)


def bench_replay(args, dev):
    import torch

    import paper_2311_00591_amd as coop
    from workloads import traces

    kc = 1 if args.config is None else args.config
    k = kc if kc < len(traces.REPLAY_CONFIGS) else len(traces.REPLAY_CONFIGS) - 1
    spec = traces.REPLAY_CONFIGS[k]
    state, trace = traces.make_replay(k, args.seed)
    P, cap, T = len(state["len"]), state["capacity"], trace["num_ops"]
    st0, tr = coop.replay_to_device(state, trace, dev)
    # compulsory bytes: each pool's slots read and written once (size, cost,
    # kind, id: 21 B), each operation read once (op, id, size, cost, flags:
    # 22 B) and its outcome written (block, window, cost, free: 40 B); the
    # replay is bound by its chain of dependent operations, not by these
    alg_bytes = 2 * 21 * P * cap + (22 + 40) * P * T
    policy = {"window": coop.POLICY_WINDOW, "greedy": coop.POLICY_GREEDY}[args.policy]
    stream = torch.cuda.current_stream(dev)
    sh = stream.cuda_stream
    cap_bytes = np.array([int(state["size"][b * cap:(b + 1) * cap].sum()) for b in range(P)],
                         dtype=np.float64)
    none = np.uint64(2**64 - 1)

    def run_once(pol):
        """One untimed replay under policy pol: its host outputs and summary."""
        s1 = {k2: (v.clone() if hasattr(v, "clone") else v) for k2, v in st0.items()}
        r1 = coop.Replay(s1, tr, policy=pol)
        r1.launch(sh)
        torch.cuda.synchronize()
        out = {"block": r1.block.cpu().numpy().view(np.uint64).reshape(P, T),
               "free": r1.free.cpu().numpy().view(np.uint64).reshape(P, T),
               "cost": r1.cost.cpu().numpy().view(np.uint64).reshape(P, T)}
        sampled = out["free"] != none
        failed = (out["block"] == none) & (np.asarray(trace["op"]).reshape(P, T) == 0)
        summary = {
            "eviction_events": int(sampled.sum()),
            "fragmentation_rate_mean": (float(np.mean(
                (out["free"].astype(np.float64) / cap_bytes[:, None])[sampled]))
                if sampled.any() else None),
            "evicted_cost_total": float(out["cost"].astype(np.float64).sum()),
            "failed_allocations": int(failed.sum()),
            "status": int(r1.status.item()),
        }
        return out, summary

    host, summary = run_once(policy)
    other = coop.POLICY_GREEDY if policy == coop.POLICY_WINDOW else coop.POLICY_WINDOW
    _, other_summary = run_once(other)
    by_policy = {args.policy: summary,
                 ("greedy" if other == coop.POLICY_GREEDY else "window"): other_summary}
    parity = None
    if not args.no_parity:
        import oracle
        _, want = oracle.replay(state, trace, threads=16, policy=policy)
        parity = bool(all(np.array_equal(host[k2], want[k2]) for k2 in ("block", "free", "cost")))
    st = {k2: (v.clone() if hasattr(v, "clone") else v) for k2, v in st0.items()}
    r = coop.Replay(st, tr, policy=policy)
    times = []
    for i in range(args.warmup + args.steps):
        for k2 in ("size", "cost", "kind", "id", "len"):
            st[k2].copy_(st0[k2])
        torch.cuda.synchronize()
        start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        start.record(stream)
        r.launch(sh)
        stop.record(stream)
        torch.cuda.synchronize()
        if i >= args.warmup:
            times.append(start.elapsed_time(stop))
    ms = float(np.median(times))
    t = ms / 1e3
    achieved = alg_bytes / t / 1e9
    cpu = None
    if args.cpu_seconds > 0:
        import oracle
        try:
            threads = len(os.sched_getaffinity(0))
        except AttributeError:
            threads = os.cpu_count() or 1
        threads = max(1, min(threads, 64))
        t0 = time.perf_counter()
        oracle.replay(state, trace, threads=threads, policy=policy)
        one = time.perf_counter() - t0
        reps = max(1, min(100, int(args.cpu_seconds / max(one, 1e-6))))
        t0 = time.perf_counter()
        for _ in range(reps):
            oracle.replay(state, trace, threads=threads, policy=policy)
        dt = time.perf_counter() - t0
        single = None
        if one * threads < args.cpu_seconds / 4:
            t0 = time.perf_counter()
            oracle.replay(state, trace, threads=1, policy=policy)
            single = P * T / (time.perf_counter() - t0)
        cpu = {"value": reps * P * T / dt, "unit": "operations/s", "cores": threads,
               "kind": "oracle", "single_thread_value": single, "cpu_model": _cpu_model(),
               "sample": f"whole replay ({P} pools x {T} operations) x {reps}, "
                         f"{dt:.1f} s, {threads} threads"}
    rec = {
        "metric": REPLAY_METRIC,
        "value": P * T / t,
        "unit": "operations/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u64",
        "data": "synthetic",
        "config": {
            "workload": f"{spec.name}: {P} pools x {T} operations ({spec.layers} layers, "
                        f"{spec.iterations} iteration(s), {spec.pattern} pattern), "
                        f"{cap} slots per pool",
            "num_pools": P, "num_ops": T, "capacity": cap, "seed": args.seed,
            "policy": args.policy,
        },
        "evictions": summary["eviction_events"],
        "fragmentation_rate_mean": summary["fragmentation_rate_mean"],
        "policies": by_policy,
        "roofline": {
            "kernel": "replay_resident_kernel (pools held in LDS)",
            "bound": "hbm",
            "achieved": achieved,
            "peak": PEAK_HBM_GBS,
            "unit": "GB/s",
            "frac": achieved / PEAK_HBM_GBS,
            "traffic": None,
            "algorithmic_bytes_per_launch": alg_bytes,
        },
        "cpu_baseline": cpu,
        "parity_vs_oracle": parity,
        "kernel_source": source_digest(os.path.join(ROOT, "paper_2311_00591_amd", "csrc",
                                                    "coop_replay.hip")),
    }
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
