"""Benchmark of the ALP allocation search on one MI355X.

    python bench.py [--steps K] [--warmup W] [--workload cfg3] [--no-cpu-baseline]

One step = one complete search, or batch of searches (per-option terms, exhaustive scan of
every candidate, final reduction and result decode) over the synthetic workload, with the
profile tables, the queries and the result records resident in HBM: alp_search_batch_async,
the steps queued back to back on the stream and the timed region closed by its
synchronisation.  The same searches through the host-buffer entry points (alp_search or
alp_search_batch: queries from host memory, results to mapped host memory, one synchronisation
per call) are timed after the timed region and reported under config.host_buffer_api.  For
``--workload multi`` a step is one alp_allocate_workflows call (every per-workflow budget
searched exhaustively, then the budget split; host buffers).  The default workload is the 5-LLM
space with G = 64 GPUs and 128 options per LLM (2^35 = 34,359,738,368 candidates per step).
Prints one JSON line.

``value`` = candidates evaluated per second.  ``roofline`` relates the scan kernel (the dominant
kernel) to the integer VALU peak of the chip: 2 int32 lane operations per candidate (the budget
comparison and the objective minimum update), 256 CUs x 64 lanes x 2.4 GHz = 39.32 Tlane-op/s;
the kernel duration is measured with HIP events on the stream the library launches on.
``cpu_baseline`` times the CPU oracle, single-threaded, on a bounded slice of the same space.

The paper's own pruned search (alp_search_pruned) has two workloads of its own, where a step is
one pruned search and ``value`` counts fraction vectors per second:
  ``pruned``        the 4,096-instance batch of the exhaustive ``cfg4`` workload (another
                    workload's instances with ``--config``), with the optimality gap against
                    the exhaustive results on the same instances;
  ``pruned-paper``  the point of the paper's scheduler micro-benchmark: ``--llms`` LLMs,
                    ``--budget`` GPUs, ``--fractions`` fractions per GPU (default 5, 16, 10).

``--workload place`` times alp_place (Section 6 placement) on the exhaustive search results of
a workload's instances (``--config``, default the 4,096-instance batch), and reports how many of
the searched optima, and of the pruned search's results, can be placed on the budget's 8-GPU
nodes.

``--workload stats`` times the workflow statistics (alp_trace_stats, Section 4 step 2) over
20,000 synthetic beam-search traces (about 15 million LLM calls, resident on the device);
``value`` counts trace calls per second and the roofline is HBM: 20 bytes read per call (LLM
index and two timestamps) and 8 per trace offset.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from workloads import CONFIGS, make_batch, make_custom, target_from_tmax  # noqa: E402

PEAK_LANE_OPS = 256 * 64 * 2.4e9        # int32 VALU lane-ops/s of MI355X
OPS_PER_CANDIDATE = 2                   # budget compare + objective min
# Kernel times are read from HIP events on the first and every TIME_EVERY-th timed step: an
# event-stamped dispatch costs the GPU a few microseconds of idle time, which would otherwise
# be part of every step of a small search.
TIME_EVERY = 8
# The wider count of lane-ops per candidate (add the last term, compare the budget, compare the
# best, select value and index), reported beside ``frac`` for comparison with that accounting.
OPS_PER_CANDIDATE_WIDE = 5
WORKLOADS = {"cfg2": 2, "cfg3": 3, "cfg4": 4, "cfg1": 1, "multi": 2, "pruned": 4,
             "pruned-paper": None, "stats": None, "place": 4}
HBM_PEAK = 8.0e12                       # MI355X HBM3E bytes/s
STATS_TRACES = 20_000                   # beam-search requests of the statistics workload
# Several workflows sharing one GPU pool: four 4-LLM workflows drawn like the 4-LLM workload
# split 32 GPUs under egalitarian welfare; each workflow's target is set at an even share.
MULTI_WORKFLOWS, MULTI_GPUS = 4, 32
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "scan_min_hbm_bytes.md")
KERNEL_SOURCES = ("alp_kernels.hip", "alp_device.h", "alp_internal.h")
STATS_TRAFFIC_FILE = os.path.join(ROOT, "profiles", "trace_stats_hbm_bytes.md")
STATS_SOURCES = ("alp_stats.hip", "alp_device.h", "alp_internal.h")
METRIC = "ALP candidate allocations evaluated/sec on 1 GPU"


def _traffic(kernel_digest: str, workload: str, path: str = TRAFFIC_FILE):
    """HBM bytes per launch (per call for the statistics) from a committed rocprofv3 counter
    summary, if it was taken on the current kernel source and this workload."""
    try:
        with open(path) as f:
            text = f.read()
        t = json.loads(text.split("```json", 1)[1].split("```", 1)[0])
    except (OSError, ValueError, IndexError):
        return None
    entry = t.get(workload)
    if not entry or t.get("kernel_source_sha256") != kernel_digest:
        return None
    return entry.get("bytes_per_launch")


def _kernel_digest(sources=KERNEL_SOURCES) -> str:
    """SHA-256 over the sources compiled into the measured kernels (the scan by default)."""
    import hashlib
    h = hashlib.sha256()
    for name in sources:
        with open(os.path.join(ROOT, "paper_2604_15186_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def host_cpu() -> str:
    """The host's CPU model and logical CPU count (the oracle uses one of them)."""
    model = "unknown CPU"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return f"{model}, {os.cpu_count()} logical CPUs"


def cpu_baseline(batch, G, lam, seconds: float):
    """Single-threaded oracle argmin over the first indices of instance 0, sized to ~seconds."""
    import oracle
    inst = oracle.Instance(batch, 0)
    n = 1 << 20
    t0 = time.perf_counter()
    oracle.argmin(inst, G, lam, 0, n)
    dt = time.perf_counter() - t0
    total = min(inst.N, max(n, int(n * seconds / max(dt, 1e-6))))
    t0 = time.perf_counter()
    oracle.argmin(inst, G, lam, 0, total)
    dt = time.perf_counter() - t0
    return {"value": total / dt, "unit": "candidates/s", "cores": 1, "kind": "oracle", "host": host_cpu(),
            "sample": f"first {total:,} candidate indices of the same instance, exhaustive "
                      f"single-threaded C oracle ({dt:.1f} s)"}


def cpu_baseline_pruned(batch, G, lam, seconds: float):
    """Single-threaded oracle pruned search over the batch's first instances, ~seconds."""
    import oracle
    vectors, done, t0 = 0, 0, time.perf_counter()
    while done < len(G) and time.perf_counter() - t0 < seconds:
        vectors += oracle.pruned(oracle.Instance(batch, done), int(G[done]), int(lam[done]))["vectors"]
        done += 1
    dt = time.perf_counter() - t0
    return {"value": vectors / dt, "unit": "fraction vectors/s", "cores": 1, "kind": "oracle", "host": host_cpu(),
            "sample": f"pruned search of the first {done} instances ({vectors:,} fraction "
                      f"vectors), single-threaded C oracle ({dt:.1f} s)"}


def timed_steps(step, ctx, steps: int, warmup: int):
    """Runs warmup + steps calls; returns (elapsed s, mean kernel ms [3] over the timed calls,
    the last timed call's kernel_times(), last output).  The library times the first and every
    TIME_EVERY-th step of the timed region with HIP events stamped on the kernel dispatches and
    sums the times itself, so the timed loop holds nothing but the calls."""
    import torch
    for _ in range(warmup):
        step()
    ctx.set_timing(TIME_EVERY)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        out = step()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    totals, timed = ctx.kernel_time_totals()
    avg = totals / max(1, timed)
    last = ctx.kernel_times()
    ctx.set_timing(False)
    return elapsed, avg, last, out


def gap_stats(pruned, exhaustive) -> dict:
    """Pruned results against exhaustive ones on the same queries."""
    ok_p = pruned["best"]["status"] == 0
    ok_e = exhaustive["status"] == 0
    both = ok_p & ok_e
    Lp = pruned["best"]["latency_us"].astype(np.float64)
    Le = exhaustive["latency_us"].astype(np.float64)
    worse = both & (Lp > Le)
    rel = (Lp[worse] / Le[worse] - 1.0) if worse.any() else np.zeros(0)
    return {"queries": int(len(ok_e)), "exhaustive_feasible": int(ok_e.sum()),
            "pruned_feasible": int(ok_p.sum()),
            "same_optimum": int((both & (Lp == Le)).sum()),
            "same_allocation": int((both & (pruned["best"]["index"] == exhaustive["index"])).sum()),
            "worse": int(worse.sum()), "pruned_infeasible_only": int((ok_e & ~ok_p).sum()),
            "mean_gap_when_worse": float(rel.mean()) if len(rel) else 0.0,
            "max_gap": float(rel.max()) if len(rel) else 0.0}


def paper_point(llms: int, budget: int, fractions: int):
    """Synthetic instance at the paper's scheduler micro-benchmark point: llms LLMs drawn like
    the 5-LLM workload (1B-70B parameters, Dirichlet 0.5 shares), budget GPUs, `fractions`
    share units per GPU; shares are up to 8 values spread over 1..fractions, 4 replica counts."""
    fq = sorted({max(1, round(fractions * k / 8)) for k in range(1, 9)})
    return make_custom(2604, llms, (1, 2, 4, 8), fq, 4, 8, budget, count=1, frac_den=fractions,
                       param_range=(1e9, 70e9), alpha=0.5)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="cfg3", choices=sorted(WORKLOADS))
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--variant", type=int, default=0)
    ap.add_argument("--config", type=int, default=4, choices=sorted(CONFIGS),
                    help="pruned: the workload whose instances are searched (default: the "
                         "4,096-instance batch)")
    ap.add_argument("--llms", type=int, default=5, help="pruned-paper: LLMs")
    ap.add_argument("--budget", type=int, default=16, help="pruned-paper: GPUs")
    ap.add_argument("--fractions", type=int, default=10, help="pruned-paper: fractions per GPU")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="after timing, run one plain device copy of this size (for scaling "
                         "hardware byte counters)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the search runs on a single MI355X; "
              "multi-GPU sharding is not built (run with --gpus 1)", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2604_15186_amd import alp

    if not torch.cuda.is_available():
        print("no GPU visible", file=sys.stderr)
        sys.exit(1)
    if args.workload.startswith("pruned"):
        line = run_pruned(args, alp)
    elif args.workload == "stats":
        line = run_stats(args, alp)
    elif args.workload == "place":
        line = run_place(args, alp)
    else:
        line = run_exhaustive(args, alp)
    if args.calib_copy_mib:
        src = torch.ones(args.calib_copy_mib << 20, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        line["calib_copy_bytes"] = args.calib_copy_mib << 20
    print(json.dumps(line), flush=True)


def _line(args, value, unit, elapsed, dtype_cfg, roofline, cpu):
    return {"metric": METRIC, "value": value, "unit": unit, "n_gpus": 1, "steps": args.steps,
            "warmup": args.warmup, "ms_per_step": elapsed / args.steps * 1e3,
            "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "u32",
            "data": "synthetic (seeded profile tables, see workloads/)", "config": dtype_cfg,
            "roofline": roofline, "cpu_baseline": cpu}


def run_exhaustive(args, alp):
    cfg_id = WORKLOADS[args.workload]
    cfg = CONFIGS[cfg_id]
    multi = args.workload == "multi"
    if multi:
        insts = list(range(MULTI_WORKFLOWS))
    else:
        insts = list(range(cfg.num_instances)) if cfg_id == 4 else [0]
    batch = make_batch(cfg_id, insts)
    ctx = alp.Context(batch)
    ctx.set_launch(args.variant)
    G = batch["G"]
    if multi:
        G = np.full(len(insts), MULTI_GPUS // MULTI_WORKFLOWS, dtype=np.uint32)
    tmax = ctx.max_throughput(G)
    lam = np.asarray([target_from_tmax(int(batch["u_ppm"][i]), int(tmax[i]))
                      for i in range(len(insts))], dtype=np.uint32)
    per_step = ctx.num_candidates * len(insts) * ((MULTI_GPUS + 1) if multi else 1)
    sync_api = None
    if multi:
        def step():
            plan = ctx.allocate_workflows(lam, MULTI_GPUS, alp.WELFARE_EGALITARIAN)[0]
            return int(plan["status"])

        elapsed, avg, last, status = timed_steps(step, ctx, args.steps, args.warmup)
        assert status in (0, 5)
    else:
        # Queries and results resident in HBM: the searches are queued on the stream back to back
        # and the timed region ends with the stream's synchronisation.
        import torch
        dev = torch.device("cuda", 0)
        Gd = torch.from_numpy(np.ascontiguousarray(G, dtype=np.uint32).view(np.int32)).to(dev)
        Ld = torch.from_numpy(lam.view(np.int32)).to(dev)
        out = torch.empty(len(insts) * alp.RESULT_DTYPE.itemsize, dtype=torch.uint8, device=dev)

        def step():
            ctx.search_batch_async(Gd, Ld, out)

        elapsed, avg, last, _ = timed_steps(step, ctx, args.steps, args.warmup)
        got = alp.results_from_device(out, len(insts))
        ref = ctx.search_batch(G, lam)                  # host-buffer path, outside the timing
        assert got.tobytes() == ref.tobytes() and set(got["status"]) <= {0, 5}
        # The same searches through the host-buffer entry points (query scalars or arrays from
        # host memory, result records to mapped host memory, one synchronisation per call).
        n_sync = max(5, args.steps // 2)
        t0 = time.perf_counter()
        for _ in range(n_sync):
            if len(insts) == 1:
                ctx.search(0, int(G[0]), int(lam[0]))
            else:
                ctx.search_batch(G, lam)
        dt = (time.perf_counter() - t0) / n_sync
        sync_api = {"ms_per_call": dt * 1e3, "value": per_step / dt,
                    "entry_point": "alp_search" if len(insts) == 1 else "alp_search_batch"}
    terms_ms, split_ms, blocks = float(avg[0]), float(avg[2]), last[3]
    value = per_step * args.steps / elapsed
    avg_scan_s = float(avg[1]) / 1e3
    achieved = per_step * OPS_PER_CANDIDATE / avg_scan_s
    config = {"workload": (f"{MULTI_WORKFLOWS} workflows of {cfg.num_llms} LLMs share "
                           f"{MULTI_GPUS} GPUs (egalitarian welfare): all "
                           f"{MULTI_WORKFLOWS * (MULTI_GPUS + 1)} per-workflow budget "
                           "searches, then the budget split") if multi
              else f"{cfg.name}: {cfg.description}",
              "candidates_per_step": per_step, "instances": len(insts),
              "llms": cfg.num_llms, "gpu_budget": MULTI_GPUS if multi else cfg.gpu_budget,
              "options_per_llm": len(cfg.tp_values) * len(cfg.frac_q) * cfg.max_replicas,
              "scan_blocks": blocks,
              "queries_and_results": "host memory (alp_allocate_workflows)" if multi
              else "HBM (alp_search_batch_async)"}
    if sync_api is not None:
        config["host_buffer_api"] = sync_api
    roofline = {"bound": "alu", "achieved": achieved / 1e12, "peak": PEAK_LANE_OPS / 1e12,
                "unit": "TOP/s", "frac": achieved / PEAK_LANE_OPS,
                "traffic": _traffic(_kernel_digest(), args.workload),
                "kernel": "scan", "kernel_ms": avg_scan_s * 1e3,
                "ops_per_candidate": OPS_PER_CANDIDATE,
                "frac_at_5_ops": per_step * OPS_PER_CANDIDATE_WIDE / avg_scan_s / PEAK_LANE_OPS,
                "other_kernels_ms": {"option_terms": terms_ms, "budget_split": split_ms}}
    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(batch, int(G[0]), int(lam[0]), args.cpu_seconds)
    ctx.close()
    return _line(args, value, "candidates/s", elapsed, config, roofline, cpu)


def run_pruned(args, alp):
    if args.workload == "pruned":
        cfg = CONFIGS[args.config]
        batch = make_batch(args.config, range(cfg.num_instances))
        what = (f"the paper's pruned search (Section 5 steps 1-3) on {cfg.name}: "
                f"{cfg.num_instances} instance(s) of {cfg.num_llms} LLMs, G={cfg.gpu_budget}, "
                f"4 share units per GPU")
    else:
        batch = paper_point(args.llms, args.budget, args.fractions)
        what = (f"the paper's pruned search at its scheduler micro-benchmark point: "
                f"{args.llms} LLMs, {args.budget} GPUs, {args.fractions} fractions per GPU")
    ctx = alp.Context(batch)
    G = np.asarray(batch["G"], dtype=np.uint32)
    tmax = ctx.max_throughput(G)
    lam = np.asarray([target_from_tmax(int(batch["u_ppm"][i]), int(tmax[i]))
                      for i in range(len(G))], dtype=np.uint32)
    first = ctx.search_pruned(G, lam)
    vectors = int(first["vectors"].sum())

    def step():
        return ctx.search_pruned(G, lam)

    elapsed, avg, last, out = timed_steps(step, ctx, args.steps, args.warmup)
    assert (out["best"]["index"] == first["best"]["index"]).all()
    avg_enum_s = float(avg[1]) / 1e3
    avg_table_ms = float(avg[2])
    # exhaustive results of the same queries for the gap, outside the timed region (skipped
    # beyond 2^36 candidates per query, a minute of scanning)
    exhaustive = ctx.search_batch(G, lam) if ctx.num_candidates <= (1 << 36) else None
    ops_per_vector = 2 * int(batch["space"]["M"])    # per LLM: add L, accumulate the index
    achieved = vectors * ops_per_vector / avg_enum_s
    config = {"workload": what, "instances": int(len(G)), "llms": int(batch["space"]["M"]),
              "units_per_gpu": int(batch["space"]["Q"]), "gpu_budget": int(G[0]),
              "fraction_vectors_per_step": vectors,
              "unpruned_vectors_per_query": int(first["unpruned"][0]),
              "gap_vs_exhaustive": None if exhaustive is None else gap_stats(out, exhaustive),
              "enumeration_blocks": last[3]}
    roofline = {"bound": "alu", "achieved": achieved / 1e12, "peak": PEAK_LANE_OPS / 1e12,
                "unit": "TOP/s", "frac": achieved / PEAK_LANE_OPS, "traffic": None,
                "kernel": "fraction enumeration", "kernel_ms": avg_enum_s * 1e3,
                "ops_per_vector": ops_per_vector,
                "other_kernels_ms": {"option_terms": float(avg[0]), "option_table": avg_table_ms}}
    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline_pruned(batch, G, lam, args.cpu_seconds)
    ctx.close()
    return _line(args, vectors * args.steps / elapsed, "fraction vectors/s", elapsed, config,
                 roofline, cpu)


def _place_args(res, M):
    return ([int(v) for v in res["tp"][:M]], [int(v) for v in res["frac_units"][:M]],
            [int(v) for v in res["replicas"][:M]])


def cpu_baseline_place(batch, res, G, seconds: float):
    """Single-threaded oracle placement of the results, about `seconds` of work."""
    import oracle
    Q, M = int(batch["space"]["Q"]), int(batch["space"]["M"])
    done, t0 = 0, time.perf_counter()
    while done < len(res) and time.perf_counter() - t0 < seconds:
        if int(res[done]["status"]) == 0:
            oracle.place(Q, int(G[done]), *_place_args(res[done], M))
        done += 1
    dt = time.perf_counter() - t0
    return {"value": done / dt, "unit": "allocations/s", "cores": 1, "kind": "oracle", "host": host_cpu(),
            "sample": f"placement of the first {done} results, single-threaded C oracle "
                      f"({dt:.2f} s, including the Python call per allocation)"}


def run_place(args, alp):
    cfg = CONFIGS[args.config]
    batch = make_batch(args.config, range(cfg.num_instances))
    ctx = alp.Context(batch)
    G = np.asarray(batch["G"], dtype=np.uint32)
    tmax = ctx.max_throughput(G)
    lam = np.asarray([target_from_tmax(int(batch["u_ppm"][i]), int(tmax[i]))
                      for i in range(len(G))], dtype=np.uint32)
    res = ctx.search_batch(G, lam)
    pruned = ctx.search_pruned(G, lam)["best"]

    def step():
        return ctx.place(res, G)

    elapsed, avg, _, out = timed_steps(step, ctx, args.steps, args.warmup)
    k_s = float(avg[1]) / 1e3
    out_p = ctx.place(pruned, G)
    replicas = int(res["replicas"].sum())
    ops = int(sum(int(res[i]["replicas"].sum()) * int(G[i]) for i in range(len(G))))
    feasible = res["status"] == 0
    config = {"workload": f"placement (Section 6) of the exhaustive optima of {cfg.name}: "
                          f"{len(G)} allocation(s) on {int(G[0])} GPUs in nodes of 8",
              "allocations": int(len(G)), "replicas": replicas,
              "optima_placed": int((out["status"] == 0).sum()),
              "optima_feasible": int(feasible.sum()),
              "pruned_placed": int((out_p["status"] == 0).sum()),
              "pruned_feasible": int((pruned["status"] == 0).sum()),
              "mean_gpus_used": float(out["gpus_used"][out["status"] == 0].mean())
              if (out["status"] == 0).any() else 0.0}
    roofline = {"bound": "alu", "achieved": ops / k_s / 1e12, "peak": PEAK_LANE_OPS / 1e12,
                "unit": "TOP/s", "frac": ops / k_s / PEAK_LANE_OPS, "traffic": None,
                "kernel": "place", "kernel_ms": k_s * 1e3,
                "ops": "one pass over the budget's GPUs per replica"}
    cpu = None if args.no_cpu_baseline else cpu_baseline_place(batch, res, G, args.cpu_seconds)
    ctx.close()
    return _line(args, len(G) * args.steps / elapsed, "allocations/s", elapsed, config, roofline,
                 cpu)


def cpu_baseline_stats(tr, seconds: float):
    """Single-threaded oracle over the first traces, about `seconds` of work."""
    import oracle
    off = tr["offsets"]
    R, done, t0 = len(off) - 1, 0, time.perf_counter()
    step = 256
    while done < R and time.perf_counter() - t0 < seconds:
        hi = min(R, done + step)
        lo_c, hi_c = int(off[done]), int(off[hi])
        oracle.trace_stats(tr["M"], off[done:hi + 1] - off[done], tr["llm"][lo_c:hi_c],
                           tr["start"][lo_c:hi_c], tr["end"][lo_c:hi_c])
        done = hi
    dt = time.perf_counter() - t0
    calls = int(off[done])
    return {"value": calls / dt, "unit": "trace calls/s", "cores": 1, "kind": "oracle", "host": host_cpu(),
            "sample": f"the first {done} traces ({calls:,} calls), single-threaded C oracle "
                      f"({dt:.1f} s)"}


def run_stats(args, alp):
    import torch
    from workloads.traces import make_traces
    tr = make_traces("beam", STATS_TRACES, 0)
    calls = int(len(tr["llm"]))
    dev = [torch.from_numpy(np.ascontiguousarray(tr[k]).view(t)).to("cuda:0")
           for k, t in (("offsets", np.int64), ("llm", np.int32), ("start", np.int64),
                        ("end", np.int64))]
    torch.cuda.synchronize()
    ctx = alp.StatsContext(0)

    def step():
        return ctx.compute(tr["M"], *dev)

    import torch as _t
    for _ in range(args.warmup):
        step()
    ctx.set_timing(True)
    kernel_ms = []
    _t.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        out = step()
        kernel_ms.append(ctx.time_ms())
    _t.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    ctx.set_timing(False)
    k_s = float(np.mean(kernel_ms)) / 1e3
    alg_bytes = 20 * calls + 8 * (STATS_TRACES + 1)
    achieved = alg_bytes / k_s
    lengths = np.diff(tr["offsets"].astype(np.int64))
    config = {"workload": f"workflow statistics (Section 4 step 2) of {STATS_TRACES} synthetic "
                          f"beam-search traces: 2 LLMs, {calls:,} calls, 24-843 generator calls "
                          "per request, 3 concurrent beams",
              "traces": STATS_TRACES, "calls": calls, "longest_trace": int(lengths.max()),
              "n_milli": [int(v) for v in out["n_milli"]],
              "p_milli": [int(v) for v in out["p_milli"]]}
    roofline = {"bound": "hbm", "achieved": achieved / 1e9, "peak": HBM_PEAK / 1e9,
                "unit": "GB/s", "frac": achieved / HBM_PEAK,
                "traffic": _traffic(_kernel_digest(STATS_SOURCES), "stats", STATS_TRAFFIC_FILE),
                "kernel": "trace statistics (all kernels)", "kernel_ms": k_s * 1e3,
                "bytes_per_call": 20}
    cpu = None if args.no_cpu_baseline else cpu_baseline_stats(tr, args.cpu_seconds)
    ctx.close()
    return _line(args, calls * args.steps / elapsed, "trace calls/s", elapsed, config, roofline,
                 cpu)


if __name__ == "__main__":
    main()
