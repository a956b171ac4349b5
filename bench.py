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
kernel) to the integer VALU peak of the chip: 2 int32 lane operations per candidate, the work the
kernel issues (the budget comparison and the objective minimum update), against CUs x 64 lanes x
the maximum engine clock, both read from rocminfo in the run (256 CUs and 2.4 GHz on MI355X:
39.32 Tlane-op/s).  The kernel duration is the median over separately timed steps after the timed
region, from HIP events stamped on the scan dispatch on the stream the library launches on.
``cpu_baseline`` times the CPU oracle on a bounded slice of the same space, in worker processes
on every host core of the job (at most 16), before the benchmark touches the GPU.

The default run also measures the other exhaustive workloads in the same process and reports
them under ``config.other_workloads``: the single 4-LLM search (cfg2) and the 4,096-search batch
(cfg4) with their scan-kernel medians and roofline fractions, and the 2- and 3-LLM searches
(cfg0, cfg1) with their HBM-resident step and ``alp_search`` call latency.  ``--only`` skips them.
``--oracle-full`` adds the oracle's full argmin of the workload's instance 0 across the host
cores (wall time and core count; about a minute for the 5-LLM space).

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

MI355X_CUS, MI355X_CLOCK_HZ = 256, 2.4e9    # published figures, used if rocminfo cannot be read
OPS_PER_CANDIDATE = 2                   # budget compare + objective min: the work issued
FRAC_BASIS = "issued VALU lane-ops (2 per candidate: budget compare, objective minimum)"
# Kernel times come from a separate pass after the timed region, every step event-stamped (an
# event-stamped dispatch costs the GPU a few microseconds of idle time, which must not be part
# of the timed steps of a small search); the figure reported is the median.
TIMING_SAMPLES = 9
# The wider count of lane-ops per candidate (add the last term, compare the budget, compare the
# best, select value and index), reported beside ``frac`` for comparison with that accounting.
OPS_PER_CANDIDATE_WIDE = 5
SQ_COUNTER_FILE = os.path.join(ROOT, "profiles", "scan_min_sq_counters.md")
# Exhaustive workloads measured besides the headline one in the default run.
OTHER_WORKLOADS = ("cfg2", "cfg4", "cfg1", "cfg0")
WORKLOADS = {"cfg0": 0, "cfg2": 2, "cfg3": 3, "cfg4": 4, "cfg1": 1, "multi": 2, "pruned": 4,
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


def _counter_entry(kernel_digest: str, workload: str, path: str):
    """A workload's entry of the machine-readable block of a committed rocprofv3 counter
    summary, if the counters were taken on the current kernel source."""
    try:
        with open(path) as f:
            text = f.read()
        t = json.loads(text.split("```json", 1)[1].split("```", 1)[0])
    except (OSError, ValueError, IndexError):
        return None
    if t.get("kernel_source_sha256") != kernel_digest:
        return None
    return t.get(workload)


def _traffic(kernel_digest: str, workload: str, path: str = TRAFFIC_FILE):
    """HBM bytes per launch (per call for the statistics) from the counter summary."""
    entry = _counter_entry(kernel_digest, workload, path)
    return entry.get("bytes_per_launch") if entry else None


def _lane_ops_per_candidate(kernel_digest: str, workload: str):
    """VALU lane-ops the scan issued per candidate (SQ_INSTS_VALU x 64 / candidates) from the
    instruction-counter summary."""
    entry = _counter_entry(kernel_digest, workload, SQ_COUNTER_FILE)
    return entry.get("valu_lane_ops_per_candidate") if entry else None


def chip_peak():
    """(CUs, maximum engine clock in Hz, source) of the gfx950 agent, read from rocminfo;
    the published MI355X figures if it cannot be read.  Runs rocminfo as a child process."""
    import subprocess
    try:
        out = subprocess.run(["rocminfo"], capture_output=True, text=True, timeout=120).stdout
    except (OSError, subprocess.SubprocessError):
        out = ""
    for agent in out.split("Agent ")[1:]:
        if "gfx950" not in agent:
            continue
        cus = clock = None
        for line in agent.splitlines():
            key, _, val = line.strip().partition(":")
            if key.strip() == "Compute Unit" and cus is None:
                cus = int(val.split()[0])
            elif key.strip() == "Max Clock Freq. (MHz)" and clock is None:
                clock = float(val.split()[0]) * 1e6
        if cus and clock:
            return cus, clock, "rocminfo"
    return MI355X_CUS, MI355X_CLOCK_HZ, "published MI355X figures (rocminfo not readable)"


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


def host_cores() -> int:
    """Cores the job may use: the CPU affinity set, at most 16 (one GPU's share of its host)."""
    try:
        n = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def _oracle_slice(task):
    """Worker: the oracle's argmin over [lo, hi) of one workload instance (wall seconds, x, L)."""
    cfg_id, inst, G, lam, lo, hi = task
    import oracle
    b = make_batch(cfg_id, [inst])
    t0 = time.perf_counter()
    r = oracle.argmin(oracle.Instance(b, 0), G, lam, lo, hi)
    return time.perf_counter() - t0, r["x"], r["L"]


def _oracle_query(cfg_id: int):
    """Instance 0 of a workload with its target rate, from the oracle alone (T_max by the
    threshold method)."""
    import oracle
    b = make_batch(cfg_id, [0])
    inst = oracle.Instance(b, 0)
    G = int(b["G"][0])
    lam = target_from_tmax(int(b["u_ppm"][0]), oracle.tmax(inst, G))
    return b, inst, G, lam


def _parallel_slices(cfg_id, G, lam, bounds, cores):
    from concurrent.futures import ProcessPoolExecutor
    from multiprocessing import get_context
    tasks = [(cfg_id, 0, G, lam, lo, hi) for lo, hi in bounds]
    t0 = time.perf_counter()
    with ProcessPoolExecutor(cores, mp_context=get_context("spawn")) as ex:
        res = list(ex.map(_oracle_slice, tasks))
    return time.perf_counter() - t0, res


def cpu_baseline(cfg_id: int, seconds: float):
    """The oracle's exhaustive argmin over a bounded slice of instance 0, split into equal
    contiguous slices over every host core of the job (worker processes, started before the
    benchmark touches the GPU); about `seconds` of wall time."""
    import oracle
    _, inst, G, lam = _oracle_query(cfg_id)
    n = 1 << 20
    t0 = time.perf_counter()
    oracle.argmin(inst, G, lam, 0, n)
    rate1 = n / max(time.perf_counter() - t0, 1e-6)
    cores = host_cores()
    per = max(n, int(rate1 * seconds))
    total = min(inst.N, per * cores)
    per = -(-total // cores)
    bounds = [(k * per, min(total, (k + 1) * per)) for k in range(cores) if k * per < total]
    wall, _ = _parallel_slices(cfg_id, G, lam, bounds, len(bounds))
    return {"value": total / wall, "unit": "candidates/s", "cores": len(bounds), "kind": "oracle",
            "host": host_cpu(), "single_core_value": rate1,
            "sample": f"first {total:,} candidate indices of the same instance in {len(bounds)} "
                      f"contiguous slices, one per worker process, exhaustive C oracle "
                      f"({wall:.1f} s wall including process start)"}


def _oracle_instances(task):
    """Worker: the oracle's full argmin of instances [a, b) of a workload (wall s, [x, ...])."""
    cfg_id, a, b, lam = task
    import oracle
    batch = make_batch(cfg_id, range(a, b))
    t0 = time.perf_counter()
    xs = [oracle.argmin(oracle.Instance(batch, i), int(batch["G"][i]), int(lam[i]))["x"]
          for i in range(b - a)]
    return time.perf_counter() - t0, xs


def oracle_full(cfg_id: int):
    """The oracle's full argmin of the workload across the host cores, in worker processes:
    a single instance in 8 contiguous index slices per core (slice winners merge on (L, x)), a
    batch as per-instance jobs.  Wall time including process start."""
    import oracle
    from concurrent.futures import ProcessPoolExecutor
    from multiprocessing import get_context
    cores = host_cores()
    cfg = CONFIGS[cfg_id]
    if cfg_id == 4:
        batch = make_batch(cfg_id, range(cfg.num_instances))
        lam = [target_from_tmax(int(batch["u_ppm"][i]),
                                oracle.tmax(oracle.Instance(batch, i), int(batch["G"][i])))
               for i in range(cfg.num_instances)]
        step = 64
        tasks = [(cfg_id, a, min(a + step, cfg.num_instances), lam[a:a + step])
                 for a in range(0, cfg.num_instances, step)]
        t0 = time.perf_counter()
        with ProcessPoolExecutor(cores, mp_context=get_context("spawn")) as ex:
            res = list(ex.map(_oracle_instances, tasks))
        wall = time.perf_counter() - t0
        xs = [x for _, part in res for x in part]
        total = cfg.num_instances * oracle.Instance(batch, 0).N
        return {"candidates": total, "cores": cores, "wall_s": wall, "value": total / wall,
                "unit": "candidates/s", "jobs": f"{len(tasks)} jobs of {step} instances",
                "host": host_cpu(), "_indices": xs}
    _, inst, G, lam = _oracle_query(cfg_id)
    parts = 8 * cores
    per = -(-inst.N // parts)
    bounds = [(k * per, min(inst.N, (k + 1) * per)) for k in range(parts) if k * per < inst.N]
    wall, res = _parallel_slices(cfg_id, G, lam, bounds, cores)
    best = min(((L, x) for _, x, L in res if x is not None), default=(None, None))
    return {"candidates": inst.N, "cores": cores, "wall_s": wall, "value": inst.N / wall,
            "unit": "candidates/s", "jobs": f"{len(bounds)} index slices", "x": best[1],
            "L": best[0], "host": host_cpu()}


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


def timed_steps(step, ctx, steps: int, warmup: int, samples: int = TIMING_SAMPLES):
    """Runs warmup + steps calls with no timing inside the timed region, then `samples` more
    calls each timed with HIP events stamped on the kernel dispatches.  Returns (elapsed s of
    the timed region, median kernel ms [3] over the samples, the last sample's kernel_times(),
    the last timed-region output)."""
    import torch
    for _ in range(warmup):
        step()
    ctx.set_timing(False)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        out = step()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    ctx.set_timing(1)
    per_call = []
    for _ in range(samples):
        step()
        per_call.append(ctx.kernel_times())
    ctx.set_timing(False)
    med = np.median(np.asarray([t[:3] for t in per_call], dtype=np.float64), axis=0)
    return elapsed, med, per_call[-1], out


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
    ap.add_argument("--only", action="store_true",
                    help="measure the named workload alone (no other workloads in the line)")
    ap.add_argument("--no-oracle-full", action="store_true",
                    help="skip the oracle's full argmin across host cores (5-LLM search and "
                         "4,096-search batch)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the search runs on a single MI355X; "
              "multi-GPU sharding is not built (run with --gpus 1)", file=sys.stderr)
        sys.exit(2)

    # Before anything touches the GPU: the chip's peak from rocminfo and the oracle legs of the
    # exhaustive workloads, which run in worker processes.
    peak_info = chip_peak()
    exhaustive = not (args.workload.startswith("pruned") or args.workload in ("stats", "place"))
    cpu, full = None, {}
    if exhaustive:
        if not args.no_cpu_baseline:
            cpu = cpu_baseline(WORKLOADS[args.workload], args.cpu_seconds)
        if not args.no_oracle_full and args.workload == "cfg3":
            for name in ("cfg3", "cfg4") if not args.only else ("cfg3",):
                full[name] = oracle_full(WORKLOADS[name])

    import torch
    from paper_2604_15186_amd import alp

    if not torch.cuda.is_available():
        print("no GPU visible", file=sys.stderr)
        sys.exit(1)
    peak = peak_info[0] * 64 * peak_info[1]
    if args.workload.startswith("pruned"):
        line = run_pruned(args, alp, peak)
    elif args.workload == "stats":
        line = run_stats(args, alp)
    elif args.workload == "place":
        line = run_place(args, alp, peak)
    else:
        line = run_exhaustive(args, alp, peak_info, cpu, full)
    if args.calib_copy_mib:
        src = torch.ones(args.calib_copy_mib << 20, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        line["calib_copy_bytes"] = args.calib_copy_mib << 20
    print(json.dumps(line), flush=True)


# The other workloads' own metrics (the exhaustive search reports METRIC).
SIDE_METRICS = {
    "fraction vectors/s": "ALP pruned-search fraction vectors evaluated/sec on 1 GPU",
    "allocations/s": "allocations placed on GPUs/sec on 1 GPU",
    "trace calls/s": "workflow-statistics trace calls processed/sec on 1 GPU",
}


def _line(args, value, unit, elapsed, dtype_cfg, roofline, cpu):
    data = ("synthetic (seeded execution traces, see workloads/traces.py)"
            if unit == "trace calls/s" else "synthetic (seeded profile tables, see workloads/)")
    return {"metric": SIDE_METRICS.get(unit, METRIC), "value": value, "unit": unit, "n_gpus": 1,
            "steps": args.steps, "warmup": args.warmup, "ms_per_step": elapsed / args.steps * 1e3,
            "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "u32",
            "data": data, "config": dtype_cfg, "roofline": roofline, "cpu_baseline": cpu}


def measure_exhaustive(alp, cfg_id: int, steps: int, warmup: int, variant: int, peak: float,
                       multi: bool = False) -> dict:
    """One exhaustive workload: the timed HBM-resident steps, the kernel medians, the roofline
    fraction and the host-buffer call latency."""
    cfg = CONFIGS[cfg_id]
    if multi:
        insts = list(range(MULTI_WORKFLOWS))
    else:
        insts = list(range(cfg.num_instances)) if cfg_id == 4 else [0]
    batch = make_batch(cfg_id, insts)
    ctx = alp.Context(batch)
    ctx.set_launch(variant)
    G = batch["G"]
    if multi:
        G = np.full(len(insts), MULTI_GPUS // MULTI_WORKFLOWS, dtype=np.uint32)
    tmax = ctx.max_throughput(G)
    lam = np.asarray([target_from_tmax(int(batch["u_ppm"][i]), int(tmax[i]))
                      for i in range(len(insts))], dtype=np.uint32)
    per_step = ctx.num_candidates * len(insts) * ((MULTI_GPUS + 1) if multi else 1)
    sync_api, argmin = None, None
    if multi:
        def step():
            plan = ctx.allocate_workflows(lam, MULTI_GPUS, alp.WELFARE_EGALITARIAN)[0]
            return int(plan["status"])

        elapsed, med, last, status = timed_steps(step, ctx, steps, warmup)
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

        elapsed, med, last, _ = timed_steps(step, ctx, steps, warmup)
        got = alp.results_from_device(out, len(insts))
        ref = ctx.search_batch(G, lam)                  # host-buffer path, outside the timing
        assert got.tobytes() == ref.tobytes() and set(got["status"]) <= {0, 5}
        # The same searches through the host-buffer entry points (query scalars or arrays from
        # host memory, result records to mapped host memory, one synchronisation per call).
        n_sync = max(9, steps // 2)
        times = []
        for _ in range(n_sync):
            t0 = time.perf_counter()
            if len(insts) == 1:
                ctx.search(0, int(G[0]), int(lam[0]))
            else:
                ctx.search_batch(G, lam)
            times.append(time.perf_counter() - t0)
        dt = float(np.median(times))
        if len(insts) == 1:
            argmin = {"index": int(got[0]["index"]), "latency_us": int(got[0]["latency_us"])}
        sync_api = {"ms_per_call": dt * 1e3, "value": per_step / dt, "calls": n_sync,
                    "statistic": "median",
                    "entry_point": "alp_search" if len(insts) == 1 else "alp_search_batch"}
    scan_s = float(med[1]) / 1e3
    ctx.close()
    r = {"workload": (f"{MULTI_WORKFLOWS} workflows of {cfg.num_llms} LLMs share "
                      f"{MULTI_GPUS} GPUs (egalitarian welfare): all "
                      f"{MULTI_WORKFLOWS * (MULTI_GPUS + 1)} per-workflow budget "
                      "searches, then the budget split") if multi
         else f"{cfg.name}: {cfg.description}",
         "candidates_per_step": per_step, "instances": len(insts), "llms": cfg.num_llms,
         "gpu_budget": MULTI_GPUS if multi else cfg.gpu_budget,
         "options_per_llm": len(cfg.tp_values) * len(cfg.frac_q) * cfg.max_replicas,
         "scan_blocks": last[3], "ms_per_step": elapsed / steps * 1e3,
         "value": per_step * steps / elapsed,
         "scan_kernel_ms": scan_s * 1e3, "option_terms_ms": float(med[0]),
         "budget_split_ms": float(med[2]), "kernel_samples": TIMING_SAMPLES,
         "frac": per_step * OPS_PER_CANDIDATE / scan_s / peak,
         "queries_and_results": "host memory (alp_allocate_workflows)" if multi
         else "HBM (alp_search_batch_async)"}
    if sync_api is not None:
        r["host_buffer_api"] = sync_api
    if argmin is not None:
        r["argmin"] = argmin
    if not multi and len(insts) > 1:
        r["_indices"] = got["index"].copy()
    return r


def run_exhaustive(args, alp, peak_info, cpu, full):
    cus, clock, source = peak_info
    peak = cus * 64 * clock
    multi = args.workload == "multi"
    cfg_id = WORKLOADS[args.workload]
    m = measure_exhaustive(alp, cfg_id, args.steps, args.warmup, args.variant, peak, multi)
    digest = _kernel_digest()
    config = {k: m[k] for k in ("workload", "candidates_per_step", "instances", "llms",
                                "gpu_budget", "options_per_llm", "scan_blocks",
                                "queries_and_results") if k in m}
    if "argmin" in m:
        config["argmin"] = m["argmin"]
    if "host_buffer_api" in m:
        config["host_buffer_api"] = m["host_buffer_api"]
    if not args.only and not multi and args.workload == "cfg3":
        others = {}
        for name in OTHER_WORKLOADS:
            o = measure_exhaustive(alp, WORKLOADS[name], args.steps, args.warmup, args.variant,
                                   peak)
            o["valu_lane_ops_per_candidate"] = _lane_ops_per_candidate(digest, name)
            others[name] = o
        config["other_workloads"] = others
    if full:
        # The oracle's full argmins, against the GPU results of the same searches.
        out = {}
        for name, f in full.items():
            f = dict(f)
            if name == args.workload:
                f["matches_gpu"] = f["x"] == m.get("argmin", {}).get("index")
            else:
                xs = f.pop("_indices")
                gpu = config.get("other_workloads", {}).get(name, {}).pop("_indices", None)
                f["matches_gpu"] = gpu is not None and [int(v) for v in gpu] == [
                    int(v) if v is not None else (1 << 64) - 1 for v in xs]
            out[name] = f
        config["oracle_full_argmin"] = out
    for o in config.get("other_workloads", {}).values():
        o.pop("_indices", None)
    scan_s = m["scan_kernel_ms"] / 1e3
    achieved = m["candidates_per_step"] * OPS_PER_CANDIDATE / scan_s
    roofline = {"bound": "alu", "achieved": achieved / 1e12, "peak": peak / 1e12,
                "unit": "TOP/s", "frac": achieved / peak,
                "traffic": _traffic(digest, args.workload),
                "kernel": "scan", "kernel_ms": m["scan_kernel_ms"],
                "kernel_ms_statistic": f"median of {TIMING_SAMPLES} event-stamped steps",
                "frac_basis": FRAC_BASIS, "ops_per_candidate": OPS_PER_CANDIDATE,
                "valu_lane_ops_per_candidate": _lane_ops_per_candidate(digest, args.workload),
                "peak_source": f"{cus} CUs x 64 lanes x {clock / 1e9:.2f} GHz ({source})",
                "frac_at_5_ops": m["candidates_per_step"] * OPS_PER_CANDIDATE_WIDE / scan_s / peak,
                "other_kernels_ms": {"option_terms": m["option_terms_ms"],
                                     "budget_split": m["budget_split_ms"]}}
    return _line(args, m["value"], "candidates/s", m["ms_per_step"] / 1e3 * args.steps, config,
                 roofline, cpu)


def run_pruned(args, alp, peak: float):
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
    roofline = {"bound": "alu", "achieved": achieved / 1e12, "peak": peak / 1e12,
                "unit": "TOP/s", "frac": achieved / peak, "traffic": None,
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


def run_place(args, alp, peak: float):
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
    roofline = {"bound": "alu", "achieved": ops / k_s / 1e12, "peak": peak / 1e12,
                "unit": "TOP/s", "frac": ops / k_s / peak, "traffic": None,
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
    ctx = alp.StatsContext(0)

    def timed(order):
        """Median kernel time (HIP events around the launches) over the timed steps, the wall
        time of those steps and the last result, for the calls taken in the given order."""
        dev = [torch.from_numpy(np.ascontiguousarray(tr[k][order]).view(t)).to("cuda:0")
               for k, t in (("llm", np.int32), ("start", np.int64), ("end", np.int64))]
        off = torch.from_numpy(tr["offsets"].view(np.int64)).to("cuda:0")
        torch.cuda.synchronize()
        for _ in range(args.warmup):
            ctx.compute(tr["M"], off, *dev)
        ctx.set_timing(True)
        kernel_ms = []
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(args.steps):
            out = ctx.compute(tr["M"], off, *dev)
            kernel_ms.append(ctx.time_ms())
        torch.cuda.synchronize()
        elapsed = time.perf_counter() - t0
        ctx.set_timing(False)
        return float(np.median(kernel_ms)), elapsed, out

    alg_bytes = 20 * calls + 8 * (STATS_TRACES + 1)
    # As logged (in order of end time): the sweep without a sort.
    k_ms, elapsed, out = timed(np.arange(calls))
    # The same calls shuffled within each trace: every trace is sorted (the context sees that the
    # traces are not in end order and sorts directly, checking the order again every 8th call).
    rng = np.random.default_rng(5)
    off = tr["offsets"].astype(np.int64)
    perm = np.concatenate([lo + rng.permutation(hi - lo) for lo, hi in zip(off[:-1], off[1:])])
    s_ms, s_elapsed, s_out = timed(perm)
    if not (s_out == out).all():
        raise SystemExit("shuffled traces gave different statistics")
    achieved = alg_bytes / (k_ms / 1e3)
    lengths = np.diff(off)
    config = {"workload": f"workflow statistics (Section 4 step 2) of {STATS_TRACES} synthetic "
                          f"beam-search traces: 2 LLMs, {calls:,} calls, 24-843 generator calls "
                          "per request, 3 concurrent beams",
              "traces": STATS_TRACES, "calls": calls, "longest_trace": int(lengths.max()),
              "n_milli": [int(v) for v in out["n_milli"]],
              "p_milli": [int(v) for v in out["p_milli"]],
              "shuffled": {"order": "calls shuffled within each trace (sorted on the GPU)",
                           "value": calls * args.steps / s_elapsed, "unit": "trace calls/s",
                           "kernel_ms": s_ms, "frac": alg_bytes / (s_ms / 1e3) / HBM_PEAK}}
    roofline = {"bound": "hbm", "achieved": achieved / 1e9, "peak": HBM_PEAK / 1e9,
                "unit": "GB/s", "frac": achieved / HBM_PEAK,
                "traffic": _traffic(_kernel_digest(STATS_SOURCES), "stats", STATS_TRAFFIC_FILE),
                "kernel": "trace statistics (all kernels)", "kernel_ms": k_ms,
                "kernel_ms_stat": "median over the timed steps", "bytes_per_call": 20}
    cpu = None if args.no_cpu_baseline else cpu_baseline_stats(tr, args.cpu_seconds)
    ctx.close()
    return _line(args, calls * args.steps / elapsed, "trace calls/s", elapsed, config, roofline,
                 cpu)


if __name__ == "__main__":
    main()
