"""Writes the expected search results of the synthetic workloads by running the oracle only.

    python tests/golden/make_golden.py --cfg 1 2 4 3 [--jobs 8] [--slices DIR]

For each instance: the oracle's maximum throughput T_max within the budget (threshold method),
the target lambda = max(1, floor(u * T_max)), and the exhaustive argmin over the whole candidate
space.  Some workloads add queries of an instance at another target fraction (EXTRA_QUERIES:
the 5-LLM instance at 2% of T_max, where tens of millions of candidates are feasible and ties
are many), stored as further rows with their own u_ppm.  Each search runs (brute force, split into index slices run in parallel single-threaded processes and
merged by lexicographic (L, x) minimum), with the winner's T_w and U, the number of feasible
candidates and the sum of their L_w modulo 2^64.  Slice results are cached as JSON files in the
slice directory so an interrupted run resumes.  Output: ``cfg<N>_argmin.json`` next to this
script.  Nothing here reads GPU results.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import multiprocessing as mp
import os
import sys
import time

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
from workloads import CONFIGS, make_batch, target_from_tmax  # noqa: E402

SLICE = 1 << 27
# Further (instance, u_ppm) queries per workload, beyond each instance at its drawn target.
EXTRA_QUERIES = {3: [(0, 20_000)]}


def table_digest(batch: dict) -> str:
    h = hashlib.sha256()
    for k in ("W", "n", "p", "allowed", "rate", "lat", "u_ppm", "G"):
        h.update(batch[k].tobytes())
    return h.hexdigest()


def _query(cfg: int, inst: int, u_ppm: int | None = None):
    b = make_batch(cfg, [inst])
    o = oracle.Instance(b, 0)
    G = int(b["G"][0])
    tmax = oracle.tmax(o, G)
    u = int(b["u_ppm"][0]) if u_ppm is None else u_ppm
    lam = target_from_tmax(u, tmax)
    return b, o, G, tmax, lam, u


def _slice_job(args):
    cfg, q, inst, u_ppm, lo, hi, cache = args
    tag = "" if u_ppm is None else f"_u{u_ppm}"
    path = os.path.join(cache, f"cfg{cfg}_i{inst}{tag}_{lo}_{hi}.json") if cache else None
    if path and os.path.exists(path):
        with open(path) as f:
            r = json.load(f)
            r["q"] = q
            return r
    _, o, G, _, lam, _ = _query(cfg, inst, u_ppm)
    r = oracle.argmin(o, G, lam, lo, hi)
    r.update({"q": q, "inst": inst, "lo": lo, "hi": hi})
    if path:
        tmp = path + ".tmp"
        with open(tmp, "w") as f:
            json.dump(r, f)
        os.replace(tmp, path)
    return r


def run_cfg(cfg: int, jobs: int, cache: str | None) -> dict:
    conf = CONFIGS[cfg]
    insts = list(range(conf.num_instances))
    b_all = make_batch(cfg, insts)
    N = (len(conf.tp_values) * len(conf.frac_q) * conf.max_replicas) ** conf.num_llms
    queries = [(inst, None) for inst in insts] + list(EXTRA_QUERIES.get(cfg, []))
    tasks = []
    for q, (inst, u_ppm) in enumerate(queries):
        for lo in range(0, N, SLICE):
            tasks.append((cfg, q, inst, u_ppm, lo, min(N, lo + SLICE), cache))
    t0 = time.time()
    parts = {}
    with mp.Pool(jobs) as pool:
        for k, r in enumerate(pool.imap_unordered(_slice_job, tasks, chunksize=1)):
            parts.setdefault(r["q"], []).append(r)
            if (k + 1) % max(1, len(tasks) // 20) == 0:
                print(f"cfg{cfg}: {k + 1}/{len(tasks)} slices, {time.time() - t0:.0f}s", flush=True)
    rows = []
    for q, (inst, u_ppm) in enumerate(queries):
        b, o, G, tmax, lam, u = _query(cfg, inst, u_ppm)
        best = oracle.merge_argmin(parts[q])
        row = {"inst": inst, "G": G, "u_ppm": u, "tmax": tmax, "lambda": lam,
               "x": best["x"], "L": best["L"], "n_feasible": best["n_feasible"],
               "sum_L": best["sum_L"]}
        if best["x"] is not None:
            ev = oracle.evaluate(o, G, lam, best["x"])
            row.update({"T": ev["T"], "U": ev["U"]})
        rows.append(row)
    return {"cfg": cfg, "name": conf.name, "candidates_per_instance": N,
            "table_sha256": table_digest(b_all), "oracle_wall_s": round(time.time() - t0, 1),
            "jobs": jobs, "command": "python tests/golden/make_golden.py --cfg %d" % cfg,
            "results": rows}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--cfg", type=int, nargs="+", required=True)
    ap.add_argument("--jobs", type=int, default=os.cpu_count())
    ap.add_argument("--slices", default=None, help="directory for resumable slice results")
    args = ap.parse_args()
    oracle.lib()
    if args.slices:
        os.makedirs(args.slices, exist_ok=True)
    for cfg in args.cfg:
        out = run_cfg(cfg, args.jobs, args.slices)
        path = os.path.join(HERE, f"cfg{cfg}_argmin.json")
        with open(path, "w") as f:
            json.dump(out, f, indent=0)
        print(f"wrote {path} ({out['oracle_wall_s']} s)", flush=True)


if __name__ == "__main__":
    main()
