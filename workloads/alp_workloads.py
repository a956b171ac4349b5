"""Seeded synthetic workloads for the Aggregate LLM Pipeline (ALP) allocation search.

This module only draws inputs: per-LLM throughput--latency profile tables (one table per
tensor-parallel degree and GPU share, as produced by the profiling step of Section 4),
per-LLM workflow statistics n_m and p_m (Section 4, the workflow statistics step), model weight
sizes for the memory-fit bound (Section 5, step 1), a GPU budget and
a target-rate fraction.  It contains none of the predictor's arithmetic (no Eq. 1 / Eq. 2
terms, no feasibility, no argmin): those live, independently, in the oracle and in the HIP
library.  The target workflow rate is stated here only as a fraction ``u_ppm`` (parts per
million) of the largest rate the budget can sustain; each side computes that maximum itself
and :func:`target_from_tmax` turns the pair into an integer rate.

The paper's real workloads (RAG with a reranker, beam search with a process reward model) and
their profiled tables are not available; the synthetic tables below stand in for them with the
same structure: small and large LLMs in one workflow, 2-5 LLM stages, latency that grows with
load up to a saturation throughput, tensor parallelism up to one 8-GPU node, fractional GPU
shares in quarters.

All values are quantised to integers (microseconds, milli-requests per second, milli-units for
n_m and p_m, bytes), so the oracle and the GPU path read identical integer inputs.

Array layout of a batch (B instances, M LLMs, |TP| degrees, |FQ| shares, K profile points):

  W        uint64 [B, M]                  model weight bytes (bf16: 2 bytes per parameter)
  n        uint32 [B, M]                  invocations per workflow request, x1000
  p        uint32 [B, M]                  request-level parallelism, x1000
  allowed  uint8  [B, M, |TP|, |FQ|]      1 if the (tp, share) pair may be deployed
  rate     uint32 [B, M, |TP|, |FQ|, K]   per-replica arrival rate of profile point k, milli-req/s,
                                          strictly ascending in k; the last point is saturation
  lat      uint32 [B, M, |TP|, |FQ|, K]   mean latency at that rate, microseconds
  G        uint32 [B]                     GPU budget (whole GPUs)
  u_ppm    uint32 [B]                     target rate as a fraction of the maximum, ppm
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

SEED_ROOT = (2604, 15186)
HBM_BYTES_MI355X = 288 * 10**9          # HBM3E bytes per GPU used by the memory-fit bound
REFERENCE_EXEC_S = 30.0                 # R: reference request execution time used to map shares to n_m


@dataclass(frozen=True)
class WorkloadConfig:
    """One synthetic workload family (shape of the search space and the value distributions)."""

    name: str
    num_llms: int
    gpu_budget: int
    tp_values: tuple
    frac_q: tuple                 # GPU shares in units of 1/frac_den
    max_replicas: int
    param_range: tuple            # model size range, parameters (log-uniform)
    sort_sizes: bool              # sort model sizes ascending (generator first, largest verifier last)
    alpha: float                  # Dirichlet concentration of the per-LLM execution shares
    target: str                   # "uniform": u ~ U(lo, hi); "loguniform": u = exp(U(ln lo, ln hi))
    target_range: tuple
    num_instances: int = 1
    frac_den: int = 4
    num_points: int = 8
    frac_tp: bool = False         # allow a GPU share below 1 together with tp > 1
    description: str = field(default="", compare=False)


CONFIGS = {
    0: WorkloadConfig(
        name="alp-2llm-g8", num_llms=2, gpu_budget=8, tp_values=(1, 2, 4, 8), frac_q=(1, 2, 4),
        max_replicas=4, param_range=(0.5e9, 70e9), sort_sizes=True, alpha=1.0,
        target="uniform", target_range=(0.1, 0.9), num_instances=1000,
        description="2-LLM generator+verifier, G=8, 48 options/LLM, 2,304 candidates"),
    1: WorkloadConfig(
        name="alp-3llm-g16", num_llms=3, gpu_budget=16, tp_values=(1, 2, 4, 8), frac_q=(1, 2, 3, 4),
        max_replicas=8, param_range=(0.5e9, 70e9), sort_sizes=True, alpha=1.0,
        target="uniform", target_range=(0.1, 0.9), num_instances=64,
        description="3-LLM beam-search shape, G=16, 128 options/LLM, 2,097,152 candidates"),
    2: WorkloadConfig(
        name="alp-4llm-g32", num_llms=4, gpu_budget=32, tp_values=(1, 2, 4, 8), frac_q=(1, 2, 3, 4),
        max_replicas=8, param_range=(1e9, 70e9), sort_sizes=False, alpha=0.5,
        target="uniform", target_range=(0.1, 0.9), num_instances=4,
        description="4-LLM workflow, G=32, skewed shares, 268,435,456 candidates"),
    3: WorkloadConfig(
        name="alp-5llm-g64", num_llms=5, gpu_budget=64, tp_values=(1, 2, 4, 8), frac_q=(1, 2, 3, 4),
        max_replicas=8, param_range=(1e9, 70e9), sort_sizes=False, alpha=0.5,
        target="uniform", target_range=(0.1, 0.9), num_instances=1,
        description="5-LLM workflow, G=64, 34,359,738,368 candidates"),
    4: WorkloadConfig(
        name="alp-batch4096-3llm-g16", num_llms=3, gpu_budget=16, tp_values=(1, 2, 4, 8),
        frac_q=(1, 2, 3, 4), max_replicas=8, param_range=(0.5e9, 70e9), sort_sizes=True, alpha=1.0,
        target="loguniform", target_range=(0.05, 1.0), num_instances=4096,
        description="4,096 independent 3-LLM instances, G=16 each, 8,589,934,592 candidates in total"),
}


def num_options(space: dict) -> int:
    """Options per LLM: |TP| * |FQ| * D (invalid combinations included)."""
    return len(space["tp"]) * len(space["fq"]) * int(space["D"])


def num_candidates(space: dict) -> int:
    """Size of the mixed-radix candidate space, O ** M."""
    return num_options(space) ** int(space["M"])


def _space_of(cfg: WorkloadConfig) -> dict:
    return {
        "M": cfg.num_llms,
        "tp": np.asarray(cfg.tp_values, dtype=np.uint32),
        "fq": np.asarray(cfg.frac_q, dtype=np.uint32),
        "Q": cfg.frac_den,
        "D": cfg.max_replicas,
        "K": cfg.num_points,
    }


def _profile_tables(space: dict, L0: float, frac_tp: bool):
    """Synthetic per-replica throughput--latency profile of one LLM for every (tp, share).

    Base latency L0 (seconds at tp=1, whole GPU, low load) is scaled by (0.2 + 0.8/tp) / f^0.8
    for tensor-parallel degree tp and GPU share f.  The per-replica saturation throughput is
    f * tp * tp^-0.15 / L requests/s.  The K profile points sit at rates T*k/K with latency
    L * (1 + 2 (k/K)^3), i.e. latency rises towards saturation as in a load sweep.
    """
    tps, fqs, Q, K = space["tp"], space["fq"], int(space["Q"]), int(space["K"])
    rate = np.zeros((len(tps), len(fqs), K), dtype=np.uint32)
    lat = np.zeros((len(tps), len(fqs), K), dtype=np.uint32)
    allowed = np.zeros((len(tps), len(fqs)), dtype=np.uint8)
    ks = np.arange(1, K + 1, dtype=np.float64)
    for i, tp in enumerate(tps):
        for j, q in enumerate(fqs):
            f = float(q) / Q
            L = L0 * (0.2 + 0.8 / float(tp)) / f ** 0.8
            T = f * float(tp) * float(tp) ** -0.15 / L
            r = np.rint(1000.0 * T * ks / K).astype(np.int64)
            r[0] = max(r[0], 1)
            for k in range(1, K):
                r[k] = max(r[k], r[k - 1] + 1)
            rate[i, j] = r
            lat[i, j] = np.maximum(1, np.rint(1e6 * L * (1.0 + 2.0 * (ks / K) ** 3))).astype(np.int64)
            allowed[i, j] = 1 if (frac_tp or q == Q or tp == 1) else 0
    return allowed, rate, lat


def _draw_instance(space: dict, rng: np.random.Generator, param_range, sort_sizes, alpha,
                   target, target_range, frac_tp):
    M = int(space["M"])
    lo, hi = param_range
    params = np.exp(rng.uniform(np.log(lo), np.log(hi), size=M))
    if sort_sizes:
        params = np.sort(params)
    L0 = np.exp(rng.uniform(np.log(0.05), np.log(5.0), size=M))
    shares = rng.dirichlet(np.full(M, float(alpha)))
    par = rng.uniform(1.0, 4.0, size=M)
    if target == "uniform":
        u = rng.uniform(*target_range)
    else:
        u = float(np.exp(rng.uniform(np.log(target_range[0]), np.log(target_range[1]))))
    out = {
        "W": np.rint(2.0 * params).astype(np.uint64),
        "n": np.maximum(1, np.rint(1000.0 * shares * REFERENCE_EXEC_S / L0)).astype(np.uint32),
        "p": np.rint(1000.0 * par).astype(np.uint32),
        "u_ppm": np.uint32(min(10**6, max(1, int(round(u * 1e6))))),
    }
    tabs = [_profile_tables(space, float(L0[m]), frac_tp) for m in range(M)]
    out["allowed"] = np.stack([t[0] for t in tabs])
    out["rate"] = np.stack([t[1] for t in tabs])
    out["lat"] = np.stack([t[2] for t in tabs])
    return out


def _stack(space: dict, parts: list, G, H: int, meta: dict) -> dict:
    batch = {"space": space, "H": int(H)}
    for key in ("W", "n", "p", "allowed", "rate", "lat"):
        batch[key] = np.ascontiguousarray(np.stack([q[key] for q in parts]))
    batch["u_ppm"] = np.asarray([q["u_ppm"] for q in parts], dtype=np.uint32)
    batch["G"] = np.broadcast_to(np.asarray(G, dtype=np.uint32), (len(parts),)).copy()
    batch.update(meta)
    return batch


def make_batch(cfg_id: int, instances) -> dict:
    """Instances ``instances`` of workload ``cfg_id``; instance i is seeded by (2604, 15186, cfg, i)."""
    cfg = CONFIGS[cfg_id]
    space = _space_of(cfg)
    parts = []
    for inst in instances:
        rng = np.random.default_rng(np.random.SeedSequence([*SEED_ROOT, cfg_id, int(inst)]))
        parts.append(_draw_instance(space, rng, cfg.param_range, cfg.sort_sizes, cfg.alpha,
                                    cfg.target, cfg.target_range, cfg.frac_tp))
    return _stack(space, parts, cfg.gpu_budget, HBM_BYTES_MI355X,
                  {"cfg": cfg_id, "instances": [int(i) for i in instances], "name": cfg.name})


def make_instance(cfg_id: int, inst: int = 0) -> dict:
    return make_batch(cfg_id, [inst])


def make_custom(seed: int, M: int, tp_values, frac_q, D: int, K: int, G, *, count: int = 1,
                frac_den: int = 4, param_range=(0.5e9, 70e9), alpha: float = 1.0,
                frac_tp: bool = False, H: int = HBM_BYTES_MI355X, deny_prob: float = 0.0) -> dict:
    """Instances of an arbitrary search-space shape (for tests: ragged option counts, K=1, M=1...).

    ``deny_prob`` additionally clears random ``allowed`` entries, to exercise invalid options.
    """
    space = {"M": int(M), "tp": np.asarray(tp_values, dtype=np.uint32),
             "fq": np.asarray(frac_q, dtype=np.uint32), "Q": int(frac_den), "D": int(D), "K": int(K)}
    parts = []
    for c in range(count):
        rng = np.random.default_rng(np.random.SeedSequence([*SEED_ROOT, 1000 + int(seed), c]))
        part = _draw_instance(space, rng, param_range, False, alpha, "uniform", (0.1, 0.9), frac_tp)
        if deny_prob > 0:
            mask = rng.uniform(size=part["allowed"].shape) < deny_prob
            part["allowed"] = np.where(mask, 0, part["allowed"]).astype(np.uint8)
        parts.append(part)
    return _stack(space, parts, G, H, {"cfg": None, "instances": list(range(count)),
                                       "name": f"custom-{seed}"})


def select(batch: dict, i: int) -> dict:
    """Single-instance view (batch dimension of length 1) of instance i of a batch."""
    out = {"space": batch["space"], "H": batch["H"]}
    for key in ("W", "n", "p", "allowed", "rate", "lat", "u_ppm", "G"):
        out[key] = np.ascontiguousarray(batch[key][i:i + 1])
    return out


def sample_indices(cfg_id: int, inst: int, count: int, N: int) -> np.ndarray:
    """``count`` candidate indices uniform over [0, N), then the two ends of the range."""
    rng = np.random.default_rng(np.random.SeedSequence([*SEED_ROOT, cfg_id, int(inst), 7]))
    idx = rng.integers(0, N, size=count, dtype=np.uint64)
    return np.concatenate([idx, np.asarray([0, N - 1], dtype=np.uint64)])


def target_from_tmax(u_ppm: int, tmax: int) -> int:
    """Target workflow rate (milli-req/s) = max(1, floor(u * T_max)), u given in ppm."""
    return max(1, (int(u_ppm) * int(tmax)) // 10**6)
