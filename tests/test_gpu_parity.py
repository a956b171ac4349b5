"""Parity of the HIP search (through the C ABI) with the oracle.  Needs an MI355X.

Integer results must be bit-identical: winning index, L_w, T_w, share units, per-LLM choices,
per-candidate evaluations, maximum throughput.  Full-size configurations compare against the
results ``golden/make_golden.py`` wrote with the oracle; small spaces compare against the oracle
directly.  Launch geometry and kernel variant must not change any result.
"""
from __future__ import annotations

import json
import os

import numpy as np
import pytest

import oracle
from workloads import make_batch, make_custom, sample_indices, target_from_tmax

from hand_cases import case_batch, load_cases

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
NONE32 = (1 << 32) - 1


@pytest.fixture(scope="module")
def alp():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2604_15186_amd import alp as binding
    binding.lib()
    return binding


def golden(cfg):
    with open(os.path.join(GOLDEN, f"cfg{cfg}_argmin.json")) as f:
        return json.load(f)


def _decode_expect(batch, i, x):
    """Per-LLM (tp, share, replicas) of candidate x, from the space description alone."""
    sp = batch["space"]
    D, nfq, O, M = int(sp["D"]), len(sp["fq"]), \
        len(sp["tp"]) * len(sp["fq"]) * int(sp["D"]), int(sp["M"])
    digits = []
    for _ in range(M):
        digits.append(x % O)
        x //= O
    digits = digits[::-1]
    tp = [int(sp["tp"][(o // D) // nfq]) for o in digits]
    fq = [int(sp["fq"][(o // D) % nfq]) for o in digits]
    d = [o % D + 1 for o in digits]
    pad = [0] * (8 - M)
    return tp + pad, fq + pad, d + pad


def check_result(batch, i, res, x, L, T=None, U=None):
    r = {k: int(res[k]) for k in ("index", "latency_us", "throughput_milli", "gpu_units", "status")}
    if x is None:
        assert r["status"] == 5 and r["index"] == (1 << 64) - 1, r
        return
    assert r["status"] == 0, r
    assert (r["index"], r["latency_us"]) == (x, L), (r, x, L)
    if T is not None:
        assert (r["throughput_milli"], r["gpu_units"]) == (T, U), (r, T, U)
    tp, fq, d = _decode_expect(batch, i, x)
    assert [int(v) for v in res["tp"]] == tp
    assert [int(v) for v in res["frac_units"]] == fq
    assert [int(v) for v in res["replicas"]] == d


def oracle_expect(batch, i, G, lam):
    inst = oracle.Instance(batch, i)
    a = oracle.argmin(inst, G, lam)
    if a["x"] is None:
        return None, None, None, None
    ev = oracle.evaluate(inst, G, lam, a["x"])
    return a["x"], a["L"], ev["T"], ev["U"]


# --------------------------------------------------------------------------------------------
CASES = load_cases()
# Scan variants: row-minimum (automatic distribution), thread-per-candidate, exact-tracking lanes,
# row-minimum with fixed per-wave rows, row-minimum with rows handed out within each block,
# row-minimum over the pair table of LLMs M-3 and M-2 (3 or more LLMs; otherwise automatic).
SEP = 16                       # ALP_LAUNCH_SEPARATE_TERMS: option terms in their own kernel
# Spaces of at most 2^25 candidates run the row-minimum scan in one launch; SEP variants keep the
# two-launch form of each work distribution.
VARIANTS = (1, 2, 3, 4, 5, 6, 1 | SEP, 4 | SEP, 5 | SEP)


@pytest.mark.parametrize("case", CASES, ids=[c["id"] for c in CASES])
def test_hand_cases(alp, case):
    b = case_batch(case)
    with alp.Context(b) as ctx:
        for variant in VARIANTS:
            ctx.set_launch(variant)
            for q in case["queries"]:
                res = ctx.search(0, q["G"], q["lambda"])
                check_result(b, 0, res, q["x"], q.get("L"), q.get("T"), q.get("U"))
        for t in case["tmax"]:
            assert int(ctx.max_throughput([t["G"]])[0]) == t["T"]
        for e in case["evals"]:
            ev = ctx.eval_candidates(0, e["G"], e["lambda"], [e["x"]])[0]
            want_L = NONE32 if e["L"] is None else e["L"]
            assert (int(ev["flags"]), int(ev["latency_us"]), int(ev["throughput_milli"]),
                    int(ev["gpu_units"])) == (e["flags"], want_L, e["T"], e["U"])


def test_cfg0_all_instances_batch_and_single(alp):
    """2-LLM workload, 1000 instances, full space: one batched call vs the oracle."""
    b = make_batch(0, range(1000))
    exp_tmax = np.asarray([oracle.tmax(oracle.Instance(b, i), int(b["G"][i])) for i in range(1000)])
    lam = np.asarray([target_from_tmax(int(b["u_ppm"][i]), exp_tmax[i]) for i in range(1000)],
                     dtype=np.uint32)
    with alp.Context(b) as ctx:
        assert np.array_equal(ctx.max_throughput(b["G"]), exp_tmax)
        out = ctx.search_batch(b["G"], lam)
        for i in range(1000):
            x, L, T, U = oracle_expect(b, i, int(b["G"][i]), int(lam[i]))
            check_result(b, i, out[i], x, L, T, U)
        for i in (0, 1, 999):
            check_result(b, i, ctx.search(i, int(b["G"][i]), int(lam[i])),
                         *oracle_expect(b, i, int(b["G"][i]), int(lam[i])))


@pytest.mark.parametrize("cfg", [1, 2, 3])
def test_full_space_matches_golden(alp, cfg):
    g = golden(cfg)
    rows = g["results"]
    b = make_batch(cfg, [r["inst"] for r in rows])
    with alp.Context(b) as ctx:
        tm = ctx.max_throughput([r["G"] for r in rows])
        assert [int(v) for v in tm] == [r["tmax"] for r in rows]
        # automatic launch (the pair table from 5 LLMs), the pair table forced, fixed row ranges
        for variant in (0, 6, 4):
            ctx.set_launch(variant)
            for i, r in enumerate(rows):
                res = ctx.search(i, r["G"], r["lambda"])
                check_result(b, i, res, r["x"], r["L"], r["T"], r["U"])
        ctx.set_launch(0)


def test_cfg4_batch_matches_golden(alp):
    """4,096 independent 3-LLM instances in one alp_search_batch call."""
    g = golden(4)
    rows = g["results"]
    b = make_batch(4, [r["inst"] for r in rows])
    with alp.Context(b) as ctx:
        tm = ctx.max_throughput([r["G"] for r in rows])
        assert [int(v) for v in tm] == [r["tmax"] for r in rows]
        want = [(r["x"], r["L"], r["T"], r["U"]) for r in rows]
        # automatic launch, then rows handed out within blocks (several blocks per item, split
        # rows), then fixed per-wave rows with one block per item
        for launch in [(0, 0, 0, 0), (5, 3, 256, 4), (4, 1, 512, 0), (SEP, 0, 0, 0),
                       (5 | SEP, 3, 256, 4)]:
            ctx.set_launch(*launch)
            out = ctx.search_batch([r["G"] for r in rows], [r["lambda"] for r in rows])
            bad = [i for i in range(len(rows))
                   if (int(out[i]["index"]), int(out[i]["latency_us"]),
                       int(out[i]["throughput_milli"]), int(out[i]["gpu_units"])) != want[i]]
            assert not bad, (launch, bad[:10])


@pytest.mark.parametrize("cfg,count", [(2, 1_000_000), (3, 10_000_000)])
def test_random_candidates_elementwise(alp, cfg, count):
    """Sampled candidates of the full-size spaces, evaluated one by one by both sides."""
    r = golden(cfg)["results"][0]
    b = make_batch(cfg, [r["inst"]])
    inst = oracle.Instance(b, 0)
    xs = sample_indices(cfg, r["inst"], count, inst.N)
    x = r["x"]
    xs = np.concatenate([xs, np.asarray([x, x - 1, x + 1], dtype=np.uint64)])
    want = oracle.evaluate_many(inst, r["G"], r["lambda"], xs)
    with alp.Context(b) as ctx:
        got = ctx.eval_candidates(0, r["G"], r["lambda"], xs)
    want_L = np.where(want["L"] == (1 << 64) - 1, NONE32, want["L"]).astype(np.uint64)
    assert np.array_equal(got["flags"], want["flags"])
    assert np.array_equal(got["latency_us"].astype(np.uint64), want_L)
    assert np.array_equal(got["throughput_milli"].astype(np.uint64), want["T"])
    assert np.array_equal(got["gpu_units"].astype(np.uint64), want["U"])


def test_launch_geometry_and_variant_do_not_change_results(alp):
    g = golden(2)["results"][1]
    b = make_batch(2, [g["inst"]])
    with alp.Context(b) as ctx:
        for variant, bpi, tpb, ch in [(1, 0, 0, 0), (1, 1, 64, 0), (1, 7, 128, 0),
                                      (1, 3000, 1024, 0), (1, 0, 0, 1), (1, 0, 0, 2),
                                      (1, 0, 0, 4), (1, 0, 0, 8), (1, 7, 128, 8),
                                      (1, 3000, 1024, 2), (1, 1, 64, 4), (2, 0, 0, 0),
                                      (2, 5, 256, 0), (0, 64, 512, 0), (3, 0, 0, 0),
                                      (3, 5, 128, 0), (4, 0, 0, 0), (4, 7, 128, 4),
                                      (4, 3000, 1024, 0), (5, 0, 0, 0), (5, 1, 64, 0),
                                      (5, 7, 128, 8), (5, 256, 1024, 4), (5, 3000, 1024, 1),
                                      (5, 512, 512, 2), (6, 0, 0, 0), (6, 1, 64, 0),
                                      (6, 7, 128, 16), (6, 300, 1024, 1024), (6, 3000, 256, 1),
                                      (SEP, 0, 0, 0), (1 | SEP, 7, 128, 8), (4 | SEP, 7, 128, 0),
                                      (5 | SEP, 3000, 1024, 1), (5 | SEP, 1, 64, 4)]:
            ctx.set_launch(variant, bpi, tpb, ch)
            res = ctx.search(0, g["G"], g["lambda"])
            check_result(b, 0, res, g["x"], g["L"], g["T"], g["U"])
        for bad in ((1, 0, 0, 3),                      # 3 does not divide 128 / 16
                    (1, 0, 0, 16),                     # 16 divides only the pair table's 1,024
                    (6, 0, 0, 3),                      # 3 does not divide 128 * 128 / 16
                    (7, 0, 0, 0), (0, 0, 96, 0),       # no variant 7; 96 threads
                    (2 | SEP, 0, 0, 0), (6 | SEP, 0, 0, 0)):   # one launch never applies there
            with pytest.raises(alp.AlpError):
                ctx.set_launch(*bad)
        ctx.set_launch(0, 0, 0)
        first = ctx.search(0, g["G"], g["lambda"])
        for _ in range(3):
            assert ctx.search(0, g["G"], g["lambda"]).tobytes() == first.tobytes()


SHAPES = [
    # seed, M, tp, fq, D, K, G, count   (O = |tp|*|fq|*D; 1..8 options per lane)
    (31, 1, (1, 2, 4, 8), (1, 2, 3, 4), 8, 8, 16, 3),      # M = 1, O = 128
    (32, 2, (1, 2), (2, 4), 3, 4, 6, 4),                   # O = 12 (ragged, one lane slot)
    (33, 3, (1, 2, 4), (1, 2, 4), 7, 3, 12, 3),            # O = 63
    (34, 3, (1, 2, 4, 8), (1, 2, 3, 4), 5, 1, 20, 2),      # O = 80, K = 1
    (35, 2, (1, 2, 4, 8), (1, 2, 3, 4), 13, 8, 24, 2),     # O = 208 (four slots)
    (36, 2, (1, 2, 4, 8, 16), (1, 2, 4, 8), 16, 6, 40, 2),  # O = 320 (eight slots), Q = 8
    (37, 4, (1, 2), (4,), 4, 2, 8, 3),                      # O = 8, M = 4
    (38, 6, (1, 2), (2, 4), 2, 2, 10, 1),                   # O = 8, M = 6 (four outer digits)
    (39, 8, (1, 2), (4,), 1, 2, 12, 1),                     # O = 2, M = 8 (largest M)
    (40, 2, (1, 2, 4, 8), (1, 2, 3, 4, 5, 6, 7, 8), 16, 16, 48, 1),  # O = 512, K = 16 (maxima)
]


@pytest.mark.parametrize("spec", SHAPES, ids=[f"seed{s[0]}" for s in SHAPES])
def test_ragged_and_degenerate_spaces(alp, spec):
    seed, M, tps, fqs, D, K, G, count = spec
    Q = 8 if max(fqs) > 4 else 4
    if len(fqs) == 8:
        Q = 8
    b = make_custom(seed, M, tps, fqs, D, K, G, count=count, frac_den=Q, deny_prob=0.1,
                    param_range=(0.5e9, 400e9))
    with alp.Context(b) as ctx:
        tms = ctx.max_throughput([G] * count)
        for i in range(count):
            inst = oracle.Instance(b, i)
            assert int(tms[i]) == oracle.tmax(inst, G)
            t = int(tms[i])
            for lam in sorted({1, target_from_tmax(int(b["u_ppm"][i]), t), t, t + 1}):
                for g in (0, G // 2, G):
                    want = oracle_expect(b, i, g, lam)
                    for variant in VARIANTS:
                        ctx.set_launch(variant)
                        check_result(b, i, ctx.search(i, g, lam), *want)
                    n16 = (inst.O + 15) // 16
                    for ch in (c for c in range(1, n16 + 1) if n16 % c == 0):
                        ctx.set_launch(1 if ch > 1 else 5, 0, 0, ch)
                        check_result(b, i, ctx.search(i, g, lam), *want)
            ctx.set_launch(0)
            xs = np.arange(min(inst.N, 50_000), dtype=np.uint64)
            lam = target_from_tmax(int(b["u_ppm"][i]), t)
            want = oracle.evaluate_many(inst, G, lam, xs)
            got = ctx.eval_candidates(i, G, lam, xs)
            assert np.array_equal(got["flags"], want["flags"])
            assert np.array_equal(got["latency_us"].astype(np.uint64),
                                  np.where(want["L"] == (1 << 64) - 1, NONE32, want["L"]))


def _extreme_batch(seed, K, count=2):
    """Instances whose inputs span the documented ranges rather than a workload's: n and p from
    1 to 2^31 - 1 (with both ends), rates anywhere below 2^31 with gaps of 1 as well as wide
    ones, latencies in any order up to what the 32-bit latency bound allows (2^31 - 1 where p / n
    permits, 0 where it does not), weights from 1 byte to 2^40 (some do not fit) and denied
    pairs.  3 LLMs of 60 options: 216,000 candidates per instance."""
    rng = np.random.default_rng([2604, 15186, 77, seed, K])
    tps, fqs, Q, D, M = (1, 2, 4, 8), (1, 2, 4), 4, 5, 3
    nt, nf, B = len(tps), len(fqs), count

    def logu(lo, hi, size):
        v = np.exp(rng.uniform(np.log(lo), np.log(hi + 1.0), size)).astype(np.int64)
        return np.clip(v, lo, hi)

    n = logu(1, 2**31 - 1, (B, M))
    p = logu(1, 2**31 - 1, (B, M))
    n[0, 0], p[0, 0], n[0, 1], p[0, 1] = 1, 2**31 - 1, 2**31 - 1, 2**31 - 1
    W = logu(1, 2**40, (B, M))
    allowed = (rng.uniform(size=(B, M, nt, nf)) < 0.85).astype(np.uint8)
    rate = np.zeros((B, M, nt, nf, K), np.int64)
    lat = np.zeros((B, M, nt, nf, K), np.int64)
    for b in range(B):
        for m in range(M):
            # every latency term of the LLM stays within (2^32 - 2) / M, so the instance passes
            # the load-time bound on the latency sum
            lmax = min(2**31 - 1, ((2**32 - 2) // M) * int(p[b, m]) // int(n[b, m]))
            for i in range(nt):
                for j in range(nf):
                    r = [int(logu(1, 2**29, 1)[0])]
                    for _ in range(K - 1):
                        gap = 1 if rng.uniform() < 0.3 else int(logu(1, 2**27, 1)[0])
                        r.append(min(r[-1] + gap, 2**31 - 1 - (K - len(r))))
                    rate[b, m, i, j] = r
                    top = lmax if rng.uniform() < 0.3 else int(rng.integers(0, lmax + 1))
                    lat[b, m, i, j] = rng.integers(0, top + 1, K)
    space = {"M": M, "tp": np.asarray(tps, np.uint32), "fq": np.asarray(fqs, np.uint32), "Q": Q,
             "D": D, "K": K}
    return {"space": space, "H": 1 << 40, "W": W.astype(np.uint64), "n": n.astype(np.uint32),
            "p": p.astype(np.uint32), "allowed": allowed, "rate": rate.astype(np.uint32),
            "lat": lat.astype(np.uint32), "u_ppm": np.full(B, 500_000, np.uint32),
            "G": np.full(B, 64, np.uint32), "cfg": None, "instances": list(range(B)),
            "name": f"extreme-{seed}-{K}"}


@pytest.mark.parametrize("K", [1, 2, 7, 16])
def test_option_terms_over_the_input_ranges(alp, K):
    """Every candidate's evaluation, the argmin (one launch and separate option terms) and the
    maximum throughput against the oracle, on inputs at the edges of their ranges: saturated
    normalised throughputs (n = 1), thresholds hit exactly (lambda = floor(1000 d T / n) and one
    more), loads on profile points and in unit-width segments, latency terms near the 32-bit
    bound, one-point curves."""
    b = _extreme_batch(5 + K, K)
    rng = np.random.default_rng([2604, 15186, 78, K])
    sp = b["space"]
    O = len(sp["tp"]) * len(sp["fq"]) * sp["D"]
    with alp.Context(b) as ctx:
        tms = ctx.max_throughput([64, 64])
        for i in range(2):
            inst = oracle.Instance(b, i)
            assert int(tms[i]) == oracle.tmax(inst, 64)
            lams = {1, 2**32 - 1, int(tms[i]) or 1}
            lams |= {int(v) for v in np.exp(rng.uniform(0, np.log(2.0**32 - 1), 4))}
            for _ in range(3):
                m, o = int(rng.integers(0, 3)), int(rng.integers(0, O))
                d, ij = o % sp["D"] + 1, o // sp["D"]
                T = int(b["rate"][i, m, ij // len(sp["fq"]), ij % len(sp["fq"]), K - 1])
                edge = 1000 * d * T // int(b["n"][i, m])
                lams |= {v for v in (edge, edge + 1) if 1 <= v < 2**32}
            xs = np.arange(inst.N, dtype=np.uint64)
            for lam in sorted(lams):
                want = oracle.evaluate_many(inst, 64, lam, xs)
                got = ctx.eval_candidates(i, 64, lam, xs)
                assert np.array_equal(got["flags"], want["flags"]), lam
                assert np.array_equal(got["latency_us"].astype(np.uint64),
                                      np.where(want["L"] == (1 << 64) - 1, NONE32, want["L"])), lam
                assert np.array_equal(got["throughput_milli"].astype(np.uint64), want["T"]), lam
                assert np.array_equal(got["gpu_units"].astype(np.uint64), want["U"]), lam
                for g in (8, 64):
                    expect = oracle_expect(b, i, g, lam)
                    for variant in (0, 1 | SEP):
                        ctx.set_launch(variant)
                        check_result(b, i, ctx.search(i, g, lam), *expect)
                    ctx.set_launch(0)


def test_batch_edge_cases(alp):
    b = make_batch(1, range(3))
    with alp.Context(b) as ctx:
        assert len(ctx.search_batch([], [])) == 0
        G = [16, 0, 16]
        t = ctx.max_throughput(G)
        assert int(t[1]) == 0
        lam = [int(t[0]), 1, int(t[2]) + 1]
        out = ctx.search_batch(G, lam, instances=[0, 1, 2])
        assert int(out[0]["status"]) == 0
        assert int(out[1]["status"]) == 5 and int(out[2]["status"]) == 5
        inst = oracle.Instance(b, 0)
        a = oracle.argmin(inst, 16, int(t[0]))
        assert int(out[0]["index"]) == a["x"]
        # repeated instance ids in one batch
        out = ctx.search_batch([16, 16], [lam[0], lam[0]], instances=[0, 0])
        assert out[0].tobytes() == out[1].tobytes()
        with pytest.raises(alp.AlpError):
            ctx.search(3, 16, 1)
        with pytest.raises(alp.AlpError):
            ctx.eval_candidates(0, 16, 1, [ctx.num_candidates])


@pytest.mark.parametrize("seed", [41, 42, 43])
def test_many_ties_keep_lowest_index(alp, seed):
    """Load-independent, option-independent latencies: every feasible candidate ties, so the
    answer is the lowest feasible index.  Exercises the tie-break at lane, wave, block and grid
    level and the row re-scan."""
    M, G = 4, 12
    b = make_custom(seed, M, (1, 2, 4, 8), (1, 2, 3, 4), 8, 1, G, count=2)
    for i in range(2):
        for m in range(M):
            b["lat"][i, m] = 1000 * (m + 1)
            b["n"][i, m] = 1000
            b["p"][i, m] = 1000
    with alp.Context(b) as ctx:
        for i in range(2):
            inst = oracle.Instance(b, i)
            t = oracle.tmax(inst, G)
            for lam in (1, max(1, t // 3), t):
                want = oracle_expect(b, i, G, lam)
                assert want[0] is not None
                for variant in VARIANTS:
                    ctx.set_launch(variant)
                    check_result(b, i, ctx.search(i, G, lam), *want)


@pytest.mark.parametrize("G,lam_frac", [(1, 0), (2, 0), (3, 2), (6, 3)])
def test_sparse_feasibility_multi_block(alp, G, lam_frac):
    """Budgets so tight that few candidates of a 4-LLM space (64 options each, 2^24 candidates,
    hundreds of blocks) fit: most blocks hold no feasible candidate, a few publish winners, and
    the item's last block must still return the lowest index at the minimum latency."""
    b = make_custom(77, 4, (1, 2, 4, 8), (1, 2, 3, 4), 4, 8, G, count=1, param_range=(0.5e9, 8e9))
    inst = oracle.Instance(b, 0)
    t = oracle.tmax(inst, G)
    lam = max(1, t * lam_frac // 4)
    want = oracle_expect(b, 0, G, lam)
    with alp.Context(b) as ctx:
        for launch in [(0, 0, 0, 0), (4, 0, 0, 0), (5, 0, 0, 0), (5, 64, 512, 0), (1, 0, 0, 4),
                       (6, 0, 0, 0), (6, 16, 256, 64), (SEP, 0, 0, 0), (5 | SEP, 64, 512, 0),
                       (4 | SEP, 0, 0, 0)]:
            ctx.set_launch(*launch)
            check_result(b, 0, ctx.search(0, G, lam), *want)
        ctx.set_launch(0)


# ------------------------------------------------------------------------------------------
# Several workflows sharing a GPU pool.
def _alloc_case(cfg, insts, G_total):
    b = make_batch(cfg, insts)
    W = len(insts)
    share = G_total // W
    lam = [target_from_tmax(int(b["u_ppm"][i]), oracle.tmax(oracle.Instance(b, i), share))
           for i in range(W)]
    return b, lam


@pytest.mark.parametrize("cfg,insts,G_total", [(0, [3, 17, 42, 99], 20), (1, [0, 7, 21], 12),
                                               (0, [5], 9), (1, [2, 11], 40)])
def test_allocate_workflows_matches_oracle(alp, cfg, insts, G_total):
    b, lam = _alloc_case(cfg, insts, G_total)
    L = oracle.workflow_latencies(b, lam, G_total)
    with alp.Context(b) as ctx:
        for policy in (oracle.EGALITARIAN, oracle.SOCIAL):
            want = oracle.allocate(L, policy)
            plan, gpus, res = ctx.allocate_workflows(lam, G_total, policy)
            assert int(plan["policy"]) == policy
            if want is None:
                assert int(plan["status"]) == 5 and gpus is None
                continue
            g, mx, sm = want
            assert int(plan["status"]) == 0
            assert [int(v) for v in gpus] == g
            assert (int(plan["max_latency_us"]), int(plan["sum_latency_us"]),
                    int(plan["gpus_used"])) == (mx, sm, sum(g))
            for w in range(len(insts)):
                check_result(b, w, res[w], *oracle_expect(b, w, g[w], lam[w]))


def test_allocate_workflows_infeasible_and_edges(alp):
    b, lam = _alloc_case(1, [0, 1, 2], 12)
    with alp.Context(b) as ctx:
        plan, gpus, res = ctx.allocate_workflows(lam, 0, oracle.EGALITARIAN)
        assert int(plan["status"]) == 5 and gpus is None
        plan, gpus, res = ctx.allocate_workflows([10**9, lam[1], lam[2]], 12, oracle.SOCIAL)
        assert int(plan["status"]) == 5
        with pytest.raises(alp.AlpError):
            ctx.allocate_workflows(lam, 12, 7)
        with pytest.raises(alp.AlpError):
            ctx.allocate_workflows([1] * 17, 12)


# ------------------------------------------------------------------------------------------
# The paper's pruned search (Section 5, steps 1-3).
from pruned_ref import EDGE_SPACES, edge_batch  # noqa: E402


def _check_pruned(b, i, rec, G, lam, flags):
    inst = oracle.Instance(b, i)
    p = oracle.pruned(inst, G, lam, flags)
    assert (int(rec["vectors"]), int(rec["unpruned"])) == (p["vectors"], p["unpruned"]), (i, G, lam, flags)
    if p["x"] is None:
        check_result(b, i, rec["best"], None, None)
        return
    ev = oracle.evaluate(inst, G, lam, p["x"])
    check_result(b, i, rec["best"], p["x"], p["L"], ev["T"], ev["U"])


def _targets(b, G):
    return [target_from_tmax(int(b["u_ppm"][i]), oracle.tmax(oracle.Instance(b, i), int(G[i])))
            for i in range(len(G))]


def test_pruned_hand_case(alp):
    case = next(c for c in load_cases() if c["id"] == "H2")
    b = case_batch(case)
    with alp.Context(b) as ctx:
        for q in case["pruned"]:
            rec = ctx.search_pruned([q["G"]], [q["lambda"]], q["flags"])[0]
            assert int(rec["vectors"]) == q["vectors"] and int(rec["unpruned"]) == q["unpruned"]
            if q["x"] is None:
                assert int(rec["best"]["status"]) == 5
            else:
                assert (int(rec["best"]["index"]), int(rec["best"]["latency_us"])) == (q["x"], q["L"])


@pytest.mark.parametrize("cfg,count", [(0, 1000), (4, 4096)])
def test_pruned_batch_matches_oracle(alp, cfg, count):
    b = make_batch(cfg, range(count))
    G = np.asarray(b["G"], dtype=np.uint32)
    lam = _targets(b, G)
    with alp.Context(b) as ctx:
        out = ctx.search_pruned(G, lam)
        for i in range(count):
            _check_pruned(b, i, out[i], int(G[i]), lam[i], 3)
        sub = list(range(0, count, max(1, count // 64)))
        for flags in (0, 1, 2):
            out = ctx.search_pruned(G[sub], [lam[i] for i in sub], flags, instances=sub)
            for k, i in enumerate(sub):
                _check_pruned(b, i, out[k], int(G[i]), lam[i], flags)


@pytest.mark.parametrize("cfg,insts", [(1, range(16)), (2, range(4)), (3, [0])])
def test_pruned_larger_spaces_match_oracle(alp, cfg, insts):
    insts = list(insts)
    b = make_batch(cfg, insts)
    G = np.asarray(b["G"], dtype=np.uint32)
    lam = _targets(b, G)
    with alp.Context(b) as ctx:
        for flags in ((0, 1, 2, 3) if cfg < 3 else (3, 1)):
            out = ctx.search_pruned(G, lam, flags)
            for i in range(len(insts)):
                _check_pruned(b, i, out[i], int(G[i]), lam[i], flags)


@pytest.mark.parametrize("M,G,Q", [(5, 16, 10), (5, 8, 10), (6, 4, 8)])
def test_pruned_paper_point_and_six_llms(alp, M, G, Q):
    """Five and six LLMs at the paper's scheduler point (M = 5, 16 GPUs, 10 fractions per GPU)
    and smaller budgets: the walk below the two fixed fractions runs three levels deep."""
    fq = sorted({max(1, round(Q * k / 8)) for k in range(1, 9)})
    b = make_custom(2604, M, (1, 2, 4, 8), fq, 4, 8, G, count=1, frac_den=Q,
                    param_range=(1e9, 70e9), alpha=0.5)
    lam = _targets(b, [G])
    with alp.Context(b) as ctx:
        for flags in ((3, 1) if G * Q > 100 else (3, 1, 0)):     # flags 0: every vector
            out = ctx.search_pruned([G], lam, flags)
            _check_pruned(b, 0, out[0], G, lam[0], flags)


@pytest.mark.parametrize("seed,variant", EDGE_SPACES)
def test_pruned_edge_spaces(alp, seed, variant):
    b, G = edge_batch(seed, variant)
    inst = oracle.Instance(b, 0)
    tmax = oracle.tmax(inst, G)
    lams = sorted({1, max(1, tmax // 4), max(1, tmax // 2), tmax, tmax + 1})
    with alp.Context(b) as ctx:
        for flags in (0, 1, 2, 3):
            out = ctx.search_pruned([G] * len(lams), lams, flags, instances=[0] * len(lams))
            for k, lam in enumerate(lams):
                _check_pruned(b, 0, out[k], G, lam, flags)
        # budgets 0..G in one batch, mixed fraction ranges
        Gs = list(range(0, G + 1))
        out = ctx.search_pruned(Gs, [lams[1]] * len(Gs), 3, instances=[0] * len(Gs))
        for k, g in enumerate(Gs):
            _check_pruned(b, 0, out[k], g, lams[1], 3)


def test_pruned_counts_the_papers_space(alp):
    # Section 5 step 1: 5 LLMs, 16 GPUs, 10 fractions per GPU: C(164, 4) fraction vectors.
    b = make_custom(50, 5, (1, 2, 4, 8), (1, 2, 5, 10), 2, 2, 16, count=1, frac_den=10,
                    param_range=(0.5e9, 70e9))
    inst = oracle.Instance(b, 0)
    lam = max(1, oracle.tmax(inst, 16) // 2)
    with alp.Context(b) as ctx:
        rec = ctx.search_pruned([16], [lam], 0)[0]
        assert int(rec["vectors"]) == 29_051_001 == int(rec["unpruned"])
        _check_pruned(b, 0, rec, 16, lam, 0)
        rec = ctx.search_pruned([16], [lam], 3)[0]
        _check_pruned(b, 0, rec, 16, lam, 3)
        assert int(rec["vectors"]) < 29_051_001


def test_pruned_rejects_out_of_range(alp):
    b = make_custom(51, 5, (1, 2), (1, 2, 4), 2, 2, 64, count=1, frac_den=16)
    with alp.Context(b) as ctx:
        with pytest.raises(alp.AlpError) as e:
            ctx.search_pruned([129], [1], 3)           # Q*G = 2064 units
        assert e.value.status == alp.ALP_EINVAL
        with pytest.raises(alp.AlpError) as e:
            ctx.search_pruned([64], [1], 0)            # C(1028, 4) > 2^34 vectors
        assert e.value.status == alp.ALP_ERANGE
        with pytest.raises(alp.AlpError) as e:
            ctx.search_pruned([4], [1], 4)
        assert e.value.status == alp.ALP_EINVAL
        assert len(ctx.search_pruned([], [], 3)) == 0
