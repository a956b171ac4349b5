"""Pins of the oracle to what the paper and the mathematics fix (CPU only).

* hand-derived cases (``golden/hand_cases.json``): option terms, candidate evaluations, argmins,
  maximum throughputs, each value worked out by hand;
* invariants the paper states or the definitions imply (throughput linear in replicas,
  latency falling with replicas, monotonicity in budget and target, separability when the
  budget does not bind, the load/throughput identity, the K=1 closed form);
* two different algorithms for the same quantity agreeing: brute-force maximum throughput vs
  the threshold method, brute-force argmin vs dynamic programming;
* the C oracle vs a naive pure-Python statement on tiny random spaces.
"""
from __future__ import annotations

import itertools

import numpy as np
import pytest

import oracle
from oracle import pyref
from workloads import CONFIGS, make_batch, make_custom, num_options, target_from_tmax

from dp_knapsack import dp_argmin
from hand_cases import case_batch, load_cases

CASES = load_cases()
NONE64 = (1 << 64) - 1


@pytest.mark.parametrize("case", CASES, ids=[c["id"] for c in CASES])
def test_hand_terms(case):
    b = case_batch(case)
    inst = oracle.Instance(b, 0)
    for t in case["terms"]:
        got = oracle.option_term(inst, t["m"], t["o"], t["lambda"])
        ref = pyref.option_term(b, 0, t["m"], t["o"], t["lambda"])
        for key in ("ok", "thr_ok", "u", "tau", "c"):
            if key in t:
                assert got[key] == t[key], (case["id"], t, key, got)
                assert ref[key] == t[key], (case["id"], t, key, ref)


@pytest.mark.parametrize("case", CASES, ids=[c["id"] for c in CASES])
def test_hand_evals(case):
    b = case_batch(case)
    inst = oracle.Instance(b, 0)
    for e in case["evals"]:
        got = oracle.evaluate(inst, e["G"], e["lambda"], e["x"])
        ref = pyref.evaluate(b, 0, e["G"], e["lambda"], e["x"])
        want = {"flags": e["flags"], "L": NONE64 if e["L"] is None else e["L"], "T": e["T"],
                "U": e["U"]}
        assert got == want, (case["id"], e, got)
        assert ref == want, (case["id"], e, ref)


@pytest.mark.parametrize("case", CASES, ids=[c["id"] for c in CASES])
def test_hand_queries(case):
    b = case_batch(case)
    inst = oracle.Instance(b, 0)
    for q in case["queries"]:
        got = oracle.argmin(inst, q["G"], q["lambda"])
        ref = pyref.argmin(b, 0, q["G"], q["lambda"])
        assert got["x"] == q["x"], (case["id"], q, got)
        assert ref["x"] == q["x"], (case["id"], q, ref)
        if q["x"] is not None:
            assert got["L"] == q["L"]
            ev = oracle.evaluate(inst, q["G"], q["lambda"], q["x"])
            assert (ev["flags"], ev["L"], ev["T"], ev["U"]) == (7, q["L"], q["T"], q["U"])


@pytest.mark.parametrize("case", CASES, ids=[c["id"] for c in CASES])
def test_hand_tmax(case):
    b = case_batch(case)
    inst = oracle.Instance(b, 0)
    for t in case["tmax"]:
        assert oracle.tmax(inst, t["G"]) == t["T"], (case["id"], t)
        assert oracle.tmax_brute(inst, t["G"]) == t["T"], (case["id"], t)


def test_hand_tmax_maximiser_count():
    case = next(c for c in CASES if "count_tmax_maximisers" in c)
    spec = case["count_tmax_maximisers"]
    inst = oracle.Instance(case_batch(case), 0)
    xs = np.arange(inst.N, dtype=np.uint64)
    ev = oracle.evaluate_many(inst, spec["G"], 0, xs)
    hits = ((ev["flags"] & 1) == 1) & ((ev["flags"] & 4) == 4) & (ev["T"] == spec["T"])
    assert int(hits.sum()) == spec["count"]


def _small_spaces():
    # (seed, M, tp, fq, D, K, G, frac_tp, deny)
    yield (1, 2, (1, 2), (1, 2, 4), 3, 4, 4, False, 0.0)
    yield (2, 3, (1, 2, 4), (2, 4), 2, 3, 6, True, 0.2)
    yield (3, 1, (1, 2, 4, 8), (1, 2, 3, 4), 5, 8, 5, False, 0.0)
    yield (4, 3, (1,), (1, 2, 3, 4), 3, 1, 3, False, 0.1)
    yield (5, 4, (1, 2), (4,), 3, 2, 4, False, 0.0)


@pytest.mark.parametrize("spec", list(_small_spaces()), ids=lambda s: f"seed{s[0]}")
def test_c_oracle_matches_python_statement(spec):
    seed, M, tps, fqs, D, K, G, frac_tp, deny = spec
    b = make_custom(seed, M, tps, fqs, D, K, G, count=2, frac_tp=frac_tp, deny_prob=deny,
                    param_range=(0.5e9, 300e9))
    for i in range(2):
        inst = oracle.Instance(b, i)
        tmax = oracle.tmax(inst, G)
        assert tmax == oracle.tmax_brute(inst, G)
        for lam in sorted({1, target_from_tmax(int(b["u_ppm"][i]), tmax), tmax, tmax + 1}):
            for m in range(M):
                for o in range(inst.O):
                    assert oracle.option_term(inst, m, o, lam) == pyref.option_term(b, i, m, o, lam)
            xs = np.arange(inst.N, dtype=np.uint64)
            ev = oracle.evaluate_many(inst, G, lam, xs)
            for x in range(0, inst.N, max(1, inst.N // 200)):
                ref = pyref.evaluate(b, i, G, lam, x)
                got = {k: int(ev[k][x]) for k in ("flags", "L", "T", "U")}
                assert got == ref
            assert oracle.argmin(inst, G, lam)["x"] == pyref.argmin(b, i, G, lam)["x"]


def _usable_terms(inst, lam):
    return [[(t["ok"] and t["thr_ok"], t["c"], t["u"]) for t in row]
            for row in oracle.option_terms(inst, lam)]


def test_cfg0_argmin_matches_dp_and_eval():
    """Brute force and DP agree on the 2-LLM workload; the winner evaluates as claimed."""
    b = make_batch(0, range(200))
    Q = int(b["space"]["Q"])
    infeasible = 0
    for i in range(200):
        inst = oracle.Instance(b, i)
        G = int(b["G"][i])
        lam = target_from_tmax(int(b["u_ppm"][i]), oracle.tmax(inst, G))
        got = oracle.argmin(inst, G, lam)
        dp = dp_argmin(_usable_terms(inst, lam), Q * G)
        if dp is None:
            infeasible += 1
            assert got["x"] is None
            continue
        assert (got["x"], got["L"]) == dp
        ev = oracle.evaluate(inst, G, lam, got["x"])
        assert ev["flags"] == 7 and ev["L"] == got["L"] and ev["T"] >= lam
    assert infeasible == 0  # lambda <= T_max always leaves a feasible candidate


def test_cfg0_tmax_threshold_equals_brute_force():
    b = make_batch(0, range(100))
    for i in range(100):
        inst = oracle.Instance(b, i)
        G = int(b["G"][i])
        assert oracle.tmax(inst, G) == oracle.tmax_brute(inst, G)


def test_target_at_tmax_is_feasible_and_above_is_not():
    """lambda = T_max is feasible, T_max + 1 is not (Eq. 2 read as T_w >= lambda)."""
    b = make_batch(0, range(50))
    for i in range(50):
        inst = oracle.Instance(b, i)
        G = int(b["G"][i])
        t = oracle.tmax(inst, G)
        assert t > 0
        assert oracle.argmin(inst, G, t)["x"] is not None
        assert oracle.argmin(inst, G, t + 1)["x"] is None


def test_throughput_linear_in_replicas_and_latency_falls():
    """tau grows with d (Section 4 step 3); with latency rising in load, c falls with d."""
    b = make_batch(1, range(4))
    sp = b["space"]
    D = int(sp["D"])
    for i in range(4):
        inst = oracle.Instance(b, i)
        lam = 1000
        terms = oracle.option_terms(inst, lam)
        for m in range(inst.M):
            for base in range(0, inst.O, D):
                row = terms[m][base:base + D]
                taus = [t["tau"] for t in row]
                assert taus == sorted(taus)
                assert taus[-1] >= D * taus[0] - D  # floor(d*x) >= d*floor(x)
                cs = [t["c"] for t in row if t["thr_ok"]]
                assert cs == sorted(cs, reverse=True)
                thr = [t["thr_ok"] for t in row]
                assert thr == sorted(thr)  # once sustainable, more replicas stay sustainable


def test_load_identity_r_le_T_iff_tau_ge_lambda():
    """r = ceil(lambda n / (1000 d)) <= T  <=>  floor(1000 d T / n) >= lambda, for all options."""
    b = make_batch(1, range(3))
    for i in range(3):
        inst = oracle.Instance(b, i)
        taus = {t["tau"] for row in oracle.option_terms(inst, 0) for t in row}
        lams = sorted({1} | {max(1, t + dlt) for t in taus for dlt in (-1, 0, 1)})[::7]
        for lam in lams:
            for row in oracle.option_terms(inst, lam):
                for t in row:
                    assert bool(t["thr_ok"]) == (t["tau"] >= lam)


def test_monotone_in_budget_and_target():
    b = make_batch(0, range(30))
    for i in range(30):
        inst = oracle.Instance(b, i)
        G = int(b["G"][i])
        t = oracle.tmax(inst, G)
        lams = [max(1, t * k // 5) for k in range(1, 6)]
        Ls = [oracle.argmin(inst, G, lam)["L"] for lam in lams]
        assert Ls == sorted(Ls)
        lam = lams[1]
        LG = [oracle.argmin(inst, g, lam)["L"] for g in range(G, G + 4)]
        assert all(x is not None for x in LG) and LG == sorted(LG, reverse=True)


def test_separable_when_budget_never_binds():
    """With a budget no candidate can exceed, the argmin is each LLM's own best option."""
    b = make_batch(1, range(3))
    for i in range(3):
        inst = oracle.Instance(b, i)
        lam = target_from_tmax(int(b["u_ppm"][i]), oracle.tmax(inst, int(b["G"][i])))
        terms = oracle.option_terms(inst, lam)
        G_big = sum(max(t["u"] for t in row) for row in terms)  # in quarters >= needed GPUs
        x = 0
        L = 0
        for row in terms:
            usable = [(t["c"], o) for o, t in enumerate(row) if t["ok"] and t["thr_ok"]]
            c, o = min(usable)
            x = x * inst.O + o
            L += c
        got = oracle.argmin(inst, G_big, lam)
        assert (got["x"], got["L"]) == (x, L)


def test_k1_closed_form_minimal_replicas():
    """With load-independent latency (K=1) more replicas never help, so each chosen d_m is the
    least replica count that sustains the target: ceil(lambda n_m / (1000 T_m))."""
    b = make_custom(11, 3, (1, 2, 4), (1, 2, 4), 6, 1, 8, count=4)
    sp = b["space"]
    D, nfq = int(sp["D"]), len(sp["fq"])
    for i in range(4):
        inst = oracle.Instance(b, i)
        G = int(b["G"][i])
        lam = target_from_tmax(int(b["u_ppm"][i]), oracle.tmax(inst, G))
        got = oracle.argmin(inst, G, lam)
        assert got["x"] is not None
        digits = pyref.digits(b, got["x"])
        for m, o in enumerate(digits):
            d = o % D + 1
            j = (o // D) % nfq
            ii = (o // D) // nfq
            T = int(b["rate"][i, m, ii, j, 0])
            n = int(b["n"][i, m])
            assert d == -((-lam * n) // (1000 * T))


def test_dp_agrees_with_brute_force_on_random_spaces():
    for seed, M, tps, fqs, D, K, G in [(21, 3, (1, 2, 4, 8), (1, 2, 4), 4, 8, 6),
                                       (22, 2, (1, 2, 4, 8), (1, 2, 3, 4), 8, 8, 5),
                                       (23, 4, (1, 2), (2, 4), 3, 2, 7)]:
        b = make_custom(seed, M, tps, fqs, D, K, G, count=3, deny_prob=0.15)
        for i in range(3):
            inst = oracle.Instance(b, i)
            for lam in (1, target_from_tmax(int(b["u_ppm"][i]), oracle.tmax(inst, G))):
                got = oracle.argmin(inst, G, lam)
                dp = dp_argmin(_usable_terms(inst, lam), int(b["space"]["Q"]) * G)
                assert (None if dp is None else dp) == (None if got["x"] is None
                                                        else (got["x"], got["L"]))


def test_sliced_argmin_merges_to_full():
    b = make_batch(1, [5])
    inst = oracle.Instance(b, 0)
    G = int(b["G"][0])
    lam = target_from_tmax(int(b["u_ppm"][0]), oracle.tmax(inst, G))
    full = oracle.argmin(inst, G, lam)
    cuts = [0, 1, 1000, inst.N // 3, inst.N // 2 + 7, inst.N]
    parts = [oracle.argmin(inst, G, lam, lo, hi) for lo, hi in zip(cuts, cuts[1:])]
    assert oracle.merge_argmin(parts) == full


def test_generator_tables_are_valid():
    for cfg in CONFIGS:
        b = make_batch(cfg, range(3))
        r = b["rate"].astype(np.int64)
        assert (np.diff(r, axis=-1) >= 1).all() and (r >= 1).all() and (r < 2**31).all()
        assert (b["lat"] < 2**31).all() and (b["lat"] >= 1).all()
        assert (b["n"] >= 1).all() and (b["p"] >= 1000).all() and (b["p"] <= 4000).all()
        assert b["rate"].shape[1:] == (CONFIGS[cfg].num_llms, 4, len(CONFIGS[cfg].frac_q), 8)
        O = num_options(b["space"])
        assert O == (48 if cfg == 0 else 128)
        # tp > 1 only with a whole GPU
        tp = b["space"]["tp"]
        fq = b["space"]["fq"]
        for ii, j in itertools.product(range(len(tp)), range(len(fq))):
            expect = 1 if (tp[ii] == 1 or fq[j] == 4) else 0
            assert (b["allowed"][:, :, ii, j] == expect).all()


def test_generator_is_deterministic():
    a = make_batch(2, [1])
    b = make_batch(2, [1])
    for k in ("W", "n", "p", "allowed", "rate", "lat", "u_ppm"):
        assert np.array_equal(a[k], b[k])


# ------------------------------------------------------------------------------------------
# Several workflows sharing a GPU pool (Section 5, scheduling multiple workflows).
import json as _json  # noqa: E402
import os as _os  # noqa: E402

from alloc_dp import split as _split_dp  # noqa: E402

_ALLOC = _json.load(open(_os.path.join(_os.path.dirname(__file__), "golden", "hand_cases.json")))[
    "allocation_cases"]


def _table(L):
    return np.asarray([[oracle.U64_NONE if v is None else v for v in row] for row in L],
                      dtype=np.uint64)


def _expect(e):
    return None if e is None else (e["g"], e["max"], e["sum"])


@pytest.mark.parametrize("case", _ALLOC["tables"], ids=[c["id"] for c in _ALLOC["tables"]])
def test_allocate_hand_tables(case):
    for name, policy in (("egalitarian", oracle.EGALITARIAN), ("social", oracle.SOCIAL)):
        got = oracle.allocate(_table(case["L"]), policy)
        assert got == _expect(case[name]), (case["id"], name, got)
        assert _split_dp(case["L"], case["G"], policy) == _expect(case[name])


def test_allocate_hand_workflows():
    spec = _ALLOC["workflows"]
    cases = {c["id"]: c for c in CASES}
    L = []
    for cid, lam in zip(spec["cases"], spec["lambda"]):
        inst = oracle.Instance(case_batch(cases[cid]), 0)
        row = []
        for g in range(len(spec["L"][0])):
            r = oracle.argmin(inst, g, lam)
            row.append(r["L"])
        L.append(row)
    assert L == spec["L"]
    for q in spec["queries"]:
        sub = [row[: q["G"] + 1] for row in L]
        for name, policy in (("egalitarian", oracle.EGALITARIAN), ("social", oracle.SOCIAL)):
            assert oracle.allocate(_table(sub), policy) == _expect(q[name]), (q, name)


def test_allocate_brute_force_equals_threshold_dp():
    rng = np.random.default_rng(5)
    for trial in range(300):
        W = int(rng.integers(1, 5))
        G = int(rng.integers(0, 9))
        L = []
        for _ in range(W):
            first = int(rng.integers(0, G + 2))           # fewest GPUs that make w feasible
            vals = sorted(rng.integers(1, 40, size=G + 1).tolist(), reverse=True)
            L.append([None if g < first else vals[g] for g in range(G + 1)])
        for policy in (oracle.EGALITARIAN, oracle.SOCIAL):
            assert oracle.allocate(_table(L), policy) == _split_dp(L, G, policy), (trial, L, G)


# ------------------------------------------------------------------------------------------
# The paper's pruned search (Section 5, steps 1-3).
import math as _math  # noqa: E402

from pruned_ref import EDGE_SPACES, edge_batch as _pruned_edge_batch  # noqa: E402
from pruned_ref import placeable as _placeable, pruned as _pruned_literal  # noqa: E402


def test_pruned_unpruned_count_is_the_papers():
    # Section 5, step 1: 5 LLMs, 16 GPUs, 10 fractions per GPU give C(164, 4), about 29 million.
    assert oracle.count_fractions(5, 160, [0] * 5, False) == 29_051_001 == _math.comb(164, 4)
    assert oracle.binomial(164, 4) == 29_051_001
    for M, total in [(1, 7), (2, 9), (3, 12), (4, 10)]:
        assert oracle.count_fractions(M, total, [0] * M, False) == _math.comb(total + M - 1, M - 1)


def _partitions_at_most(n, k):
    # partitions of n into at most k parts: p(n, k) = p(n, k - 1) + p(n - k, k)
    if n == 0:
        return 1
    if n < 0 or k == 0:
        return 0
    return _partitions_at_most(n, k - 1) + _partitions_at_most(n - k, k)


def test_pruned_ordered_count_is_partitions():
    assert oracle.count_fractions(3, 10, [0] * 3, True) == 14
    for M in range(1, 6):
        for n in range(0, 30):
            assert oracle.count_fractions(M, n, [0] * M, True) == _partitions_at_most(n, M)


def test_pruned_count_with_bounds_by_brute_force():
    rng = np.random.default_rng(5)
    for _ in range(60):
        M = int(rng.integers(1, 5))
        total = int(rng.integers(0, 14))
        lo = [int(v) for v in rng.integers(0, 4, size=M)]
        for ordered in (False, True):
            want = 0
            for f in itertools.product(range(total + 1), repeat=M):
                if sum(f) != total or any(f[k] < lo[k] for k in range(M)):
                    continue
                if any(f[k] > total - sum(lo[k + 1:]) for k in range(M)):
                    continue
                if ordered and any(f[k] > f[k - 1] for k in range(1, M)):
                    continue
                want += 1
            assert oracle.count_fractions(M, total, lo, ordered) == want, (M, total, lo, ordered)


def test_pruned_placement_rule_matches_backtracking():
    checked = 0
    for Q in (2, 4, 5):
        for a in range(0, 2 * Q):
            for f in range(1, 3 * Q + 1):
                for tp in (1, 2, 3, 4):
                    for q in range(1, Q + 1):
                        for d in range(1, 5):
                            want = _placeable(Q, a, f, tp, q, d)
                            assert oracle.fits(Q, a, f, tp, q, d) == want, (Q, a, f, tp, q, d)
                            checked += want
    assert checked > 100


def test_pruned_hand_case():
    case = next(c for c in load_cases() if c["id"] == "H2")
    b = case_batch(case)
    inst = oracle.Instance(b, 0)
    for q in case["pruned"]:
        got = oracle.pruned(inst, q["G"], q["lambda"], q["flags"])
        assert got["x"] == q["x"] and got["vectors"] == q["vectors"], (q, got)
        assert got["unpruned"] == q["unpruned"]
        if q["x"] is not None:
            assert got["L"] == q["L"]
        assert _pruned_literal(b, 0, q["G"], q["lambda"], q["flags"]) == \
            {k: got[k] for k in ("x", "L", "vectors")}


def _pruned_spaces():
    # (seed, M, tp, fq, Q, D, K, G)
    yield (11, 2, (1, 2), (1, 2, 4), 4, 3, 3, 3)
    yield (12, 3, (1, 2), (2, 4), 4, 2, 2, 2)
    yield (13, 2, (1, 2, 4), (1, 2, 3, 4), 4, 4, 4, 4)
    yield (14, 3, (1,), (1, 2, 3), 3, 3, 1, 3)
    yield (15, 1, (1, 2), (1, 2, 4), 4, 4, 3, 3)


@pytest.mark.parametrize("spec", list(_pruned_spaces()), ids=lambda s: f"seed{s[0]}")
def test_pruned_matches_literal_statement(spec):
    seed, M, tps, fqs, Q, D, K, G = spec
    b = make_custom(seed, M, tps, fqs, D, K, G, count=2, frac_den=Q, param_range=(0.5e9, 150e9))
    for i in range(2):
        inst = oracle.Instance(b, i)
        tmax = oracle.tmax(inst, G)
        for lam in sorted({1, max(1, tmax // 3), max(1, tmax // 2), tmax}):
            for flags in (0, 1, 2, 3):
                got = oracle.pruned(inst, G, lam, flags)
                assert {k: got[k] for k in ("x", "L", "vectors")} == \
                    _pruned_literal(b, i, G, lam, flags), (i, lam, flags)




@pytest.mark.parametrize("seed,variant", EDGE_SPACES)
def test_pruned_matches_literal_statement_on_edge_spaces(seed, variant):
    b, G = _pruned_edge_batch(seed, variant)
    inst = oracle.Instance(b, 0)
    tmax = oracle.tmax(inst, G)
    for lam in sorted({1, max(1, tmax // 4), max(1, tmax // 2), tmax}):
        for flags in (0, 1, 2, 3):
            got = oracle.pruned(inst, G, lam, flags)
            assert {k: got[k] for k in ("x", "L", "vectors")} == \
                _pruned_literal(b, 0, G, lam, flags), (seed, variant, lam, flags)


@pytest.mark.parametrize("cfg,count", [(0, 40), (1, 16)])
def test_pruned_result_is_a_full_budget_candidate_no_better_than_exhaustive(cfg, count):
    b = make_batch(cfg, range(count))
    found = missed = 0
    for i in range(count):
        inst = oracle.Instance(b, i)
        G = int(b["G"][i])
        lam = target_from_tmax(int(b["u_ppm"][i]), oracle.tmax(inst, G))
        p = oracle.pruned(inst, G, lam)
        ex = oracle.argmin(inst, G, lam)
        assert p["unpruned"] == _math.comb(4 * G + inst.M - 1, inst.M - 1)
        assert p["vectors"] <= p["unpruned"]
        if p["x"] is None:
            missed += ex["x"] is not None
            continue
        found += 1
        e = oracle.evaluate(inst, G, lam, p["x"])
        assert e["flags"] == 7 and e["L"] == p["L"] and e["U"] == 4 * G
        assert ex["x"] is not None and ex["L"] <= p["L"]
        missed += p["L"] > ex["L"]
    assert found > count // 2
    if cfg == 1:
        assert missed > 0       # the pruned search is a heuristic: it misses some optima here
