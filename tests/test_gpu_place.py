"""Parity of the HIP placement (Section 6) with the oracle, through the C ABI.  Needs an MI355X.
Every field must be identical: status, replicas placed, GPUs and nodes used, and every
replica's node and GPU set."""
from __future__ import annotations

import json
import os

import numpy as np
import pytest

import oracle
from workloads import make_batch, make_custom, target_from_tmax

pytestmark = pytest.mark.gpu

CASES = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "hand_cases.json")))[
    "placement_cases"]


@pytest.fixture(scope="module")
def alp():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2604_15186_amd import alp as binding
    binding.lib()
    return binding


def _ctx(alp, M, Q=4):
    b = make_custom(60 + M, M, (1, 2, 4, 8), tuple(range(1, Q + 1)) if Q <= 8 else (1, 2, 4, Q),
                    16, 1, 8, count=1, frac_den=Q)
    return alp.Context(b)


def _records(alp, allocs):
    """allocs: list of (tp, q, d) lists per LLM, or None for an infeasible result."""
    res = np.zeros(len(allocs), dtype=alp.RESULT_DTYPE)
    for i, a in enumerate(allocs):
        if a is None:
            res[i]["status"] = 5
            continue
        for m, (t, q, d) in enumerate(zip(*a)):
            res[i]["tp"][m], res[i]["frac_units"][m], res[i]["replicas"][m] = t, q, d
    return res


def _compare(Q, G, tp, q, d, rec):
    want = oracle.place(Q, G, tp, q, d)
    n = sum(d)
    assert (int(rec["status"]) == 0) == want["placed"]
    assert (int(rec["replicas"]), int(rec["gpus_used"]), int(rec["nodes_used"])) == \
        (want["replicas"], want["gpus_used"], want["nodes_used"])
    assert [int(v) for v in rec["slot"][:n]] == want["slot"]
    assert all(int(v) == 0xFFFF for v in rec["slot"][n:])


def test_hand_cases(alp):
    for case in CASES:
        M = len(case["tp"])
        with _ctx(alp, M, case["Q"]) as ctx:
            res = _records(alp, [(case["tp"], case["q"], case["d"])])
            rec = ctx.place(res, [case["G"]])[0]
            _compare(case["Q"], case["G"], case["tp"], case["q"], case["d"], rec)


@pytest.mark.parametrize("M", [1, 3, 5])
def test_random_allocations(alp, M):
    rng = np.random.default_rng(100 + M)
    allocs, Gs = [], []
    for _ in range(3000):
        tp = [int(rng.choice([1, 2, 4, 8])) for _ in range(M)]
        q = [int(rng.integers(1, 5)) for _ in range(M)]
        d = [int(rng.integers(1, 17)) for _ in range(M)]
        allocs.append((tp, q, d))
        Gs.append(int(rng.choice([1, 3, 4, 8, 9, 12, 16, 24, 32, 40, 64])))
    with _ctx(alp, M) as ctx:
        out = ctx.place(_records(alp, allocs), Gs)
    placed = 0
    for (tp, q, d), G, rec in zip(allocs, Gs, out):
        _compare(4, G, tp, q, d, rec)
        placed += int(rec["status"]) == 0
    assert 0 < placed < len(allocs)


def test_search_results_of_the_batch(alp):
    b = make_batch(4, range(4096))
    G = np.asarray(b["G"], dtype=np.uint32)
    with alp.Context(b) as ctx:
        tmax = ctx.max_throughput(G)
        lam = [target_from_tmax(int(b["u_ppm"][i]), int(tmax[i])) for i in range(len(G))]
        res = ctx.search_batch(G, lam)
        out = ctx.place(res, G)
    for i in range(len(G)):
        M = 3
        tp = [int(v) for v in res[i]["tp"][:M]]
        q = [int(v) for v in res[i]["frac_units"][:M]]
        d = [int(v) for v in res[i]["replicas"][:M]]
        _compare(4, int(G[i]), tp, q, d, out[i])


def test_infeasible_and_rejected(alp):
    with _ctx(alp, 2) as ctx:
        out = ctx.place(_records(alp, [None, ([1, 2], [4, 4], [1, 1])]), [8, 8])
        assert int(out[0]["status"]) == 5 and int(out[0]["replicas"]) == 0
        assert all(int(v) == 0xFFFF for v in out[0]["slot"])
        assert int(out[1]["status"]) == 0
        with pytest.raises(alp.AlpError):
            ctx.place(_records(alp, [([1, 1], [4, 4], [1, 1])]), [65])
        with pytest.raises(alp.AlpError):
            ctx.place(_records(alp, [([3, 1], [4, 4], [1, 1])]), [8])     # tp 3 not in the space
        with pytest.raises(alp.AlpError):
            ctx.place(_records(alp, [([1, 1], [4, 4], [1, 17])]), [8])    # 17 replicas
        assert len(ctx.place(np.zeros(0, alp.RESULT_DTYPE), [])) == 0
