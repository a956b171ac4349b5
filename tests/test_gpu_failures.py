"""Failure paths of the C ABI on an MI355X: every failing call returns its documented status,
and the search context it failed on still gives the oracle's results afterwards (the ABI
promises that a failed call leaves the context unchanged).  Allocation failure is forced from
the host with the library's ALP_TEST_FAIL_ALLOC hook, so no kernel runs in a broken state."""
from __future__ import annotations

import ctypes as C

import numpy as np
import pytest

from workloads import make_batch, target_from_tmax

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def env():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2604_15186_amd import alp
    import oracle
    alp.lib()
    b = make_batch(1, range(12))
    G = np.asarray(b["G"], dtype=np.uint32)
    lam = np.asarray([target_from_tmax(int(b["u_ppm"][i]),
                                       oracle.tmax(oracle.Instance(b, i), int(G[i])))
                      for i in range(len(G))], dtype=np.uint32)
    want = [oracle.argmin(oracle.Instance(b, i), int(G[i]), int(lam[i])) for i in range(len(G))]
    return alp, torch, b, G, lam, want


def _matches_oracle(alp, ctx, G, lam, want):
    out = ctx.search_batch(G, lam)
    for i, w in enumerate(want):
        assert int(out[i]["index"]) == (w["x"] if w["x"] is not None else alp.NO_INDEX), i
        if w["x"] is not None:
            assert int(out[i]["latency_us"]) == w["L"]
    one = ctx.search(3, int(G[3]), int(lam[3]))
    assert one.tobytes() == out[3].tobytes()
    return out


def _raises(alp, status, fn, *args, **kw):
    with pytest.raises(alp.AlpError) as err:
        fn(*args, **kw)
    assert err.value.status == status, str(err.value)


def test_failing_calls_leave_the_context_unchanged(env):
    alp, torch, b, G, lam, want = env
    lib = alp.lib()
    with alp.Context(b) as ctx:
        ref = _matches_oracle(alp, ctx, G, lam, want)
        raw = ctx._ctx
        failing = [
            (alp.ALP_EINVAL, lambda: ctx.search(99, 16, 1)),                      # instance
            (alp.ALP_EINVAL, lambda: ctx.search_batch(G, lam, instances=np.full(12, 40))),
            (alp.ALP_EINVAL, lambda: ctx.max_throughput(G, instances=np.full(12, 40))),
            (alp.ALP_EINVAL, lambda: ctx.set_launch(7)),                          # variant
            (alp.ALP_EINVAL, lambda: ctx.set_launch(1, 0, 96 + 1)),               # block size
            (alp.ALP_EINVAL, lambda: ctx.eval_candidates(0, 16, 1, np.asarray([1 << 40]))),
            (alp.ALP_EINVAL, lambda: ctx.allocate_workflows(np.ones(17, np.uint32), 8)),
            (alp.ALP_EINVAL, lambda: ctx.allocate_workflows(lam[:2], 2000)),
            (alp.ALP_EINVAL, lambda: ctx.search_pruned(G, lam, flags=8)),
            (alp.ALP_EINVAL, lambda: ctx.place(ref, np.full(12, 65, np.uint32))),
        ]
        for status, call in failing:
            with pytest.raises(alp.AlpError) as err:
                call()
            assert err.value.status == status, str(err.value)
            out = ctx.search_batch(G, lam)
            assert out.tobytes() == ref.tobytes()
        # raw calls with missing pointers
        assert lib.alp_search(raw, 0, 16, 1, None) == alp.ALP_EINVAL
        assert lib.alp_search_batch(raw, 3, None, None, None, None) == alp.ALP_EINVAL
        assert lib.alp_search_batch_async(raw, 3, None, None, None, None) == alp.ALP_EINVAL
        assert lib.alp_max_throughput(raw, 3, None, None, None) == alp.ALP_EINVAL
        assert lib.alp_eval_candidates(raw, 0, 16, 1, None, 3, None) == alp.ALP_EINVAL
        assert lib.alp_kernel_times(raw, None, None) == alp.ALP_EINVAL
        assert lib.alp_set_timing(raw, -1) == alp.ALP_EINVAL
        _matches_oracle(alp, ctx, G, lam, want)


def test_forced_allocation_failure_is_enomem(env, monkeypatch):
    alp, torch, b, G, lam, want = env
    with alp.Context(b) as ctx:
        small = ctx.search(0, int(G[0]), int(lam[0]))         # scratch for one search
        monkeypatch.setenv("ALP_TEST_FAIL_ALLOC", "1")
        # a batch needs larger scratch: ENOMEM, nothing launched
        _raises(alp, alp.ALP_ENOMEM, ctx.search_batch, G, lam)
        _raises(alp, alp.ALP_ENOMEM, ctx.search_pruned, G, lam)
        none = np.zeros(12, alp.RESULT_DTYPE)
        none["status"] = alp.ALP_INFEASIBLE                    # valid records, nothing to place
        _raises(alp, alp.ALP_ENOMEM, ctx.place, none, G)
        assert "out of memory" in alp.last_error().lower() or "hipMalloc" in alp.last_error()
        # what needs no new memory still works while allocations fail
        again = ctx.search(0, int(G[0]), int(lam[0]))
        assert again.tobytes() == small.tobytes()
        # a new context cannot be created, and says so
        _raises(alp, alp.ALP_ENOMEM, alp.Context, make_batch(0, range(2)))
        sctx = C.c_void_p()
        assert alp.lib().alp_stats_create(C.byref(sctx), 0, None) == alp.ALP_ENOMEM
        assert not sctx.value
        monkeypatch.delenv("ALP_TEST_FAIL_ALLOC")
        _matches_oracle(alp, ctx, G, lam, want)


def test_forced_allocation_failure_in_statistics(env, monkeypatch):
    alp, torch, *_ = env
    from workloads.traces import make_traces
    import oracle
    tr = make_traces("beam", 64, 3)
    dev = [torch.from_numpy(np.ascontiguousarray(tr[k]).view(t)).cuda()
           for k, t in (("offsets", np.int64), ("llm", np.int32), ("start", np.int64),
                        ("end", np.int64))]
    want = oracle.trace_stats(tr["M"], tr["offsets"], tr["llm"], tr["start"], tr["end"])
    with alp.StatsContext(0) as sc:
        monkeypatch.setenv("ALP_TEST_FAIL_ALLOC", "1")
        _raises(alp, alp.ALP_ENOMEM, sc.compute, tr["M"], *dev)   # offsets buffer cannot grow
        monkeypatch.delenv("ALP_TEST_FAIL_ALLOC")
        out = sc.compute(tr["M"], *dev)
        for m in range(tr["M"]):
            assert int(out[m]["n_milli"]) == want[m]["n_milli"]
            assert int(out[m]["p_milli"]) == want[m]["p_milli"]
