"""alp_search_batch_async_noalloc, the entry point for callers that cannot allocate: on an
MI355X, through the C ABI, its result records equal those of alp_search_batch_async byte for
byte, on two calls in a row with the second smaller, across the scan's launch forms (claimed
sub-rows, fixed row ranges, the pair table); a batch beyond the fixed array is rejected before
anything is queued and leaves the context working."""
from __future__ import annotations

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
    alp.lib()
    return alp, torch


def _device_queries(alp, torch, ctx, b, idx):
    G = np.asarray(b["G"], dtype=np.uint32)[idx]
    tmax = ctx.max_throughput(G, instances=np.asarray(idx, dtype=np.uint32))
    lam = np.asarray([target_from_tmax(int(b["u_ppm"][i]), int(t)) for i, t in zip(idx, tmax)],
                     dtype=np.uint32)
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a, np.uint32).view(np.int32)).cuda()  # noqa: E731
    return dev(G), dev(lam), dev(np.asarray(idx, np.uint32))


def _both(alp, torch, ctx, G, lam, inst):
    n = int(G.numel())
    out_ref = torch.zeros(n * alp.RESULT_DTYPE.itemsize, dtype=torch.uint8, device="cuda")
    out_new = torch.full_like(out_ref, 0xA5)          # leftovers must not leak into results
    ctx.search_batch_async(G, lam, out_ref, instances=inst)
    ctx.search_batch_async(G, lam, out_new, instances=inst, noalloc=True)
    torch.cuda.synchronize()
    return alp.results_from_device(out_ref, n), alp.results_from_device(out_new, n)


@pytest.mark.parametrize("cfg,first,second", [
    (1, 64, 8),          # 3 LLMs: claimed sub-rows
    (2, 4, 1),           # 4 LLMs: claimed whole rows
    (0, 600, 37),        # 2 LLMs, many items: fixed row ranges
])
def test_matches_async_on_two_calls(env, cfg, first, second):
    alp, torch = env
    b = make_batch(cfg, range(first))
    with alp.Context(b) as ctx:
        for n in (first, second):
            idx = list(range(first - n, first))[::-1]       # a different instance order each call
            G, lam, inst = _device_queries(alp, torch, ctx, b, idx)
            ref, got = _both(alp, torch, ctx, G, lam, inst)
            assert got.tobytes() == ref.tobytes(), (cfg, n)
            assert set(got["status"]) <= {alp.ALP_OK, alp.ALP_INFEASIBLE}


def test_pair_form_then_a_smaller_space(env):
    alp, torch = env
    b3 = make_batch(3, [0])
    with alp.Context(b3) as ctx:
        G, lam, inst = _device_queries(alp, torch, ctx, b3, [0])
        ref, got = _both(alp, torch, ctx, G, lam, inst)
        assert got.tobytes() == ref.tobytes()
        assert got[0]["status"] == alp.ALP_OK
    b0 = make_batch(0, range(5))
    with alp.Context(b0) as ctx:
        G, lam, inst = _device_queries(alp, torch, ctx, b0, [4, 0, 2])
        ref, got = _both(alp, torch, ctx, G, lam, inst)
        assert got.tobytes() == ref.tobytes()


def test_rejected_queries_and_oversized_batch(env):
    alp, torch = env
    b = make_batch(1, range(4))
    with alp.Context(b) as ctx:
        G, lam, inst = _device_queries(alp, torch, ctx, b, [0, 1, 2, 3])
        inst[2] = 99                                       # out of range: an EINVAL record
        ref, got = _both(alp, torch, ctx, G, lam, inst)
        assert got.tobytes() == ref.tobytes()
        assert got[2]["status"] == alp.ALP_EINVAL
        # 4,096 3-LLM searches need about 24 MiB of scratch: rejected, nothing queued
        n = 4096
        big = torch.zeros(n, dtype=torch.int32, device="cuda")
        out = torch.zeros(n * alp.RESULT_DTYPE.itemsize, dtype=torch.uint8, device="cuda")
        with pytest.raises(alp.AlpError) as err:
            ctx.search_batch_async(big + 16, big + 1, out, instances=big, noalloc=True)
        assert err.value.status == alp.ALP_ERANGE
        assert "fixed array holds" in str(err.value)
        torch.cuda.synchronize()
        assert int(out.sum()) == 0
        # the context and the array still work
        G, lam, inst = _device_queries(alp, torch, ctx, b, [3, 1])
        ref, got = _both(alp, torch, ctx, G, lam, inst)
        assert got.tobytes() == ref.tobytes()
