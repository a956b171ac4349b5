"""The C ABI's promises about streams and contexts, on an MI355X: work ordered on a caller's
HIP stream, distinct contexts independent (also from two threads at once), and results that
do not depend on either."""
from __future__ import annotations

import threading

import numpy as np
import pytest

from workloads import make_batch, target_from_tmax
from workloads.traces import make_traces

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def alp():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2604_15186_amd import alp as binding
    binding.lib()
    return binding


def _queries(alp, b):
    G = np.asarray(b["G"], dtype=np.uint32)
    with alp.Context(b) as ctx:
        tmax = ctx.max_throughput(G)
        lam = np.asarray([target_from_tmax(int(b["u_ppm"][i]), int(tmax[i]))
                          for i in range(len(G))], dtype=np.uint32)
        ref = ctx.search_batch(G, lam)
    return G, lam, ref


def test_search_on_a_caller_stream(alp):
    import torch
    b = make_batch(1, range(16))
    G, lam, ref = _queries(alp, b)
    s = torch.cuda.Stream()
    with alp.Context(b, stream=s.cuda_stream) as ctx:
        # device work queued on the caller's stream before the search must not disturb it
        x = torch.ones(1 << 24, device="cuda")
        with torch.cuda.stream(s):
            y = x * 2
        out = ctx.search_batch(G, lam)
        assert out.tobytes() == ref.tobytes()
        assert float(y[0]) == 2.0
        one = ctx.search(5, int(G[5]), int(lam[5]))
        assert one.tobytes() == ref[5].tobytes()
        pr = ctx.search_pruned(G, lam)
        assert (pr["best"]["status"] <= 5).all()


def test_contexts_in_two_threads(alp):
    import torch
    batches = [make_batch(1, range(8)), make_batch(0, range(64))]
    refs = [_queries(alp, b) for b in batches]
    errors = []

    def work(k):
        try:
            s = torch.cuda.Stream()
            with alp.Context(batches[k], stream=s.cuda_stream) as ctx:
                G, lam, ref = refs[k]
                for _ in range(20):
                    out = ctx.search_batch(G, lam)
                    if out.tobytes() != ref.tobytes():
                        errors.append(f"context {k}: results differ")
                        return
                with pytest.raises(alp.AlpError):
                    ctx.search(10_000, 1, 1)               # instance out of range
        except Exception as e:                              # reported by the main thread
            errors.append(f"context {k}: {e!r}")

    threads = [threading.Thread(target=work, args=(k,)) for k in range(2)]
    for t in threads:
        t.start()
    for t in threads:
        t.join(timeout=120)
    assert not any(t.is_alive() for t in threads)
    assert errors == []


def test_statistics_on_a_caller_stream(alp):
    import torch
    tr = make_traces("rag", 500, 2)
    s = torch.cuda.Stream()
    with alp.StatsContext(0) as c0, alp.StatsContext(0, stream=s.cuda_stream) as c1:
        a = c0.compute(tr["M"], tr["offsets"], tr["llm"], tr["start"], tr["end"])
        with torch.cuda.stream(s):
            b = c1.compute(tr["M"], tr["offsets"], tr["llm"], tr["start"], tr["end"])
        assert a.tobytes() == b.tobytes()


def test_kernel_time_totals_sum_the_calls(alp):
    b = make_batch(1, range(2))
    G, lam, _ = _queries(alp, b)
    with alp.Context(b) as ctx:
        ctx.set_timing(True)
        per_call = np.zeros(3)
        for _ in range(5):
            ctx.search(0, int(G[0]), int(lam[0]))
            per_call += np.asarray(ctx.kernel_times()[:3], dtype=np.float64)
        tot, calls = ctx.kernel_time_totals()
        assert calls == 5 and tot[1] > 0 and np.allclose(tot, per_call, rtol=1e-6, atol=1e-9)
        ctx.set_timing(True)                           # setting again starts new sums
        assert (ctx.kernel_time_totals()[0] == 0).all()
        ctx.set_timing(False)
        ctx.search(0, int(G[0]), int(lam[0]))          # untimed calls add nothing
        tot, calls = ctx.kernel_time_totals()
        assert (tot == 0).all() and calls == 0
        ctx.set_timing(3)                              # calls 0, 3, 6 of the next 8 are timed
        for _ in range(8):
            ctx.search(0, int(G[0]), int(lam[0]))
        tot, calls = ctx.kernel_time_totals()
        assert calls == 3 and tot[1] > 0
        with pytest.raises(alp.AlpError):
            ctx.set_timing(-1)


def test_async_batch_matches_the_synchronous_batch(alp):
    import torch
    b = make_batch(4, range(64))
    G, lam, ref = _queries(alp, b)
    dev = torch.device("cuda", 0)
    s = torch.cuda.Stream()
    with alp.Context(b, stream=s.cuda_stream) as ctx:
        Gd = torch.from_numpy(G.view(np.int32)).to(dev)
        Ld = torch.from_numpy(lam.view(np.int32)).to(dev)
        torch.cuda.synchronize()
        outs = []
        # several calls queued back to back on the context stream, one wait at the end
        for k in range(3):
            o = torch.empty(len(G) * alp.RESULT_DTYPE.itemsize, dtype=torch.uint8, device=dev)
            ctx.search_batch_async(Gd, Ld, o)
            outs.append(o)
        s.synchronize()
        for o in outs:
            assert alp.results_from_device(o, len(G)).tobytes() == ref.tobytes()
        # then a synchronous search on the same context is ordered after them
        assert ctx.search(3, int(G[3]), int(lam[3])).tobytes() == ref[3].tobytes()


def test_async_batch_rejects_bad_instances_per_record(alp):
    import torch
    b = make_batch(1, range(4))
    G, lam, ref = _queries(alp, b)
    dev = torch.device("cuda", 0)
    with alp.Context(b) as ctx:
        inst = np.array([0, 1, 7, 3], dtype=np.uint32)           # 7: only 4 instances loaded
        o = torch.empty(4 * alp.RESULT_DTYPE.itemsize, dtype=torch.uint8, device=dev)
        ctx.search_batch_async(torch.from_numpy(G.view(np.int32)).to(dev),
                               torch.from_numpy(lam.view(np.int32)).to(dev), o,
                               instances=torch.from_numpy(inst.view(np.int32)).to(dev))
        torch.cuda.synchronize()
        got = alp.results_from_device(o, 4)
        assert got[2]["status"] == alp.ALP_EINVAL and got[2]["index"] == (1 << 64) - 1
        for i in (0, 1, 3):
            assert got[i].tobytes() == ref[i].tobytes()
        # a larger batch than before grows the scratch buffers (after waiting for the stream)
        b2 = np.tile(G, 50)
        l2 = np.tile(lam, 50)
        o2 = torch.empty(len(b2) * alp.RESULT_DTYPE.itemsize, dtype=torch.uint8, device=dev)
        ctx.search_batch_async(torch.from_numpy(b2.view(np.int32)).to(dev),
                               torch.from_numpy(l2.view(np.int32)).to(dev), o2,
                               instances=torch.from_numpy(np.tile(np.arange(4, dtype=np.uint32),
                                                                  50).view(np.int32)).to(dev))
        torch.cuda.synchronize()
        assert alp.results_from_device(o2, len(b2)).tobytes() == np.tile(ref, 50).tobytes()
        with pytest.raises(ValueError):
            ctx.search_batch_async(torch.zeros(3, dtype=torch.int64, device=dev),
                                   torch.zeros(3, dtype=torch.int64, device=dev), o)


def test_async_kernel_times_are_collected(alp):
    import torch
    b = make_batch(1, range(2))
    G, lam, _ = _queries(alp, b)
    dev = torch.device("cuda", 0)
    Gd = torch.from_numpy(G.view(np.int32)).to(dev)
    Ld = torch.from_numpy(lam.view(np.int32)).to(dev)
    o = torch.empty(2 * alp.RESULT_DTYPE.itemsize, dtype=torch.uint8, device=dev)
    with alp.Context(b) as ctx:
        # one launch (no option-term kernel), then the two-launch form
        for variant, terms in ((0, False), (16, True)):
            ctx.set_launch(variant)
            ctx.set_timing(True)
            for _ in range(4):
                ctx.search_batch_async(Gd, Ld, o)
            tot, calls = ctx.kernel_time_totals()      # waits for the four queued searches
            last = ctx.kernel_times()
            assert calls == 4 and tot[1] > 0 and (tot[0] > 0) == terms and tot[2] == 0
            assert 0 < last[1] < tot[1]                  # one call's scan, four calls' sum
            ctx.set_timing(True)
            assert (ctx.kernel_time_totals()[0] == 0).all()


def test_wave_row_count_beyond_32_bits_is_rejected(alp):
    """The fixed-range scan counts a wave's rows in 32 bits: an override that would give one
    wave 2^32 rows or more (8 LLMs of 128 options, one 64-thread block: 128^6 = 2^42 rows) is
    rejected with ERANGE before anything is launched, not answered."""
    import torch
    from workloads import make_custom
    b = make_custom(3, 8, (1, 2, 4, 8), (1, 2, 3, 4), 8, 2, 64)
    with alp.Context(b) as ctx:
        assert ctx.num_candidates == 1 << 56
        ctx.set_launch(4, 1, 64, 0)
        with pytest.raises(alp.AlpError) as err:
            ctx.search(0, 64, 1)
        assert err.value.status == alp.ALP_ERANGE and "rows" in str(err.value)
        G = torch.full((1,), 64, dtype=torch.int32, device="cuda")
        out = torch.zeros(alp.RESULT_DTYPE.itemsize, dtype=torch.uint8, device="cuda")
        with pytest.raises(alp.AlpError) as err:
            ctx.search_batch_async(G, G, out)
        assert err.value.status == alp.ALP_ERANGE
        torch.cuda.synchronize()
        assert int(out.sum()) == 0
