"""Parity of the HIP workflow statistics (Section 4, step 2) with the oracle, through the C ABI.
Needs an MI355X.  Every field of every LLM's record must be identical: n_m, p_m, call counts,
summed durations and covered time."""
from __future__ import annotations

import numpy as np
import pytest

import oracle
from workloads.traces import make_traces

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ctx():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2604_15186_amd import alp
    with alp.StatsContext(0) as c:
        yield c


def _pack(traces):
    offsets = [0]
    llm, s, e = [], [], []
    for tr in traces:
        for m, a, b in tr:
            llm.append(m), s.append(a), e.append(b)
        offsets.append(len(llm))
    return (np.asarray(offsets, np.uint64), np.asarray(llm, np.uint32), np.asarray(s, np.uint64),
            np.asarray(e, np.uint64))


def _same(ctx, M, offsets, llm, start, end):
    got = ctx.compute(M, offsets, llm, start, end)
    want = oracle.trace_stats(M, offsets, llm, start, end)
    for f in want.dtype.names:
        assert [int(v) for v in got[f]] == [int(v) for v in want[f]], f
    return got


@pytest.mark.parametrize("shape,R", [("beam", 300), ("rag", 2000), ("beam", 3000)])
def test_synthetic_traces(ctx, shape, R):
    tr = make_traces(shape, R, 11)
    print(f"{shape} R={R} calls={len(tr['llm'])}", flush=True)
    _same(ctx, tr["M"], tr["offsets"], tr["llm"], tr["start"], tr["end"])


def test_long_traces_mixed_with_short(ctx):
    rng = np.random.default_rng(5)
    traces = []
    for n in (3, 2048, 2049, 5000, 0, 20000, 700, 4096, 4097):
        tr = []
        for _ in range(n):
            a = int(rng.integers(0, 1 << 22))
            tr.append((int(rng.integers(0, 4)), a, a + int(rng.integers(0, 50_000))))
        traces.append(tr)
    _same(ctx, 4, *_pack(traces))


def test_wide_and_narrow_time_spans(ctx):
    # short traces whose calls span more than 2^29 us take the (key, end) sort, narrow ones the
    # packed key; both in one launch, with a long trace of each kind
    rng = np.random.default_rng(9)
    traces = []
    for span_bits, n in ((40, 300), (22, 300), (31, 1500), (29, 2048), (30, 2), (35, 3000),
                         (20, 5000), (28, 1)):
        tr = []
        for _ in range(n):
            a = int(rng.integers(0, 1 << span_bits))
            tr.append((int(rng.integers(0, 3)), a, a + int(rng.integers(0, 1 << 20))))
        traces.append(tr)
    _same(ctx, 3, *_pack(traces))


def test_edge_cases(ctx):
    # empty traces, zero-length calls, identical calls, unused LLMs, a single call
    traces = [[], [(0, 5, 5), (0, 7, 7)], [(3, 0, 10)] * 7, [], [(5, 1 << 59, (1 << 59) + 3)],
              [(1, 0, (1 << 32) - 1)]]
    got = _same(ctx, 8, *_pack(traces))
    assert int(got[2]["n_milli"]) == 0 and int(got[2]["p_milli"]) == 0
    assert int(got[3]["p_milli"]) == 7000
    _same(ctx, 1, *_pack([[]]))
    _same(ctx, 1, *_pack([[(0, 0, 1)]]))


def test_call_order_and_time_shift_do_not_matter(ctx):
    tr = make_traces("beam", 200, 4)
    base = _same(ctx, tr["M"], tr["offsets"], tr["llm"], tr["start"], tr["end"])
    rng = np.random.default_rng(2)
    off = tr["offsets"].astype(np.int64)
    perm = np.concatenate([lo + rng.permutation(hi - lo) for lo, hi in zip(off[:-1], off[1:])])
    shift = np.repeat(rng.integers(0, 1 << 30, len(off) - 1), np.diff(off)).astype(np.uint64)
    got = ctx.compute(tr["M"], tr["offsets"], tr["llm"][perm], tr["start"][perm] + shift[perm],
                      tr["end"][perm] + shift[perm])
    assert (got == base).all()


def test_malformed_input_is_rejected(ctx):
    from paper_2604_15186_amd import alp
    cases = [
        (alp.ALP_EINVAL, 2, _pack([[(2, 0, 5)]])),                     # llm out of range
        (alp.ALP_EINVAL, 2, _pack([[(0, 5, 4)]])),                     # ends before it starts
        (alp.ALP_ERANGE, 2, _pack([[(0, 0, 1 << 32)]])),               # duration of 2^32 us
        (alp.ALP_ERANGE, 2, _pack([[(0, 1 << 60, (1 << 60) + 1)]])),   # start beyond 2^60 us
        # a trace of 2^24 + 1 calls (rejected from the offsets alone; the call arrays are not read)
        (alp.ALP_ERANGE, 2, (np.asarray([0, (1 << 24) + 1], np.uint64), np.zeros(1, np.uint32),
                             np.zeros(1, np.uint64), np.ones(1, np.uint64))),
    ]
    for status, M, arrays in cases:
        with pytest.raises(alp.AlpError) as e:
            ctx.compute(M, *arrays)
        assert e.value.status == status
    off, llm, s, e_ = _pack([[(0, 0, 5)], [(0, 1, 2)]])
    for bad in (np.asarray([1, 1, 2], np.uint64), np.asarray([0, 2, 1], np.uint64)):
        with pytest.raises(alp.AlpError) as e:
            ctx.compute(1, bad, llm, s, e_)
        assert e.value.status == alp.ALP_EINVAL
    with pytest.raises(alp.AlpError):
        ctx.compute(9, off, llm, s, e_)
    # the context still works after rejected calls
    _same(ctx, 1, off, llm, s, e_)


def test_trace_of_the_maximum_length(ctx):
    """One trace of 2^24 calls (the most a trace may hold; the long-trace pass sorts it in a
    global scratch region), in random order, between short traces."""
    rng = np.random.default_rng(41)
    n = 1 << 24
    m = rng.integers(0, 3, n).astype(np.uint32)
    s = np.uint64(1 << 35) + rng.integers(0, 1 << 30, n).astype(np.uint64)
    e = s + rng.integers(0, 100_000, n).astype(np.uint64)
    offsets = np.asarray([0, 3, 3 + n, 3 + n + 5], np.uint64)
    llm = np.concatenate([np.zeros(3, np.uint32), m, np.ones(5, np.uint32)])
    start = np.concatenate([np.asarray([1, 2, 3], np.uint64), s,
                            np.asarray([9, 8, 7, 6, 5], np.uint64)])
    end = np.concatenate([np.asarray([4, 5, 6], np.uint64), e,
                          np.asarray([19, 18, 17, 16, 15], np.uint64)])
    print(f"trace of {n} calls", flush=True)
    _same(ctx, 3, offsets, llm, start, end)


def test_every_sort_size_and_input_order(ctx):
    """Trace lengths at each power-of-two boundary of the in-register sort (256, 512, 1,024 and
    2,048 slots per workgroup), in sorted, reversed, constant and random order, with repeated
    keys and all 8 LLM indices."""
    rng = np.random.default_rng(23)
    traces = []
    for n in (1, 2, 255, 256, 257, 511, 512, 513, 1023, 1024, 1025, 2047, 2048):
        m = rng.integers(0, 8, n)
        s = rng.integers(0, 1 << 20, n)
        s[: n // 4] = s[0]                               # repeated starts
        d = rng.integers(0, 30_000, n)
        for order in ("random", "sorted", "reversed", "constant"):
            if order == "sorted":
                idx = np.lexsort((s, m))
            elif order == "reversed":
                idx = np.lexsort((s, m))[::-1]
            else:
                idx = rng.permutation(n)
            mm, ss, dd = m[idx], s[idx], d[idx]
            if order == "constant":
                mm, ss, dd = np.full(n, 3), np.full(n, 777), np.full(n, 5)
            traces.append([(int(a), int(b), int(b + c)) for a, b, c in zip(mm, ss, dd)])
    _same(ctx, 8, *_pack(traces))


def test_traces_in_end_order(ctx):
    """Traces already in order of end time (as logged on completion) take a sweep without a sort
    (one wave per trace, rows of 64 calls from the end); ties of end time, zero-length and nested
    calls, all 8 LLMs, spans below 2^29 us, just below 2^32 us (the sweep's 32-bit times) and
    above, at row boundaries (1, 63, 64, 65, ... 2,048 calls).  Copies with one pair of
    neighbours swapped (inside a row, across two rows, at either end) must take the sort and
    agree.  Traces whose calls lie 2^32 - 1 and 2^32 us before the last end, or whose last call
    ends at 2^60 us or later, must agree as well."""
    rng = np.random.default_rng(31)
    traces = []
    for n in (1, 2, 3, 63, 64, 65, 255, 256, 257, 511, 512, 513, 1023, 1024, 1025, 2047, 2048):
        for span_bits in (20, 31, 34):
            m = rng.integers(0, 8, n)
            s = rng.integers(0, 1 << span_bits, n)
            d = rng.integers(0, 40_000, n)
            d[rng.random(n) < 0.1] = 0                       # zero-length calls
            e = s + d
            e[rng.random(n) < 0.2] = e[0] if n else 0        # ties of end time
            s = np.maximum(np.minimum(s, e), e - np.minimum(e, 40_000))   # durations < 2^32
            idx = np.lexsort((s, e))
            calls = [(int(a), int(b), int(c)) for a, b, c in zip(m[idx], s[idx], e[idx])]
            traces.append(calls)
            for pos in (0, 63, 127, 255, 511, n // 2, n - 2, n - 65, n - 66, n - 129):
                # swap calls pos and pos + 1
                if pos < 0:
                    continue
                if pos + 1 < n and calls[pos][2] != calls[pos + 1][2]:
                    sw = list(calls)
                    sw[pos], sw[pos + 1] = sw[pos + 1], sw[pos]
                    traces.append(sw)
    # one LLM only, nested calls all ending together
    traces.append([(0, 1000 - i, 1000) for i in range(700)])
    # the first call starts 2^32 - 1 us (sweep) or 2^32 us (sort) before the last end
    for last in ((1 << 32) - 1, 1 << 32):
        traces.append([(0, 0, 5), (1, 3, 9), (0, last - 10, last - 2), (1, last - 7, last)])
    # the last call ends at 2^60 us or later (starts below it): the sort takes the trace
    traces.append([(0, (1 << 60) - 10, (1 << 60) - 5), (1, (1 << 60) - 8, (1 << 60) + 3)])
    _same(ctx, 8, *_pack(traces))


def test_order_adaptive_passes_agree():
    """A context whose sweep finds most traces out of end order sorts every trace on its next
    calls (then checks the order again): both kinds of call, on traces in either order, must
    match the oracle."""
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2604_15186_amd import alp
    tr = make_traces("beam", 300, 7)
    off = tr["offsets"].astype(np.int64)
    rng = np.random.default_rng(8)
    perm = np.concatenate([lo + rng.permutation(hi - lo) for lo, hi in zip(off[:-1], off[1:])])
    orders = [(tr["llm"][perm], tr["start"][perm], tr["end"][perm]),
              (tr["llm"], tr["start"], tr["end"])]
    with alp.StatsContext(0) as c:
        for k in range(12):                    # shuffled, in order, shuffled, ...
            llm, s, e = orders[k % 2]
            _same(c, tr["M"], tr["offsets"], llm, s, e)


def test_work_list_longer_than_the_sort_grid_with_long_traces():
    """On a fresh context the first call sweeps: 2,500 of 3,000 beam traces shuffled within the
    trace fill a work list longer than the sort pass's grid of 1,024 blocks (blocks take several
    entries in turn), and three traces beyond 2,048 calls make the long-trace pass the one whose
    last block finishes.  The next calls sort every trace directly (most were out of order),
    with the long traces again; every call must match the oracle."""
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2604_15186_amd import alp
    tr = make_traces("beam", 3000, 13)
    off = tr["offsets"].astype(np.int64)
    rng = np.random.default_rng(14)
    parts = []
    for r, (lo, hi) in enumerate(zip(off[:-1], off[1:])):
        idx = lo + (rng.permutation(hi - lo) if r < 2500 else np.arange(hi - lo))
        parts.append([(int(tr["llm"][i]), int(tr["start"][i]), int(tr["end"][i])) for i in idx])
    for n in (2049, 6000, 4096):                       # long traces, in random order
        t0 = int(rng.integers(0, 1 << 30))
        s = t0 + rng.integers(0, 1 << 24, n)
        parts.append([(int(m), int(a), int(a + d)) for m, a, d in
                      zip(rng.integers(0, 2, n), s, rng.integers(0, 100_000, n))])
    arrays = _pack(parts)
    with alp.StatsContext(0) as c:
        for _ in range(3):                             # sweep + list, then direct sorts
            _same(c, tr["M"], *arrays)


def test_direct_sort_of_every_trace_length_and_span():
    """After a call whose traces are mostly out of end order, the context sorts every trace
    directly, by groups of one to four waves per trace of at most 2,048 calls (the group sizes
    change at 512, 1,024 and 1,536 calls).  A group keys each call by its start
    relative to the trace's first call and keeps the trace only if every start lies in
    [first - 2^28, first + 2^28); other traces go to the block sort.  Traces at both edges of
    that range and just beyond its upper end, spans of 2^29 us or more, narrow traces of every
    group size, empty, single-call and long traces must all match the oracle, on two direct
    calls in a row."""
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2604_15186_amd import alp
    rng = np.random.default_rng(31)
    tr = make_traces("beam", 400, 17)
    off = tr["offsets"].astype(np.int64)
    perm = np.concatenate([lo + rng.permutation(hi - lo) for lo, hi in zip(off[:-1], off[1:])])
    shuffled = (tr["offsets"], tr["llm"][perm], tr["start"][perm], tr["end"][perm])
    traces = [[]]
    base = 1 << 40
    for n in (1, 2, 63, 64, 65, 200, 511, 512, 513, 1000, 1024, 1025, 1536, 1537, 1700, 2048,
              2049, 3000):
        for lo_off, hi_off in ((0, 1 << 20), (-(1 << 28) + 1, (1 << 28) - 1),
                               (-(1 << 28), 0), (0, 1 << 28), (-(1 << 30), 1 << 30)):
            s = base + rng.integers(lo_off, hi_off + 1, n)
            s[0] = base                                  # the wave's reference call
            if n > 1:
                s[1] = base + lo_off                     # both ends of the range present
            if n > 2:
                s[2] = base + hi_off
            m = rng.integers(0, 4, n)
            d = rng.integers(0, 50_000, n)
            traces.append([(int(a), int(b), int(b + c)) for a, b, c in zip(m, s, d)])
    arrays = _pack(traces)
    with alp.StatsContext(0) as c:
        _same(c, tr["M"], *shuffled)                   # sweeps, finds the order mixed
        for _ in range(2):
            _same(c, 4, *arrays)
