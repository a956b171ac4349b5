"""Pins of the oracle's workflow statistics (Section 4, step 2) against what the paper and the
mathematics fix: the paper's beam example (three concurrent generator beams give p = 3, two
concurrent verifier calls give p = 2), closed forms (disjoint calls: p = 1; k identical calls:
p = k), a brute-force count of covered time on a unit grid, and invariances (call order within
a trace, a time shift of a trace, splitting traces)."""
from __future__ import annotations

import numpy as np
import pytest

import oracle


def _pack(traces):
    """traces: list of lists of (llm, start, end) -> arrays."""
    offsets = [0]
    llm, s, e = [], [], []
    for tr in traces:
        for m, a, b in tr:
            llm.append(m), s.append(a), e.append(b)
        offsets.append(len(llm))
    return (np.asarray(offsets, np.uint64), np.asarray(llm, np.uint32), np.asarray(s, np.uint64),
            np.asarray(e, np.uint64))


def test_paper_beam_example():
    # Section 4 step 2: three beams of the generator run concurrently (p_GEN ~ 3); the verifier
    # scores two candidates when two beams produced the same value (p_VER ~ 2).  Two rounds.
    trace = []
    t = 1000
    for _ in range(2):
        trace += [(0, t, t + 500)] * 3
        trace += [(1, t + 600, t + 700)] * 2
        t += 800
    st = oracle.trace_stats(2, *_pack([trace]))
    assert (int(st[0]["n_milli"]), int(st[0]["p_milli"])) == (6000, 3000)
    assert (int(st[1]["n_milli"]), int(st[1]["p_milli"])) == (4000, 2000)
    assert (int(st[0]["busy_us"]), int(st[0]["active_us"])) == (3000, 1000)


def test_closed_forms():
    # disjoint calls: p = 1; k identical: p = k; nested [0,10) and [2,4): busy 12, active 10
    st = oracle.trace_stats(3, *_pack([[(0, 0, 10), (0, 10, 20), (0, 30, 35),
                                        (1, 5, 9), (1, 5, 9), (1, 5, 9), (1, 5, 9),
                                        (2, 0, 10), (2, 2, 4)]]))
    assert [int(v) for v in st["p_milli"]] == [1000, 4000, 1200]
    assert [int(v) for v in st["calls"]] == [3, 4, 2]
    # two traces: n is per trace, p pools durations and covered time over traces
    st = oracle.trace_stats(2, *_pack([[(0, 0, 10), (0, 0, 10)], [(0, 0, 30)]]))
    assert (int(st[0]["n_milli"]), int(st[0]["p_milli"])) == (1500, 1250)   # 50 / 40
    assert (int(st[1]["n_milli"]), int(st[1]["p_milli"])) == (0, 0)          # no calls
    # calls of zero length only: p = 1 by convention; n still counts them
    st = oracle.trace_stats(1, *_pack([[(0, 5, 5), (0, 7, 7)], []]))
    assert (int(st[0]["n_milli"]), int(st[0]["p_milli"])) == (1000, 1000)


def _grid_stats(M, traces):
    """Brute force on a unit grid: covered time = number of unit slots [t, t+1) inside at least
    one of the LLM's calls, per trace."""
    calls = np.zeros(M, np.int64)
    busy = np.zeros(M, np.int64)
    active = np.zeros(M, np.int64)
    for tr in traces:
        for m in range(M):
            cover = set()
            for mm, a, b in tr:
                if mm == m:
                    calls[m] += 1
                    busy[m] += b - a
                    cover.update(range(a, b))
            active[m] += len(cover)
    R = len(traces)
    n = [int(c * 1000 // R) for c in calls]
    p = [0 if c == 0 else 1000 if a == 0 else int(b * 1000 // a)
         for c, b, a in zip(calls, busy, active)]
    return n, p, calls.tolist(), busy.tolist(), active.tolist()


@pytest.mark.parametrize("seed", range(8))
def test_grid_brute_force(seed):
    rng = np.random.default_rng(seed)
    M = int(rng.integers(1, 6))
    traces = []
    for _ in range(int(rng.integers(1, 12))):
        tr = []
        for _ in range(int(rng.integers(0, 25))):
            a = int(rng.integers(0, 60))
            tr.append((int(rng.integers(0, M)), a, a + int(rng.integers(0, 15))))
        traces.append(tr)
    st = oracle.trace_stats(M, *_pack(traces))
    n, p, calls, busy, active = _grid_stats(M, traces)
    assert [int(v) for v in st["n_milli"]] == n
    assert [int(v) for v in st["p_milli"]] == p
    assert [int(v) for v in st["calls"]] == calls
    assert [int(v) for v in st["busy_us"]] == busy
    assert [int(v) for v in st["active_us"]] == active


def test_invariances():
    from workloads.traces import make_traces
    tr = make_traces("beam", 30, 3)
    base = oracle.trace_stats(tr["M"], tr["offsets"], tr["llm"], tr["start"], tr["end"])
    rng = np.random.default_rng(1)
    off = tr["offsets"].astype(np.int64)
    perm = np.concatenate([lo + rng.permutation(hi - lo) for lo, hi in zip(off[:-1], off[1:])])
    shift = np.repeat(rng.integers(0, 1 << 30, len(off) - 1), np.diff(off)).astype(np.uint64)
    st = oracle.trace_stats(tr["M"], tr["offsets"], tr["llm"][perm], tr["start"][perm] + shift[perm],
                            tr["end"][perm] + shift[perm])
    assert (st == base).all()
    # p is at least 1 when calls have length; never above the largest concurrency (3 beams)
    assert (base["p_milli"] >= 1000).all() and (base["p_milli"] <= 3000).all()


def test_malformed_traces_rejected():
    with pytest.raises(ValueError):
        oracle.trace_stats(1, *_pack([[(1, 0, 5)]]))       # llm out of range
    with pytest.raises(ValueError):
        oracle.trace_stats(1, *_pack([[(0, 5, 4)]]))       # ends before it starts
