"""Seeded synthetic execution traces for the workflow statistics (Section 4, step 2).

A trace is one workflow-level request: the LLM-level calls it made, each (llm, start, end) in
microseconds, in the order a logging proxy sees them complete.  Two workflow shapes from the
paper's evaluation stand in for its recorded traces (which are not available):

* ``beam``: LLM 0 = generator, LLM 1 = verifier (process reward model).  A request runs S rounds,
  S ~ U[8, 281] (so 24..843 generator calls, as the paper reports 24..844 for its beam-search
  trace).  Each round the generator extends 3 beams concurrently, then the verifier scores the
  distinct candidates concurrently (1..3 calls: beams that produced the same text are scored
  once), then the next round starts.
* ``rag``: LLM 0 = embedding model, LLM 1 = reranker, LLM 2 = generator.  A request embeds the
  query, reranks 5..20 retrieved documents concurrently and generates once; with probability 0.3
  it retrieves and reranks a second time before generating.

Durations are log-normal around per-LLM means; tools (retrieval, orchestration) are the gaps
between rounds and produce no calls.  Arrays: offsets (uint64, R + 1), llm (uint32), start and
end (uint64).
"""
from __future__ import annotations

import numpy as np

SEED_ROOT = (2604, 15186, 77)


def _lognormal(rng, mean_us, size, sigma=0.5):
    mu = np.log(mean_us) - sigma * sigma / 2
    return np.maximum(1, np.rint(rng.lognormal(mu, sigma, size))).astype(np.int64)


def _beam_request(rng, t0):
    S = int(rng.integers(8, 282))
    gen = _lognormal(rng, 300_000, (S, 3))                    # generator: ~0.3 s per call
    gen_jit = rng.integers(0, 2_000, (S, 3))
    k = rng.choice([1, 2, 3], size=S, p=[0.1, 0.5, 0.4])      # distinct candidates per round
    ver = _lognormal(rng, 80_000, (S, 3))                     # verifier: ~80 ms per call
    ver_jit = rng.integers(0, 1_000, (S, 3))
    ver_used = np.arange(3)[None, :] < k[:, None]
    gap1 = rng.integers(100, 5_000, S)
    gap2 = rng.integers(100, 5_000, S)
    gen_span = (gen_jit + gen).max(axis=1)
    ver_span = np.where(ver_used, ver_jit + ver, 0).max(axis=1)
    round_len = gen_span + gap1 + ver_span + gap2
    rstart = t0 + np.concatenate([[0], np.cumsum(round_len)[:-1]])
    g_s = rstart[:, None] + gen_jit
    g_e = g_s + gen
    v_base = rstart + gen_span + gap1
    v_s = v_base[:, None] + ver_jit
    v_e = v_s + ver
    llm = np.concatenate([np.zeros(3 * S, np.uint32), np.ones(int(ver_used.sum()), np.uint32)])
    s = np.concatenate([g_s.ravel(), v_s[ver_used]])
    e = np.concatenate([g_e.ravel(), v_e[ver_used]])
    return llm, s, e


def _rag_request(rng, t0):
    llm, s, e = [], [], []
    t = t0
    for _ in range(2 if rng.random() < 0.3 else 1):
        d = int(_lognormal(rng, 10_000, 1)[0])                # embedding of the query
        llm.append(0), s.append(t), e.append(t + d)
        t += d + int(rng.integers(2_000, 20_000))             # retrieval (a tool)
        k = int(rng.integers(5, 21))
        jit = rng.integers(0, 500, k)
        dur = _lognormal(rng, 30_000, k)
        for j in range(k):
            llm.append(1), s.append(t + int(jit[j])), e.append(t + int(jit[j]) + int(dur[j]))
        t = max(e) + int(rng.integers(100, 2_000))
    d = int(_lognormal(rng, 2_000_000, 1)[0])                 # generation
    llm.append(2), s.append(t), e.append(t + d)
    return np.asarray(llm, np.uint32), np.asarray(s, np.int64), np.asarray(e, np.int64)


SHAPES = {"beam": (2, _beam_request), "rag": (3, _rag_request)}


def make_traces(shape: str, R: int, seed: int = 0) -> dict:
    """R traces of the given shape ("beam" or "rag"); calls in completion order per trace."""
    M, request = SHAPES[shape]
    rng = np.random.default_rng(np.random.SeedSequence([*SEED_ROOT, seed, R, len(shape)]))
    parts, offsets = [], [0]
    for r in range(R):
        t0 = int(rng.integers(0, 1 << 40))                    # requests at arbitrary times
        llm, s, e = request(rng, t0)
        order = np.lexsort((s, e))                            # completion order
        parts.append((llm[order], s[order], e[order]))
        offsets.append(offsets[-1] + len(llm))
    return {"M": M, "R": R, "shape": shape,
            "offsets": np.asarray(offsets, dtype=np.uint64),
            "llm": np.concatenate([p[0] for p in parts]).astype(np.uint32),
            "start": np.concatenate([p[1] for p in parts]).astype(np.uint64),
            "end": np.concatenate([p[2] for p in parts]).astype(np.uint64)}
