"""Literal statement of the most-constrained-first placement (Section 6) for tests: every set of
tp GPUs of a node is enumerated (no windows), scored as the reading states, and single-GPU
replicas follow the occupied-first rule.  Shares nothing with the C oracle."""
from __future__ import annotations

import itertools

NODE = 8


def place(Q, G, tp, q, d):
    free = [Q] * G
    nodes = [list(range(n, min(n + NODE, G))) for n in range(0, G, NODE)]
    order = sorted((m for m in range(len(tp)) if d[m] > 0),
                   key=lambda m: (tp[m] == 1, -tp[m] * q[m], m))
    first = [sum(d[:m]) for m in range(len(tp))]
    slot = [0xFFFF] * sum(d)
    placed = True
    for m in order:
        for r in range(d[m]):
            choice = None
            if tp[m] > 1:
                best = None
                for n, gpus in enumerate(nodes):
                    dom = sum(free[g] for g in gpus)
                    room = sorted((g for g in gpus if free[g] >= q[m]), key=lambda g: (free[g], g))
                    rank = {g: i for i, g in enumerate(room)}
                    for sub in itertools.combinations(room, tp[m]):
                        fr = [free[g] for g in sub]
                        key = (max(fr) - min(fr), dom, sum(fr), n, sorted(rank[g] for g in sub))
                        if best is None or key < best[0]:
                            best = (key, sub)
                if best is not None:
                    choice = best[1]
            else:
                occ = [g for g in range(G) if q[m] <= free[g] < Q]
                if occ:
                    choice = (min(occ, key=lambda g: (free[g], g)),)
                else:
                    cands = [(sum(free[g] for g in gpus), n, min(g for g in gpus if free[g] == Q))
                             for n, gpus in enumerate(nodes) if any(free[g] == Q for g in gpus)]
                    if cands and q[m] <= Q:
                        choice = (min(cands)[2],)
            if choice is None:
                placed = False
                break
            for g in choice:
                free[g] -= q[m]
            n = choice[0] // NODE
            slot[first[m] + r] = n << 8 | sum(1 << (g - n * NODE) for g in choice)
        if not placed:
            break
    return placed, slot, free
