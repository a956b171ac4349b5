"""Independent statement of the multi-workflow split (test helper): threshold, then DP.

Egalitarian welfare: the smallest largest-latency t* is found by thresholds (workflow w needs the
fewest GPUs g with L[w][g] <= t; t is reachable iff those fit together, and t* is one of the
table's values); then, among splits whose latencies are all <= t*, a knapsack DP over the
budget minimises the latency sum, and the smallest budget of each workflow in turn that stays
optimal gives the lexicographically smallest vector.  Social welfare is the same DP without the
threshold.  A different algorithm from the oracle's brute force over budget vectors.
"""
from __future__ import annotations

NONE = None


def split(L, G: int, policy: int):
    W = len(L)
    if policy == 0:
        t_star = None
        for t in sorted({v for row in L for v in row if v is not None}):
            need = 0
            for row in L:
                g = next((g for g, v in enumerate(row) if v is not None and v <= t), None)
                if g is None:
                    need = None
                    break
                need += g
            if need is not None and need <= G:
                t_star = t
                break
        if t_star is None:
            return None
        allowed = [[v is not None and v <= t_star for v in row] for row in L]
    else:
        allowed = [[v is not None for v in row] for row in L]
    INF = float("inf")
    best = [[INF] * (G + 1) for _ in range(W + 1)]
    best[W] = [0] * (G + 1)
    for w in range(W - 1, -1, -1):
        for b in range(G + 1):
            best[w][b] = min((L[w][g] + best[w + 1][b - g] for g in range(b + 1) if allowed[w][g]),
                             default=INF)
    if best[0][G] == INF:
        return None
    g_vec, b = [], G
    for w in range(W):
        for g in range(b + 1):
            if allowed[w][g] and L[w][g] + best[w + 1][b - g] == best[w][b]:
                g_vec.append(g)
                b -= g
                break
    lat = [L[w][g] for w, g in enumerate(g_vec)]
    return g_vec, max(lat), sum(lat)
