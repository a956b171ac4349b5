"""Independent check of the search result by dynamic programming (test helper).

The constrained argmin is a multiple-choice knapsack: pick one option per LLM, total share
units <= Q*G, minimise the summed latency contribution (Eq. 1), options that are not deployable
or cannot sustain the target rate excluded.  Suffix tables best[m][b] (lowest total latency of
LLMs m..M-1 within b units) give the optimum in O(M * O * Q*G); reconstructing from LLM 0
upwards and taking the smallest option that stays optimal at each step gives the
lexicographically smallest digit vector, i.e. the lowest candidate index among ties.

This is a different algorithm from the exhaustive enumeration, so agreement pins the
enumeration's combination, budget and tie-break logic at sizes brute force cannot reach in a
test.  It takes the per-option terms as input.
"""
from __future__ import annotations

import numpy as np

INF = 1 << 62


def dp_argmin(terms, capacity: int):
    """terms[m][o] = (usable, c, u).  Returns (x, L) or None if nothing is feasible."""
    M, O = len(terms), len(terms[0])
    B = int(capacity)
    best = [None] * (M + 1)
    best[M] = np.zeros(B + 1, dtype=np.int64)
    for m in range(M - 1, -1, -1):
        cur = np.full(B + 1, INF, dtype=np.int64)
        nxt = best[m + 1]
        for usable, c, u in terms[m]:
            if not usable or u > B:
                continue
            cand = np.minimum(nxt[: B + 1 - u] + int(c), INF)
            np.minimum(cur[u:], cand, out=cur[u:])
        best[m] = cur
    if best[0][B] >= INF:
        return None
    b, x = B, 0
    for m in range(M):
        target = int(best[m][b])
        for o, (usable, c, u) in enumerate(terms[m]):
            if usable and u <= b and int(c) + int(best[m + 1][b - u]) == target:
                x = x * O + o
                b -= u
                break
        else:  # pragma: no cover - the optimum always reconstructs
            raise AssertionError("reconstruction failed")
    return x, int(best[0][B])
