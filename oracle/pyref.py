"""ORACLE (pure Python) -- test infrastructure only; small cases only.

A second, deliberately naive statement of the same definitions as ``alp_oracle.c``, in Python
integers (no fixed-width wrap-around), used to cross-check the C oracle on tiny spaces.

Definitions (Section 4, steps 4-5, Eq. 1 and Eq. 2; Section 5 step 1):
  per-replica LLM rate     r   = ceil(lambda * n_m / (1000 d))        (milli-req/s)
  sustainable              r  <= T = rate[K-1]                         (saturation point)
  latency at r             flat below rate[0], linear between points, floored
  contribution             c   = floor(latency * n_m / p_m)            (Eq. 1 term)
  normalised throughput    tau = floor(1000 d T / n_m)                 (Eq. 2 term)
  share units              u   = tp * q * d
  fits                     W_m * Q <= tp * q * H  and the (tp, q) pair is allowed
"""
from __future__ import annotations


def _get(batch, key, i):
    return batch[key][i]


def option_term(batch: dict, i: int, m: int, o: int, lam: int) -> dict:
    sp = batch["space"]
    tps, fqs, D, K, Q = [int(v) for v in sp["tp"]], [int(v) for v in sp["fq"]], int(sp["D"]), \
        int(sp["K"]), int(sp["Q"])
    d = o % D + 1
    jj = o // D
    j = jj % len(fqs)
    ii = jj // len(fqs)
    tp, q = tps[ii], fqs[j]
    rate = [int(v) for v in batch["rate"][i][m][ii][j]]
    lat = [int(v) for v in batch["lat"][i][m][ii][j]]
    n, p, W = int(batch["n"][i][m]), int(batch["p"][i][m]), int(batch["W"][i][m])
    ok = bool(batch["allowed"][i][m][ii][j]) and W * Q <= tp * q * int(batch["H"])
    T = rate[-1]
    tau = min(1000 * d * T // n, 2**32 - 1)
    r = -((-lam * n) // (1000 * d))
    thr_ok = r <= T
    c = 0
    if thr_ok:
        if r <= rate[0]:
            ell = lat[0]
        else:
            k = next(k for k in range(1, K) if r <= rate[k])
            ell = (lat[k - 1] * (rate[k] - r) + lat[k] * (r - rate[k - 1])) // (rate[k] - rate[k - 1])
        c = ell * n // p
    return {"ok": int(ok), "thr_ok": int(thr_ok), "c": c, "u": tp * q * d, "tau": tau}


def num_options(batch: dict) -> int:
    sp = batch["space"]
    return len(sp["tp"]) * len(sp["fq"]) * int(sp["D"])


def digits(batch: dict, x: int) -> list:
    M, O = int(batch["space"]["M"]), num_options(batch)
    out = []
    for _ in range(M):
        out.append(x % O)
        x //= O
    return out[::-1]


def evaluate(batch: dict, i: int, G: int, lam: int, x: int) -> dict:
    terms = [option_term(batch, i, m, o, lam) for m, o in enumerate(digits(batch, x))]
    all_ok = all(t["ok"] for t in terms)
    all_thr = all(t["thr_ok"] for t in terms)
    U = sum(t["u"] for t in terms)
    budget_ok = U <= int(batch["space"]["Q"]) * G
    return {"flags": int(all_ok) | int(all_thr) << 1 | int(budget_ok) << 2,
            "L": sum(t["c"] for t in terms) if all_ok and all_thr else (1 << 64) - 1,
            "T": min(t["tau"] for t in terms) if all_ok else 0,
            "U": U}


def argmin(batch: dict, i: int, G: int, lam: int) -> dict:
    O, M = num_options(batch), int(batch["space"]["M"])
    best = None
    for x in range(O ** M):
        e = evaluate(batch, i, G, lam, x)
        if e["flags"] == 7 and (best is None or e["L"] < best[0]):
            best = (e["L"], x)
    return {"x": None if best is None else best[1], "L": None if best is None else best[0]}
