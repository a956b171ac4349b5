"""ORACLE -- test infrastructure only.

Only the test suite, the smoke check and the benchmark's CPU-baseline leg may import this
package.  The GPU library and its Python binding never import, link or call it, and it shares
no code with them.  It wraps ``liborc.so`` (built from ``alp_oracle.c`` by :func:`build`) with
ctypes and adds a slow pure-Python statement of the same definitions for tiny cases
(:mod:`oracle.pyref`).

Functions take a batch dictionary as produced by :mod:`workloads` and an instance number.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
SOURCE = os.path.join(_HERE, "alp_oracle.c")
BUILT_PATH = os.path.join(_HERE, "liborc.so")
# ALP_ORACLE_LIB names another build of the same source to load instead (the test suite uses it
# for sanitizer builds and for planted-mistake copies of the oracle).
LIB_PATH = os.environ.get("ALP_ORACLE_LIB", BUILT_PATH)
U64_NONE = (1 << 64) - 1


def build() -> str:
    """Compile ``liborc.so`` with gcc (always rebuilds)."""
    tmp = BUILT_PATH + ".tmp"
    subprocess.run(["gcc", "-std=c11", "-O2", "-Wall", "-Wextra", "-shared", "-fPIC", SOURCE, "-o",
                    tmp], check=True)
    os.replace(tmp, BUILT_PATH)
    return BUILT_PATH


class _Inst(C.Structure):
    _fields_ = [("M", C.c_uint32), ("n_tp", C.c_uint32), ("n_fq", C.c_uint32), ("D", C.c_uint32),
                ("K", C.c_uint32), ("Q", C.c_uint32),
                ("tp", C.c_void_p), ("fq", C.c_void_p), ("W", C.c_void_p), ("n", C.c_void_p),
                ("p", C.c_void_p), ("allowed", C.c_void_p), ("rate", C.c_void_p),
                ("lat", C.c_void_p), ("H", C.c_uint64)]


class _Term(C.Structure):
    _fields_ = [("ok", C.c_uint32), ("thr_ok", C.c_uint32), ("c", C.c_uint64), ("u", C.c_uint64),
                ("tau", C.c_uint64)]


class _Eval(C.Structure):
    _fields_ = [("flags", C.c_uint32), ("L", C.c_uint64), ("T", C.c_uint64), ("U", C.c_uint64)]


class _Argmin(C.Structure):
    _fields_ = [("best_x", C.c_uint64), ("best_L", C.c_uint64), ("n_feasible", C.c_uint64),
                ("sum_L", C.c_uint64)]


class _Placement(C.Structure):
    _fields_ = [("placed", C.c_uint32), ("replicas", C.c_uint32), ("gpus_used", C.c_uint32),
                ("nodes_used", C.c_uint32), ("slot", C.c_uint16 * 128)]


class _Pruned(C.Structure):
    _fields_ = [("best_x", C.c_uint64), ("best_L", C.c_uint64), ("vectors", C.c_uint64),
                ("unpruned", C.c_uint64)]


EVAL_DTYPE = np.dtype([("flags", np.uint32), ("L", np.uint64), ("T", np.uint64), ("U", np.uint64)],
                      align=True)

_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH) and LIB_PATH == BUILT_PATH:
            build()
        L = C.CDLL(LIB_PATH)
        P = C.POINTER
        L.orc_num_options.argtypes = [P(_Inst)]
        L.orc_num_options.restype = C.c_uint32
        L.orc_option_term.argtypes = [P(_Inst), C.c_uint32, C.c_uint32, C.c_uint32, P(_Term)]
        L.orc_eval.argtypes = [P(_Inst), C.c_uint32, C.c_uint32, C.c_uint64, P(_Eval)]
        L.orc_eval_many.argtypes = [P(_Inst), C.c_uint32, C.c_uint32, C.c_void_p, C.c_uint64,
                                    C.c_void_p]
        L.orc_argmin.argtypes = [P(_Inst), C.c_uint32, C.c_uint32, C.c_uint64, C.c_uint64,
                                 C.c_void_p, P(_Argmin)]
        L.orc_tmax_brute.argtypes = [P(_Inst), C.c_uint32, C.c_uint64, C.c_uint64,
                                     P(C.c_uint64)]
        L.orc_tmax_threshold.argtypes = [P(_Inst), C.c_uint32, C.c_void_p, P(C.c_uint64)]
        L.orc_allocate.argtypes = [C.c_uint32, C.c_uint32, C.c_void_p, C.c_uint32, C.c_void_p,
                                   P(C.c_uint64), P(C.c_uint64)]
        L.orc_pruned.argtypes = [P(_Inst), C.c_uint32, C.c_uint32, C.c_uint32, C.c_void_p,
                                 P(_Pruned)]
        L.orc_fits.argtypes = [C.c_uint32, C.c_uint64, C.c_uint64, C.c_uint64, C.c_uint64,
                               C.c_uint64]
        L.orc_count_fractions.argtypes = [C.c_uint32, C.c_uint64, C.c_void_p, C.c_int]
        L.orc_count_fractions.restype = C.c_uint64
        L.orc_binomial.argtypes = [C.c_uint64, C.c_uint64]
        L.orc_binomial.restype = C.c_uint64
        L.orc_place.argtypes = [C.c_uint32, C.c_uint32, C.c_uint32, C.c_void_p, C.c_void_p,
                                C.c_void_p, P(_Placement)]
        L.orc_place_exact.argtypes = [C.c_uint32, C.c_uint32, C.c_uint32, C.c_void_p,
                                      C.c_void_p, C.c_void_p]
        L.orc_place.restype = C.c_int
        L.orc_place_exact.restype = C.c_int
        L.orc_trace_stats.argtypes = [C.c_uint32, C.c_uint32, C.c_void_p, C.c_void_p, C.c_void_p,
                                      C.c_void_p, C.c_void_p, C.c_void_p]
        for f in (L.orc_option_term, L.orc_eval, L.orc_eval_many, L.orc_argmin, L.orc_tmax_brute,
                  L.orc_tmax_threshold, L.orc_allocate, L.orc_pruned, L.orc_fits,
                  L.orc_trace_stats):
            f.restype = C.c_int
        _lib = L
    return _lib


class Instance:
    """Keeps the numpy arrays of one instance alive and exposes them as an ``orc_instance``."""

    def __init__(self, batch: dict, i: int = 0):
        sp = batch["space"]
        self.arrays = {
            "tp": np.ascontiguousarray(sp["tp"], dtype=np.uint32),
            "fq": np.ascontiguousarray(sp["fq"], dtype=np.uint32),
            "W": np.ascontiguousarray(batch["W"][i], dtype=np.uint64),
            "n": np.ascontiguousarray(batch["n"][i], dtype=np.uint32),
            "p": np.ascontiguousarray(batch["p"][i], dtype=np.uint32),
            "allowed": np.ascontiguousarray(batch["allowed"][i], dtype=np.uint8),
            "rate": np.ascontiguousarray(batch["rate"][i], dtype=np.uint32),
            "lat": np.ascontiguousarray(batch["lat"][i], dtype=np.uint32),
        }
        a = self.arrays
        self.M, self.K = int(sp["M"]), int(sp["K"])
        self.O = len(a["tp"]) * len(a["fq"]) * int(sp["D"])
        self.N = self.O ** self.M
        self.G = int(batch["G"][i])
        self.u_ppm = int(batch["u_ppm"][i])
        self.c = _Inst(self.M, len(a["tp"]), len(a["fq"]), int(sp["D"]), self.K, int(sp["Q"]),
                       *(a[k].ctypes.data for k in ("tp", "fq", "W", "n", "p", "allowed", "rate",
                                                     "lat")),
                       int(batch["H"]))
        self._scratch = (_Term * (self.M * self.O))()


def option_term(inst: Instance, m: int, o: int, lam: int) -> dict:
    t = _Term()
    if lib().orc_option_term(C.byref(inst.c), m, o, lam, C.byref(t)) != 0:
        raise ValueError("option out of range")
    return {"ok": int(t.ok), "thr_ok": int(t.thr_ok), "c": int(t.c), "u": int(t.u),
            "tau": int(t.tau)}


def option_terms(inst: Instance, lam: int) -> list:
    """[m][o] -> term dictionaries."""
    return [[option_term(inst, m, o, lam) for o in range(inst.O)] for m in range(inst.M)]


def evaluate(inst: Instance, G: int, lam: int, x: int) -> dict:
    e = _Eval()
    if lib().orc_eval(C.byref(inst.c), G, lam, x, C.byref(e)) != 0:
        raise ValueError("candidate index out of range")
    return {"flags": int(e.flags), "L": int(e.L), "T": int(e.T), "U": int(e.U)}


def evaluate_many(inst: Instance, G: int, lam: int, xs: np.ndarray) -> np.ndarray:
    xs = np.ascontiguousarray(xs, dtype=np.uint64)
    out = np.zeros(len(xs), dtype=EVAL_DTYPE)
    assert EVAL_DTYPE.itemsize == C.sizeof(_Eval)
    if lib().orc_eval_many(C.byref(inst.c), G, lam, xs.ctypes.data, len(xs), out.ctypes.data) != 0:
        raise ValueError("candidate index out of range")
    return out


def argmin(inst: Instance, G: int, lam: int, lo: int = 0, hi: int | None = None) -> dict:
    hi = inst.N if hi is None else hi
    if not (0 <= lo <= hi <= inst.N):
        raise ValueError("range outside the candidate space")
    r = _Argmin()
    if lib().orc_argmin(C.byref(inst.c), G, lam, lo, hi, inst._scratch, C.byref(r)) != 0:
        raise ValueError("bad instance")
    return {"x": None if r.best_x == U64_NONE else int(r.best_x),
            "L": None if r.best_x == U64_NONE else int(r.best_L),
            "n_feasible": int(r.n_feasible), "sum_L": int(r.sum_L)}


def tmax_brute(inst: Instance, G: int, lo: int = 0, hi: int | None = None) -> int:
    hi = inst.N if hi is None else hi
    out = C.c_uint64()
    if lib().orc_tmax_brute(C.byref(inst.c), G, lo, hi, C.byref(out)) != 0:
        raise ValueError("bad range")
    return int(out.value)


def tmax(inst: Instance, G: int) -> int:
    """Largest T_w reachable within budget G (threshold method)."""
    out = C.c_uint64()
    lib().orc_tmax_threshold(C.byref(inst.c), G, inst._scratch, C.byref(out))
    return int(out.value)


def merge_argmin(parts: list) -> dict:
    """Merges argmin results of disjoint index slices (lexicographic (L, x) minimum)."""
    best = {"x": None, "L": None, "n_feasible": 0, "sum_L": 0}
    for r in parts:
        best["n_feasible"] += r["n_feasible"]
        best["sum_L"] = (best["sum_L"] + r["sum_L"]) % (1 << 64)
        if r["x"] is not None and (best["x"] is None or (r["L"], r["x"]) < (best["L"], best["x"])):
            best["x"], best["L"] = r["x"], r["L"]
    return best


def workflow_latencies(batch: dict, lambdas, G_total: int) -> np.ndarray:
    """L[w][g]: the search result's latency of workflow (instance) w at g GPUs, g = 0..G_total;
    U64_NONE where infeasible.  Brute force per (w, g)."""
    W = len(lambdas)
    L = np.full((W, G_total + 1), U64_NONE, dtype=np.uint64)
    for w in range(W):
        inst = Instance(batch, w)
        for g in range(G_total + 1):
            r = argmin(inst, g, int(lambdas[w]))
            if r["x"] is not None:
                L[w, g] = r["L"]
    return L


EGALITARIAN, SOCIAL = 0, 1


def allocate(L: np.ndarray, policy: int):
    """Budget split over workflows for latency table L[w][g] (see orc_allocate).  Returns
    (budgets, max latency, latency sum) or None if no split makes every workflow feasible."""
    L = np.ascontiguousarray(L, dtype=np.uint64)
    W, G1 = L.shape
    g = np.zeros(W, dtype=np.uint32)
    mx, sm = C.c_uint64(), C.c_uint64()
    rc = lib().orc_allocate(W, G1 - 1, L.ctypes.data, policy, g.ctypes.data, C.byref(mx), C.byref(sm))
    if rc < 0:
        raise ValueError("bad arguments")
    if rc == 1:
        return None
    return [int(v) for v in g], int(mx.value), int(sm.value)


PRUNE_ORDER, PRUNE_MIN = 1, 2


def pruned(inst: Instance, G: int, lam: int, flags: int = PRUNE_ORDER | PRUNE_MIN) -> dict:
    """The paper's pruned fraction-enumeration search (see orc_pruned)."""
    r = _Pruned()
    if lib().orc_pruned(C.byref(inst.c), G, lam, flags, inst._scratch, C.byref(r)) != 0:
        raise ValueError("bad arguments")
    none = r.best_x == U64_NONE
    return {"x": None if none else int(r.best_x), "L": None if none else int(r.best_L),
            "vectors": int(r.vectors), "unpruned": int(r.unpruned)}


def fits(Q: int, a: int, f: int, tp: int, q: int, d: int) -> bool:
    """Placement test of step 3 (see orc_fits)."""
    return bool(lib().orc_fits(Q, a, f, tp, q, d))


def count_fractions(M: int, total: int, lo, ordered: bool) -> int:
    """Number of step-1 fraction vectors for lower bounds lo (per position)."""
    lo = np.ascontiguousarray(lo, dtype=np.uint64)
    assert len(lo) == M
    return int(lib().orc_count_fractions(M, total, lo.ctypes.data, 1 if ordered else 0))


def binomial(n: int, k: int) -> int:
    return int(lib().orc_binomial(n, k))


STATS_DTYPE = np.dtype([("n_milli", np.uint32), ("p_milli", np.uint32), ("calls", np.uint64),
                        ("busy_us", np.uint64), ("active_us", np.uint64)])


def trace_stats(M: int, offsets, llm, start, end) -> np.ndarray:
    """Workflow statistics n_m, p_m per LLM from traces (see orc_trace_stats)."""
    offsets = np.ascontiguousarray(offsets, dtype=np.uint64)
    llm = np.ascontiguousarray(llm, dtype=np.uint32)
    start = np.ascontiguousarray(start, dtype=np.uint64)
    end = np.ascontiguousarray(end, dtype=np.uint64)
    R = len(offsets) - 1
    longest = int(np.diff(offsets.astype(np.int64)).max()) if R > 0 else 0
    scratch = np.zeros(2 * max(1, longest), dtype=np.uint64)
    out = np.zeros(M, dtype=STATS_DTYPE)
    if lib().orc_trace_stats(M, R, offsets.ctypes.data, llm.ctypes.data, start.ctypes.data,
                             end.ctypes.data, scratch.ctypes.data, out.ctypes.data) != 0:
        raise ValueError("malformed traces")
    return out


def place(Q: int, G: int, tp, q, d) -> dict:
    """The most-constrained-first placement of an allocation (see orc_place): placed flag,
    replicas placed, GPUs and nodes used, and per replica (LLM-major) node << 8 | GPU mask
    (0xFFFF if not placed)."""
    M = len(tp)
    a = [np.ascontiguousarray(v, dtype=np.uint32) for v in (tp, q, d)]
    r = _Placement()
    if lib().orc_place(Q, G, M, a[0].ctypes.data, a[1].ctypes.data, a[2].ctypes.data,
                       C.byref(r)) != 0:
        raise ValueError("bad allocation")
    n = int(sum(int(v) for v in d))
    return {"placed": bool(r.placed), "replicas": int(r.replicas), "gpus_used": int(r.gpus_used),
            "nodes_used": int(r.nodes_used), "slot": [int(v) for v in r.slot[:n]]}


def place_exact(Q: int, G: int, tp, q, d) -> bool:
    """Whether any placement exists (backtracking; small cases)."""
    a = [np.ascontiguousarray(v, dtype=np.uint32) for v in (tp, q, d)]
    r = lib().orc_place_exact(Q, G, len(tp), a[0].ctypes.data, a[1].ctypes.data, a[2].ctypes.data)
    if r < 0:
        raise ValueError("bad allocation")
    return bool(r)
