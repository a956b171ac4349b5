"""The stored full-size results (written by ``golden/make_golden.py`` from the oracle) still match
the generator, and agree with an independent dynamic program (CPU only)."""
from __future__ import annotations

import json
import os

import numpy as np
import pytest

import oracle
from workloads import make_batch, target_from_tmax

from dp_knapsack import dp_argmin

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def load_golden(cfg: int) -> dict:
    with open(os.path.join(GOLDEN, f"cfg{cfg}_argmin.json")) as f:
        return json.load(f)


def _import_digest():
    import importlib.util
    spec = importlib.util.spec_from_file_location("make_golden", os.path.join(GOLDEN, "make_golden.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod.table_digest


@pytest.mark.parametrize("cfg", [1, 2, 3, 4])
def test_golden_tables_unchanged(cfg):
    g = load_golden(cfg)
    b = make_batch(cfg, sorted({r["inst"] for r in g["results"]}))
    assert _import_digest()(b) == g["table_sha256"]


@pytest.mark.parametrize("cfg,sample", [(1, None), (2, None), (3, None), (4, 160)])
def test_golden_matches_dp_and_eval(cfg, sample):
    g = load_golden(cfg)
    rows = g["results"]
    if sample:
        rows = rows[:: max(1, len(rows) // sample)]
    b = make_batch(cfg, [r["inst"] for r in rows])
    Q = int(b["space"]["Q"])
    for i, r in enumerate(rows):
        inst = oracle.Instance(b, i)
        assert oracle.tmax(inst, r["G"]) == r["tmax"]
        assert r["lambda"] == target_from_tmax(r["u_ppm"], r["tmax"])
        terms = [[(t["ok"] and t["thr_ok"], t["c"], t["u"]) for t in row]
                 for row in oracle.option_terms(inst, r["lambda"])]
        dp = dp_argmin(terms, Q * r["G"])
        assert dp == (r["x"], r["L"]), (cfg, r)
        ev = oracle.evaluate(inst, r["G"], r["lambda"], r["x"])
        assert (ev["flags"], ev["L"], ev["T"], ev["U"]) == (7, r["L"], r["T"], r["U"])
        assert r["n_feasible"] >= 1


def test_golden_cfg1_rerun_matches():
    """A few config-1 instances re-run through the oracle's brute force give the stored rows."""
    g = load_golden(1)
    for r in g["results"][:3]:
        b = make_batch(1, [r["inst"]])
        inst = oracle.Instance(b, 0)
        got = oracle.argmin(inst, r["G"], r["lambda"])
        assert (got["x"], got["L"], got["n_feasible"], got["sum_L"]) == (
            r["x"], r["L"], r["n_feasible"], r["sum_L"])
