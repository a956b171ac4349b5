"""Loads the hand-derived cases of ``tests/golden/hand_cases.json`` as batches (test helper)."""
from __future__ import annotations

import json
import os

import numpy as np

PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "hand_cases.json")


def load_cases() -> list:
    with open(PATH) as f:
        return json.load(f)["cases"]


def case_batch(case: dict, G: int = 0) -> dict:
    sp = case["space"]
    space = {"M": sp["M"], "tp": np.asarray(sp["tp"], dtype=np.uint32),
             "fq": np.asarray(sp["fq"], dtype=np.uint32), "Q": sp["Q"], "D": sp["D"], "K": sp["K"]}
    return {
        "space": space, "H": int(case["H"]),
        "W": np.asarray([case["W"]], dtype=np.uint64),
        "n": np.asarray([case["n"]], dtype=np.uint32),
        "p": np.asarray([case["p"]], dtype=np.uint32),
        "allowed": np.asarray([case["allowed"]], dtype=np.uint8),
        "rate": np.asarray([case["rate"]], dtype=np.uint32),
        "lat": np.asarray([case["lat"]], dtype=np.uint32),
        "G": np.asarray([G], dtype=np.uint32),
        "u_ppm": np.asarray([10**6], dtype=np.uint32),
        "cfg": None, "instances": [0], "name": case["id"],
    }
