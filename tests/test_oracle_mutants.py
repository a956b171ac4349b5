"""Each planted mistake of ``tests/oracle_mutants.py`` fails the pins it names (CPU only).

The mistake is applied to a copy of ``oracle/alp_oracle.c`` in a temporary directory, the copy
is built with gcc, and the named pin tests run against it in a child process (the oracle loads
the build that ``ALP_ORACLE_LIB`` names).  A pin that still passes on a planted mistake does not
pin what it claims to.
"""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

import pytest

from oracle_mutants import MUTANTS

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SOURCE = os.path.join(ROOT, "oracle", "alp_oracle.c")


def _mutated(src: str, old: str, new: str, nth: int) -> str:
    pos = -1
    for _ in range(nth + 1):
        pos = src.index(old, pos + 1)
    return src[:pos] + new + src[pos + len(old):]


def _run(k: int, tmp: str):
    name, old, new, nth, pins = MUTANTS[k]
    with open(SOURCE) as f:
        src = f.read()
    c = os.path.join(tmp, f"mutant{k}.c")
    so = os.path.join(tmp, f"mutant{k}.so")
    with open(c, "w") as f:
        f.write(_mutated(src, old, new, nth))
    b = subprocess.run(["gcc", "-std=c11", "-O1", "-shared", "-fPIC", c, "-o", so],
                       capture_output=True, text=True)
    if b.returncode != 0:
        return name, "build failed: " + b.stderr[-500:]
    env = dict(os.environ, ALP_ORACLE_LIB=so)
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-m", "not gpu",
                        "-p", "no:cacheprovider", *pins], cwd=ROOT, env=env, capture_output=True,
                       text=True, timeout=600)
    # 1: tests ran and some failed; anything else (0 = all passed, 4/5 = no such test) is a miss
    if r.returncode != 1:
        return name, f"pytest exit {r.returncode}: {r.stdout[-800:]}"
    return name, None


def test_mutants_apply_to_the_current_source():
    with open(SOURCE) as f:
        src = f.read()
    for name, old, new, nth, pins in MUTANTS:
        assert src.count(old) > nth, name
        assert pins, name


def test_every_planted_mistake_fails_its_pins(tmp_path):
    workers = max(1, min(8, len(os.sched_getaffinity(0))))
    with ThreadPoolExecutor(workers) as ex:
        results = list(ex.map(lambda k: _run(k, str(tmp_path)), range(len(MUTANTS))))
    missed = [(name, why) for name, why in results if why]
    assert not missed, missed
