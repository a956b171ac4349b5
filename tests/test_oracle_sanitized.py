"""The oracle's pins under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

``oracle/alp_oracle.c`` is built with ``-fsanitize=address,undefined -fno-sanitize-recover=all``
and the ``-m "not gpu"`` pin suites run against that build in a child process (the Python
interpreter is not instrumented, so the ASan runtime is preloaded; leak checking is off because
the interpreter itself keeps memory until exit).  Any out-of-bounds access, use after free,
signed overflow, misaligned access or shift past the width aborts the child and fails here.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PIN_SUITES = ["tests/test_oracle_pins.py", "tests/test_place_pins.py", "tests/test_stats_pins.py"]


def _runtime(name: str) -> str:
    path = subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True, text=True,
                          check=True).stdout.strip()
    if not os.path.isabs(path) or not os.path.exists(path):
        pytest.skip(f"{name} is not available to gcc here")
    return path


@pytest.fixture(scope="module")
def sanitized_lib(tmp_path_factory):
    if shutil.which("gcc") is None:
        pytest.skip("gcc not available")
    out = tmp_path_factory.mktemp("asan") / "liborc_asan_ubsan.so"
    subprocess.run(["gcc", "-std=c11", "-O1", "-g", "-fsanitize=address,undefined",
                    "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-shared", "-fPIC",
                    os.path.join(ROOT, "oracle", "alp_oracle.c"), "-o", str(out)], check=True)
    syms = subprocess.run(["nm", "-D", str(out)], capture_output=True, text=True, check=True).stdout
    assert "__asan_report" in syms and "__ubsan_handle" in syms   # really instrumented
    return str(out)


def test_pins_pass_under_asan_and_ubsan(sanitized_lib):
    env = dict(os.environ)
    env.update({
        "ALP_ORACLE_LIB": sanitized_lib,
        "LD_PRELOAD": f"{_runtime('libasan.so')} {_runtime('libubsan.so')}",
        "ASAN_OPTIONS": "detect_leaks=0:abort_on_error=1",
        "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1",
    })
    check = ("import oracle, sys; oracle.lib(); "
             "sys.exit(0 if oracle.LIB_PATH == sys.argv[1] else 3)")
    r = subprocess.run([sys.executable, "-c", check, sanitized_lib], cwd=ROOT, env=env,
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr[-2000:]
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-m", "not gpu",
                        "-p", "no:cacheprovider", *PIN_SUITES], cwd=ROOT, env=env,
                       capture_output=True, text=True, timeout=900)
    assert r.returncode == 0, (r.stdout[-3000:], r.stderr[-3000:])
    assert " passed" in r.stdout and "ERROR: AddressSanitizer" not in r.stderr
