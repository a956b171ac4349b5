"""The C ABI library loads, exports every function ``include/alp.h`` declares, has the documented
struct layout, and rejects malformed arguments before touching a device (CPU only)."""
from __future__ import annotations

import ctypes as C
import os
import re
import subprocess

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "alp.h")

alp = pytest.importorskip("paper_2604_15186_amd.alp")


def declared_functions() -> list:
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(alp_[a-z_]+)\s*\(", text)))


def test_header_and_binding_agree():
    assert declared_functions() == sorted(alp.EXPORTS)


def _prototype(name: str) -> str:
    text = re.sub(r"/\*.*?\*/", "", open(HEADER).read(), flags=re.S)
    m = re.search(r"^([\w \*]+?)\b" + name + r"\s*\(([^)]*)\)\s*;", text, re.M)
    assert m, name
    return " ".join((m.group(1) + " " + name + "(" + m.group(2) + ")").split())


def test_documented_boundary_form():
    """The load call takes the six tables as flat arrays and every status comes back as int32_t
    (the form the design documents in place of a per-instance struct and an enum return)."""
    assert _prototype("alp_load_profiles") == (
        "int32_t alp_load_profiles(alp_ctx **out, const alp_space_t *space, uint32_t "
        "num_instances, const uint64_t *weight_bytes, const uint32_t *n_milli, const uint32_t "
        "*p_milli, const uint8_t *allowed, const uint32_t *rate_milli, const uint32_t *lat_us, "
        "uint64_t hbm_bytes_per_gpu, int32_t device, void *hip_stream)")
    assert _prototype("alp_search") == (
        "int32_t alp_search(alp_ctx *ctx, uint32_t instance, uint32_t gpu_budget, uint32_t "
        "target_milli, alp_result_t *out)")
    assert _prototype("alp_eval_candidates") == (
        "int32_t alp_eval_candidates(alp_ctx *ctx, uint32_t instance, uint32_t gpu_budget, "
        "uint32_t target_milli, const uint64_t *indices, uint64_t count, alp_eval_t *out)")
    void_or_str = {"alp_free", "alp_stats_free", "alp_status_str", "alp_last_error"}
    for name in declared_functions():
        if name not in void_or_str:
            assert _prototype(name).startswith("int32_t "), name
    text = open(HEADER).read()
    for name, cite in (("alp_search", "Eq. 1"), ("alp_search", "Section 3"),
                       ("alp_eval_candidates", "Eq. 2")):
        block = text[:text.index("int32_t " + name + "(")]
        assert cite in block[block.rindex("/*"):], (name, cite)


def test_library_exports_every_declared_symbol():
    lib = alp.lib()
    for name in declared_functions():
        assert hasattr(lib, name), name
    out = subprocess.run(["nm", "-D", "--defined-only", alp.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r"\bT (alp_[a-z_]+)\b", out))
    assert set(declared_functions()) <= exported


def test_struct_layout_matches_header(tmp_path):
    src = tmp_path / "layout.c"
    src.write_text(r'''
#include <stdio.h>
#include <stddef.h>
#include "alp.h"
int main(void) {
  printf("%zu %zu %zu %zu %zu %zu %zu\n", sizeof(alp_space_t), sizeof(alp_result_t), sizeof(alp_eval_t),
         sizeof(alp_plan_t), sizeof(alp_pruned_t), sizeof(alp_stats_t), sizeof(alp_placement_t));
  printf("%zu %zu %zu %zu\n", offsetof(alp_plan_t, max_latency_us), offsetof(alp_plan_t, sum_latency_us),
         offsetof(alp_pruned_t, fraction_vectors), offsetof(alp_pruned_t, unpruned_vectors));
  printf("%zu %zu %zu %zu %zu %zu %zu %zu\n", offsetof(alp_result_t, index),
         offsetof(alp_result_t, latency_us), offsetof(alp_result_t, throughput_milli),
         offsetof(alp_result_t, gpu_units), offsetof(alp_result_t, status),
         offsetof(alp_result_t, tp), offsetof(alp_result_t, frac_units),
         offsetof(alp_result_t, replicas));
  return 0;
}
''')
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-std=c11", "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe)],
                   check=True)
    lines = subprocess.run([str(exe)], capture_output=True, text=True, check=True).stdout.split("\n")
    sizes = [int(v) for v in lines[0].split()]
    assert sizes == [C.sizeof(alp.Space), alp.RESULT_DTYPE.itemsize, alp.EVAL_DTYPE.itemsize,
                     alp.PLAN_DTYPE.itemsize, alp.PRUNED_DTYPE.itemsize, alp.STATS_DTYPE.itemsize,
                     alp.PLACEMENT_DTYPE.itemsize]
    assert [int(v) for v in lines[1].split()] == [
        alp.PLAN_DTYPE.fields["max_latency_us"][1], alp.PLAN_DTYPE.fields["sum_latency_us"][1],
        alp.PRUNED_DTYPE.fields["vectors"][1], alp.PRUNED_DTYPE.fields["unpruned"][1]]
    offs = [int(v) for v in lines[2].split()]
    names = ["index", "latency_us", "throughput_milli", "gpu_units", "status", "tp", "frac_units",
             "replicas"]
    assert offs == [alp.RESULT_DTYPE.fields[n][1] for n in names]


def test_status_strings():
    names = ["ALP_OK", "ALP_EINVAL", "ALP_ERANGE", "ALP_ENOMEM", "ALP_EDEVICE", "ALP_INFEASIBLE"]
    for code, name in enumerate(names):
        assert alp.status_str(code) == name
    assert alp.status_str(99) == "ALP_UNKNOWN"


def _arrays(M=2, ntp=1, nfq=1, K=2, B=1):
    return {
        "W": np.ones((B, M), np.uint64), "n": np.full((B, M), 1000, np.uint32),
        "p": np.full((B, M), 1000, np.uint32), "allowed": np.ones((B, M, ntp, nfq), np.uint8),
        "rate": np.tile(np.arange(1, K + 1, dtype=np.uint32) * 100, (B, M, ntp, nfq, 1)),
        "lat": np.full((B, M, ntp, nfq, K), 1000, np.uint32),
    }


def _load(space: dict, a: dict, H=10**12, B=1, device=0):
    lib = alp.lib()
    s = alp.space_struct(space)
    ctx = C.c_void_p()
    ptr = lambda v: v.ctypes.data_as(C.c_void_p)  # noqa: E731
    st = lib.alp_load_profiles(C.byref(ctx), C.byref(s), B, ptr(a["W"]), ptr(a["n"]), ptr(a["p"]),
                               ptr(a["allowed"]), ptr(a["rate"]), ptr(a["lat"]), H, device, None)
    return st, ctx


BASE = {"M": 2, "tp": [1], "fq": [4], "Q": 4, "D": 2, "K": 2}


@pytest.mark.parametrize("change,why", [
    ({"M": 0}, "num_llms"), ({"M": 9}, "num_llms"), ({"tp": [2, 1]}, "ascending"),
    ({"tp": [0]}, "tp_values"), ({"fq": [5]}, "frac_units"), ({"Q": 17}, "units_per_gpu"),
    ({"D": 17}, "max_replicas"), ({"K": 0}, "num_points"),
    ({"tp": [1, 2, 3, 4, 5, 6, 7, 8], "fq": [1, 2, 3, 4, 5, 6, 7, 8], "Q": 8, "D": 16}, "options"),
])
def test_invalid_space_rejected(change, why):
    space = dict(BASE, **change)
    M = space["M"] if 1 <= space["M"] <= 8 else 2
    a = _arrays(M=M, ntp=len(space["tp"]), nfq=len(space["fq"]), K=max(space["K"], 1))
    st, ctx = _load(space, a)
    assert st == alp.ALP_EINVAL and not ctx.value
    assert why in alp.last_error()


def test_candidate_space_beyond_2_63_is_erange():
    # O = 4 * 8 * 8 = 256 options, 256^8 = 2^64 candidates
    space = {"M": 8, "tp": [1, 2, 4, 8], "fq": [1, 2, 3, 4, 5, 6, 7, 8], "Q": 8, "D": 8, "K": 1}
    a = _arrays(M=8, ntp=4, nfq=8, K=1)
    st, _ = _load(space, a)
    assert st == alp.ALP_ERANGE


@pytest.mark.parametrize("field,value,why", [
    ("n", 0, "n_milli"), ("p", 0, "p_milli"), ("allowed", 2, "allowed"),
    ("rate", None, "ascending"), ("lat", 1 << 31, "2^31"), ("W", 1 << 48, "weight_bytes"),
])
def test_invalid_tables_rejected(field, value, why):
    a = _arrays()
    if field == "rate":
        a["rate"][0, 1, 0, 0, :] = [500, 500]
    else:
        a[field].flat[1] = value
    st, ctx = _load(BASE, a)
    assert st == alp.ALP_EINVAL and not ctx.value
    assert why in alp.last_error()


def test_objective_overflow_is_erange():
    a = _arrays()
    a["lat"][:] = (1 << 31) - 1
    a["n"][:] = 4000
    a["p"][:] = 1000                    # 4 * 2^31 per LLM > 2^32
    st, _ = _load(BASE, a)
    assert st == alp.ALP_ERANGE
    assert "32-bit" in alp.last_error()


@pytest.mark.skipif(os.path.exists("/dev/kfd"), reason="a GPU driver is present on this machine")
def test_no_device_is_edevice():
    """Without a GPU driver no HIP device can be visible: a valid load is EDEVICE, exactly, and
    so is a statistics context."""
    st, ctx = _load(BASE, _arrays())
    assert st == alp.ALP_EDEVICE and not ctx.value
    assert "device" in alp.last_error()
    sctx = C.c_void_p()
    assert alp.lib().alp_stats_create(C.byref(sctx), 0, None) == alp.ALP_EDEVICE
    assert not sctx.value


def test_unfit_options_do_not_count_towards_overflow():
    a = _arrays()
    a["lat"][:] = (1 << 31) - 1
    a["n"][:] = 4000
    a["W"][:] = 10**6                  # H = 10 bytes below: nothing fits, so nothing can overflow
    st, ctx = _load(BASE, a, H=10)
    if st == alp.ALP_OK:
        alp.lib().alp_free(ctx)
    assert st in (alp.ALP_OK, alp.ALP_EDEVICE)   # EDEVICE on a machine without a GPU


def test_null_arguments_rejected():
    lib = alp.lib()
    assert lib.alp_load_profiles(None, None, 1, None, None, None, None, None, None, 1, 0, None) \
        == alp.ALP_EINVAL
    out = np.zeros(1, alp.RESULT_DTYPE)
    assert lib.alp_search(None, 0, 1, 1, out.ctypes.data_as(C.c_void_p)) == alp.ALP_EINVAL
    assert lib.alp_search_batch(None, 1, None, None, None, None) == alp.ALP_EINVAL
    assert lib.alp_search_batch_async(None, 1, None, None, None, None) == alp.ALP_EINVAL
    assert lib.alp_set_launch(None, 0, 0, 0, 0) == alp.ALP_EINVAL
    assert lib.alp_kernel_time_totals(None, (C.c_double * 3)(), None) == alp.ALP_EINVAL
    assert lib.alp_set_timing(None, 1) == alp.ALP_EINVAL
    assert lib.alp_search_pruned(None, 1, None, None, None, 3, None) == alp.ALP_EINVAL
    assert lib.alp_trace_stats(None, 2, 1, None, None, None, None, None) == alp.ALP_EINVAL
    assert lib.alp_stats_create(None, 0, None) == alp.ALP_EINVAL
    assert lib.alp_place(None, 1, None, None, None) == alp.ALP_EINVAL
    lib.alp_stats_free(None)
    assert lib.alp_allocate_workflows(None, 1, None, None, 4, 0, None, None, None) == alp.ALP_EINVAL
    lib.alp_free(None)
