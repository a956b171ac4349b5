"""Python binding of the gfx950 ALP allocation-search library (``libalp.so``).

Argument marshalling only: every step of the search runs in the HIP kernels behind the C ABI
declared in ``include/alp.h``.  PyTorch supplies the HIP stream the library orders its work on.
If the library has not been built, :func:`lib` raises -- there is no other implementation to
fall back to.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libalp.so")

ALP_OK, ALP_EINVAL, ALP_ERANGE, ALP_ENOMEM, ALP_EDEVICE, ALP_INFEASIBLE = range(6)
NO_INDEX = (1 << 64) - 1
NO_LATENCY = (1 << 32) - 1
MAX_LLMS = 8

# Symbols declared in include/alp.h.
EXPORTS = ("alp_load_profiles", "alp_search", "alp_search_batch", "alp_search_batch_async",
           "alp_search_batch_async_noalloc",
           "alp_max_throughput", "alp_allocate_workflows", "alp_search_pruned", "alp_stats_create",
           "alp_trace_stats", "alp_stats_set_timing", "alp_stats_time", "alp_stats_free", "alp_place",
           "alp_eval_candidates",
           "alp_set_launch", "alp_set_timing", "alp_kernel_times", "alp_kernel_time_totals",
           "alp_num_candidates", "alp_free",
           "alp_status_str", "alp_last_error")


class AlpError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{status_str(status)}: {message}")
        self.status = status


class Space(C.Structure):
    _fields_ = [("num_llms", C.c_uint32), ("num_tp", C.c_uint32), ("tp_values", C.c_uint32 * 8),
                ("num_frac", C.c_uint32), ("frac_units", C.c_uint32 * 8),
                ("units_per_gpu", C.c_uint32), ("max_replicas", C.c_uint32),
                ("num_points", C.c_uint32)]


RESULT_DTYPE = np.dtype([("index", np.uint64), ("latency_us", np.uint32),
                         ("throughput_milli", np.uint32), ("gpu_units", np.uint32),
                         ("status", np.uint32), ("tp", np.uint8, 8), ("frac_units", np.uint8, 8),
                         ("replicas", np.uint8, 8)])
EVAL_DTYPE = np.dtype([("flags", np.uint32), ("latency_us", np.uint32),
                       ("throughput_milli", np.uint32), ("gpu_units", np.uint32)])
PLAN_DTYPE = np.dtype([("status", np.uint32), ("policy", np.uint32), ("max_latency_us", np.uint32),
                       ("gpus_used", np.uint32), ("sum_latency_us", np.uint64)])
PRUNED_DTYPE = np.dtype([("best", RESULT_DTYPE), ("vectors", np.uint64), ("unpruned", np.uint64)])
assert RESULT_DTYPE.itemsize == 48 and EVAL_DTYPE.itemsize == 16 and PLAN_DTYPE.itemsize == 24
assert PRUNED_DTYPE.itemsize == 64
STATS_DTYPE = np.dtype([("n_milli", np.uint32), ("p_milli", np.uint32), ("calls", np.uint64),
                        ("busy_us", np.uint64), ("active_us", np.uint64)])
assert STATS_DTYPE.itemsize == 32
PLACEMENT_DTYPE = np.dtype([("status", np.uint32), ("replicas", np.uint32),
                            ("gpus_used", np.uint32), ("nodes_used", np.uint32),
                            ("slot", np.uint16, 128)])
assert PLACEMENT_DTYPE.itemsize == 272
PLACE_NONE = 0xFFFF
WELFARE_EGALITARIAN, WELFARE_SOCIAL = 0, 1
PRUNE_ORDER, PRUNE_MIN_FRACTION = 1, 2

_lib = None


def lib():
    """Loads ``libalp.so``; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build() first")
        L = C.CDLL(LIB_PATH)
        vp, u32, u64, i32 = C.c_void_p, C.c_uint32, C.c_uint64, C.c_int32
        L.alp_load_profiles.argtypes = [C.POINTER(vp), C.POINTER(Space), u32, vp, vp, vp, vp, vp,
                                        vp, u64, i32, vp]
        L.alp_search.argtypes = [vp, u32, u32, u32, vp]
        L.alp_search_batch.argtypes = [vp, u32, vp, vp, vp, vp]
        L.alp_search_batch_async.argtypes = [vp, u32, vp, vp, vp, vp]
        L.alp_search_batch_async_noalloc.argtypes = [vp, u32, vp, vp, vp, vp]
        L.alp_max_throughput.argtypes = [vp, u32, vp, vp, vp]
        L.alp_eval_candidates.argtypes = [vp, u32, u32, u32, vp, u64, vp]
        L.alp_allocate_workflows.argtypes = [vp, u32, vp, vp, u32, u32, vp, vp, vp]
        L.alp_search_pruned.argtypes = [vp, u32, vp, vp, vp, u32, vp]
        L.alp_place.argtypes = [vp, u32, vp, vp, vp]
        L.alp_stats_create.argtypes = [C.POINTER(vp), i32, vp]
        L.alp_trace_stats.argtypes = [vp, u32, u32, vp, vp, vp, vp, vp]
        L.alp_stats_set_timing.argtypes = [vp, i32]
        L.alp_stats_time.argtypes = [vp, C.POINTER(C.c_float)]
        L.alp_stats_free.argtypes = [vp]
        L.alp_stats_free.restype = None
        L.alp_set_launch.argtypes = [vp, u32, u32, u32, u32]
        L.alp_set_timing.argtypes = [vp, i32]
        L.alp_kernel_times.argtypes = [vp, C.POINTER(C.c_float), C.POINTER(u32)]
        L.alp_kernel_time_totals.argtypes = [vp, C.POINTER(C.c_double), C.POINTER(u64)]
        L.alp_num_candidates.argtypes = [vp, C.POINTER(u64)]
        for name in ("alp_load_profiles", "alp_search", "alp_search_batch",
                     "alp_search_batch_async", "alp_search_batch_async_noalloc",
                     "alp_max_throughput",
                     "alp_allocate_workflows", "alp_search_pruned", "alp_stats_create",
                     "alp_trace_stats", "alp_stats_set_timing", "alp_stats_time", "alp_place",
                     "alp_eval_candidates", "alp_set_launch", "alp_set_timing",
                     "alp_kernel_times", "alp_kernel_time_totals", "alp_num_candidates"):
            getattr(L, name).restype = i32
        L.alp_free.argtypes = [vp]
        L.alp_free.restype = None
        L.alp_status_str.argtypes = [i32]
        L.alp_status_str.restype = C.c_char_p
        L.alp_last_error.argtypes = []
        L.alp_last_error.restype = C.c_char_p
        _lib = L
    return _lib


def status_str(status: int) -> str:
    return lib().alp_status_str(status).decode()


def last_error() -> str:
    return lib().alp_last_error().decode()


def _check(status: int, allowed=(ALP_OK,)) -> int:
    if status not in allowed:
        raise AlpError(status, last_error())
    return status


def _ptr(a: np.ndarray) -> int:
    # The address as an int (ctypes converts it for c_void_p arguments); data_as() costs several
    # microseconds per call, which a single small search can notice.
    return a.ctypes.data


def space_struct(space: dict) -> Space:
    s = Space()
    s.num_llms = int(space["M"])
    tp = [int(v) for v in space["tp"]]
    fq = [int(v) for v in space["fq"]]
    s.num_tp, s.num_frac = len(tp), len(fq)
    for i, v in enumerate(tp[:8]):
        s.tp_values[i] = v
    for j, v in enumerate(fq[:8]):
        s.frac_units[j] = v
    s.units_per_gpu, s.max_replicas, s.num_points = int(space["Q"]), int(space["D"]), int(space["K"])
    return s


def torch_stream(device: int = 0) -> int:
    """Handle of torch's current HIP stream on ``device`` (0 if torch sees no GPU)."""
    try:
        import torch
    except ImportError:
        return 0
    if not torch.cuda.is_available():
        return 0
    return int(torch.cuda.current_stream(device).cuda_stream)


class Context:
    """Profiles of a batch of workflow instances resident on one GPU (``alp_load_profiles``)."""

    def __init__(self, batch: dict, device: int = 0, stream: int | None = None):
        self._keep = {
            "W": np.ascontiguousarray(batch["W"], dtype=np.uint64),
            "n": np.ascontiguousarray(batch["n"], dtype=np.uint32),
            "p": np.ascontiguousarray(batch["p"], dtype=np.uint32),
            "allowed": np.ascontiguousarray(batch["allowed"], dtype=np.uint8),
            "rate": np.ascontiguousarray(batch["rate"], dtype=np.uint32),
            "lat": np.ascontiguousarray(batch["lat"], dtype=np.uint32),
        }
        k = self._keep
        self.space = space_struct(batch["space"])
        self.num_instances = int(k["W"].shape[0])
        self.M = int(batch["space"]["M"])
        self.stream = torch_stream(device) if stream is None else int(stream)
        self._ctx = C.c_void_p()
        _check(lib().alp_load_profiles(C.byref(self._ctx), C.byref(self.space), self.num_instances,
                                       _ptr(k["W"]), _ptr(k["n"]), _ptr(k["p"]),
                                       _ptr(k["allowed"]), _ptr(k["rate"]), _ptr(k["lat"]),
                                       int(batch["H"]), device, self.stream))
        n = C.c_uint64()
        _check(lib().alp_num_candidates(self._ctx, C.byref(n)))
        self.num_candidates = int(n.value)

    def close(self):
        if self._ctx:
            lib().alp_free(self._ctx)
            self._ctx = C.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    def search(self, instance: int, gpu_budget: int, target_milli: int) -> np.void:
        out = np.zeros(1, dtype=RESULT_DTYPE)
        _check(lib().alp_search(self._ctx, instance, gpu_budget, target_milli, _ptr(out)),
               (ALP_OK, ALP_INFEASIBLE))
        return out[0]

    def search_batch(self, gpu_budget, target_milli, instances=None) -> np.ndarray:
        G = np.ascontiguousarray(gpu_budget, dtype=np.uint32)
        lam = np.ascontiguousarray(target_milli, dtype=np.uint32)
        count = len(G)
        assert len(lam) == count
        inst = None if instances is None else np.ascontiguousarray(instances, dtype=np.uint32)
        out = np.zeros(count, dtype=RESULT_DTYPE)
        _check(lib().alp_search_batch(self._ctx, count, None if inst is None else _ptr(inst),
                                      _ptr(G), _ptr(lam), _ptr(out)))
        return out

    def search_batch_async(self, gpu_budget, target_milli, out, instances=None,
                           noalloc: bool = False) -> None:
        """alp_search_batch_async: torch tensors on the context's device -- gpu_budget,
        target_milli (and instances) of int32 or uint32, out of uint8 with count * 48 bytes.
        Queued on the context stream; read out after that stream's work is done (see
        results_from_device).  noalloc: alp_search_batch_async_noalloc instead (scratch in the
        library's fixed device array)."""
        count = int(gpu_budget.numel())
        tensors = [gpu_budget, target_milli] + ([] if instances is None else [instances])
        for t in tensors:
            if not t.is_cuda or not t.is_contiguous() or t.element_size() != 4 or t.numel() != count:
                raise ValueError("queries must be contiguous 32-bit device tensors of one length")
        if not out.is_cuda or not out.is_contiguous() or out.numel() * out.element_size() < \
                count * RESULT_DTYPE.itemsize:
            raise ValueError(f"out must be a contiguous device tensor of {count} x "
                             f"{RESULT_DTYPE.itemsize} bytes")
        fn = lib().alp_search_batch_async_noalloc if noalloc else lib().alp_search_batch_async
        _check(fn(self._ctx, count, None if instances is None else instances.data_ptr(),
                  gpu_budget.data_ptr(), target_milli.data_ptr(), out.data_ptr()))

    def max_throughput(self, gpu_budget, instances=None) -> np.ndarray:
        G = np.ascontiguousarray(gpu_budget, dtype=np.uint32)
        inst = None if instances is None else np.ascontiguousarray(instances, dtype=np.uint32)
        out = np.zeros(len(G), dtype=np.uint32)
        _check(lib().alp_max_throughput(self._ctx, len(G), None if inst is None else _ptr(inst),
                                        _ptr(G), _ptr(out)))
        return out

    def allocate_workflows(self, target_milli, total_gpus: int, policy: int = WELFARE_EGALITARIAN,
                           instances=None):
        """Splits total_gpus over workflows (alp_allocate_workflows).  Returns (plan record,
        budgets, per-workflow results); budgets and results are None when infeasible."""
        lam = np.ascontiguousarray(target_milli, dtype=np.uint32)
        W = len(lam)
        inst = None if instances is None else np.ascontiguousarray(instances, dtype=np.uint32)
        plan = np.zeros(1, dtype=PLAN_DTYPE)
        gpus = np.zeros(W, dtype=np.uint32)
        res = np.zeros(W, dtype=RESULT_DTYPE)
        st = _check(lib().alp_allocate_workflows(self._ctx, W, None if inst is None else _ptr(inst),
                                                 _ptr(lam), total_gpus, policy, _ptr(plan),
                                                 _ptr(gpus), _ptr(res)), (ALP_OK, ALP_INFEASIBLE))
        if st == ALP_INFEASIBLE:
            return plan[0], None, None
        return plan[0], gpus, res

    def search_pruned(self, gpu_budget, target_milli, flags: int = PRUNE_ORDER | PRUNE_MIN_FRACTION,
                      instances=None) -> np.ndarray:
        """The paper's pruned search for each query (alp_search_pruned); PRUNED_DTYPE records."""
        G = np.ascontiguousarray(gpu_budget, dtype=np.uint32)
        lam = np.ascontiguousarray(target_milli, dtype=np.uint32)
        assert len(lam) == len(G)
        inst = None if instances is None else np.ascontiguousarray(instances, dtype=np.uint32)
        out = np.zeros(len(G), dtype=PRUNED_DTYPE)
        _check(lib().alp_search_pruned(self._ctx, len(G), None if inst is None else _ptr(inst),
                                       _ptr(G), _ptr(lam), flags, _ptr(out)))
        return out

    def place(self, allocations, gpu_budget) -> np.ndarray:
        """Places search results (RESULT_DTYPE records) on their GPU budgets (alp_place)."""
        res = np.ascontiguousarray(allocations, dtype=RESULT_DTYPE)
        G = np.ascontiguousarray(gpu_budget, dtype=np.uint32)
        assert len(G) == len(res)
        out = np.zeros(len(res), dtype=PLACEMENT_DTYPE)
        _check(lib().alp_place(self._ctx, len(res), _ptr(res), _ptr(G), _ptr(out)))
        return out

    def eval_candidates(self, instance: int, gpu_budget: int, target_milli: int, indices) -> np.ndarray:
        idx = np.ascontiguousarray(indices, dtype=np.uint64)
        out = np.zeros(len(idx), dtype=EVAL_DTYPE)
        _check(lib().alp_eval_candidates(self._ctx, instance, gpu_budget, target_milli, _ptr(idx),
                                         len(idx), _ptr(out)))
        return out

    def set_launch(self, variant: int = 0, blocks_per_item: int = 0, threads_per_block: int = 0,
                   inner_chunks: int = 0):
        _check(lib().alp_set_launch(self._ctx, variant, blocks_per_item, threads_per_block,
                                    inner_chunks))

    def set_timing(self, enable: bool | int):
        """False/0: off; True/1: every call timed; N: the first and every N-th call timed."""
        _check(lib().alp_set_timing(self._ctx, int(enable)))

    def kernel_time_totals(self) -> tuple[np.ndarray, int]:
        """(sums of kernel_times()' three figures, number of timed calls) since timing was set."""
        ms = (C.c_double * 3)()
        calls = C.c_uint64()
        _check(lib().alp_kernel_time_totals(self._ctx, ms, C.byref(calls)))
        return np.array([ms[0], ms[1], ms[2]]), int(calls.value)

    def kernel_times(self):
        """(option-term ms, scan ms, third-kernel ms, grid blocks) of the last call; the third
        kernel is the budget split or the pruned search's option table."""
        ms = (C.c_float * 3)()
        blocks = C.c_uint32()
        _check(lib().alp_kernel_times(self._ctx, ms, C.byref(blocks)))
        return float(ms[0]), float(ms[1]), float(ms[2]), int(blocks.value)


class StatsContext:
    """Workflow statistics from execution traces on one GPU (alp_stats_create / alp_trace_stats).

    ``compute`` takes torch tensors already on the device (offsets and timestamps 64-bit, llm
    32-bit), or numpy arrays, which it copies to the device first with torch."""

    def __init__(self, device: int = 0, stream: int | None = None):
        self.device = device
        self.stream = torch_stream(device) if stream is None else int(stream)
        self._ctx = C.c_void_p()
        _check(lib().alp_stats_create(C.byref(self._ctx), device, self.stream))

    @staticmethod
    def _device_array(a, dtype, device):
        import torch
        if isinstance(a, torch.Tensor):
            assert a.is_cuda and a.is_contiguous() and a.element_size() == np.dtype(dtype).itemsize
            return a
        a = np.ascontiguousarray(a, dtype=dtype)
        signed = {np.dtype(np.uint64): np.int64, np.dtype(np.uint32): np.int32}[a.dtype]
        return torch.from_numpy(a.view(signed)).to(f"cuda:{device}")

    def compute(self, num_llms: int, offsets, llm, start, end) -> np.ndarray:
        dev = [self._device_array(a, t, self.device) for a, t in
               ((offsets, np.uint64), (llm, np.uint32), (start, np.uint64), (end, np.uint64))]
        out = np.zeros(num_llms, dtype=STATS_DTYPE)
        R = int(dev[0].numel()) - 1
        _check(lib().alp_trace_stats(self._ctx, num_llms, R,
                                     *(C.c_void_p(t.data_ptr()) for t in dev), _ptr(out)))
        return out

    def set_timing(self, enable: bool):
        _check(lib().alp_stats_set_timing(self._ctx, 1 if enable else 0))

    def time_ms(self) -> float:
        ms = C.c_float()
        _check(lib().alp_stats_time(self._ctx, C.byref(ms)))
        return float(ms.value)

    def close(self):
        if self._ctx:
            lib().alp_stats_free(self._ctx)
            self._ctx = C.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()


def results_from_device(out, count: int) -> np.ndarray:
    """The first count records of a device tensor written by search_batch_async (copies to the
    host; call after the stream's work is done)."""
    import torch
    raw = out.reshape(-1).view(torch.uint8)[: count * RESULT_DTYPE.itemsize]
    return raw.cpu().numpy().view(RESULT_DTYPE).copy()


def result_dict(r) -> dict:
    """Plain-Python view of one RESULT_DTYPE record."""
    d = {k: int(r[k]) for k in ("index", "latency_us", "throughput_milli", "gpu_units", "status")}
    d["x"] = None if d["index"] == NO_INDEX else d["index"]
    for k in ("tp", "frac_units", "replicas"):
        d[k] = [int(v) for v in r[k]]
    return d
