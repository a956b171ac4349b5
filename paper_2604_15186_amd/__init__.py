"""MI355X (gfx950) implementation of the Aggregate LLM Pipeline allocation search of Scepsy
(arXiv 2604.15186): exhaustive evaluation of the latency / throughput predictor over every
per-LLM choice of tensor-parallel degree, GPU share and replica count, and the constrained
argmin.  The computation runs in HIP kernels behind the C ABI of ``include/alp.h``;
:mod:`paper_2604_15186_amd.alp` is the Python binding.
"""
from .alp import (  # noqa: F401
    ALP_EDEVICE,
    ALP_EINVAL,
    ALP_ENOMEM,
    ALP_ERANGE,
    ALP_INFEASIBLE,
    ALP_OK,
    AlpError,
    Context,
    EVAL_DTYPE,
    RESULT_DTYPE,
    lib,
    result_dict,
)
