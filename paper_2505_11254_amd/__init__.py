"""MI355X-native Delta Attention prefill (arXiv 2505.11254).

The compute path is a C-ABI shared library of hand-written gfx950 HIP kernels
(``csrc/``, declared in ``include/delta_attn.h``).  ``binding`` marshals torch
tensors into those calls; torch only supplies device memory and streams.
Importing this package loads nothing: the library is loaded on first call.
"""
from .workloads import WORKLOADS, HEADLINE, Workload  # noqa: F401

__all__ = ["WORKLOADS", "HEADLINE", "Workload"]
