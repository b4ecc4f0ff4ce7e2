"""Seeded synthetic inputs shared by the tests, the benchmark and the oracle checks.

Holds input generation only (lengths, page placement, N(0,1) bf16 tensors); none of
the attention arithmetic lives here.
"""
from .configs import (KILO, SPECS, TENSOR_K, TENSOR_Q, TENSOR_V, Spec, Workload,
                      custom_group_workload, custom_prune_workload, custom_workload,
                      make_workload)
from ._native import build, host_threads, normal_bf16, normal_f32, philox4x32_10

__all__ = ["KILO", "SPECS", "TENSOR_K", "TENSOR_Q", "TENSOR_V", "Spec", "Workload",
           "custom_group_workload", "custom_prune_workload", "custom_workload", "make_workload",
           "build", "host_threads", "normal_bf16", "normal_f32", "philox4x32_10"]
