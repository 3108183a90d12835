"""Seeded synthetic inputs shared by the tests, the benchmark and the oracle.

This module holds no part of the attention method's arithmetic: it draws
Q/K/V, draws and packs routing maps, and picks rows to sample.  Both the HIP
path and the CPU oracle receive exactly the arrays it returns.
"""

from .configs import WorkloadConfig, MaskSpec, WORKLOADS, workload, small_workload
from .generate import (
    make_qkv,
    make_route_bits,
    decode_route_bits,
    legal_group_table,
    route_stats,
    sample_rows,
    pack_route_bits,
)

__all__ = [
    "WorkloadConfig",
    "MaskSpec",
    "WORKLOADS",
    "workload",
    "small_workload",
    "make_qkv",
    "make_route_bits",
    "decode_route_bits",
    "legal_group_table",
    "route_stats",
    "sample_rows",
    "pack_route_bits",
]
