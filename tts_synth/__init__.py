"""Seeded synthetic beam-search workloads for prefix-shared decode attention.

This package only *generates inputs*: beam trees, paged block tables,
sequence lengths, and the query / key / value tensors in their storage
formats. It holds none of the attention arithmetic and none of the prefix
metadata logic, so both the CPU oracle and the HIP library can consume it
without sharing any of the method's code.
"""

from .workload import (  # noqa: F401
    CONFIGS,
    AttnShape,
    ReqSpec,
    WorkloadConfig,
    Workload,
    BeamTree,
    build_tree,
    make_workload,
    workload_from_tree,
)
