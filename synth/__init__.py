"""Seeded synthetic inputs shared by the HIP path, the oracle and the benchmark.

This package draws weights and coordinate weights only.  It holds none of
the codec's arithmetic (no backbone, no basis, no fit): both sides of every
parity check receive the very same tensors from here.
"""
from .workloads import (  # noqa: F401
    Module,
    Workload,
    WORKLOADS,
    workload,
    gen_module_inputs,
    gen_records,
    round_half_even_count,
)
