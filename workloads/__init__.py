"""Seeded synthetic request batches shared by the tests, the benchmark and the oracle harness.

This package only produces input data (token ids, request boundaries, provenance
descriptors as raw (name, value) byte fields, locations).  It performs no hashing, no
encoding and no table logic, so the GPU path and the CPU oracle can both consume it
without sharing any of the method's arithmetic.
"""

from .recipes import (  # noqa: F401
    Batch,
    Workload,
    CORE_NAMES,
    make_workload,
    locations,
    WORKLOADS,
    OmissionCase,
    OMISSION_CASES,
    make_omission,
    make_omission_tiny,
    make_budget,
    identity_shapes,
)
