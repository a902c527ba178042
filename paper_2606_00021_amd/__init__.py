"""SENSE retrieval + soft-gated evaluation hot path for one AMD MI355X (gfx950).

The kernels live in ``libsense.so`` (HIP, built from ``csrc/``); ``sense``
is its Python binding and ``synth`` the seeded workload generator.
"""
from .sense import (  # noqa: F401
    Index,
    SenseError,
    load_library,
    sense_build_index,
    sense_retrieve,
    sense_retrieve_workspace_size,
    sense_soft_gate_verify,
    sense_soft_gate_verify_workspace_size,
)
