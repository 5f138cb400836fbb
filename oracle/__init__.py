"""CPU oracle for Scattered Linear Attention -- test infrastructure only.

Only the test suite, the smoke check and the benchmark's CPU-baseline leg may use
this package.  It shares no code with the HIP library and imports nothing from it.
"""
from .sla_ref import (  # noqa: F401
    FEATURE_MAPS,
    chunk_plan_ref,
    cwi_backward_ref,
    cwi_forward_ref,
    dphi,
    dphi_relu,
    feature_map,
    phi,
    phi_relu,
    segments_ref,
    sla_backward_ref,
    sla_forward_ref,
    sla_projected_backward_ref,
    sla_projected_forward_ref,
    widen,
    xca_backward_ref,
    xca_forward_ref,
)
