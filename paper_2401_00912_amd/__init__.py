"""Scattered Linear Attention (SLA, arXiv 2401.00912) on AMD Instinct MI355X.

The compute path is libsla.so (hand-written HIP for gfx950, C ABI in
include/sla.h); ``paper_2401_00912_amd.sla`` is its Python binding.
"""
from . import sla  # noqa: F401
from .sla import backward, build_segments, forward, plan_bytes, plan_layout  # noqa: F401
