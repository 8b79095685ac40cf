"""CPU oracle for the SMoES MoE layer: test infrastructure, not the product.

Only tests/, the smoke entry and the benchmark's CPU-baseline leg may import
this package. It is plain float64 NumPy written from the paper's equations and
shares no code with the HIP path (which must never fall back to it).
"""
from .smoes_oracle import *  # noqa: F401,F403
from .smoes_oracle import GaussState, GmmState  # noqa: F401
