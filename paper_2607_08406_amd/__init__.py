"""MI355X (gfx950) implementation of the hot path of the Monte Carlo
mutation-selection method (MCA): single-parameter mutation, incremental loss
evaluation from cached local fields, greedy accept or roll back.

The computation lives in the HIP library ``libmca.so`` (C ABI in
``include/mca.h``); ``paper_2607_08406_amd.mca`` is its ctypes binding.
"""
from . import mca  # noqa: F401
from .mca import Context, MCAError, TransformerContext, mlp_desc, transformer_desc  # noqa: F401

__all__ = ["mca", "Context", "MCAError", "TransformerContext", "mlp_desc", "transformer_desc"]
