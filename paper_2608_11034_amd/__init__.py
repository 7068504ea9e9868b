"""MI355X (gfx950) hot path of Consensus Collective Communication (C3).

The work runs in libc3.so (HIP kernels behind the C ABI of include/c3.h);
``paper_2608_11034_amd.c3`` is its Python binding for torch device tensors.
"""
from . import c3  # noqa: F401
from .c3 import (signature, tensor_signature, consensus, localize, confirm, num_chunks,  # noqa: F401
                 adamw_slice, OptimizerBoundaryCheck, timing_consensus, SignaturePlan,
                 C3Error)
