"""MI355X-native Higher-order Linear Attention (arXiv 2510.27258).

The computation lives in libhla.so (HIP for gfx950, C ABI in include/hla.h).
`capi` mirrors the C entry points one to one; `hla` wraps them for torch
tensors (torch provides device memory and the current stream only).
"""
from . import capi  # noqa: F401
from .hla import (HLA2, State, ahla_forward, backward, chunk_summaries, forward, forward_decay,  # noqa: F401
                  hla2_attention, hla3_forward, prefill, scan, split_state, state_floats, step, workspace_bytes)
