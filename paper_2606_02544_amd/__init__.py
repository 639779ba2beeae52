"""SimSD verification step on AMD MI355X (gfx950).

The compute lives in ``libsimsd.so`` (HIP kernels behind the C ABI of
include/simsd.h); ``binding`` marshals torch tensors into those calls.
"""

from . import binding
from .binding import (SimsdError, verify_attention, verify_accept, validate_step_map,
                      attention_desc, accept_desc, attention_workspace_size,
                      accept_workspace_size)

__all__ = ["binding", "SimsdError", "verify_attention", "verify_accept", "validate_step_map",
           "attention_desc", "accept_desc", "attention_workspace_size", "accept_workspace_size"]
