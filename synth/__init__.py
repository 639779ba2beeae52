"""Seeded synthetic inputs for the SimSD verification step.

This package only *makes* inputs: tensors of the shapes, dtypes and value
distributions of the verification workloads, from fixed seeds.  It holds none of
the verification arithmetic (no mask, no attention, no argmax): the CPU oracle
and the GPU path both consume what it produces and neither is imported here.
"""

from .configs import CONFIGS, VerifyConfig, config_by_id
from .generate import (VerifyInputs, generate, generate_draft_side, generate_lmhead_side,
                       bf16_bits_from_f32)

__all__ = ["CONFIGS", "VerifyConfig", "config_by_id", "VerifyInputs", "generate",
           "generate_draft_side", "generate_lmhead_side", "bf16_bits_from_f32"]
