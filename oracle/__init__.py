"""CPU oracle for the SimSD verification step -- TEST INFRASTRUCTURE ONLY.

A plain, slow, float64 numpy statement of what the GPU path computes:

  * ``mask``      slot labels and the token-level temporal attention mask of
                  Sec. 3.1 (eq. 1), with the prompt visible to every response row
                  and padding rows/columns removed;
  * ``attention`` softmax attention of every new row over [cached prefix | new
                  slots] under that mask (Sec. 3.2, "Target Model Verification");
  * ``accept``    the greedy (temperature-0) form of the acceptance rule of
                  eq. 2: argmax with lowest-index ties, softmax confidence, the
                  target probability of each draft and the accepted prefix length;
  * ``rope``      rotary embedding at the RoPE-copy positions of Sec. 3.1-3.2,
                  applied to the new slots' queries and keys when asked for;
  * ``lmhead``    the verification logits written out as hidden . weight^T
                  (float64) and handed to the greedy acceptance;
  * ``sampled``   the stochastic form of eq. 2 at temperature T: acceptance with
                  probability min(1, p_theta/p_phi) from caller-supplied uniforms
                  and the residual draw at the first rejection.

Only the test-suite, the smoke check and the benchmark's CPU-baseline leg may
import this package.  The product path (the C-ABI library and its Python
binding) never imports, links or calls it, and shares no code with it.  Inputs
come from the ``synth`` generator; bfloat16 tensors arrive as uint16 bit
patterns and are widened exactly to float64 here.
"""

from .widen import widen
from .mask import slot_labels, new_slot_visibility, DATA, MASK
from .attention import attend, verify_attention
from .accept import verify_accept
from .sampled import verify_accept_sampled
from .lmhead import lmhead_logits, verify_accept_lmhead

__all__ = ["widen", "slot_labels", "new_slot_visibility", "DATA", "MASK", "attend",
           "verify_attention", "verify_accept", "verify_accept_sampled", "lmhead_logits",
           "verify_accept_lmhead"]
