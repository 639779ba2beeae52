"""Verification logits from the LM head (oracle; test infrastructure only).

Sec. 3.2: the target distribution at each verification slot is the target
model's prediction there, i.e. the LM head applied to the slot's final hidden
state.  Here that product is written out in float64 -- logits[b, k, v] =
hidden[b, k, :] . weight[v, :] -- and handed to the greedy acceptance oracle,
so the fused kernel (which never stores the logits) is checked against the
plain definition.
"""

from __future__ import annotations

import numpy as np

from .accept import verify_accept
from .widen import widen


def lmhead_logits(hidden, weight, dtype: str) -> np.ndarray:
    """float64 logits [b, B, V] of hidden [b, B, H] and weight [V, H]."""
    h = widen(np.asarray(hidden), dtype)
    V = weight.shape[0]
    out = np.empty(h.shape[:-1] + (V,), np.float64)
    step = 1 << 13                              # bounded float64 copies of the weight
    for v0 in range(0, V, step):
        out[..., v0:v0 + step] = h @ widen(weight[v0:v0 + step], dtype).T
    return out


def verify_accept_lmhead(hidden, weight, draft_ids, step_map, num_ref, dtype: str):
    """Greedy acceptance (eq. 2 at temperature 0) on the LM-head logits:
    (target_ids, confidence, draft_prob, accept_len) as ``accept.verify_accept``;
    also the float64 logits for tie checks."""
    logits = lmhead_logits(hidden, weight, dtype)
    out = verify_accept(logits, draft_ids, step_map, num_ref, "f64")
    return out + (logits,)
