"""Greedy acceptance over the verification logits (oracle; test infrastructure only).

Sec. 3.2 ("Target Model Verification"), eq. 2: draft r is accepted with
probability min(1, p_theta(r)(D_r) / p_phi(r)(D_r)), in draft order, and the
longest prefix before the first rejection is kept.  At temperature 0 both
distributions are one-hot on their argmax, so alpha_r is 1 when the target's
argmax equals the draft and 0 otherwise; the token the target supplies at the
first rejection is its argmax.  That limit is what is computed here.

Per scanned block row (step_map >= 1; rows at or below 0 are committed or
padding and are not scanned):
  target_id   smallest vocabulary index whose stored logit equals the row maximum
  confidence  exp(max - logsumexp(row)), the largest softmax probability (T = 1)
Per draft r < gamma:
  draft_prob  exp(x[draft] - logsumexp(row)), 0 for an id outside [0, V)
Per sequence:
  accept_len  the largest a <= gamma with target_id(row of draft r) == draft r
              for every r < a.
"""

from __future__ import annotations

import math

import numpy as np

from .widen import widen


def scan_row(x: np.ndarray):
    """(target_id, max, logsumexp) of one float64 logit row."""
    m = x.max()
    target = int(np.flatnonzero(x == m)[0])
    lse = m + math.log(np.exp(x - m).sum())
    return target, m, lse


def verify_accept(logits, draft_ids, step_map, num_ref, dtype: str):
    """Returns target_ids int32 [b, B], confidence float64 [b, B],
    draft_prob float64 [b, L] and accept_len int32 [b]."""
    logits = np.asarray(logits)
    b, B, V = logits.shape
    L = draft_ids.shape[1]
    target_ids = np.full((b, B), -1, np.int32)
    confidence = np.zeros((b, B))
    row_lse = np.full((b, B), np.nan)
    draft_prob = np.zeros((b, L))
    accept_len = np.zeros((b,), np.int32)
    for s in range(b):
        for k in range(B):
            if step_map[s, k] >= 1:
                x = widen(logits[s, k], dtype)
                t, m, lse = scan_row(x)
                target_ids[s, k] = t
                confidence[s, k] = math.exp(m - lse)
                row_lse[s, k] = lse
        gamma = int(num_ref[s])
        accepting = True
        for r in range(gamma):
            k_r = int(np.flatnonzero(step_map[s] == r + 1)[0])
            tok = int(draft_ids[s, r])
            if 0 <= tok < V:
                draft_prob[s, r] = math.exp(float(widen(logits[s, k_r, tok], dtype))
                                            - row_lse[s, k_r])
            if accepting and target_ids[s, k_r] == tok:
                accept_len[s] += 1
            else:
                accepting = False
    return target_ids, confidence, draft_prob, accept_len
