"""Stochastic acceptance of eq. 2 (oracle; test infrastructure only).

Sec. 3.2 ("Target Model Verification"), eq. 2: draft r is accepted with
probability alpha_r = min(1, p_theta(r)(D_r) / p_phi(r)(D_r)), in the
draft-induced order, and the longest prefix before the first rejection is
kept; at the first rejection the target supplies the token at that position
and the drafted suffix is dropped.  The paper runs it at temperature 1.0
(Sec. 4.1, configurations).  Readings (the paper states the rule, not
these details):

  * p_theta(r) = softmax(logits[b, k_r] / T), k_r the block slot verified at
    step r (its verification row); p_phi(r) = softmax(draft_logits[b, r-1] / T),
    the drafter's distribution when it proposed draft r.
  * The draw behind alpha_r is a caller-supplied uniform u_r = uniforms[b, r-1]
    in [0, 1): draft r is accepted iff u_r * p_phi(D_r) < p_theta(D_r), which
    happens with probability min(1, p_theta/p_phi).  A draft id outside [0, V)
    is a rejection.
  * The token at the first rejection (draft a+1) is the standard speculative
    sampling residual, q(x) = max(0, p_theta(x) - p_phi(x)) / Z: drawn by
    inverse CDF in vocabulary order with w = uniforms[b, L], i.e. the smallest
    x whose running sum of q exceeds w * Z.  If Z is 0 the draw uses p_theta.
    With every draft accepted there is no draw (-1).

Everything is float64; bfloat16 logits are widened exactly.
"""

from __future__ import annotations

import numpy as np

from .widen import widen


def softmax_t(x: np.ndarray, temperature: float) -> np.ndarray:
    """softmax(x / T) of one float64 row."""
    z = x / temperature
    e = np.exp(z - z.max())
    return e / e.sum()


def accept_draft(u: float, p_target: float, p_draft: float) -> bool:
    """u * p_phi(D) < p_theta(D): probability min(1, p_theta / p_phi) for u ~ U[0, 1)."""
    return u * p_draft < p_target


def residual(pt: np.ndarray, pd: np.ndarray):
    """The residual weights max(0, p_theta - p_phi), or p_theta where they sum to 0;
    returns (weights, used_target)."""
    q = np.maximum(pt - pd, 0.0)
    if q.sum() > 0.0:
        return q, False
    return pt.copy(), True


def draw(q: np.ndarray, w: float) -> int:
    """Smallest x with sum_{y <= x} q(y) > w * sum(q) (inverse CDF, index order)."""
    c = np.cumsum(q)
    hit = np.flatnonzero(c > w * c[-1])
    return int(hit[0]) if hit.size else int(np.flatnonzero(q > 0)[-1])


def rows_of_steps(step_row: np.ndarray, gamma: int):
    """k_r for r = 1..gamma: the block slot whose step is r."""
    return [int(np.flatnonzero(step_row == r + 1)[0]) for r in range(gamma)]


def residual_row(logits_row, draft_row, temperature: float, dtype: str):
    """(weights, used_target) of the residual of one (target row, draft row) pair."""
    pt = softmax_t(widen(logits_row, dtype), temperature)
    pd = softmax_t(widen(draft_row, dtype), temperature)
    return residual(pt, pd)


def verify_accept_sampled(logits, draft_logits, draft_ids, step_map, num_ref, uniforms,
                          temperature: float, dtype: str):
    """Returns p_target float64 [b, L], p_draft float64 [b, L], accept_len int32 [b]
    and correction int32 [b] (-1 when every draft was accepted).

    logits [b, B, V] and draft_logits [b, L, V] are in `dtype` ("f32" or "bf16"
    bit patterns); uniforms [b, L + 1] float."""
    logits = np.asarray(logits)
    b, B, V = logits.shape
    L = draft_ids.shape[1]
    p_target = np.zeros((b, L))
    p_draft = np.zeros((b, L))
    accept_len = np.zeros((b,), np.int32)
    correction = np.full((b,), -1, np.int32)
    for s in range(b):
        gamma = int(num_ref[s])
        rows = rows_of_steps(step_map[s], gamma)
        dists = []
        for r in range(gamma):
            pt = softmax_t(widen(logits[s, rows[r]], dtype), temperature)
            pd = softmax_t(widen(draft_logits[s, r], dtype), temperature)
            tok = int(draft_ids[s, r])
            if 0 <= tok < V:
                p_target[s, r] = pt[tok]
                p_draft[s, r] = pd[tok]
            dists.append((pt, pd, 0 <= tok < V))
        a = 0
        while a < gamma:
            pt, pd, ok = dists[a]
            if not (ok and accept_draft(float(uniforms[s, a]), p_target[s, a], p_draft[s, a])):
                break
            a += 1
        accept_len[s] = a
        if a < gamma:
            pt, pd, _ = dists[a]
            q, _ = residual(pt, pd)
            correction[s] = draw(q, float(uniforms[s, L]))
    return p_target, p_draft, accept_len, correction
