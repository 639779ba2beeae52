"""Slot labels and the temporal attention mask (oracle; test infrastructure only).

Follows Sec. 3.1 ("Input Layout Prepare", "Temporal Attention Mask") and the
verification layout of Sec. 3.2 ("Target Model Verification").

New slots of one sequence, in storage order:
  block slots     k = 0..B-1   the mask section (prediction / verification slots)
  reference slots B + r, r = 0..L-1   the data section; slot r holds the r-th
                  drafted token, so its temporal label is r + 1.

Readings where the paper is silent (each listed with its reason in the design
notes of the repository):
  * step_map[k] == 0: a block position committed before this step.  It behaves
    like the prompt (label 0): visible to every non-padded row.
  * step_map[k] > gamma: a block position not drafted in this step; it stays a
    mask placeholder at every draft step, i.e. label gamma + 1.
  * step_map[k] < 0, and reference slots r >= gamma: padding.  Padding rows see
    nothing and padding columns are seen by no row.
  * Self-visibility follows eq. 1 literally (<= and >=): every slot sees itself.
"""

from __future__ import annotations

import numpy as np

MASK = 0    # block slot: prediction position (the paper's D-tilde section)
DATA = 1    # reference slot: drafted token (the paper's D section)


def slot_labels(step_row, gamma: int, L: int):
    """Section, temporal label and validity of the B + L new slots of one sequence.

    Returns (section, tau, valid): int arrays section/tau and a bool array valid,
    each of length B + L.  Labels follow Sec. 3.2: the data slot of the r-th
    draft and its paired verification slot share tau = r.
    """
    step_row = np.asarray(step_row, np.int64)
    B = step_row.shape[0]
    n = B + L
    section = np.empty(n, np.int64)
    tau = np.empty(n, np.int64)
    valid = np.empty(n, bool)
    for k in range(B):
        section[k] = MASK
        t = int(step_row[k])
        if t < 0:
            valid[k], tau[k] = False, -1
        else:
            valid[k], tau[k] = True, min(t, gamma + 1)
    for r in range(L):
        section[B + r] = DATA
        tau[B + r] = r + 1
        valid[B + r] = r < gamma
    return section, tau, valid


def visible(sec_i: int, tau_i: int, sec_j: int, tau_j: int) -> bool:
    """Eq. 1 for two non-padded new slots i (query) and j (key)."""
    if sec_j == MASK and tau_j == 0:
        return True                      # committed: visible like the prompt
    if sec_i == DATA and sec_j == DATA:
        return tau_j <= tau_i            # case 1
    if sec_i == DATA and sec_j == MASK:
        return tau_j > tau_i             # case 2
    if sec_i == MASK and sec_j == DATA:
        return tau_j < tau_i             # case 3
    return tau_j >= tau_i                # case 4: both in the mask section


def new_slot_visibility(step_row, gamma: int, L: int) -> np.ndarray:
    """Dense bool matrix A[i, j] over the B + L new slots of one sequence."""
    section, tau, valid = slot_labels(step_row, gamma, L)
    n = len(section)
    A = np.zeros((n, n), bool)
    for i in range(n):
        if not valid[i]:
            continue                     # padding row: zeroed
        for j in range(n):
            if valid[j]:
                A[i, j] = visible(section[i], tau[i], section[j], tau[j])
    return A


def row_valid(step_row, gamma: int, L: int) -> np.ndarray:
    """Non-padded rows; only these see the prompt (the cached prefix)."""
    return slot_labels(step_row, gamma, L)[2]
