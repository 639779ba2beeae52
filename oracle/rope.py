"""Rotary position embedding with the RoPE-copy positions (oracle; test
infrastructure only).

Sec. 3.1 (RoPE copy): a data position and its paired mask position refer to
the same response position, so the mask position reuses the RoPE index of its
data position while prompt and data tokens keep their own absolute indices;
Sec. 3.2 applies the same alignment between each drafted token and its
verification slot.  Readings (the paper gives the rule, not these details):

  * Block slot k of sequence b (the mask section) stands for response position
    k of the block: index prefix_len + k.  Reference slot r holds draft r+1,
    the token proposed for block slot k_{r+1} (the slot whose step is r+1), so
    it carries that position's index, prefix_len + k_{r+1}, which its
    verification slot shares.  Padding reference slots (r >= gamma) take
    prefix_len; they see and are seen by nothing.
  * The rotary embedding of the SDAR (Qwen-family) models: dims i and
    i + d/2 form a pair rotated by the angle pos * theta^(-2i/d).
  * The cached prefix keys are stored already rotated at indices
    0..prefix_len-1; q and the new keys arrive unrotated.
"""

from __future__ import annotations

import numpy as np


def positions(step_row: np.ndarray, gamma: int, L: int, prefix_len: int) -> np.ndarray:
    """RoPE indices of the B + L new slots of one sequence."""
    B = len(step_row)
    pos = np.full(B + L, prefix_len, np.int64)
    pos[:B] = prefix_len + np.arange(B)
    for r in range(gamma):
        k = int(np.flatnonzero(step_row == r + 1)[0])
        pos[B + r] = prefix_len + k
    return pos


def inv_freq(d: int, theta: float) -> np.ndarray:
    """theta^(-2i/d) for i = 0..d/2-1."""
    return theta ** (-2.0 * np.arange(d // 2) / d)


def rotate(x: np.ndarray, pos: np.ndarray, theta: float) -> np.ndarray:
    """Rotate rows x [n, d] (float64) by their positions pos [n]."""
    d = x.shape[-1]
    ang = pos.astype(np.float64)[:, None] * inv_freq(d, theta)[None, :]
    c, s = np.cos(ang), np.sin(ang)
    lo, hi = x[:, : d // 2], x[:, d // 2:]
    return np.concatenate([lo * c - hi * s, hi * c + lo * s], axis=1)
