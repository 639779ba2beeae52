"""Verification attention (oracle; test infrastructure only).

Sec. 3.2 ("Target Model Verification"): one target forward pass scores every
drafted token at once; inside each attention layer every new row attends to the
cached prompt prefix (visible to all response rows, Sec. 3.1) and to the new
slots allowed by eq. 1.  With the KV cache the prefix keys and values are reused
and only the new slots are computed (Sec. 3.3, "Adaptation under Blockwise
Decoding and KV Cache").

Grouped-query attention maps query head h to KV head h // (Hq // Hkv).
Scores are scale * q.k with scale = 1/sqrt(d) unless given.  A padded row has no
visible key: its output is 0 and its log-sum-exp is -inf.  With rope_theta > 0
the new slots' queries and keys are rotated first, at the RoPE-copy positions
of ``rope.positions`` (the cached prefix keys arrive rotated).
"""

from __future__ import annotations

import math
from typing import Iterable, Optional, Tuple

import numpy as np

from .mask import new_slot_visibility, row_valid
from .rope import positions, rotate
from .widen import widen


def attend(q: np.ndarray, k: np.ndarray, v: np.ndarray, vis: np.ndarray, scale: float):
    """Masked softmax attention, written out.

    q [R, d], k [N, d], v [N, d], vis bool [R, N].
    Returns out [R, d] and lse [R] (natural log of sum_j exp(s_j) over visible j).
    """
    R = q.shape[0]
    out = np.zeros((R, v.shape[1]), np.float64)
    lse = np.full((R,), -np.inf, np.float64)
    s = scale * (q @ k.T)
    for i in range(R):
        cols = np.flatnonzero(vis[i])
        if cols.size == 0:
            continue
        si = s[i, cols]
        m = si.max()
        p = np.exp(si - m)
        l = p.sum()
        out[i] = (p @ v[cols]) / l
        lse[i] = m + math.log(l)
    return out, lse


def prefix_kv(inp, b: int, kvh: int) -> Tuple[np.ndarray, np.ndarray]:
    """The cached prefix keys/values of sequence b, KV head kvh, in token order."""
    dt = inp.cfg.dtype
    n = int(inp.prefix_lens[b])
    if inp.block_table is None:
        kc = inp.k_cache[b, :n, kvh]
        vc = inp.v_cache[b, :n, kvh]
    else:
        P = inp.k_cache.shape[1]
        t = np.arange(n)
        pages = inp.block_table[b, t // P]
        kc = inp.k_cache[pages, t % P, kvh]
        vc = inp.v_cache[pages, t % P, kvh]
    return widen(kc, dt), widen(vc, dt)


def pair_attention(inp, b: int, kvh: int, scale: Optional[float] = None, rope_theta: float = 0.0):
    """All rows of the G query heads sharing KV head kvh in sequence b.

    Returns out [n_new, G, d] and lse [G, n_new].
    """
    cfg = inp.cfg
    dt = cfg.dtype
    G, d, L = cfg.group, cfg.head_dim, cfg.max_ref
    sc = 1.0 / math.sqrt(d) if not scale else float(scale)
    gamma = int(inp.num_ref[b])
    A = new_slot_visibility(inp.step_map[b], gamma, L)
    valid = row_valid(inp.step_map[b], gamma, L)
    kp, vp = prefix_kv(inp, b, kvh)
    kn = widen(inp.k_new[b, :, kvh], dt)
    pos = positions(inp.step_map[b], gamma, L, int(inp.prefix_lens[b]))
    if rope_theta:
        kn = rotate(kn, pos, rope_theta)
    keys = np.concatenate([kp, kn], axis=0)
    vals = np.concatenate([vp, widen(inp.v_new[b, :, kvh], dt)], axis=0)
    n_new = A.shape[0]
    vis = np.concatenate([np.repeat(valid[:, None], kp.shape[0], axis=1), A], axis=1)
    out = np.zeros((n_new, G, d))
    lse = np.zeros((G, n_new))
    for g in range(G):
        h = kvh * G + g
        qh = widen(inp.q[b, :, h], dt)
        if rope_theta:
            qh = rotate(qh, pos, rope_theta)
        o, l = attend(qh, keys, vals, vis, sc)
        out[:, g] = o
        lse[g] = l
    return out, lse


def verify_attention(inp, scale: Optional[float] = None,
                     pairs: Optional[Iterable[Tuple[int, int]]] = None, rope_theta: float = 0.0):
    """Outputs of the verification attention.

    Returns out [batch, B+L, Hq, d] and lse [batch, Hq, B+L] (float64).  With
    ``pairs`` only those (sequence, KV head) pairs are computed; the other
    entries are NaN.
    """
    cfg = inp.cfg
    b, Hq, Hkv, G, n_new, d = (cfg.batch, cfg.num_q_heads, cfg.num_kv_heads, cfg.group,
                              cfg.n_new, cfg.head_dim)
    out = np.full((b, n_new, Hq, d), np.nan)
    lse = np.full((b, Hq, n_new), np.nan)
    todo = pairs if pairs is not None else [(s, h) for s in range(b) for h in range(Hkv)]
    for s, kvh in todo:
        o, l = pair_attention(inp, s, kvh, scale, rope_theta)
        out[s, :, kvh * G:(kvh + 1) * G] = o
        lse[s, kvh * G:(kvh + 1) * G] = l
    return out, lse
