"""Brute-force statement of the verification attention, for pinning the oracle.

Built from the paper's prose, not from eq. 1: every verification row sees the
prompt plus *one version of every block position*, namely the version that
position has in the block's state at that row's step (Sec. 3.1, "Masked Token
Prediction"; Sec. 3.2, "Target Model Verification"):

  * a prediction (mask) row of step t sees the data version of positions decoded
    before t and the mask placeholder of every other position;
  * a data row of step t sees the data version of positions decoded at or
    before t (itself included) and placeholders for the rest.

The data version of the r-th drafted position is reference slot B + r - 1; its
placeholder is its block slot.  A committed position (step 0) has only its block
slot, which holds the decoded token; an undrafted position stays a placeholder
and its row is evaluated after every draft.  Padding is dropped.

Each row then runs its own attention over that explicit key list, one row at a
time, with ``math.fsum`` sums.  Nothing here is shared with ``oracle``.
"""

from __future__ import annotations

import math

import numpy as np


def _f64(a, dtype):
    if dtype == "f32":
        return np.asarray(a, np.float32).astype(np.float64)
    return (np.asarray(a, np.uint16).astype(np.uint32) << np.uint32(16)).view(
        np.float32).astype(np.float64)


def row_context(step_row, gamma, L, row):
    """Indices into the new slots that new row ``row`` sees (or None if padding)."""
    B = len(step_row)
    INF = 10 ** 9

    def decoded_at(p):              # step at which block position p becomes data
        s = int(step_row[p])
        return 0 if s == 0 else (s if 1 <= s <= gamma else INF)

    if row < B:
        s = int(step_row[row])
        if s < 0:
            return None
        kind, t = "mask", (0 if s == 0 else (s if s <= gamma else gamma + 1))
    else:
        r = row - B
        if r >= gamma:
            return None
        kind, t = "data", r + 1
    ctx = []
    for p in range(B):
        s = int(step_row[p])
        if s < 0:
            continue                                  # padding position
        known = decoded_at(p) < t if kind == "mask" else decoded_at(p) <= t
        if s == 0 or not known:
            ctx.append(p)                             # block slot (token or [MASK])
        else:
            ctx.append(B + s - 1)                     # reference slot of draft s
    return ctx


def brute_attention(inp, scale=None):
    """float64 out [b, B+L, Hq, d] and lse [b, Hq, B+L], one row at a time."""
    cfg = inp.cfg
    dt = cfg.dtype
    b, Hq, G, d, B, L = (cfg.batch, cfg.num_q_heads, cfg.group, cfg.head_dim,
                         cfg.block_size, cfg.max_ref)
    sc = scale or 1.0 / math.sqrt(d)
    out = np.zeros((b, B + L, Hq, d))
    lse = np.full((b, Hq, B + L), -math.inf)
    for s in range(b):
        gamma = int(inp.num_ref[s])
        n = int(inp.prefix_lens[s])
        for row in range(B + L):
            ctx = row_context(inp.step_map[s], gamma, L, row)
            if ctx is None:
                continue
            for h in range(Hq):
                kvh = h // G
                keys, vals = [], []
                for t in range(n):
                    if inp.block_table is None:
                        keys.append(_f64(inp.k_cache[s, t, kvh], dt))
                        vals.append(_f64(inp.v_cache[s, t, kvh], dt))
                    else:
                        P = inp.k_cache.shape[1]
                        pg = int(inp.block_table[s, t // P])
                        keys.append(_f64(inp.k_cache[pg, t % P, kvh], dt))
                        vals.append(_f64(inp.v_cache[pg, t % P, kvh], dt))
                for j in ctx:
                    keys.append(_f64(inp.k_new[s, j, kvh], dt))
                    vals.append(_f64(inp.v_new[s, j, kvh], dt))
                qv = _f64(inp.q[s, row, h], dt)
                scores = [sc * math.fsum(qv * kv) for kv in keys]
                top = max(scores)
                w = [math.exp(x - top) for x in scores]
                z = math.fsum(w)
                out[s, row, h] = [math.fsum(wi * vv[c] for wi, vv in zip(w, vals)) / z
                                  for c in range(d)]
                lse[s, h, row] = top + math.log(z)
    return out, lse
