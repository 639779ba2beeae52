"""Pins of the LM-head oracle: the logits are the plain product hidden . weight^T.

* A hand-worked 2-dim head over 3 tokens.
* Element sums with math.fsum on small random shapes, bf16 and f32 (and the
  chunked product across the 8192-token chunk boundary).
* The acceptance on top is the greedy oracle (pinned in test_oracle_accept).
"""

import math

import numpy as np

import oracle
from synth import bf16_bits_from_f32


def test_hand_example():
    hidden = np.array([[[1.0, 2.0], [0.0, -1.0]]], np.float32)          # b=1, B=2, H=2
    weight = np.array([[1.0, 0.0], [0.5, 0.5], [-1.0, 3.0]], np.float32)  # V=3
    lg = oracle.lmhead_logits(hidden, weight, "f32")
    np.testing.assert_array_equal(lg[0], [[1.0, 1.5, 5.0], [0.0, -0.5, -3.0]])
    t, c, p, a, _ = oracle.verify_accept_lmhead(hidden, weight, np.array([[2, 0]]),
                                                np.array([[1, 2]]), np.array([2]), "f32")
    assert list(t[0]) == [2, 0] and a[0] == 2


def test_logits_against_element_sums():
    rng = np.random.default_rng(0)
    for dt, V in (("f32", 37), ("bf16", 8200)):
        b, B, H = 2, 3, 24
        h = rng.standard_normal((b, B, H)).astype(np.float32)
        w = rng.standard_normal((V, H)).astype(np.float32)
        if dt == "bf16":
            h, w = bf16_bits_from_f32(h), bf16_bits_from_f32(w)
        lg = oracle.lmhead_logits(h, w, dt)
        hf = oracle.widen(h, dt)
        wf = oracle.widen(w, dt)
        for s in range(b):
            for k in range(B):
                for v in (0, 1, V // 2, 8191 if V > 8192 else V - 2, V - 1):
                    want = math.fsum(hf[s, k, i] * wf[v, i] for i in range(H))
                    assert abs(lg[s, k, v] - want) <= 1e-12 * max(1.0, abs(want))
