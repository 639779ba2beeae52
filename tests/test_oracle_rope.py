"""Pins of the oracle's rotary embedding and RoPE-copy positions.

* The rotation against a complex-number statement of it: pair (x_i, x_{i+d/2})
  as z_i = x_i + i x_{i+d/2}, multiplied by exp(i pos theta^(-2i/d)).
* Scores depend only on position differences; norms are kept; position 0 is
  the identity.
* Hand-worked RoPE-copy positions (block slots at their own index, reference
  slots at their verification slot's index, padding slots at the prefix).
* Attention with rope_theta equals attention on inputs rotated here with the
  complex form (prefix keys untouched), and a verification slot sees its own
  draft's key at relative position 0.
"""

import numpy as np
import pytest

import oracle
from oracle import rope
from synth import VerifyConfig, generate


def complex_rotate(x, pos, theta):
    d = x.shape[1]
    h = d // 2
    z = x[:, :h] + 1j * x[:, h:]
    w = np.exp(1j * np.outer(pos, theta ** (-np.arange(0, d, 2) / d)))
    r = z * w
    return np.concatenate([r.real, r.imag], axis=1)


@pytest.mark.parametrize("d,theta", [(2, 10000.0), (8, 10000.0), (64, 1e6), (128, 1e6)])
def test_rotation_matches_complex_form(d, theta):
    rng = np.random.default_rng(d)
    x = rng.standard_normal((7, d))
    pos = np.array([0, 1, 5, 100, 4097, 32767, 32800])
    np.testing.assert_allclose(rope.rotate(x, pos, theta), complex_rotate(x, pos, theta),
                               rtol=0, atol=1e-9)
    # d = 2: one pair rotated by pos radians
    if d == 2:
        got = rope.rotate(np.array([[1.0, 0.0]]), np.array([np.pi / 2]) * 0 + 1, theta)
        np.testing.assert_allclose(got, [[np.cos(1.0), np.sin(1.0)]], atol=1e-15)


def test_relative_positions_norms_identity():
    rng = np.random.default_rng(1)
    d, theta = 64, 1e6
    q, k = rng.standard_normal((1, d)), rng.standard_normal((1, d))
    base = (rope.rotate(q, np.array([40]), theta) @ rope.rotate(k, np.array([13]), theta).T).item()
    for c in (1, 77, 30000):
        s = (rope.rotate(q, np.array([40 + c]), theta) @ rope.rotate(k, np.array([13 + c]), theta).T).item()
        assert abs(s - base) < 1e-9 * max(1.0, abs(base))
    x = rng.standard_normal((5, d))
    pos = np.array([0, 3, 9, 1000, 20000])
    np.testing.assert_allclose(np.linalg.norm(rope.rotate(x, pos, theta), axis=1),
                               np.linalg.norm(x, axis=1), rtol=1e-12)
    np.testing.assert_allclose(rope.rotate(x, np.zeros(5, int), theta), x, atol=0)


def test_copy_positions_hand_example():
    # B = 4, step map (2, 0, 1, 5): draft 1 at slot 2, draft 2 at slot 0,
    # slot 1 committed, slot 3 not drafted; gamma = 2, L = 3, prefix 10.
    pos = rope.positions(np.array([2, 0, 1, 5]), 2, 3, 10)
    assert list(pos) == [10, 11, 12, 13, 12, 10, 10]


def _rope_inputs(seed, paged=0):
    cfg = VerifyConfig(0, "rope", "f32", batch=3, num_q_heads=4, num_kv_heads=2, head_dim=16,
                       prefix=(0, 9), block_size=5, max_ref=4, vocab=64, page_size=paged,
                       step_mode="mixed")
    return generate(cfg, seed=seed)


@pytest.mark.parametrize("seed,paged", [(3, 0), (4, 4)])
def test_attention_with_rope_equals_prerotated_inputs(seed, paged):
    theta = 500.0
    inp = _rope_inputs(seed, paged)
    got_o, got_l = oracle.verify_attention(inp, rope_theta=theta)
    cfg = inp.cfg
    q = inp.q.astype(np.float64).copy()
    kn = inp.k_new.astype(np.float64).copy()
    for s in range(cfg.batch):
        pos = rope.positions(inp.step_map[s], int(inp.num_ref[s]), cfg.max_ref, int(inp.prefix_lens[s]))
        for h in range(cfg.num_q_heads):
            q[s, :, h] = complex_rotate(q[s, :, h], pos, theta)
        for h in range(cfg.num_kv_heads):
            kn[s, :, h] = complex_rotate(kn[s, :, h], pos, theta)
    inp.q, inp.k_new = q, kn
    want_o, want_l = oracle.verify_attention(inp)
    # (the "f32" inputs are read through float32, so the pre-rotated copies
    # lose about 1e-7 relative)
    np.testing.assert_allclose(got_o, want_o, rtol=0, atol=1e-6)
    np.testing.assert_allclose(got_l, want_l, rtol=0, atol=1e-6)


def test_verification_slot_sees_its_draft_at_distance_zero():
    """With q of a verification slot equal to k of its draft's reference slot,
    their score is |q|^2 under RoPE copy (same index), not under physical
    indices."""
    theta, d = 100.0, 8
    rng = np.random.default_rng(2)
    v = rng.standard_normal((1, d))
    step = np.array([0, 1, 2])                 # slot 1 verifies draft 1, slot 2 draft 2
    pos = rope.positions(step, 2, 2, 50)
    k_slot, r_slot = 1, 3 + 0                  # draft 1 sits in reference slot 0
    s = (rope.rotate(v, pos[[k_slot]], theta) @ rope.rotate(v, pos[[r_slot]], theta).T).item()
    assert abs(s - (v @ v.T).item()) < 1e-12
    phys = np.arange(5) + 50
    s2 = (rope.rotate(v, phys[[k_slot]], theta) @ rope.rotate(v, phys[[r_slot]], theta).T).item()
    assert abs(s2 - (v @ v.T).item()) > 1e-3
