"""Pins of the oracle's greedy acceptance (temperature-0 form of eq. 2).

Hand-worked rows, scipy's softmax for the probabilities, lowest-index ties
(including -0.0 == +0.0), out-of-range drafts, constant rows, gamma = 0 and the
generator's planted drafts."""

import numpy as np
import pytest
from scipy.special import softmax

import oracle
from synth import VerifyConfig, generate, bf16_bits_from_f32


def check_hand_example():
    # V = 6, B = 3, gamma = 3, step map (2, 3, 1): draft 1 is verified by row 2,
    # draft 2 by row 0, draft 3 by row 1.
    logits = np.array([[[0.5, 3.0, -1.0, 3.0, 2.0, 0.0],      # row 0: max 3.0 at 1 and 3
                        [1.0, 1.0, 1.0, 1.0, 1.0, 1.0],       # row 1: constant
                        [-2.0, -1.0, 4.0, 0.0, 4.0, -3.0]]],  # row 2: max 4.0 at 2 and 4
                      np.float32)
    step = np.array([[2, 3, 1]], np.int32)
    for drafts, want_len in (([2, 1, 0], 3),    # all three equal the lowest-index maxima
                             ([2, 3, 0], 1),    # draft 2 is a tied maximum but not the lowest
                             ([4, 1, 0], 0),    # draft 1 rejected at once
                             ([2, 1, 5], 2)):
        t, c, p, a = oracle.verify_accept(logits, np.array([drafts], np.int32), step,
                                          np.array([3]), "f32")
        assert list(t[0]) == [1, 0, 2]
        assert a[0] == want_len, (drafts, a[0])
        sm = softmax(logits[0].astype(np.float64), axis=-1)
        np.testing.assert_allclose(c[0], sm.max(-1), rtol=1e-14)
        rows = [2, 0, 1]
        np.testing.assert_allclose(p[0], [sm[rows[r], drafts[r]] for r in range(3)], rtol=1e-14)
    np.testing.assert_allclose(c[0, 1], 1 / 6, rtol=1e-14)


def check_signed_zero_tie():
    x = np.full((1, 1, 5), -1.0, np.float32)
    x[0, 0, 1] = -0.0
    x[0, 0, 3] = 0.0
    t, _, _, a = oracle.verify_accept(x, np.array([[3]]), np.array([[1]]), np.array([1]), "f32")
    assert t[0, 0] == 1 and a[0] == 0


def check_out_of_range_and_unscanned():
    rng = np.random.default_rng(0)
    x = rng.standard_normal((1, 4, 9)).astype(np.float32)
    step = np.array([[1, 0, -1, 2]], np.int32)
    am = int(np.argmax(x[0, 0]))
    t, c, p, a = oracle.verify_accept(x, np.array([[am, 9, -1]]), step, np.array([2]), "f32")
    assert a[0] == 1 and p[0, 1] == 0 and p[0, 2] == 0
    assert t[0, 1] == -1 and t[0, 2] == -1 and c[0, 1] == 0 and c[0, 2] == 0
    assert t[0, 3] == int(np.argmax(x[0, 3]))


def check_zero_gamma():
    x = np.zeros((2, 3, 4), np.float32)
    t, c, p, a = oracle.verify_accept(x, np.full((2, 3), -1), np.array([[4, 4, 0], [0, 0, 0]]),
                                      np.array([0, 0]), "f32")
    assert list(a) == [0, 0]
    assert list(t[0]) == [0, 0, -1] and np.allclose(c[0, :2], 0.25)


def check_bf16_widening():
    bits = np.array([0x3F80, 0xC000, 0x3FC0, 0x0000, 0x8000, 0x4149], np.uint16)
    np.testing.assert_array_equal(oracle.widen(bits, "bf16"),
                                  [1.0, -2.0, 1.5, 0.0, -0.0, 12.5625])
    np.testing.assert_array_equal(bf16_bits_from_f32(np.array([1.0, 1.00390625, 1.01171875],
                                                              np.float32)),
                                  [0x3F80, 0x3F80, 0x3F82])   # ties to even


def check_planted_drafts_match():
    cfg = VerifyConfig(0, "acc-test", "bf16", batch=4, num_q_heads=2, num_kv_heads=1,
                       head_dim=8, prefix=1, block_size=6, max_ref=6, vocab=3001, plant=0.8)
    inp = generate(cfg, seed=4)
    t, c, p, a = oracle.verify_accept(inp.logits, inp.draft_ids, inp.step_map, inp.num_ref,
                                      "bf16")
    for s in range(cfg.batch):
        for r in range(int(inp.num_ref[s])):
            row = int(np.flatnonzero(inp.step_map[s] == r + 1)[0])
            if inp.planted[s, r]:
                assert t[s, row] == inp.draft_ids[s, r]
        n = 0
        while n < inp.num_ref[s] and inp.planted[s, n]:
            n += 1
        assert a[s] >= n


PINS = [check_hand_example, check_signed_zero_tie, check_out_of_range_and_unscanned,
        check_zero_gamma, check_bf16_widening, check_planted_drafts_match]


def all_pins_pass():
    try:
        for f in PINS:
            f()
    except AssertionError:
        return False
    return True


@pytest.mark.parametrize("pin", PINS, ids=lambda f: f.__name__)
def test_accept_pin(pin):
    pin()
