"""Pins of the oracle's stochastic acceptance (eq. 2 at temperature T).

* The speculative-sampling identity: a draft sampled from p_phi, accepted with
  probability min(1, p_theta/p_phi) and otherwise replaced by a draw from the
  residual, is distributed as p_theta (Monte Carlo, first and second draft).
* Hand-worked three-token rows (acceptance thresholds, a residual with one
  token, the p_theta fallback when the residual is empty).
* Probabilities against scipy's softmax at the given temperature.
* The temperature -> 0 limit against the greedy oracle.
"""

import numpy as np
import pytest
from scipy.special import softmax

import oracle
from oracle import sampled as osmp


def run(logits, draft_logits, drafts, step, gamma, uniforms, T=1.0):
    return osmp.verify_accept_sampled(np.asarray(logits, np.float32),
                                      np.asarray(draft_logits, np.float32),
                                      np.asarray(drafts, np.int32), np.asarray(step, np.int32),
                                      np.asarray(gamma), np.asarray(uniforms, np.float64), T, "f32")


def output_frequencies(pt_logits, pd_logits, T, n, seed, position=1):
    """Empirical distribution of the token the step commits at draft `position`
    (1 or 2), with drafts sampled from p_phi by numpy and uniforms drawn here."""
    rng = np.random.default_rng(seed)
    V = len(pt_logits[0])
    B = L = 2
    pd = [softmax(np.asarray(x, np.float64) / T) for x in pd_logits]
    drafts = np.stack([rng.choice(V, size=n, p=pd[0]), rng.choice(V, size=n, p=pd[1])], 1)
    # Block slot 0 verifies draft 2, slot 1 draft 1.
    logits = np.broadcast_to(np.array([pt_logits[1], pt_logits[0]], np.float32), (n, B, V))
    dlog = np.broadcast_to(np.array(pd_logits, np.float32), (n, L, V))
    step = np.broadcast_to(np.array([2, 1], np.int32), (n, B))
    u = rng.random((n, L + 1))
    _, _, a, c = run(logits, dlog, drafts, step, np.full(n, 2), u, T)
    if position == 1:
        tok = np.where(a >= 1, drafts[:, 0], c)
    else:
        assert np.all(a >= 1)
        tok = np.where(a >= 2, drafts[:, 1], c)
    return np.bincount(tok, minlength=V) / n


@pytest.mark.parametrize("T", [1.0, 0.6])
def test_first_draft_output_is_target_distribution(T):
    pt = [1.5, -0.5, 0.3, 2.0, -1.0]
    pd = [-0.2, 1.8, 0.9, 0.1, 1.0]           # far from p_theta: many rejections
    n = 20000
    freq = output_frequencies([pt, pt], [pd, pd], T, n, seed=7)
    want = softmax(np.array(pt) / T)
    sigma = np.sqrt(want * (1 - want) / n)
    assert np.all(np.abs(freq - want) < 5 * sigma + 1e-12), (freq, want)
    # The drafts alone are far from p_theta, so the check has teeth.
    assert np.max(np.abs(softmax(np.array(pd) / T) - want)) > 20 * sigma.max()


def test_second_draft_output_is_its_target_distribution():
    pt2 = [0.0, 2.0, -1.0, 0.5, 1.0]
    pd2 = [1.0, -1.0, 1.5, 0.0, -0.5]
    same = [0.3, 0.1, -0.4, 0.9, 0.0]          # draft 1: p_phi == p_theta, always accepted
    n = 20000
    freq = output_frequencies([same, pt2], [same, pd2], 1.0, n, seed=11, position=2)
    want = softmax(np.array(pt2))
    sigma = np.sqrt(want * (1 - want) / n)
    assert np.all(np.abs(freq - want) < 5 * sigma + 1e-12), (freq, want)


def test_hand_example():
    # p_theta = (1, 2, 3)/6, p_phi = (3, 2, 1)/6 at T = 1.
    pt = np.log([1.0, 2.0, 3.0])
    pd = np.log([3.0, 2.0, 1.0])
    one = lambda d, u, w: run([[pt]], [[pd]], [[d]], [[1]], [1], [[u, w]])
    # Draft 0: alpha = (1/6)/(3/6) = 1/3.
    p_t, p_d, a, c = one(0, 0.30, 0.9)
    np.testing.assert_allclose([p_t[0, 0], p_d[0, 0]], [1 / 6, 3 / 6], rtol=1e-6)
    assert a[0] == 1 and c[0] == -1
    _, _, a, c = one(0, 0.34, 0.0)
    # Residual max(0, p_theta - p_phi) = (0, 0, 2/6): the correction is token 2.
    assert a[0] == 0 and c[0] == 2
    _, _, a, c = one(0, 0.99, 0.999)
    assert a[0] == 0 and c[0] == 2
    # Draft 2: alpha = min(1, 3) = 1, accepted for every u < 1.
    for u in (0.0, 0.5, 0.999999):
        assert one(2, u, 0.5)[2][0] == 1
    # Draft 1: alpha = 1 (equal probabilities).
    assert one(1, 0.999999, 0.5)[2][0] == 1


def test_empty_residual_draws_from_target():
    # p_phi == p_theta and an out-of-range draft: rejected, residual all zero,
    # the draw uses p_theta = (1, 2, 3)/6 with cumulative (1/6, 1/2, 1).
    pt = np.log([1.0, 2.0, 3.0])
    for w, want in ((0.0, 0), (0.16, 0), (0.2, 1), (0.49, 1), (0.51, 2), (0.999, 2)):
        _, p_d, a, c = run([[pt]], [[pt]], [[7]], [[1]], [1], [[0.0, w]])
        assert a[0] == 0 and c[0] == want and p_d[0, 0] == 0, (w, c[0])


def test_probabilities_match_softmax_and_gamma_zero():
    rng = np.random.default_rng(3)
    b, B, L, V = 3, 4, 3, 11
    logits = rng.normal(0, 2, (b, B, V)).astype(np.float32)
    dlog = rng.normal(0, 2, (b, L, V)).astype(np.float32)
    step = np.array([[2, 0, 1, 3], [1, 2, -1, 0], [4, 4, 4, 4]], np.int32)
    gamma = np.array([3, 2, 0])
    drafts = rng.integers(0, V, (b, L)).astype(np.int32)
    u = rng.random((b, L + 1))
    T = 0.7
    p_t, p_d, a, c = run(logits, dlog, drafts, step, gamma, u, T)
    for s in range(b):
        for r in range(gamma[s]):
            k = int(np.flatnonzero(step[s] == r + 1)[0])
            np.testing.assert_allclose(p_t[s, r], softmax(logits[s, k].astype(np.float64) / T)[drafts[s, r]], rtol=1e-12)
            np.testing.assert_allclose(p_d[s, r], softmax(dlog[s, r].astype(np.float64) / T)[drafts[s, r]], rtol=1e-12)
    assert a[2] == 0 and c[2] == -1 and np.all(p_t[2] == 0)


def test_small_temperature_is_greedy():
    """At T -> 0 both distributions are one-hot: with drafts at the draft rows'
    argmax the sampled rule accepts exactly where the greedy rule does, and the
    correction is the target's argmax at the first rejected row."""
    rng = np.random.default_rng(5)
    b, B, L, V = 40, 4, 4, 9
    logits = rng.normal(0, 3, (b, B, V)).astype(np.float32)
    dlog = rng.normal(0, 3, (b, L, V)).astype(np.float32)
    step = np.array([rng.permutation(B) + 1 for _ in range(b)], np.int32)
    gamma = np.full(b, L)
    # Agree with the target argmax on about half the drafts.
    for s in range(b):
        for r in range(L):
            if rng.random() < 0.6:
                k = int(np.flatnonzero(step[s] == r + 1)[0])
                dlog[s, r] = logits[s, k] + rng.normal(0, 0.01, V).astype(np.float32)
    drafts = dlog.argmax(-1).astype(np.int32)
    u = rng.random((b, L + 1))
    _, _, a, c = run(logits, dlog, drafts, step, gamma, u, T=1e-6)
    t, _, _, ga = oracle.verify_accept(logits, drafts, step, gamma, "f32")
    np.testing.assert_array_equal(a, ga)
    for s in range(b):
        if ga[s] < L:
            k = int(np.flatnonzero(step[s] == ga[s] + 1)[0])
            assert c[s] == t[s, k]
        else:
            assert c[s] == -1
    assert 0 < np.mean(ga) < L                 # both outcomes occur
