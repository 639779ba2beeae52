"""The pins must bite: plant a plausible mistake in the oracle (on the CPU, via
monkeypatching) and check that the golden masks or the brute force reject it."""

import math

import numpy as np
import pytest

import oracle
from oracle import mask as omask, attention as oattn, accept as oacc
from brute import brute_attention
from synth import generate
from test_oracle_mask import small_cfg, read_golden
import test_oracle_accept as tacc

MASK, DATA = omask.MASK, omask.DATA


def golden_ok():
    for name in ("mask_B3_mu231.txt", "mask_B5_mixed.txt"):
        rows, meta = read_golden(name)
        B, L, gamma = meta["block_size"][0], meta["max_ref"][0], meta["num_ref"][0]
        order = [f"M{k}" for k in range(B)] + [f"D{r + 1}" for r in range(L)]
        want = np.array([rows[k] for k in order], bool)
        got = omask.new_slot_visibility(np.array(meta["step_map"]), gamma, L)
        if not np.array_equal(got, want):
            return False
    return True


def brute_ok(seeds=(1, 2, 3)):
    for seed in seeds:
        cfg = small_cfg(batch=2, block_size=5, max_ref=4, prefix=(0, 6),
                        num_q_heads=4, num_kv_heads=2, head_dim=8)
        inp = generate(cfg, seed=seed, poison=True)
        out, lse = oracle.verify_attention(inp)
        bo, bl = brute_attention(inp)
        if not (np.allclose(out, bo, atol=1e-12, rtol=0) and
                np.allclose(lse, bl, atol=1e-12, rtol=0)):
            return False
    return True


def _vis_variant(which):
    def vis(si, ti, sj, tj):
        if sj == MASK and tj == 0 and which != "committed_hidden":
            return True
        if si == DATA and sj == DATA:
            return tj < ti if which == "case1_strict" else tj <= ti
        if si == DATA and sj == MASK:
            return tj >= ti if which == "case2_loose" else tj > ti
        if si == MASK and sj == DATA:
            return tj <= ti if which == "case3_loose" else tj < ti
        return tj > ti if which == "case4_strict" else tj >= ti
    return vis


@pytest.mark.parametrize("which", ["case1_strict", "case2_loose", "case3_loose",
                                   "case4_strict", "committed_hidden"])
def test_mask_mutation_caught(monkeypatch, which):
    assert golden_ok() and brute_ok()
    monkeypatch.setattr(omask, "visible", _vis_variant(which))
    assert not (golden_ok() and brute_ok())


def test_transposed_mask_caught(monkeypatch):
    real = omask.new_slot_visibility
    monkeypatch.setattr(oattn, "new_slot_visibility", lambda *a: real(*a).T.copy())
    assert not brute_ok()


def test_gqa_map_mutation_caught(monkeypatch):
    """Query head h must use KV head h // G, not h % Hkv."""
    real = oattn.pair_attention

    def wrong(inp, b, kvh, scale=None, rope_theta=0.0):
        cfg = inp.cfg
        G, Hkv = cfg.group, cfg.num_kv_heads
        out = np.zeros((cfg.n_new, G, cfg.head_dim))
        lse = np.zeros((G, cfg.n_new))
        for g in range(G):
            h = kvh * G + g
            o, l = real(inp, b, h % Hkv, scale)
            out[:, g], lse[g] = o[:, h % G], l[h % G]
        return out, lse
    monkeypatch.setattr(oattn, "pair_attention", wrong)
    assert not brute_ok()


def test_dropped_scale_caught(monkeypatch):
    real = oattn.attend
    monkeypatch.setattr(oattn, "attend", lambda q, k, v, vis, scale: real(q, k, v, vis, 1.0))
    assert not brute_ok()


def test_hidden_prefix_caught(monkeypatch):
    monkeypatch.setattr(oattn, "row_valid", lambda *a: np.zeros(len(a[0]) + a[2], bool))
    assert not brute_ok()


def test_accept_mutations_caught(monkeypatch):
    """Highest-index ties, or a missing max shift in the log-sum-exp, fail the
    accept pins."""
    assert tacc.all_pins_pass()

    def last_tie(x):
        m = x.max()
        t = int(np.flatnonzero(x == m)[-1])
        return t, m, m + math.log(np.exp(x - m).sum())
    monkeypatch.setattr(oacc, "scan_row", last_tie)
    assert not tacc.all_pins_pass()
    monkeypatch.undo()

    def no_log(x):
        m = x.max()
        return int(np.flatnonzero(x == m)[0]), m, m + np.exp(x - m).sum()
    monkeypatch.setattr(oacc, "scan_row", no_log)
    assert not tacc.all_pins_pass()


# ---- stochastic acceptance ----------------------------------------------------

import test_oracle_sampled as tsmp
from oracle import sampled as osmp


def sampled_pins_ok():
    try:
        tsmp.test_first_draft_output_is_target_distribution(1.0)
        tsmp.test_first_draft_output_is_target_distribution(0.6)
        tsmp.test_second_draft_output_is_its_target_distribution()
        tsmp.test_hand_example()
        tsmp.test_empty_residual_draws_from_target()
        tsmp.test_probabilities_match_softmax_and_gamma_zero()
        tsmp.test_small_temperature_is_greedy()
    except AssertionError:
        return False
    return True


def _sampled_variant(monkeypatch, which):
    if which == "inverted_ratio":
        monkeypatch.setattr(osmp, "accept_draft", lambda u, pt, pd: u * pt < pd)
    elif which == "unclamped_residual":
        monkeypatch.setattr(osmp, "residual", lambda pt, pd: ((pt - pd), False))
    elif which == "target_not_residual":
        monkeypatch.setattr(osmp, "residual", lambda pt, pd: (pt.copy(), True))
    elif which == "temperature_ignored":
        real = osmp.softmax_t
        monkeypatch.setattr(osmp, "softmax_t", lambda x, T: real(x, 1.0))
    elif which == "row_by_draft_index":
        monkeypatch.setattr(osmp, "rows_of_steps", lambda step_row, gamma: list(range(gamma)))
    elif which == "draw_reuses_accept_uniform":
        real = osmp.verify_accept_sampled

        def wrong(logits, dl, drafts, step, nref, u, T, dtype):
            u = np.array(u, np.float64, copy=True)
            L = drafts.shape[1]
            # the draw takes the uniform of the first draft instead of its own
            u[:, L] = u[:, 0]
            return real(logits, dl, drafts, step, nref, u, T, dtype)
        monkeypatch.setattr(osmp, "verify_accept_sampled", wrong)


@pytest.mark.parametrize("which", ["inverted_ratio", "unclamped_residual", "target_not_residual",
                                   "temperature_ignored", "row_by_draft_index",
                                   "draw_reuses_accept_uniform"])
def test_sampled_mutation_caught(monkeypatch, which):
    assert sampled_pins_ok()
    _sampled_variant(monkeypatch, which)
    assert not sampled_pins_ok()


# ---- rotary embedding --------------------------------------------------------

import test_oracle_rope as trope
from oracle import rope as orope


def rope_pins_ok():
    try:
        for d, th in [(2, 10000.0), (8, 10000.0), (64, 1e6), (128, 1e6)]:
            trope.test_rotation_matches_complex_form(d, th)
        trope.test_relative_positions_norms_identity()
        trope.test_copy_positions_hand_example()
        trope.test_attention_with_rope_equals_prerotated_inputs(3, 0)
        trope.test_attention_with_rope_equals_prerotated_inputs(4, 4)
        trope.test_verification_slot_sees_its_draft_at_distance_zero()
    except AssertionError:
        return False
    return True


@pytest.mark.parametrize("which", ["physical_positions", "interleaved_pairs", "half_frequency",
                                   "prefix_rotated_again"])
def test_rope_mutation_caught(monkeypatch, which):
    assert rope_pins_ok()
    if which == "physical_positions":
        def phys(step_row, gamma, L, prefix_len):
            return prefix_len + np.arange(len(step_row) + L)
        monkeypatch.setattr(orope, "positions", phys)
        monkeypatch.setattr(oattn, "positions", phys)
    elif which == "interleaved_pairs":
        def inter(x, pos, theta):
            d = x.shape[-1]
            ang = pos.astype(np.float64)[:, None] * orope.inv_freq(d, theta)[None, :]
            c, s = np.cos(ang), np.sin(ang)
            out = x.copy()
            out[:, 0::2] = x[:, 0::2] * c - x[:, 1::2] * s
            out[:, 1::2] = x[:, 1::2] * c + x[:, 0::2] * s
            return out
        monkeypatch.setattr(orope, "rotate", inter)
        monkeypatch.setattr(oattn, "rotate", inter)
    elif which == "half_frequency":
        monkeypatch.setattr(orope, "inv_freq", lambda d, theta: theta ** (-1.0 * np.arange(d // 2) / d))
    elif which == "prefix_rotated_again":
        real_prefix = oattn.prefix_kv
        real_pair = oattn.pair_attention

        def pair(inp, b, kvh, scale=None, rope_theta=0.0):
            if rope_theta:
                def pk(inp_, b_, kvh_):
                    k, v = real_prefix(inp_, b_, kvh_)
                    return orope.rotate(k, np.arange(k.shape[0]), rope_theta), v
                monkeypatch.setattr(oattn, "prefix_kv", pk)
            try:
                return real_pair(inp, b, kvh, scale, rope_theta)
            finally:
                monkeypatch.setattr(oattn, "prefix_kv", real_prefix)
        monkeypatch.setattr(oattn, "pair_attention", pair)
    assert not rope_pins_ok()


import test_oracle_lmhead as tlm
from oracle import lmhead as olm
from oracle.widen import widen as _widen


def lmhead_pins_ok():
    try:
        tlm.test_hand_example()
        tlm.test_logits_against_element_sums()
    except AssertionError:
        return False
    return True


@pytest.mark.parametrize("which", ["dropped_last_term", "first_chunk_repeated", "slots_reversed",
                                   "weight_rows_shifted"])
def test_lmhead_mutation_caught(monkeypatch, which):
    assert lmhead_pins_ok()
    real = olm.lmhead_logits

    def mutant(hidden, weight, dtype):
        h = _widen(np.asarray(hidden), dtype)
        w = _widen(np.asarray(weight), dtype)
        if which == "dropped_last_term":
            return h[..., :-1] @ w[:, :-1].T
        if which == "first_chunk_repeated":            # chunk loop always reads chunk 0
            step = 1 << 13
            out = real(hidden, weight, dtype)
            for v0 in range(step, w.shape[0], step):
                n = min(step, w.shape[0] - v0)
                out[..., v0:v0 + n] = h @ w[:n].T
            return out
        if which == "slots_reversed":
            return h[:, ::-1] @ w.T
        return h @ np.roll(w, 1, axis=0).T             # weight row v taken for token v + 1

    monkeypatch.setattr(olm, "lmhead_logits", mutant)
    monkeypatch.setattr(oracle, "lmhead_logits", mutant)
    assert not lmhead_pins_ok()
