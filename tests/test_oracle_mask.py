"""Pins of the oracle's mask and attention against things other than itself.

* hand-derived golden masks (tests/golden, from the paper's prose);
* brute force: each row's own context, built from the block state at its step;
* structural invariants: one representative per block position, row counts;
* special cases that reduce to textbook attention (zero draft length = plain
  bidirectional block attention, B = gamma = 1 = causal decoding, single key,
  zero query) and torch's scaled_dot_product_attention (float64, CPU);
* permutation consistency of the step map.
"""

import math
import os

import numpy as np
import pytest
import torch
from hypothesis import given, settings, strategies as st, HealthCheck

import oracle
from oracle import mask as omask
from brute import brute_attention, row_context
from synth import VerifyConfig, generate

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def small_cfg(**kw):
    base = dict(cid=0, name="tiny-test", dtype="f32", batch=2, num_q_heads=4, num_kv_heads=2,
                head_dim=16, prefix=5, block_size=4, max_ref=4, vocab=37, plant=0.5,
                qkv_std=1.0, step_mode="mixed")
    base.update(kw)
    return VerifyConfig(**base)


def read_golden(name):
    rows, meta = {}, {}
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.split("#")[0].strip()
            if not line:
                continue
            key, *vals = line.split()
            if key[0] in "MD" and key[1:].isdigit():
                rows[key] = [int(v) for v in vals]
            else:
                meta[key] = [int(v) for v in vals]
    return rows, meta


@pytest.mark.parametrize("name", ["mask_B3_mu231.txt", "mask_B5_mixed.txt"])
def test_golden_mask(name):
    rows, meta = read_golden(name)
    B, L, gamma = meta["block_size"][0], meta["max_ref"][0], meta["num_ref"][0]
    step = np.array(meta["step_map"], np.int32)
    order = [f"M{k}" for k in range(B)] + [f"D{r + 1}" for r in range(L)]
    want = np.array([rows[k] for k in order], bool)
    got = omask.new_slot_visibility(step, gamma, L)
    np.testing.assert_array_equal(got, want)
    np.testing.assert_array_equal(omask.row_valid(step, gamma, L),
                                  np.array(meta["prefix_rows"], bool))
    # the brute-force context lists agree with the same hand-made table
    for i, key in enumerate(order):
        ctx = row_context(step, gamma, L, i)
        seen = np.zeros(B + L, bool)
        if ctx is not None:
            seen[ctx] = True
        np.testing.assert_array_equal(seen, want[i], err_msg=key)


@settings(max_examples=60, deadline=None, suppress_health_check=[HealthCheck.too_slow])
@given(B=st.integers(1, 8), Lfrac=st.floats(0, 1), G=st.sampled_from([1, 2, 4]),
       Hkv=st.sampled_from([1, 2]), d=st.sampled_from([8, 16]),
       prefix=st.integers(0, 9), seed=st.integers(0, 10 ** 6),
       mode=st.sampled_from(["mixed", "full"]), paged=st.booleans())
def test_oracle_equals_brute_force(B, Lfrac, G, Hkv, d, prefix, seed, mode, paged):
    L = int(round(Lfrac * B))
    cfg = small_cfg(batch=2, num_q_heads=G * Hkv, num_kv_heads=Hkv, head_dim=d,
                    prefix=(0, prefix) if prefix else 0, block_size=B, max_ref=L,
                    step_mode=mode, page_size=3 if paged else 0)
    inp = generate(cfg, seed=seed, poison=True)
    out, lse = oracle.verify_attention(inp)
    bo, bl = brute_attention(inp)
    np.testing.assert_allclose(out, bo, rtol=0, atol=1e-12)
    np.testing.assert_allclose(lse, bl, rtol=0, atol=1e-12)


@settings(max_examples=200, deadline=None)
@given(B=st.integers(1, 32), Lfrac=st.floats(0, 1), seed=st.integers(0, 10 ** 6))
def test_one_representative_per_position(B, Lfrac, seed):
    """Every non-padded row sees exactly one version of every non-padded block
    position: so its key count is prefix + #non-padded block slots."""
    L = int(round(Lfrac * B))
    rng = np.random.default_rng(seed)
    cfg = small_cfg(batch=1, block_size=B, max_ref=L)
    from synth.generate import _step_maps
    step, gam = _step_maps(rng, cfg)
    step, gamma = step[0], int(gam[0])
    A = omask.new_slot_visibility(step, gamma, L)
    valid = omask.row_valid(step, gamma, L)
    nonpad = [p for p in range(B) if step[p] >= 0]
    for i in range(B + L):
        if not valid[i]:
            assert not A[i].any()
            continue
        assert A[i].sum() == len(nonpad)
        for p in nonpad:
            s = step[p]
            reps = A[i, p] + (A[i, B + s - 1] if 1 <= s <= gamma else 0)
            assert reps == 1
    assert not A[:, ~valid].any()


def _sdpa(q, k, v, mask=None, scale=None):
    """torch float64 CPU scaled_dot_product_attention for [H, R, d] x [H, N, d]."""
    return torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q)[None], torch.from_numpy(k)[None], torch.from_numpy(v)[None],
        attn_mask=None if mask is None else torch.from_numpy(mask)[None, None],
        scale=scale)[0].numpy()


def test_zero_draft_length_is_block_attention():
    """gamma = 0: every block row sees the prefix and the whole block (plain
    bidirectional block-diffusion attention with KV cache, Sec. 2 "Blockwise
    Decoding"); reference slots are padding."""
    cfg = small_cfg(batch=3, block_size=6, max_ref=3, prefix=7, step_mode="full")
    inp = generate(cfg, seed=5)
    inp.num_ref[:] = 0
    inp.step_map[:] = np.array([[0, 1, 4, 2, 0, 9], [1, 1, 1, 1, 1, 1], [0] * 6])
    out, lse = oracle.verify_attention(inp)
    G, B = cfg.group, cfg.block_size
    for s in range(cfg.batch):
        for kvh in range(cfg.num_kv_heads):
            k = np.concatenate([inp.k_cache[s, :7, kvh], inp.k_new[s, :B, kvh]]).astype(np.float64)
            v = np.concatenate([inp.v_cache[s, :7, kvh], inp.v_new[s, :B, kvh]]).astype(np.float64)
            for g in range(G):
                h = kvh * G + g
                q = inp.q[s, :B, h].astype(np.float64)
                want = _sdpa(q[None], k[None], v[None])[0]
                np.testing.assert_allclose(out[s, :B, h], want, atol=1e-12, rtol=0)
    assert np.all(out[:, B:] == 0) and np.all(np.isneginf(lse[:, :, B:]))


def test_single_draft_is_causal_decoding():
    """B = gamma = 1: the verification row and the drafted token's row each see
    the prefix and their own slot only (autoregressive decoding of one token)."""
    cfg = small_cfg(batch=2, block_size=1, max_ref=1, prefix=6, step_mode="full")
    inp = generate(cfg, seed=11)
    out, _ = oracle.verify_attention(inp)
    for s in range(2):
        for h in range(cfg.num_q_heads):
            kvh = h // cfg.group
            for slot in (0, 1):
                k = np.concatenate([inp.k_cache[s, :6, kvh], inp.k_new[s, slot:slot + 1, kvh]])
                v = np.concatenate([inp.v_cache[s, :6, kvh], inp.v_new[s, slot:slot + 1, kvh]])
                q = inp.q[s, slot:slot + 1, h]
                want = _sdpa(q[None].astype(np.float64), k[None].astype(np.float64),
                             v[None].astype(np.float64))[0]
                np.testing.assert_allclose(out[s, slot, h], want[0], atol=1e-12, rtol=0)


def test_single_visible_key_returns_its_value():
    cfg = small_cfg(batch=1, block_size=1, max_ref=1, prefix=0, step_mode="full")
    inp = generate(cfg, seed=3)
    out, lse = oracle.verify_attention(inp)
    for h in range(cfg.num_q_heads):
        kvh = h // cfg.group
        np.testing.assert_array_equal(out[0, 0, h], inp.v_new[0, 0, kvh].astype(np.float64))
        np.testing.assert_array_equal(out[0, 1, h], inp.v_new[0, 1, kvh].astype(np.float64))
        s = float(np.dot(inp.q[0, 1, h].astype(np.float64), inp.k_new[0, 1, kvh])) / 4.0
        assert abs(lse[0, h, 1] - s) < 1e-12


def test_zero_query_is_mean_of_visible_values():
    cfg = small_cfg(batch=2, block_size=5, max_ref=4, prefix=(0, 6))
    inp = generate(cfg, seed=21, poison=True)
    inp.q[:] = 0
    out, lse = oracle.verify_attention(inp)
    for s in range(cfg.batch):
        gamma, n = int(inp.num_ref[s]), int(inp.prefix_lens[s])
        for row in range(cfg.n_new):
            ctx = row_context(inp.step_map[s], gamma, cfg.max_ref, row)
            for h in range(cfg.num_q_heads):
                kvh = h // cfg.group
                if ctx is None:
                    assert np.all(out[s, row, h] == 0)
                    continue
                vals = np.concatenate([inp.v_cache[s, :n, kvh], inp.v_new[s, ctx, kvh]])
                np.testing.assert_allclose(out[s, row, h], vals.astype(np.float64).mean(0),
                                           atol=1e-12, rtol=0)
                assert abs(lse[s, h, row] - math.log(len(vals))) < 1e-12


@pytest.mark.parametrize("seed", [1, 2, 3])
def test_matches_torch_sdpa_with_gqa(seed):
    """Attention arithmetic (scale, softmax, GQA head map, LSE) against torch's
    float64 scaled_dot_product_attention given the same boolean mask."""
    cfg = small_cfg(batch=2, num_q_heads=8, num_kv_heads=2, head_dim=16, block_size=6,
                    max_ref=5, prefix=(0, 9))
    inp = generate(cfg, seed=seed, poison=True)
    out, lse = oracle.verify_attention(inp)
    B, L = cfg.block_size, cfg.max_ref
    for s in range(cfg.batch):
        gamma, n = int(inp.num_ref[s]), int(inp.prefix_lens[s])
        A = omask.new_slot_visibility(inp.step_map[s], gamma, L)
        valid = omask.row_valid(inp.step_map[s], gamma, L)
        mask = np.concatenate([np.repeat(valid[:, None], n, 1), A], 1)
        k = np.concatenate([inp.k_cache[s, :n], inp.k_new[s]]).astype(np.float64)  # [N,Hkv,d]
        v = np.concatenate([inp.v_cache[s, :n], inp.v_new[s]]).astype(np.float64)
        q = inp.q[s].astype(np.float64).transpose(1, 0, 2)                          # [Hq,R,d]
        got = torch.nn.functional.scaled_dot_product_attention(
            torch.from_numpy(q)[None], torch.from_numpy(k.transpose(1, 0, 2))[None],
            torch.from_numpy(v.transpose(1, 0, 2))[None],
            attn_mask=torch.from_numpy(mask)[None, None], enable_gqa=True)[0].numpy()
        rows = np.flatnonzero(valid)
        np.testing.assert_allclose(out[s][rows].transpose(1, 0, 2), got[:, rows], atol=1e-12)
        sc = 1 / math.sqrt(cfg.head_dim)
        G = cfg.group
        for h in range(cfg.num_q_heads):
            S = sc * q[h] @ k[:, h // G].T
            S[~mask] = -np.inf
            want = torch.logsumexp(torch.from_numpy(S[rows]), dim=-1).numpy()
            np.testing.assert_allclose(lse[s, h, rows], want, atol=1e-12)


def test_paged_equals_contiguous():
    cfg = small_cfg(batch=3, page_size=4, prefix=(1, 13), block_size=4, max_ref=3)
    inp = generate(cfg, seed=8, poison=True)
    out_p, lse_p = oracle.verify_attention(inp)
    P = cfg.page_size
    cap = 13
    kc = np.full((3, cap) + inp.k_cache.shape[2:], np.nan, np.float32)
    vc = np.full_like(kc, np.nan)
    for s in range(3):
        for t in range(int(inp.prefix_lens[s])):
            pg = inp.block_table[s, t // P]
            kc[s, t], vc[s, t] = inp.k_cache[pg, t % P], inp.v_cache[pg, t % P]
    inp.block_table, inp.k_cache, inp.v_cache = None, kc, vc
    out_c, lse_c = oracle.verify_attention(inp)
    np.testing.assert_array_equal(out_p, out_c)
    np.testing.assert_array_equal(lse_p, lse_c)


@pytest.mark.parametrize("seed", [0, 1, 2, 3])
def test_step_map_permutation_consistency(seed):
    """Permuting block slots together with their step-map entries permutes the
    block-row outputs and leaves the reference rows unchanged; in particular any
    step map equals the left-to-right one after ordering block slots by draft
    order (Sec. 3.1: left-to-right order is mu = (1, ..., B))."""
    cfg = small_cfg(batch=2, block_size=6, max_ref=6, prefix=4, step_mode="full")
    inp = generate(cfg, seed=seed)
    out, lse = oracle.verify_attention(inp)
    B = cfg.block_size
    for s in range(cfg.batch):
        perm = np.argsort(inp.step_map[s])          # block slots in draft order
        inp.step_map[s] = inp.step_map[s][perm]
        for a in (inp.q, inp.k_new, inp.v_new):
            a[s, :B] = a[s, perm]
        out_blk_perm = out[s, :B][perm]
        assert list(inp.step_map[s]) == list(range(1, B + 1))
        o2, _ = oracle.verify_attention(inp, pairs=[(s, h) for h in range(cfg.num_kv_heads)])
        np.testing.assert_allclose(o2[s, :B], out_blk_perm, atol=1e-14, rtol=0)
        np.testing.assert_allclose(o2[s, B:], out[s, B:], atol=1e-14, rtol=0)
