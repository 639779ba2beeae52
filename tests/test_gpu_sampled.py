"""GPU parity of the stochastic acceptance (eq. 2 at temperature T) against the
oracle, through the C ABI.

Exact: accept lengths, and the correction token wherever the draw's target
w * Z lies more than 1e-4 * Z from a boundary of the oracle's float64 CDF.
The kernel computes probabilities and running sums in float32, so the two
sides may take a different side of a threshold only within rounding of it:
the uniforms are moved 2e-3 away from each acceptance threshold before the
run, and a draw within 1e-4 * Z of a CDF boundary is checked for validity
(either neighbouring token) instead of equality.  p_theta(D_r) and p_phi(D_r)
within 1e-4 relative.
"""

import numpy as np
import pytest
import torch

import oracle
from oracle import sampled as osmp
from oracle.widen import widen
from synth import VerifyConfig, config_by_id, generate, generate_draft_side
from gpu_util import dev_tensor, int_tensor

pytestmark = pytest.mark.gpu


def run_sampled(inp, dlog, u, T, chunks_per_row=0):
    from paper_2606_02544_amd import binding
    dt = inp.cfg.dtype
    logits = dev_tensor(inp.logits, dt)
    draft_logits = dev_tensor(dlog, dt)
    pt, pd, a, c = binding.verify_accept_sampled(
        logits, draft_logits, int_tensor(inp.draft_ids), int_tensor(inp.step_map),
        int_tensor(inp.num_ref), torch.from_numpy(np.ascontiguousarray(u, np.float32)).cuda(),
        temperature=T, chunks_per_row=chunks_per_row)
    torch.cuda.synchronize()
    return (pt.cpu().double().numpy(), pd.cpu().double().numpy(), a.cpu().numpy(),
            c.cpu().numpy())


def nudge(inp, dlog, u, T):
    """Move each acceptance uniform at least 2e-3 away from its threshold
    alpha_r = p_theta / p_phi (computed here in float64)."""
    u = np.array(u, np.float64, copy=True)
    b, L = inp.draft_ids.shape
    V = inp.cfg.vocab
    for s in range(b):
        g = int(inp.num_ref[s])
        rows = osmp.rows_of_steps(inp.step_map[s], g)
        for r in range(g):
            tok = int(inp.draft_ids[s, r])
            if not 0 <= tok < V:
                continue
            pt = osmp.softmax_t(widen(inp.logits[s, rows[r]], inp.cfg.dtype), T)[tok]
            pd = osmp.softmax_t(widen(dlog[s, r], inp.cfg.dtype), T)[tok]
            alpha = pt / pd
            if abs(u[s, r] - alpha) < 2e-3:
                u[s, r] = alpha - 2e-3 if alpha > 4e-3 else min(alpha + 2e-3, 0.999)
    return u.astype(np.float32)


def check_sampled(inp, dlog, u, T, got):
    pt, pd, a, c = got
    dt = inp.cfg.dtype
    rpt, rpd, ra, rc = oracle.verify_accept_sampled(inp.logits, dlog, inp.draft_ids, inp.step_map,
                                                    inp.num_ref, u.astype(np.float64), T, dt)
    np.testing.assert_array_equal(a, ra)
    np.testing.assert_allclose(pt, rpt, rtol=1e-4, atol=1e-30)
    np.testing.assert_allclose(pd, rpd, rtol=1e-4, atol=1e-30)
    L = inp.draft_ids.shape[1]
    loose = 0
    for s in range(len(a)):
        if ra[s] >= int(inp.num_ref[s]):
            assert c[s] == -1 and rc[s] == -1, s
            continue
        k = osmp.rows_of_steps(inp.step_map[s], int(inp.num_ref[s]))[ra[s]]
        q, _ = osmp.residual_row(inp.logits[s, k], dlog[s, ra[s]], T, dt)
        cdf = np.cumsum(q)
        Z = cdf[-1]
        t = float(u[s, L]) * Z
        x = int(c[s])
        assert 0 <= x < inp.cfg.vocab, (s, x)
        if x == rc[s]:
            continue
        # Only a target within rounding of a CDF boundary may pick a neighbour.
        tol = 1e-4 * Z
        lo = cdf[x - 1] if x > 0 else 0.0
        assert lo - tol <= t <= cdf[x] + tol and q[x] > 0, (s, x, rc[s], t, lo, cdf[x])
        loose += 1
    return loose


SAMPLED_CASES = [
    # (config, T, chunks_per_row, seed): cfg 1 is fp32 V=1000; the mixed configs
    # have gamma < B, committed/undrafted/padding slots and out-of-range drafts.
    ("cfg1", 1.0, 0, 1),
    ("cfg1", 0.7, 3, 2),
    ("mixed_bf16", 1.0, 0, 3),
    ("mixed_bf16", 0.8, 5, 4),
    ("mixed_bf16_v1021", 1.0, 2, 5),      # V not a multiple of 8: scalar path
    ("mixed_f32", 1.3, 0, 6),
]


def make_inputs(name, seed):
    if name == "cfg1":
        return generate(config_by_id(1), seed=seed)
    dt = "f32" if name == "mixed_f32" else "bf16"
    V = 1021 if name.endswith("v1021") else 4096
    cfg = VerifyConfig(0, name, dt, batch=9, num_q_heads=4, num_kv_heads=2, head_dim=64,
                       prefix=(0, 8), block_size=16, max_ref=12, vocab=V, plant=0.6,
                       step_mode="mixed")
    return generate(cfg, seed=seed, bad_draft_rate=0.2)


@pytest.mark.parametrize("case", SAMPLED_CASES, ids=lambda c: "-".join(map(str, c)))
def test_sampled_parity(case):
    name, T, cpr, seed = case
    inp = make_inputs(name, seed)
    dlog, u = generate_draft_side(inp)
    u = nudge(inp, dlog, u, T)
    got = run_sampled(inp, dlog, u, T, cpr)
    check_sampled(inp, dlog, u, T, got)
    if inp.cfg.batch > 4:                      # both outcomes occur
        assert np.any(got[2] < inp.num_ref) and np.any(got[2] > 0)


def test_sampled_all_accepted_and_empty_residual():
    """Uniforms 0 accept every in-range draft with p_theta > 0; an out-of-range
    draft with draft rows equal to the target rows leaves an empty residual,
    and the draw falls back to p_theta."""
    inp = make_inputs("mixed_bf16", 8)
    dlog, u = generate_draft_side(inp)
    u0 = np.zeros_like(u)
    u0[:, -1] = 0.37
    got = run_sampled(inp, dlog, u0, 1.0)
    check_sampled(inp, dlog, u0, 1.0, got)
    # Draft rows := target rows; every draft id out of range.
    same = dlog.copy()
    for s in range(inp.cfg.batch):
        g = int(inp.num_ref[s])
        for r, k in enumerate(osmp.rows_of_steps(inp.step_map[s], g)):
            same[s, r] = inp.logits[s, k]
    inp.draft_ids[:] = inp.cfg.vocab + 5
    for w in (0.0, 0.5, 0.999):
        uu = np.full_like(u, 0.5)
        uu[:, -1] = w
        got = run_sampled(inp, same, uu, 1.0)
        check_sampled(inp, same, uu, 1.0, got)
        assert np.all(got[2] == 0)


def test_sampled_large_vocab_bf16():
    """The SDAR-8B-shaped workload (vocab 151936, bf16) at T = 1."""
    cfg = VerifyConfig(0, "vocab151936", "bf16", batch=8, num_q_heads=4, num_kv_heads=2,
                       head_dim=64, prefix=(0, 8), block_size=16, max_ref=16, vocab=151936,
                       plant=0.6)
    inp = generate(cfg, seed=12)
    dlog, u = generate_draft_side(inp)
    u = nudge(inp, dlog, u, 1.0)
    got = run_sampled(inp, dlog, u, 1.0)
    check_sampled(inp, dlog, u, 1.0, got)
