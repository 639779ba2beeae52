"""GPU parity of the LM head fused with the vocabulary scan against the oracle
(logits = hidden . weight^T in float64, then the greedy acceptance), through
the C ABI.  The kernel accumulates fp32 from bf16 products: a target id may
differ from the oracle's only where the oracle's top two logits lie within
1e-4 of each other (checked for validity instead); accept lengths follow the
target ids; confidence and draft probabilities within 1e-4 relative."""

import numpy as np
import pytest
import torch

import oracle
from gpu_util import dev_tensor, int_tensor, walk_accept
from synth import VerifyConfig, config_by_id, generate, generate_lmhead_side

pytestmark = pytest.mark.gpu


def run_lmhead(inp, hidden, weight):
    from paper_2606_02544_amd import binding
    t, c, p, a = binding.verify_accept_lmhead(
        dev_tensor(hidden, "bf16"), dev_tensor(weight, "bf16"), int_tensor(inp.draft_ids),
        int_tensor(inp.step_map), int_tensor(inp.num_ref))
    torch.cuda.synchronize()
    return t.cpu().numpy(), c.cpu().double().numpy(), p.cpu().double().numpy(), a.cpu().numpy()


def check_lmhead(inp, hidden, weight, got):
    t, c, p, a = got
    rt, rc, rp, ra, logits = oracle.verify_accept_lmhead(hidden, weight, inp.draft_ids,
                                                         inp.step_map, inp.num_ref, "bf16")
    scanned = inp.step_map >= 1
    near = 0
    for s, k in zip(*np.nonzero(scanned)):
        if t[s, k] != rt[s, k]:
            row = logits[s, k]
            assert 0 <= t[s, k] < row.size and row.max() - row[t[s, k]] <= 1e-4 * max(1.0, abs(row.max())), \
                (s, k, t[s, k], rt[s, k])
            near += 1
    assert np.all(t[~scanned] == -1)
    # The accepted length always follows the ids the GPU produced; where none
    # differs from the oracle's it is also the oracle's length.
    np.testing.assert_array_equal(a, walk_accept(t, inp.draft_ids, inp.step_map, inp.num_ref))
    if near == 0:
        np.testing.assert_array_equal(a, ra)
    np.testing.assert_allclose(c, rc, rtol=1e-4, atol=1e-30)
    np.testing.assert_allclose(p, rp, rtol=1e-4, atol=1e-30)


LMHEAD_CASES = [
    # batch, B, L, V, H, step_mode, seed: ragged vocabulary and row tiles, mixed step
    # maps.  Rows R = batch * B pick the kernel variant: R <= 32 (32-wide stages),
    # R <= 128 (64-wide stages), more (256-row tiles, two-stage ring).
    (3, 8, 6, 1000, 256, "mixed", 1),
    (5, 16, 16, 2051, 512, "full", 2),
    (9, 32, 24, 777, 128, "mixed", 3),       # 288 rows: two 256-row tiles
    (1, 4, 4, 151936, 2048, "full", 4),      # SDAR-1.7B-shaped head
    (2, 8, 8, 3000, 64, "mixed", 5),         # one reduction stage
    (4, 16, 12, 1500, 192, "full", 6),       # as many stages as the ring holds
    (6, 16, 8, 900, 64, "mixed", 7),         # 96 rows, one stage
    (10, 16, 16, 1200, 64, "mixed", 8),      # 160 rows, one stage
    (20, 32, 32, 2500, 320, "full", 9),      # 640 rows: three row tiles, odd stage count
]


@pytest.mark.parametrize("case", LMHEAD_CASES, ids=lambda c: "-".join(map(str, c)))
def test_lmhead_parity(case):
    b, B, L, V, H, mode, seed = case
    cfg = VerifyConfig(0, "lmhead", "bf16", batch=b, num_q_heads=2, num_kv_heads=1, head_dim=64,
                       prefix=4, block_size=B, max_ref=L, vocab=V, plant=0.6, step_mode=mode)
    inp = generate(cfg, seed=seed, bad_draft_rate=0.2 if mode == "mixed" else 0.0)
    hidden, weight = generate_lmhead_side(inp, H)
    check_lmhead(inp, hidden, weight, run_lmhead(inp, hidden, weight))


def test_lmhead_graph_replays_match_eager():
    """The LM-head entry point captured in a HIP graph: every replay, with eager
    work and synchronisation in between, reproduces the eager outputs bit for
    bit (two row-count variants)."""
    from paper_2606_02544_amd import binding
    for b, B, L, V, H, seed in ((2, 8, 8, 3000, 256, 21), (12, 16, 16, 2051, 128, 22)):
        cfg = VerifyConfig(0, "lmhead", "bf16", batch=b, num_q_heads=2, num_kv_heads=1,
                           head_dim=64, prefix=4, block_size=B, max_ref=L, vocab=V, plant=0.6,
                           step_mode="mixed")
        inp = generate(cfg, seed=seed, bad_draft_rate=0.2)
        hidden, weight = generate_lmhead_side(inp, H)
        hd, wd = dev_tensor(hidden, "bf16"), dev_tensor(weight, "bf16")
        ids, sm, nr = int_tensor(inp.draft_ids), int_tensor(inp.step_map), int_tensor(inp.num_ref)
        eager = binding.verify_accept_lmhead(hd, wd, ids, sm, nr)
        torch.cuda.synchronize()
        outs = [torch.zeros_like(t) for t in eager]
        s = torch.cuda.Stream()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.stream(s):
            binding.verify_accept_lmhead(hd, wd, ids, sm, nr, target_ids=outs[0],
                                         confidence=outs[1], draft_prob=outs[2],
                                         accept_len=outs[3], stream=s)      # workspace exists
            torch.cuda.synchronize()
            with torch.cuda.graph(g, stream=s):
                binding.verify_accept_lmhead(hd, wd, ids, sm, nr, target_ids=outs[0],
                                             confidence=outs[1], draft_prob=outs[2],
                                             accept_len=outs[3], stream=s)
        for rep in range(3):
            for t in outs:
                t.zero_()
            torch.cuda.synchronize()
            g.replay()
            torch.cuda.synchronize()
            for x, y in zip(outs, eager):
                assert torch.equal(x, y), (b, rep)
            binding.verify_accept_lmhead(hd, wd, ids, sm, nr)    # eager work between replays
            torch.cuda.synchronize()
        check_lmhead(inp, hidden, weight, tuple(t.cpu().numpy() if t.dtype == torch.int32
                                                else t.cpu().double().numpy() for t in outs))


@pytest.mark.parametrize("gamma,committed,batch", [(0, 0, 3), (0, 3, 6), (3, 2, 6), (5, 0, 3)])
def test_lmhead_steps_inside_a_block(gamma, committed, batch):
    """Fewer drafts than block slots, committed slots, and the plain block step
    (gamma = 0: no reference slots, draft_ids may be empty) on the LM-head path."""
    cfg = VerifyConfig(0, "steps", "bf16", batch=batch, num_q_heads=2, num_kv_heads=1,
                       head_dim=64, prefix=4, block_size=8, max_ref=gamma, vocab=3000,
                       plant=0.6, committed=committed)
    inp = generate(cfg, seed=90 + 7 * gamma + committed)
    assert np.all(inp.num_ref == gamma)
    hidden, weight = generate_lmhead_side(inp, 128)
    got = run_lmhead(inp, hidden, weight)
    check_lmhead(inp, hidden, weight, got)
    if gamma == 0:
        assert np.all(got[3] == 0)


@pytest.mark.parametrize("batch,B", [(8, 16), (16, 32)])
def test_lmhead_8b_head(batch, B):
    """The SDAR-8B-shaped head (H = 4096, V = 151936) at the row counts of the
    8B layer (128 rows: 64-wide stages) and the long-context step (512 rows:
    256-row tiles), gamma = B as in the workloads."""
    cfg = VerifyConfig(0, "lmhead8b", "bf16", batch=batch, num_q_heads=2, num_kv_heads=1,
                       head_dim=64, prefix=4, block_size=B, max_ref=B, vocab=151936,
                       plant=0.6, step_mode="full")
    inp = generate(cfg, seed=100 + B)
    hidden, weight = generate_lmhead_side(inp, 4096)
    check_lmhead(inp, hidden, weight, run_lmhead(inp, hidden, weight))
