"""GPU parity: the HIP path through the C ABI against the float64 oracle.

Attention outputs: bf16 within 2e-2 of each row's largest |value|, f32 within
1e-5 absolute, LSE within 1e-4.  target_ids and accept_len: bit-exact.
Confidence and draft probabilities: 1e-4 relative.
"""

import numpy as np
import pytest
import torch

import oracle
from gpu_util import (DeviceInputs, run_attention, run_accept, check_attention, check_accept,
                      oracle_accept)
from synth import CONFIGS, VerifyConfig, generate

pytestmark = pytest.mark.gpu


def _full_parity(inp, kv_chunk=0, chunks_per_row=0):
    d = DeviceInputs(inp)
    out, lse = run_attention(d, kv_chunk)
    ref_out, ref_lse = oracle.verify_attention(inp)
    check_attention(out, lse, ref_out, ref_lse, inp.cfg.dtype)
    check_accept(run_accept(d, chunks_per_row), oracle_accept(inp))


@pytest.mark.parametrize("cid", [1, 2, 3])
def test_config_full(cid):
    inp = generate(CONFIGS[cid], poison=True)
    _full_parity(inp)


@pytest.mark.parametrize("gamma,committed", [(8, 0), (3, 0), (3, 2), (0, 0), (0, 5)])
def test_steps_inside_a_block(gamma, committed):
    """A verification step with gamma < B drafts (the paper's gamma ablation,
    Table 3, at B = 8), later steps of the block with committed slots, and the
    plain block step (gamma = 0) once fewer than gamma positions remain."""
    cfg = VerifyConfig(0, "steps", "bf16", batch=6, num_q_heads=8, num_kv_heads=2,
                       head_dim=128, prefix=(0, 300), block_size=8, max_ref=gamma,
                       vocab=3000, plant=0.6, qkv_std=0.3, committed=committed)
    inp = generate(cfg, seed=60 + 7 * gamma + committed, poison=True)
    assert np.all(inp.num_ref == gamma)
    assert np.all(np.sum(inp.step_map == 0, axis=1) == committed)
    for chunk in (0, 64, -1):
        _full_parity(inp, kv_chunk=chunk)


class _FullSizeRuns:
    """One GPU run per full-size workload (the benchmark's launch
    configuration), kept on the host for the tests that check its pairs.  Only
    the latest workload is held, so host memory stays bounded."""

    def __init__(self):
        self.cid, self.val = None, None

    def get(self, cid):
        if self.cid != cid:
            self.cid, self.val = None, None
            inp = generate(CONFIGS[cid], poison=True)
            d = DeviceInputs(inp)
            out, lse = run_attention(d)
            acc = run_accept(d)
            del d
            torch.cuda.empty_cache()
            self.cid, self.val = cid, (inp, out, lse, acc)
        return self.val


@pytest.fixture(scope="module")
def full_size():
    runs = _FullSizeRuns()
    yield runs
    runs.val = None


def _check_pairs(inp, out, lse, pairs):
    ref_out, ref_lse = oracle.verify_attention(inp, pairs=pairs)
    G = inp.cfg.group
    for s, h in pairs:
        sl = slice(h * G, (h + 1) * G)
        check_attention(out[s, :, sl], lse[s, sl], ref_out[s, :, sl], ref_lse[s, sl], "bf16")


def _ragged_sequences(inp):
    lens = inp.prefix_lens
    b = inp.cfg.batch
    seqs = [int(np.argmin(lens)), int(np.argmax(lens)), 0, b - 1]
    rng = np.random.default_rng(2024)
    for s in rng.permutation(b):
        if len(seqs) == 8:
            break
        if int(s) not in seqs:
            seqs.append(int(s))
    return seqs


@pytest.mark.parametrize("part", range(4))
def test_long_context_every_pair(full_size, part):
    """Long-context workload (16 sequences x 8 KV heads, prefix 16384): the
    attention of every (sequence, KV head) pair against the oracle, a quarter
    of them per test; the accept step on every row."""
    inp, out, lse, acc = full_size.get(4)
    seqs = range(4 * part, 4 * part + 4)
    _check_pairs(inp, out, lse, [(s, h) for s in seqs for h in range(inp.cfg.num_kv_heads)])
    assert np.all(np.isfinite(out)) and np.all(np.isfinite(lse))
    if part == 0:
        check_accept(acc, oracle_accept(inp))


@pytest.mark.parametrize("part", range(2))
def test_ragged_paged_eight_sequences(full_size, part):
    """Ragged-paged workload (64 sequences, prefixes U[512, 32768], 16-token
    pages in random order): every KV head of eight sequences, including the
    shortest and the longest prefix; the accept step on every row."""
    inp, out, lse, acc = full_size.get(5)
    seqs = _ragged_sequences(inp)[4 * part:4 * part + 4]
    _check_pairs(inp, out, lse, [(s, h) for s in seqs for h in range(inp.cfg.num_kv_heads)])
    assert np.all(np.isfinite(out)) and np.all(np.isfinite(lse))
    if part == 0:
        check_accept(acc, oracle_accept(inp))


MIXED = [
    # dtype, head_dim, Hq, Hkv, B, L, prefix, page, kv_chunk, seed
    ("bf16", 128, 8, 2, 8, 8, (0, 300), 0, 64, 1),
    ("bf16", 128, 4, 4, 5, 3, (1, 200), 16, 128, 2),
    ("bf16", 64, 6, 2, 4, 4, (60, 130), 0, 64, 3),
    ("bf16", 64, 16, 1, 16, 16, (0, 150), 7, 64, 4),
    ("bf16", 128, 2, 2, 1, 1, (0, 70), 0, 0, 5),
    ("bf16", 128, 32, 8, 8, 0, (64, 64), 0, 0, 6),
    ("bf16", 128, 12, 4, 3, 2, (0, 0), 0, 0, 7),
    ("bf16", 128, 16, 2, 32, 32, (100, 400), 16, 64, 8),
    ("bf16", 64, 8, 2, 16, 16, (100, 300), 16, 64, 13),     # 128 rows: 4 row waves x 2
    ("bf16", 128, 12, 3, 24, 8, (0, 700), 32, 128, 14),     # 128 rows, paged, tail tiles
    # stream decomposition at small sizes: fewer tiles than groups (one-tile
    # ranges, many partials per pair), ragged and empty prefixes, paged
    ("bf16", 128, 8, 2, 8, 8, (0, 300), 0, -1, 15),
    ("bf16", 64, 8, 2, 16, 16, (100, 3000), 16, -1, 16),
    ("bf16", 128, 4, 4, 4, 4, (0, 9000), 0, -1, 17),
    ("bf16", 128, 12, 3, 24, 8, (0, 2500), 32, -1, 18),
    ("bf16", 64, 4, 2, 4, 4, (0, 0), 0, -1, 19),           # stream, new-slot tiles only
    ("bf16", 64, 16, 2, 8, 8, (0, 500), 8, -1, 20),        # stream, 128 rows, d 64, 8-token pages
    ("bf16", 128, 16, 2, 4, 4, (0, 700), 64, 0, 21),       # pages of exactly one tile
    ("bf16", 64, 4, 4, 8, 8, (0, 400), 4, 64, 22),         # 4-token pages (one page per 4 rows)
    ("bf16", 128, 8, 2, 8, 8, (600, 1100), 0, 64, 23),     # 10-18 splits: 4-dim merge, two rounds
    ("f32", 64, 2, 1, 4, 4, (0, 100), 0, 64, 9),
    ("f32", 128, 8, 2, 6, 4, (1, 90), 5, 64, 10),
    ("f32", 128, 4, 1, 8, 8, (0, 0), 0, 0, 11),
    ("f32", 64, 16, 2, 16, 16, (30, 150), 0, 0, 12),
    ("f32", 128, 4, 2, 4, 4, (500, 1100), 16, 64, 24),     # up to 18 splits, paged
]


@pytest.mark.parametrize("case", MIXED, ids=lambda c: "-".join(map(str, c)))
def test_mixed_step_maps(case):
    """Per-sequence gamma < B, committed, undrafted and padding slots, ragged
    prefixes (including empty), paged caches, forced small chunks (several
    splits and ragged tails), NaN-poisoned cache tails, out-of-range drafts."""
    dt, d, hq, hkv, B, L, prefix, page, kv_chunk, seed = case
    cfg = VerifyConfig(0, "mixed", dt, batch=5, num_q_heads=hq, num_kv_heads=hkv, head_dim=d,
                       prefix=prefix, block_size=B, max_ref=L, vocab=1000 + 8 * seed,
                       page_size=page, plant=0.6, qkv_std=0.3 if dt == "bf16" else 1.0,
                       step_mode="mixed")
    inp = generate(cfg, seed=seed, poison=True, bad_draft_rate=0.3)
    _full_parity(inp, kv_chunk=kv_chunk, chunks_per_row=0)


def test_max_new_slots_and_group():
    """B + L = 64 new slots and 16 query heads per KV head: 1024 packed rows,
    several row blocks."""
    cfg = VerifyConfig(0, "wide", "bf16", batch=2, num_q_heads=32, num_kv_heads=2,
                       head_dim=128, prefix=(200, 333), block_size=32, max_ref=32,
                       vocab=4096, qkv_std=0.25, step_mode="mixed")
    _full_parity(generate(cfg, seed=31, poison=True), kv_chunk=128)


def test_stream_largest_batch():
    """The stream decomposition at its largest batch (256 sequences): the
    per-sequence tile offsets are scanned over all 256 entries; ragged
    prefixes, paged cache."""
    cfg = VerifyConfig(0, "stream256", "bf16", batch=256, num_q_heads=8, num_kv_heads=2,
                       head_dim=128, prefix=(0, 300), block_size=8, max_ref=8, vocab=512,
                       page_size=16, qkv_std=0.3, step_mode="mixed")
    inp = generate(cfg, seed=41, poison=True)
    d = DeviceInputs(inp)
    ref_out, ref_lse = oracle.verify_attention(inp)
    for chunk in (-1, 0):
        out, lse = run_attention(d, chunk)
        check_attention(out, lse, ref_out, ref_lse, "bf16")


def test_split_count_invariance_and_determinism():
    inp = generate(CONFIGS[3].replace(batch=2, prefix=1000), seed=77, poison=True)
    d = DeviceInputs(inp)
    ref_out, ref_lse = oracle.verify_attention(inp)
    outs = []
    for chunk in (64, 192, 1024, -1, 0, 0):
        out, lse = run_attention(d, chunk)
        check_attention(out, lse, ref_out, ref_lse, "bf16")
        outs.append((out, lse))
    np.testing.assert_array_equal(outs[-1][0], outs[-2][0])   # same launch: same bits
    np.testing.assert_array_equal(outs[-1][1], outs[-2][1])
    ref = oracle_accept(inp)
    for cpr in (1, 3, 17, 0):
        check_accept(run_accept(d, cpr), ref)


def test_optional_outputs_null():
    """lse, confidence and draft_prob are optional (NULL): the other outputs
    are unchanged, with one split and with several (the merge kernel)."""
    import ctypes
    from paper_2606_02544_amd import binding
    from gpu_util import dev_tensor
    inp = generate(CONFIGS[3].replace(batch=2, prefix=700), seed=91, poison=True)
    d = DeviceInputs(inp)
    cfg = inp.cfg
    for chunk in (1024, 128, -1):
        ref_out, _ = run_attention(d, chunk)
        out, lse = binding.verify_attention(
            d.q, d.k_new, d.v_new, d.k_cache, d.v_cache, d.block_table, d.prefix_lens,
            d.step_map, d.num_ref, block_size=cfg.block_size, max_ref=cfg.max_ref,
            max_prefix_len=cfg.max_prefix, page_size=cfg.page_size, kv_chunk=chunk,
            want_lse=False)
        torch.cuda.synchronize()
        assert lse is None
        np.testing.assert_array_equal(out.float().cpu().double().numpy(), ref_out)
    t_ref, _, _, a_ref = run_accept(d)
    b, B = cfg.batch, cfg.block_size
    tid = torch.empty((b, B), dtype=torch.int32, device="cuda")
    alen = torch.empty((b,), dtype=torch.int32, device="cuda")
    desc = binding.accept_desc(d.logits, cfg.max_ref)
    ws = torch.zeros(max(binding.accept_workspace_size(desc), 16), dtype=torch.uint8, device="cuda")
    P = lambda t: ctypes.c_void_p(t.data_ptr())
    st = binding.lib().simsd_verify_accept(
        ctypes.byref(desc), P(d.logits), P(d.draft_ids), P(d.step_map), P(d.num_ref), P(tid),
        None, None, P(alen), P(ws), ws.numel(), None)
    torch.cuda.synchronize()
    assert st == 0, binding.lib().simsd_last_error()
    np.testing.assert_array_equal(tid.cpu().numpy(), t_ref)
    np.testing.assert_array_equal(alen.cpu().numpy(), a_ref)


def test_workspace_reuse_many_launches():
    """Repeated launches sharing one workspace keep producing the same bits."""
    inp = generate(CONFIGS[2], seed=5)
    d = DeviceInputs(inp)
    first = run_attention(d, 64)
    acc0 = run_accept(d, 0)
    for _ in range(20):
        out, lse = run_attention(d, 64)
        np.testing.assert_array_equal(out, first[0])
        np.testing.assert_array_equal(lse, first[1])
        acc = run_accept(d, 0)
        np.testing.assert_array_equal(acc[0], acc0[0])
        np.testing.assert_array_equal(acc[3], acc0[3])


def _accept_case(logits, drafts, step, gamma, dtype, cprs=(0, 1, 2, 5)):
    from synth import bf16_bits_from_f32
    x = logits.astype(np.float32)
    stored = bf16_bits_from_f32(x) if dtype == "bf16" else x
    ref = oracle.verify_accept(stored, drafts, step, gamma, dtype)
    from gpu_util import dev_tensor, int_tensor
    from paper_2606_02544_amd import binding
    for cpr in cprs:
        got = binding.verify_accept(dev_tensor(stored, dtype), int_tensor(drafts),
                                    int_tensor(step), int_tensor(gamma), chunks_per_row=cpr)
        torch.cuda.synchronize()
        got = tuple(t.cpu().numpy().astype(np.float64) if t.dtype == torch.float32
                    else t.cpu().numpy() for t in got)
        check_accept(got, ref)
    return ref


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("V", [5, 8, 1003, 4096, 151936])
def test_accept_ties_zeros_and_bad_drafts(dtype, V):
    rng = np.random.default_rng(V)
    b, B, L = 3, 6, 5
    x = np.round(rng.standard_normal((b, B, V)) * 4) / 4          # many exact ties
    x[0, 1, :] = -1.0
    x[0, 1, [V // 3, V - 1]] = 0.0                                # +0 / -0 tie
    x[0, 1, V - 1] = -0.0
    x[1, 2, :] = 3.0                                              # constant row
    x[2, 0, V - 1] = 50.0                                         # max in the last element
    step = np.array([[2, 1, 3, 4, 5, 0], [1, -1, 2, 0, 6, 3], [1, 2, 3, 4, 5, 6]], np.int32)
    gamma = np.array([5, 3, 0], np.int32)
    argmax = lambda s, k: int(np.argmax(x[s, k].astype(np.float32)))
    drafts = np.full((b, L), -1, np.int32)
    drafts[0] = [argmax(0, 1), argmax(0, 0), V, argmax(0, 3), -3]
    drafts[1, :3] = [argmax(1, 0), 0, argmax(1, 5)]
    ref = _accept_case(x, drafts, step, gamma, dtype)
    assert ref[3][2] == 0


def test_accept_bench_shape_chunking():
    inp = generate(CONFIGS[2], seed=11)
    d = DeviceInputs(inp)
    ref = oracle_accept(inp)
    for cpr in (1, 7, 64, 600, 1500, 0):     # 600, 1500: the long-row merge
        check_accept(run_accept(d, cpr), ref)


@pytest.mark.parametrize("kv_chunk", [128, -1])
def test_hip_graph_replays_match_eager(kv_chunk):
    """Both entry points captured in one HIP graph (the benchmark's timing
    mode), chunked and stream decompositions: every replay, with eager work and
    synchronisation in between, reproduces the eager outputs bit for bit."""
    from paper_2606_02544_amd import binding
    inp = generate(CONFIGS[3].replace(batch=2, prefix=700), seed=3, poison=True)
    d = DeviceInputs(inp)
    cfg = inp.cfg
    kw = dict(block_size=cfg.block_size, max_ref=cfg.max_ref, max_prefix_len=cfg.max_prefix,
              kv_chunk=kv_chunk)
    args = (d.q, d.k_new, d.v_new, d.k_cache, d.v_cache, d.block_table, d.prefix_lens,
            d.step_map, d.num_ref)
    eager_out, eager_lse = binding.verify_attention(*args, **kw)
    eager_acc = binding.verify_accept(d.logits, d.draft_ids, d.step_map, d.num_ref)
    torch.cuda.synchronize()
    out = torch.zeros_like(eager_out)
    lse = torch.zeros_like(eager_lse)
    acc = [torch.zeros_like(t) for t in eager_acc]
    s = torch.cuda.Stream()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(s):
        binding.verify_attention(*args, out=out, lse=lse, stream=s, **kw)   # workspaces exist
        binding.verify_accept(d.logits, d.draft_ids, d.step_map, d.num_ref, target_ids=acc[0],
                              confidence=acc[1], draft_prob=acc[2], accept_len=acc[3], stream=s)
        torch.cuda.synchronize()
        with torch.cuda.graph(g, stream=s):
            binding.verify_attention(*args, out=out, lse=lse, stream=s, **kw)
            binding.verify_accept(d.logits, d.draft_ids, d.step_map, d.num_ref,
                                  target_ids=acc[0], confidence=acc[1], draft_prob=acc[2],
                                  accept_len=acc[3], stream=s)
    for rep in range(4):
        out.zero_()
        lse.zero_()
        for t in acc:
            t.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, eager_out) and torch.equal(lse, eager_lse), rep
        for a, b in zip(acc, eager_acc):
            assert torch.equal(a, b), rep
        binding.verify_attention(*args, **kw)       # eager work between replays
        torch.cuda.synchronize()
