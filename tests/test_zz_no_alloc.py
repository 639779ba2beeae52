"""GPU: the allocation-free accept entry point (simsd_verify_accept_noalloc)
through the C ABI against simsd_verify_accept with a workspace, on two calls in
a row (the second with a smaller input) and on a second stream: the outputs are
the same bits, and both match the oracle.  Also captured in a HIP graph, with
eager calls on other inputs between the replays."""

import ctypes

import numpy as np
import pytest
import torch

from gpu_util import DeviceInputs, check_accept, oracle_accept
from synth import CONFIGS, VerifyConfig, generate

pytestmark = pytest.mark.gpu


def _noalloc(d, stream=None):
    from paper_2606_02544_amd import binding
    lib = binding.lib()
    b, B = d.step_map.shape
    L = d.draft_ids.shape[1]
    outs = (torch.full((b, B), -7, dtype=torch.int32, device="cuda"),
            torch.full((b, B), -7.0, dtype=torch.float32, device="cuda"),
            torch.full((b, L), -7.0, dtype=torch.float32, device="cuda"),
            torch.full((b,), -7, dtype=torch.int32, device="cuda"))
    desc = binding.accept_desc(d.logits, L)
    P = lambda t: ctypes.c_void_p(t.data_ptr())
    s = stream if stream is not None else torch.cuda.current_stream()
    st = lib.simsd_verify_accept_noalloc(ctypes.byref(desc), P(d.logits), P(d.draft_ids),
                                         P(d.step_map), P(d.num_ref), *map(P, outs),
                                         ctypes.c_void_p(s.cuda_stream))
    assert st == 0, lib.simsd_last_error().decode()
    s.synchronize()
    return outs


def _with_workspace(d):
    from paper_2606_02544_amd import binding
    outs = binding.verify_accept(d.logits, d.draft_ids, d.step_map, d.num_ref)
    torch.cuda.synchronize()
    return outs


def _same(a, b):
    for x, y in zip(a, b):
        assert torch.equal(x, y)


def _host(outs):
    return tuple(t.cpu().numpy().astype(np.float64) if t.dtype == torch.float32
                 else t.cpu().numpy() for t in outs)


def test_noalloc_matches_workspace_entry_point():
    big = generate(CONFIGS[5].replace(prefix=(16, 32)), seed=7)      # 512 rows, V 151936
    small = generate(VerifyConfig(0, "small", "f32", batch=3, num_q_heads=2, num_kv_heads=1,
                                  head_dim=64, prefix=8, block_size=6, max_ref=4, vocab=1003,
                                  step_mode="mixed"), seed=8, bad_draft_rate=0.3)
    for inp in (big, small):                  # two calls in a row, the second smaller
        d = DeviceInputs(inp)
        got = _noalloc(d)
        _same(got, _with_workspace(d))
        check_accept(_host(got), oracle_accept(inp))
    # again on another stream, after the smaller call left its partials behind
    d = DeviceInputs(big)
    s = torch.cuda.Stream()
    _same(_noalloc(d, s), _with_workspace(d))


def test_noalloc_in_a_captured_graph():
    """The allocation-free accept captured in a HIP graph (its callers include
    code under graph capture): every replay reproduces the eager outputs bit
    for bit, also after eager calls on another input have overwritten the
    shared scratch in between."""
    from paper_2606_02544_amd import binding
    a = DeviceInputs(generate(CONFIGS[3].replace(batch=2, prefix=64), seed=21))
    other = DeviceInputs(generate(VerifyConfig(0, "other", "bf16", batch=4, num_q_heads=2,
                                               num_kv_heads=1, head_dim=64, prefix=8,
                                               block_size=8, max_ref=8, vocab=5003,
                                               step_mode="mixed"), seed=22))
    eager = binding.verify_accept_noalloc(a.logits, a.draft_ids, a.step_map, a.num_ref)
    torch.cuda.synchronize()
    outs = [torch.zeros_like(t) for t in eager]
    kw = dict(target_ids=outs[0], confidence=outs[1], draft_prob=outs[2], accept_len=outs[3])
    s = torch.cuda.Stream()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(s):
        binding.verify_accept_noalloc(a.logits, a.draft_ids, a.step_map, a.num_ref, stream=s, **kw)
        torch.cuda.synchronize()
        with torch.cuda.graph(g, stream=s):
            binding.verify_accept_noalloc(a.logits, a.draft_ids, a.step_map, a.num_ref,
                                          stream=s, **kw)
    for rep in range(4):
        for t in outs:
            t.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        _same(outs, eager)
        # eager work on another input between replays, through the same scratch
        binding.verify_accept_noalloc(other.logits, other.draft_ids, other.step_map,
                                      other.num_ref)
        torch.cuda.synchronize()


def test_noalloc_refuses_oversized_shapes():
    from paper_2606_02544_amd import binding
    lib = binding.lib()
    t = torch.zeros(16, dtype=torch.int32, device="cuda")
    P = ctypes.c_void_p(t.data_ptr())
    desc = binding.AcceptDesc(batch=65535, block_size=64, max_ref=64, vocab=1000,
                              chunks_per_row=0, logits_dtype=binding.SIMSD_BF16)
    st = lib.simsd_verify_accept_noalloc(ctypes.byref(desc), P, P, P, P, P, None, None, P, None)
    assert st == 5, st                        # refused on the host, nothing enqueued
    assert "scratch" in lib.simsd_last_error().decode()
