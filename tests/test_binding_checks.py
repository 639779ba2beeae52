"""The Python binding rejects tensors whose shape, dtype, device or layout the
C library cannot see, before any call (CPU; no kernel is launched: every case
raises ValueError in the checks that precede the library call)."""

import pytest
import torch

from paper_2606_02544_amd import binding

BF = torch.bfloat16


def attn_args(b=2, B=4, L=4, hq=8, hkv=2, d=64, cap=100, paged=False, dtype=BF):
    n = B + L
    a = dict(q=torch.zeros(b, n, hq, d, dtype=dtype), k_new=torch.zeros(b, n, hkv, d, dtype=dtype),
             v_new=torch.zeros(b, n, hkv, d, dtype=dtype),
             prefix_lens=torch.zeros(b, dtype=torch.int32),
             step_map=torch.zeros(b, B, dtype=torch.int32), num_ref=torch.zeros(b, dtype=torch.int32))
    if paged:
        a["k_cache"] = torch.zeros(20, 16, hkv, d, dtype=dtype)
        a["v_cache"] = torch.zeros(20, 16, hkv, d, dtype=dtype)
        a["block_table"] = torch.zeros(b, 7, dtype=torch.int32)
    else:
        a["k_cache"] = torch.zeros(b, cap, hkv, d, dtype=dtype)
        a["v_cache"] = torch.zeros(b, cap, hkv, d, dtype=dtype)
        a["block_table"] = None
    kw = dict(block_size=B, max_ref=L, max_prefix_len=100, page_size=16 if paged else 0)
    return a, kw


def check(a, kw, out=None, lse=None):
    return binding.check_attention_tensors(
        a["q"], a["k_new"], a["v_new"], a["k_cache"], a["v_cache"], a["block_table"],
        a["prefix_lens"], a["step_map"], a["num_ref"], out, lse, **kw)


def call(a, kw, **extra):
    return binding.verify_attention(a["q"], a["k_new"], a["v_new"], a["k_cache"], a["v_cache"],
                                    a["block_table"], a["prefix_lens"], a["step_map"],
                                    a["num_ref"], **kw, **extra)


def test_valid_arguments_pass_the_checks():
    for paged in (False, True):
        a, kw = attn_args(paged=paged)
        assert check(a, kw) == 2
    a, kw = attn_args(dtype=torch.float32)
    assert check(a, kw, out=torch.zeros_like(a["q"]), lse=torch.zeros(2, 8, 8)) == 2


@pytest.mark.parametrize("mutate,match", [
    (lambda a: a.update(q=a["q"].transpose(2, 3).contiguous().transpose(2, 3)), "q must be contiguous"),
    (lambda a: a.update(k_new=a["k_new"].float()), "k_new must be torch.bfloat16"),
    (lambda a: a.update(v_new=a["v_new"][:, :7]), "v_new has shape"),
    (lambda a: a.update(k_cache=a["k_cache"].float()), "k_cache must be torch.bfloat16"),
    (lambda a: a.update(v_cache=torch.zeros(2, 100, 64, 2, dtype=BF).transpose(2, 3)),
     "v_cache must have a unit stride"),
    (lambda a: a.update(v_cache=torch.zeros(2, 120, 2, 64, dtype=BF)[:, :100]),
     "strides differ"),
    (lambda a: a.update(k_cache=torch.zeros(2, 50, 2, 64, dtype=BF),
                        v_cache=torch.zeros(2, 50, 2, 64, dtype=BF)), "holds 50 tokens"),
    (lambda a: a.update(k_cache=torch.zeros(2, 100, 4, 64, dtype=BF)), "need \\[\\*, \\*, 2, 64\\]"),
    (lambda a: a.update(k_cache=torch.zeros(3, 100, 2, 64, dtype=BF),
                        v_cache=torch.zeros(3, 100, 2, 64, dtype=BF)), "dimension 0 is 3"),
    (lambda a: a.update(step_map=torch.zeros(2, 5, dtype=torch.int32)), "step_map has shape"),
    (lambda a: a.update(step_map=torch.zeros(2, 4, dtype=torch.int64)), "step_map must be torch.int32"),
    (lambda a: a.update(num_ref=torch.zeros(3, dtype=torch.int32)), "num_ref has shape"),
    (lambda a: a.update(prefix_lens=torch.zeros(4, dtype=torch.int32)[::2]),
     "prefix_lens must be contiguous"),
    (lambda a: a.update(q=torch.zeros(2, 8, 8, 64, dtype=torch.float16)), "q must be bfloat16 or float32"),
])
def test_attention_rejections(mutate, match):
    a, kw = attn_args()
    mutate(a)
    with pytest.raises(ValueError, match=match):
        call(a, kw)


def test_attention_slot_count_and_outputs():
    a, kw = attn_args()
    with pytest.raises(ValueError, match="block_size \\+ max_ref"):
        call(a, dict(kw, max_ref=3))
    with pytest.raises(ValueError, match="out must be torch.bfloat16"):
        call(a, kw, out=torch.zeros(2, 8, 8, 64))
    with pytest.raises(ValueError, match="out must be contiguous"):
        call(a, kw, out=torch.zeros(2, 8, 64, 8, dtype=BF).transpose(2, 3))
    with pytest.raises(ValueError, match="lse has shape"):
        call(a, kw, lse=torch.zeros(2, 8, 9))


def test_paged_cache_rejections():
    a, kw = attn_args(paged=True)
    with pytest.raises(ValueError, match="needs a block_table"):
        call(dict(a, block_table=None), kw)
    with pytest.raises(ValueError, match="too few pages"):
        call(dict(a, block_table=torch.zeros(2, 6, dtype=torch.int32)), kw)
    with pytest.raises(ValueError, match="page_size is 8"):
        call(a, dict(kw, page_size=8))
    with pytest.raises(ValueError, match="block_table must be torch.int32"):
        call(dict(a, block_table=torch.zeros(2, 7, dtype=torch.int64)), kw)


def accept_args(b=2, B=4, L=3, V=100):
    return (torch.zeros(b, B, V, dtype=BF), torch.zeros(b, L, dtype=torch.int32),
            torch.zeros(b, B, dtype=torch.int32), torch.zeros(b, dtype=torch.int32))


def test_accept_rejections():
    logits, ids, sm, nr = accept_args()
    with pytest.raises(ValueError, match="logits must be contiguous"):
        binding.verify_accept(logits.transpose(0, 1).contiguous().transpose(0, 1), ids, sm, nr)
    with pytest.raises(ValueError, match="draft_ids must be torch.int32"):
        binding.verify_accept(logits, ids.long(), sm, nr)
    with pytest.raises(ValueError, match="step_map has shape"):
        binding.verify_accept(logits, ids, sm[:, :3].contiguous(), nr)
    with pytest.raises(ValueError, match="target_ids has shape"):
        binding.verify_accept(logits, ids, sm, nr, target_ids=torch.zeros(2, 3, dtype=torch.int32))
    with pytest.raises(ValueError, match="draft_prob must be torch.float32"):
        binding.verify_accept(logits, ids, sm, nr, draft_prob=torch.zeros(2, 3, dtype=BF))
    with pytest.raises(ValueError, match="logits must be bfloat16 or float32"):
        binding.verify_accept(logits.half(), ids, sm, nr)


def test_accept_sampled_rejections():
    logits, ids, sm, nr = accept_args()
    dl = torch.zeros(2, 3, 100, dtype=BF)
    u = torch.zeros(2, 4)
    with pytest.raises(ValueError, match="draft_logits has shape"):
        binding.verify_accept_sampled(logits, dl[:, :2].contiguous(), ids, sm, nr, u)
    with pytest.raises(ValueError, match="draft_logits must be torch.bfloat16"):
        binding.verify_accept_sampled(logits, dl.float(), ids, sm, nr, u)
    with pytest.raises(ValueError, match="uniforms has shape"):
        binding.verify_accept_sampled(logits, dl, ids, sm, nr, torch.zeros(2, 3))
    with pytest.raises(ValueError, match="correction has shape"):
        binding.verify_accept_sampled(logits, dl, ids, sm, nr, u,
                                      correction=torch.zeros(3, dtype=torch.int32))


def test_lmhead_rejections():
    hidden = torch.zeros(2, 4, 128, dtype=BF)
    weight = torch.zeros(1000, 128, dtype=BF)
    ids, sm, nr = (torch.zeros(2, 3, dtype=torch.int32), torch.zeros(2, 4, dtype=torch.int32),
                   torch.zeros(2, dtype=torch.int32))
    with pytest.raises(ValueError, match="weight has shape"):
        binding.verify_accept_lmhead(hidden, torch.zeros(1000, 64, dtype=BF), ids, sm, nr)
    with pytest.raises(ValueError, match="weight must be contiguous"):
        binding.verify_accept_lmhead(hidden, torch.zeros(128, 1000, dtype=BF).t(), ids, sm, nr)
    with pytest.raises(ValueError, match="hidden must be torch.bfloat16"):
        binding.verify_accept_lmhead(hidden.float(), weight, ids, sm, nr)
    with pytest.raises(ValueError, match="weight must be torch.bfloat16"):
        binding.verify_accept_lmhead(hidden, weight.float(), ids, sm, nr)
    with pytest.raises(ValueError, match="num_ref has shape"):
        binding.verify_accept_lmhead(hidden, weight, ids, sm, torch.zeros(1, dtype=torch.int32))
    with pytest.raises(ValueError, match="must be a 3-D tensor"):
        binding.verify_accept_lmhead(hidden[0], weight, ids, sm, nr)


def test_workspace_cache_keyed_by_stream_and_grown_buffers_kept():
    ws = binding._Workspaces()
    cpu = torch.device("cpu")
    a = ws.get(cpu, 1, "attn", 100)
    b = ws.get(cpu, 2, "attn", 100)
    assert a.data_ptr() != b.data_ptr()               # other stream: other buffer
    assert ws.get(cpu, 1, "attn", 64) is a            # fits: reused
    c = ws.get(cpu, 1, "attn", 1000)                  # grows: a new buffer ...
    assert c is not a and c.numel() >= 1000
    assert any(r is a for r in ws._retired)           # ... and the old one stays alive
    assert ws.get(cpu, 1, "accept", 10) is not c      # other kind: other buffer
    assert ws.get(cpu, 1, "attn", 0) is None
    ws.clear()
    assert not ws._retired
