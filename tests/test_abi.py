"""The C ABI on the CPU: the library loads, exports every declared symbol,
sizes workspaces, and rejects bad arguments before any device work.

Every compute call made here fails host validation, so no kernel is ever
launched (pointer values are small aligned fakes that are never dereferenced)."""

import ctypes
import os
import re

import numpy as np
import pytest

from paper_2606_02544_amd import binding
from paper_2606_02544_amd.binding import LmheadDesc, AttnDesc, AcceptDesc

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "simsd.h")

FAKE = ctypes.c_void_p(0x10000)     # aligned, never dereferenced


def _no_gpu():
    """The fake-pointer calls below must fail host validation; as a second
    guard they only run where no GPU is visible, so a validation bug can never
    launch a kernel on bogus pointers."""
    import torch
    if torch.cuda.is_available():
        pytest.skip("host-validation tests run only without a visible GPU")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(simsd_[a-z_]+)\s*\(", text)))


def test_exports_every_declared_symbol():
    lib = binding.lib()
    names = declared_functions()
    assert len(names) >= 8
    for n in names:
        assert hasattr(lib, n), n
    assert lib.simsd_version() == 100


def test_missing_library_fails_loudly(monkeypatch):
    monkeypatch.setattr(binding, "_lib", None)
    monkeypatch.setattr(binding, "LIB_PATH", "/nonexistent/libsimsd.so")
    with pytest.raises(RuntimeError, match="missing"):
        binding.lib()


def cfg_desc(cid, **kw):
    from synth import CONFIGS
    c = CONFIGS[cid]
    d = c.head_dim
    if c.page_size:
        strides = (c.page_size * c.num_kv_heads * d, c.num_kv_heads * d, d)
        pages = -(-c.max_prefix // c.page_size)
    else:
        strides = (c.max_prefix * c.num_kv_heads * d, c.num_kv_heads * d, d)
        pages = 0
    base = dict(batch=c.batch, num_q_heads=c.num_q_heads, num_kv_heads=c.num_kv_heads,
                head_dim=d, block_size=c.block_size, max_ref=c.max_ref,
                max_prefix_len=c.max_prefix, page_size=c.page_size, max_pages_per_seq=pages,
                kv_chunk=0, cache_stride_seq=strides[0], cache_stride_token=strides[1],
                cache_stride_head=strides[2], scale=0.0,
                dtype=binding.SIMSD_F32 if c.dtype == "f32" else binding.SIMSD_BF16)
    base.update(kw)
    return AttnDesc(**base)


def test_workspace_sizes_follow_the_plan():
    # config 4: 16 x 8 pairs, 256 packed rows in 8 waves -> chunk 8192 -> 2 splits;
    # 128 * 2 partials of 256 rows x (128 + 2) floats.
    assert binding.attention_workspace_size(cfg_desc(4)) == 128 * 2 * 256 * 130 * 4
    assert binding.attention_workspace_size(cfg_desc(4, kv_chunk=4096)) == 128 * 4 * 256 * 130 * 4
    # a single split needs no workspace
    assert binding.attention_workspace_size(cfg_desc(1, kv_chunk=64)) == 0
    assert binding.attention_workspace_size(cfg_desc(2)) > 0
    assert binding.attention_workspace_size(cfg_desc(1, head_dim=96)) == 0   # invalid -> 0
    # stream decomposition (kv_chunk -1): two partial slots per resident group
    # plus 257 int64 sequence offsets; config 2 packs 128 rows -> 8 waves, 256 groups
    assert binding.attention_workspace_size(cfg_desc(2, kv_chunk=-1)) == \
        256 * 2 * 128 * 130 * 4 + 257 * 8
    assert binding.attention_workspace_size(cfg_desc(2, kv_chunk=-1, dtype=binding.SIMSD_F32)) == 0
    assert binding.attention_workspace_size(cfg_desc(4, kv_chunk=-1)) == 0   # 256 rows: no stream
    acc = AcceptDesc(batch=16, block_size=32, max_ref=32, vocab=151936, chunks_per_row=0,
                     logits_dtype=binding.SIMSD_BF16)
    # 512 rows -> 1 chunk per row (about 512 scan work-groups); 16-byte partials
    assert binding.accept_workspace_size(acc) == 512 * 1 * 16


def call_attention(desc, **over):
    _no_gpu()
    args = dict(q=FAKE, k_new=FAKE, v_new=FAKE, k_cache=FAKE, v_cache=FAKE, block_table=FAKE,
                prefix_lens=FAKE, step_map=FAKE, num_ref=FAKE, out=FAKE, lse=None,
                workspace=None, ws_bytes=0)
    args.update(over)
    lib = binding.lib()
    st = lib.simsd_verify_attention(ctypes.byref(desc), args["q"], args["k_new"], args["v_new"],
                                    args["k_cache"], args["v_cache"], args["block_table"],
                                    args["prefix_lens"], args["step_map"], args["num_ref"],
                                    args["out"], args["lse"], args["workspace"],
                                    args["ws_bytes"], None)
    return st, lib.simsd_last_error().decode()


@pytest.mark.parametrize("field,value,status", [
    ("head_dim", 96, 3), ("head_dim", 256, 3), ("num_q_heads", 6, 2), ("num_kv_heads", 0, 2),
    ("num_q_heads", 136, 3), ("block_size", 0, 2), ("max_ref", 5, 2), ("block_size", 40, 2),
    ("batch", 0, 2), ("batch", 70000, 2), ("max_prefix_len", -1, 2), ("kv_chunk", 100, 2),
    ("kv_chunk", -64, 2), ("kv_chunk", -2, 2), ("page_size", -2, 2),
    ("stream_f32", -1, 3), ("stream_batch", -1, 3), ("stream_rows", -1, 3), ("cache_stride_token", 12, 4),
    ("cache_stride_head", -8, 2), ("scale", -1.0, 2), ("scale", float("inf"), 2),
    ("dtype", 7, 3), ("rope_theta", -1.0, 2), ("rope_theta", float("nan"), 2),
    ("rope_theta", float("inf"), 2),
])
def test_attention_descriptor_errors(field, value, status):
    desc = cfg_desc(2)
    if field == "block_size" and value == 40:
        desc.max_ref = 30                  # B + L = 70 > 64
    if field.startswith("stream_"):        # kv_chunk -1 outside what it supports
        desc.kv_chunk = value
        if field == "stream_f32":
            desc.dtype = binding.SIMSD_F32
        elif field == "stream_batch":
            desc.batch = 257
        else:
            desc = cfg_desc(4, kv_chunk=value)       # 256 packed rows
    else:
        setattr(desc, field, value)
    st, msg = call_attention(desc, workspace=FAKE, ws_bytes=1 << 40)
    assert st == status, (st, msg)
    assert msg


def test_attention_pointer_alignment_and_workspace_errors():
    desc = cfg_desc(2, kv_chunk=64)          # needs a workspace
    ws = binding.attention_workspace_size(desc)
    assert call_attention(desc, q=None, workspace=FAKE, ws_bytes=ws)[0] == 1
    assert call_attention(desc, k_cache=None, workspace=FAKE, ws_bytes=ws)[0] == 1
    assert call_attention(desc, out=ctypes.c_void_p(0x10008), workspace=FAKE, ws_bytes=ws)[0] == 4
    assert call_attention(desc, lse=ctypes.c_void_p(0x10002), workspace=FAKE, ws_bytes=ws)[0] == 4
    assert call_attention(desc, workspace=None, ws_bytes=0)[0] == 5
    assert call_attention(desc, workspace=FAKE, ws_bytes=ws - 1)[0] == 5
    paged = cfg_desc(5)
    assert call_attention(paged, block_table=None,
                          workspace=FAKE, ws_bytes=1 << 40)[0] == 1
    paged.max_pages_per_seq = 3
    assert call_attention(paged, workspace=FAKE, ws_bytes=1 << 40)[0] == 2


def call_accept(desc, **over):
    _no_gpu()
    a = dict(logits=FAKE, draft_ids=FAKE, step_map=FAKE, num_ref=FAKE, target_ids=FAKE,
             confidence=None, draft_prob=None, accept_len=FAKE, workspace=FAKE, ws=1 << 30)
    a.update(over)
    lib = binding.lib()
    return lib.simsd_verify_accept(ctypes.byref(desc), a["logits"], a["draft_ids"],
                                   a["step_map"], a["num_ref"], a["target_ids"],
                                   a["confidence"], a["draft_prob"], a["accept_len"],
                                   a["workspace"], a["ws"], None)


def test_accept_errors():
    good = dict(batch=2, block_size=4, max_ref=4, vocab=1000, chunks_per_row=0,
                logits_dtype=binding.SIMSD_BF16)
    for k, v, st in [("batch", 0, 2), ("block_size", 65, 2), ("max_ref", 5, 2),
                     ("vocab", 0, 2), ("chunks_per_row", -1, 2), ("logits_dtype", 3, 3)]:
        d = AcceptDesc(**dict(good, **{k: v}))
        assert call_accept(d) == st, k
    d = AcceptDesc(**good)
    assert call_accept(d, logits=None) == 1
    assert call_accept(d, draft_ids=None) == 1
    assert call_accept(d, logits=ctypes.c_void_p(0x10004)) == 4
    assert call_accept(d, workspace=None) == 5
    assert call_accept(d, ws=binding.accept_workspace_size(d) - 1) == 5


def call_accept_sampled(desc, temperature=1.0, **over):
    _no_gpu()
    a = dict(logits=FAKE, draft_logits=FAKE, draft_ids=FAKE, step_map=FAKE, num_ref=FAKE,
             uniforms=FAKE, p_target=None, p_draft=None, accept_len=FAKE, correction=FAKE,
             workspace=FAKE, ws=1 << 30)
    a.update(over)
    lib = binding.lib()
    return lib.simsd_verify_accept_sampled(
        ctypes.byref(desc), ctypes.c_float(temperature), a["logits"], a["draft_logits"],
        a["draft_ids"], a["step_map"], a["num_ref"], a["uniforms"], a["p_target"], a["p_draft"],
        a["accept_len"], a["correction"], a["workspace"], a["ws"], None)


def test_accept_sampled_errors_and_workspace():
    good = dict(batch=2, block_size=4, max_ref=4, vocab=1000, chunks_per_row=0,
                logits_dtype=binding.SIMSD_BF16)
    d = AcceptDesc(**good)
    # the scan covers B verification rows and L draft rows per sequence (16-byte
    # partials), then 256-byte alignment, one 32-byte draw row per sequence and
    # 16-byte draw partials per vocabulary chunk (V = 1000: one chunk)
    rows = 2 * 8 * d_cpr(d, 8) * 16
    assert binding.accept_sampled_workspace_size(d) == -(-rows // 256) * 256 + 2 * 32 + 2 * 1 * 16
    big = AcceptDesc(batch=16, block_size=32, max_ref=32, vocab=151936, chunks_per_row=0,
                     logits_dtype=binding.SIMSD_BF16)
    # 1024 scanned rows -> 1 chunk each; 32 draw chunks per sequence (about 512 groups)
    assert binding.accept_sampled_workspace_size(big) == 16 * 64 * 16 + 16 * 32 + 16 * 32 * 16
    for k, v, st in [("batch", 0, 2), ("max_ref", 5, 2), ("vocab", 0, 2), ("logits_dtype", 3, 3)]:
        assert call_accept_sampled(AcceptDesc(**dict(good, **{k: v}))) == st, k
    for t in (0.0, -1.0, float("inf"), float("nan")):
        assert call_accept_sampled(d, temperature=t) == 2, t
    for k in ("logits", "draft_logits", "draft_ids", "step_map", "num_ref", "uniforms",
              "accept_len", "correction"):
        assert call_accept_sampled(d, **{k: None}) == 1, k
    assert call_accept_sampled(d, draft_logits=ctypes.c_void_p(0x10008)) == 4
    assert call_accept_sampled(d, workspace=None) == 5
    assert call_accept_sampled(d, ws=binding.accept_sampled_workspace_size(d) - 1) == 5
    # with L = 0 the draft inputs may be NULL
    d0 = AcceptDesc(**dict(good, max_ref=0))
    assert call_accept_sampled(d0, draft_logits=None, draft_ids=None, ws=0) in (0, 5)


def call_lmhead(desc, **over):
    _no_gpu()
    a = dict(hidden=FAKE, weight=FAKE, draft_ids=FAKE, step_map=FAKE, num_ref=FAKE,
             target_ids=FAKE, confidence=None, draft_prob=None, accept_len=FAKE, workspace=FAKE,
             ws=1 << 30)
    a.update(over)
    return binding.lib().simsd_verify_accept_lmhead(
        ctypes.byref(desc), a["hidden"], a["weight"], a["draft_ids"], a["step_map"], a["num_ref"],
        a["target_ids"], a["confidence"], a["draft_prob"], a["accept_len"], a["workspace"], a["ws"],
        None)


def test_lmhead_errors_and_workspace():
    good = dict(batch=2, block_size=4, max_ref=4, vocab=1000, hidden=128, dtype=binding.SIMSD_BF16)
    d = LmheadDesc(**good)
    # one 16-byte partial per (row, vocabulary tile: 128 entries up to 32 rows, else 256),
    # 256-byte alignment, the merged partial of each row, alignment, then one float per
    # draft slot
    R, vt = 2 * 4, -(-1000 // 128)
    merged_off = -(-(R * vt * 16) // 256) * 256
    xdraft_off = -(-(merged_off + R * 16) // 256) * 256
    assert binding.lmhead_workspace_size(d) == xdraft_off + 2 * 4 * 4
    big = LmheadDesc(**dict(good, batch=16, block_size=32, max_ref=32, vocab=151936))
    R, vt = 16 * 32, -(-151936 // 256)
    merged_off = -(-(R * vt * 16) // 256) * 256
    xdraft_off = -(-(merged_off + R * 16) // 256) * 256
    assert binding.lmhead_workspace_size(big) == xdraft_off + 16 * 32 * 4
    for k, v, st in [("batch", 0, 2), ("block_size", 65, 2), ("max_ref", 5, 2), ("vocab", 0, 2),
                     ("hidden", 0, 2), ("hidden", 96, 2), ("dtype", binding.SIMSD_F32, 3)]:
        bad = LmheadDesc(**dict(good, **{k: v}))
        assert call_lmhead(bad) == st, (k, v)
        assert binding.lib().simsd_verify_accept_lmhead_workspace_size(ctypes.byref(bad)) == 0
    for k in ("hidden", "weight", "step_map", "num_ref", "target_ids", "accept_len", "draft_ids"):
        assert call_lmhead(d, **{k: None}) == 1, k
    assert call_lmhead(d, hidden=ctypes.c_void_p(0x10008)) == 4
    assert call_lmhead(d, weight=ctypes.c_void_p(0x10004)) == 4
    assert call_lmhead(d, workspace=None) == 5
    assert call_lmhead(d, workspace=ctypes.c_void_p(0x10008)) == 4
    assert call_lmhead(d, ws=binding.lmhead_workspace_size(d) - 1) == 5


def d_cpr(desc, rows_per_seq):
    """Chunks per row the plan picks: about 512 scan work-groups, at least 256
    vectors per chunk."""
    vec = 8 if desc.vocab % 8 == 0 else 1
    nvec = -(-desc.vocab // vec)
    cpr = -(-512 // (desc.batch * rows_per_seq))
    return max(1, min(cpr, max(1, nvec // 256), nvec))


def test_validate_step_map():
    ok = np.array([[2, 1, 0, -1, 9], [1, 2, 3, 4, 5]])
    binding.validate_step_map(ok, [2, 5], max_ref=5)
    for sm, nr in [([[1, 1, 0, 0, 0]], [2]), ([[2, 3, 0, 0, 0]], [2]), ([[1, 2, 0, 0, 0]], [6]),
                   ([[1, 0, 0, 0, 0]], [-1])]:
        with pytest.raises(binding.SimsdError) as e:
            binding.validate_step_map(np.array(sm), nr, max_ref=5)
        assert e.value.status == 6


def test_status_strings():
    lib = binding.lib()
    for code, name in binding.STATUS.items():
        assert lib.simsd_status_string(code).decode() == name


def call_accept_noalloc(desc, **over):
    _no_gpu()
    a = dict(logits=FAKE, draft_ids=FAKE, step_map=FAKE, num_ref=FAKE, target_ids=FAKE,
             confidence=None, draft_prob=None, accept_len=FAKE)
    a.update(over)
    lib = binding.lib()
    st = lib.simsd_verify_accept_noalloc(ctypes.byref(desc), a["logits"], a["draft_ids"],
                                         a["step_map"], a["num_ref"], a["target_ids"],
                                         a["confidence"], a["draft_prob"], a["accept_len"], None)
    return st, lib.simsd_last_error().decode()


def test_accept_noalloc_errors():
    """The allocation-free accept: argument errors as simsd_verify_accept, a
    shape whose partials exceed the fixed scratch is refused, and with no
    device visible a valid call reports the HIP error after validation."""
    good = dict(batch=2, block_size=4, max_ref=4, vocab=1000, chunks_per_row=0,
                logits_dtype=binding.SIMSD_BF16)
    for k, v, st in [("batch", 0, 2), ("block_size", 65, 2), ("vocab", 0, 2),
                     ("logits_dtype", 3, 3)]:
        assert call_accept_noalloc(AcceptDesc(**dict(good, **{k: v})))[0] == st, k
    d = AcceptDesc(**good)
    assert call_accept_noalloc(d, logits=None)[0] == 1
    assert call_accept_noalloc(d, draft_ids=None)[0] == 1
    assert call_accept_noalloc(d, logits=ctypes.c_void_p(0x10004))[0] == 4
    # 65535 x 64 rows of 16-byte partials: 64 MiB, beyond the 4 MiB scratch
    big = AcceptDesc(**dict(good, batch=65535, block_size=64, max_ref=64))
    st, msg = call_accept_noalloc(big)
    assert st == 5 and "scratch" in msg, msg
    # largest shape that fits: partials of 262144 rows of one chunk each
    fits = AcceptDesc(**dict(good, batch=4096, block_size=64, max_ref=64, vocab=151936))
    assert binding.accept_workspace_size(fits) <= binding.NOALLOC_SCRATCH_BYTES
    st, msg = call_accept_noalloc(fits)
    assert st == 7 and "device" in msg, msg
