"""ctypes binding of libsimsd.so: argument marshalling only.

Every computation runs in the HIP kernels behind the C ABI declared in
include/simsd.h.  torch is used for device memory (tensors, workspace) and for
the current HIP stream handle.  If the shared library is missing this module
raises at load time; there is no fallback path.
"""

from __future__ import annotations

import ctypes
import os
from typing import Optional

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libsimsd.so")

SIMSD_F32, SIMSD_BF16 = 0, 1
STATUS = {0: "SIMSD_OK", 1: "SIMSD_ERR_NULL_POINTER", 2: "SIMSD_ERR_BAD_SHAPE",
          3: "SIMSD_ERR_UNSUPPORTED", 4: "SIMSD_ERR_ALIGNMENT", 5: "SIMSD_ERR_WORKSPACE",
          6: "SIMSD_ERR_INVALID_STEP_MAP", 7: "SIMSD_ERR_HIP"}


class AttnDesc(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("num_q_heads", ctypes.c_int32),
                ("num_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("block_size", ctypes.c_int32), ("max_ref", ctypes.c_int32),
                ("max_prefix_len", ctypes.c_int32), ("page_size", ctypes.c_int32),
                ("max_pages_per_seq", ctypes.c_int32), ("kv_chunk", ctypes.c_int32),
                ("cache_stride_seq", ctypes.c_int64), ("cache_stride_token", ctypes.c_int64),
                ("cache_stride_head", ctypes.c_int64), ("scale", ctypes.c_float),
                ("dtype", ctypes.c_int), ("rope_theta", ctypes.c_float)]


class AcceptDesc(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("block_size", ctypes.c_int32),
                ("max_ref", ctypes.c_int32), ("vocab", ctypes.c_int32),
                ("chunks_per_row", ctypes.c_int32), ("logits_dtype", ctypes.c_int)]


class LmheadDesc(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("block_size", ctypes.c_int32),
                ("max_ref", ctypes.c_int32), ("vocab", ctypes.c_int32),
                ("hidden", ctypes.c_int32), ("dtype", ctypes.c_int)]


class SimsdError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS.get(status, status)}: {message}")
        self.status = status


_lib = None
_P = ctypes.c_void_p
_I32P = ctypes.POINTER(ctypes.c_int32)


def lib() -> ctypes.CDLL:
    """The loaded C library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build()")
        L = ctypes.CDLL(LIB_PATH)
        L.simsd_verify_attention_workspace_size.argtypes = [ctypes.POINTER(AttnDesc)]
        L.simsd_verify_attention_workspace_size.restype = ctypes.c_size_t
        L.simsd_verify_accept_workspace_size.argtypes = [ctypes.POINTER(AcceptDesc)]
        L.simsd_verify_accept_workspace_size.restype = ctypes.c_size_t
        L.simsd_verify_attention.argtypes = [ctypes.POINTER(AttnDesc)] + [_P] * 5 + [_P] * 4 + \
            [_P, _P, _P, ctypes.c_size_t, _P]
        L.simsd_verify_attention.restype = ctypes.c_int
        L.simsd_verify_accept.argtypes = [ctypes.POINTER(AcceptDesc)] + [_P] * 8 + \
            [_P, ctypes.c_size_t, _P]
        L.simsd_verify_accept.restype = ctypes.c_int
        L.simsd_verify_accept_noalloc.argtypes = [ctypes.POINTER(AcceptDesc)] + [_P] * 9
        L.simsd_verify_accept_noalloc.restype = ctypes.c_int
        L.simsd_verify_accept_sampled_workspace_size.argtypes = [ctypes.POINTER(AcceptDesc)]
        L.simsd_verify_accept_sampled_workspace_size.restype = ctypes.c_size_t
        L.simsd_verify_accept_sampled.argtypes = [ctypes.POINTER(AcceptDesc), ctypes.c_float] + \
            [_P] * 10 + [_P, ctypes.c_size_t, _P]
        L.simsd_verify_accept_sampled.restype = ctypes.c_int
        L.simsd_verify_accept_lmhead_workspace_size.argtypes = [ctypes.POINTER(LmheadDesc)]
        L.simsd_verify_accept_lmhead_workspace_size.restype = ctypes.c_size_t
        L.simsd_verify_accept_lmhead.argtypes = [ctypes.POINTER(LmheadDesc)] + [_P] * 9 + \
            [_P, ctypes.c_size_t, _P]
        L.simsd_verify_accept_lmhead.restype = ctypes.c_int
        L.simsd_validate_step_map.argtypes = [_I32P, _I32P, ctypes.c_int32, ctypes.c_int32,
                                              ctypes.c_int32]
        L.simsd_validate_step_map.restype = ctypes.c_int
        L.simsd_status_string.argtypes = [ctypes.c_int]
        L.simsd_status_string.restype = ctypes.c_char_p
        L.simsd_last_error.argtypes = []
        L.simsd_last_error.restype = ctypes.c_char_p
        L.simsd_version.argtypes = []
        L.simsd_version.restype = ctypes.c_int
        _lib = L
    return _lib


def _check(status: int):
    if status != 0:
        raise SimsdError(status, lib().simsd_last_error().decode())


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _dtype_code(dt: torch.dtype) -> int:
    if dt == torch.bfloat16:
        return SIMSD_BF16
    if dt == torch.float32:
        return SIMSD_F32
    raise ValueError(f"unsupported dtype {dt}")


def _stream_of(stream, device: torch.device):
    """The torch stream a call runs on: the given one, else the current stream
    of the tensors' device."""
    if stream is None:
        stream = torch.cuda.current_stream(device)
    return stream


# ----------------------------------------------------------------------------
# Argument checks.  The C library checks sizes, alignment and the workspace,
# but it only sees pointers: shapes, dtypes, strides and devices of the
# tensors are checked here, before any call, and raise ValueError.
# ----------------------------------------------------------------------------
def _need(cond: bool, msg: str):
    if not cond:
        raise ValueError(msg)


def _tensor(name: str, t, shape, dtype=None, device=None):
    """t is a contiguous tensor of the given shape (None entries: any size),
    dtype and device."""
    _need(isinstance(t, torch.Tensor), f"{name} must be a torch.Tensor")
    _need(t.dim() == len(shape), f"{name} must have {len(shape)} dimensions, got shape {tuple(t.shape)}")
    for i, n in enumerate(shape):
        _need(n is None or t.shape[i] == n,
              f"{name} has shape {tuple(t.shape)}, expected {tuple('*' if x is None else x for x in shape)}")
    if dtype is not None:
        _need(t.dtype == dtype, f"{name} must be {dtype}, got {t.dtype}")
    if device is not None:
        _need(t.device == device, f"{name} is on {t.device}, expected {device}")
    _need(t.is_contiguous(), f"{name} must be contiguous")


def _int32(name, t, shape, device):
    _tensor(name, t, shape, torch.int32, device)


def _out(name, t, shape, dtype, device):
    if t is not None:
        _tensor(name, t, shape, dtype, device)


def _check_cache(k_cache, v_cache, dtype, device, hkv, d, page_size, max_prefix_len,
                 batch, block_table):
    """k/v caches: same dtype as q, same shape and strides as each other, head
    dim innermost with stride 1 (other strides are passed to the library)."""
    for name, t in (("k_cache", k_cache), ("v_cache", v_cache)):
        _need(isinstance(t, torch.Tensor) and t.dim() == 4,
              f"{name} must be a 4-D tensor [seq or page, token, Hkv, d]")
        _need(t.dtype == dtype, f"{name} must be {dtype} (the dtype of q), got {t.dtype}")
        _need(t.device == device, f"{name} is on {t.device}, expected {device}")
        _need(t.shape[2] == hkv and t.shape[3] == d,
              f"{name} has shape {tuple(t.shape)}: need [*, *, {hkv}, {d}]")
        _need(t.stride(3) == 1, f"{name} must have a unit stride over the head dimension")
    _need(tuple(k_cache.shape) == tuple(v_cache.shape), "k_cache and v_cache shapes differ")
    _need(k_cache.stride() == v_cache.stride(), "k_cache and v_cache strides differ")
    if page_size > 0:
        _need(k_cache.shape[1] == page_size,
              f"paged cache: dimension 1 is {k_cache.shape[1]}, page_size is {page_size}")
        _need(block_table is not None, "paged cache needs a block_table")
        _int32("block_table", block_table, (batch, None), device)
        _need(block_table.shape[1] * page_size >= max_prefix_len,
              "block_table has too few pages per sequence for max_prefix_len")
    else:
        _need(k_cache.shape[0] == batch,
              f"contiguous cache: dimension 0 is {k_cache.shape[0]}, batch is {batch}")
        _need(k_cache.shape[1] >= max_prefix_len,
              f"contiguous cache holds {k_cache.shape[1]} tokens, max_prefix_len is {max_prefix_len}")


class _Workspaces:
    """Scratch buffers for the workspace argument, one per (device, stream,
    kind), grown on demand.  The library needs no initialised contents.

    Keyed by stream so that calls on different streams never share a buffer
    (they could overlap on the device).  A buffer that is replaced by a larger
    one is kept alive (in ``_retired``) rather than freed: a HIP graph captured
    earlier may still launch kernels on it, and freed memory would be handed
    to other tensors by the caching allocator.  ``clear()`` drops everything
    and is only safe once no captured graph that used these buffers will be
    replayed again."""

    def __init__(self):
        self._bufs = {}
        self._retired = []

    def get(self, device: torch.device, stream_handle: int, kind: str,
            nbytes: int) -> Optional[torch.Tensor]:
        if nbytes == 0:
            return None
        key = (str(device), int(stream_handle), kind)
        buf = self._bufs.get(key)
        if buf is None or buf.numel() < nbytes:
            if buf is not None:
                self._retired.append(buf)
            buf = torch.empty(nbytes, dtype=torch.uint8, device=device)
            self._bufs[key] = buf
        return buf

    def clear(self):
        self._bufs.clear()
        self._retired.clear()


WORKSPACES = _Workspaces()


def attention_desc(q: torch.Tensor, k_cache: torch.Tensor, *, num_kv_heads: int,
                   block_size: int, max_ref: int, max_prefix_len: int, page_size: int = 0,
                   max_pages_per_seq: int = 0, kv_chunk: int = 0,
                   scale: float = 0.0, rope_theta: float = 0.0) -> AttnDesc:
    """Descriptor for q [batch, B+L, Hq, d] and a cache laid out as
    [batch, cap, Hkv, d] (contiguous) or [pages, page_size, Hkv, d] (paged)."""
    b, n_new, hq, d = q.shape
    st = k_cache.stride()
    return AttnDesc(batch=b, num_q_heads=hq, num_kv_heads=num_kv_heads, head_dim=d,
                    block_size=block_size, max_ref=max_ref, max_prefix_len=max_prefix_len,
                    page_size=page_size, max_pages_per_seq=max_pages_per_seq,
                    kv_chunk=kv_chunk, cache_stride_seq=st[0], cache_stride_token=st[1],
                    cache_stride_head=st[2], scale=scale, dtype=_dtype_code(q.dtype),
                    rope_theta=rope_theta)


def attention_workspace_size(desc: AttnDesc) -> int:
    return int(lib().simsd_verify_attention_workspace_size(ctypes.byref(desc)))


def accept_workspace_size(desc: AcceptDesc) -> int:
    return int(lib().simsd_verify_accept_workspace_size(ctypes.byref(desc)))


def _workspace(workspace, device, stream, kind, nbytes):
    """The caller's workspace (checked), or a cached one for this stream."""
    if workspace is None:
        return WORKSPACES.get(device, stream.cuda_stream, kind, nbytes)
    _tensor("workspace", workspace, (None,), None, device)
    return workspace


def _nbytes(t: Optional[torch.Tensor]) -> int:
    return 0 if t is None else t.numel() * t.element_size()


def check_attention_tensors(q, k_new, v_new, k_cache, v_cache, block_table, prefix_lens,
                            step_map, num_ref, out, lse, *, block_size: int, max_ref: int,
                            max_prefix_len: int, page_size: int):
    """Shapes, dtypes, devices and layouts of the attention arguments."""
    _need(isinstance(q, torch.Tensor) and q.dim() == 4, "q must be a 4-D tensor [batch, B+L, Hq, d]")
    _need(q.dtype in (torch.bfloat16, torch.float32), f"q must be bfloat16 or float32, got {q.dtype}")
    b, n_new, hq, d = q.shape
    dev = q.device
    _need(n_new == block_size + max_ref, f"q has {n_new} slots, block_size + max_ref is {block_size + max_ref}")
    _tensor("q", q, (b, n_new, hq, d), q.dtype, dev)
    _need(isinstance(k_new, torch.Tensor) and k_new.dim() == 4, "k_new must be a 4-D tensor")
    hkv = k_new.shape[2]
    _tensor("k_new", k_new, (b, n_new, hkv, d), q.dtype, dev)
    _tensor("v_new", v_new, (b, n_new, hkv, d), q.dtype, dev)
    if max_prefix_len > 0:
        _check_cache(k_cache, v_cache, q.dtype, dev, hkv, d, page_size, max_prefix_len, b,
                     block_table)
    _int32("prefix_lens", prefix_lens, (b,), dev)
    _int32("step_map", step_map, (b, block_size), dev)
    _int32("num_ref", num_ref, (b,), dev)
    _out("out", out, (b, n_new, hq, d), q.dtype, dev)
    _out("lse", lse, (b, hq, n_new), torch.float32, dev)
    return hkv


def verify_attention(q, k_new, v_new, k_cache, v_cache, block_table, prefix_lens, step_map,
                     num_ref, *, block_size: int, max_ref: int, max_prefix_len: int,
                     page_size: int = 0, kv_chunk: int = 0, scale: float = 0.0,
                     rope_theta: float = 0.0,
                     out: Optional[torch.Tensor] = None, lse: Optional[torch.Tensor] = None,
                     want_lse: bool = True, workspace: Optional[torch.Tensor] = None,
                     stream=None, desc: Optional[AttnDesc] = None):
    """simsd_verify_attention on torch tensors.  Returns (out, lse).

    Raises ValueError on tensors whose shape, dtype, device or layout does not
    match (before anything is launched), SimsdError if the library rejects
    the call."""
    hkv = check_attention_tensors(q, k_new, v_new, k_cache, v_cache, block_table, prefix_lens,
                                  step_map, num_ref, out, lse, block_size=block_size,
                                  max_ref=max_ref, max_prefix_len=max_prefix_len,
                                  page_size=page_size)
    if desc is None:
        desc = attention_desc(q, k_cache if max_prefix_len > 0 else k_new, num_kv_heads=hkv,
                              block_size=block_size, max_ref=max_ref,
                              max_prefix_len=max_prefix_len, page_size=page_size,
                              max_pages_per_seq=(block_table.shape[1]
                                                 if block_table is not None and page_size > 0
                                                 else 0),
                              kv_chunk=kv_chunk, scale=scale, rope_theta=rope_theta)
    dev = q.device
    if out is None:
        out = torch.empty(q.shape, dtype=q.dtype, device=dev)
    if lse is None and want_lse:
        lse = torch.empty((q.shape[0], q.shape[2], q.shape[1]), dtype=torch.float32, device=dev)
    st = _stream_of(stream, dev)
    workspace = _workspace(workspace, dev, st, "attn", attention_workspace_size(desc))
    _check(lib().simsd_verify_attention(
        ctypes.byref(desc), _ptr(q), _ptr(k_new), _ptr(v_new), _ptr(k_cache), _ptr(v_cache),
        _ptr(block_table), _ptr(prefix_lens), _ptr(step_map), _ptr(num_ref), _ptr(out),
        _ptr(lse), _ptr(workspace), _nbytes(workspace), ctypes.c_void_p(st.cuda_stream)))
    return out, lse


def accept_desc(logits: torch.Tensor, max_ref: int, chunks_per_row: int = 0) -> AcceptDesc:
    b, B, V = logits.shape
    return AcceptDesc(batch=b, block_size=B, max_ref=max_ref, vocab=V,
                      chunks_per_row=chunks_per_row, logits_dtype=_dtype_code(logits.dtype))


def _check_accept_inputs(logits, draft_ids, step_map, num_ref):
    _need(isinstance(logits, torch.Tensor) and logits.dim() == 3, "logits must be a 3-D tensor [batch, B, V]")
    _need(logits.dtype in (torch.bfloat16, torch.float32),
          f"logits must be bfloat16 or float32, got {logits.dtype}")
    b, B, V = logits.shape
    dev = logits.device
    _tensor("logits", logits, (b, B, V), logits.dtype, dev)
    _need(isinstance(draft_ids, torch.Tensor) and draft_ids.dim() == 2,
          "draft_ids must be a 2-D tensor [batch, L]")
    _int32("draft_ids", draft_ids, (b, None), dev)
    _int32("step_map", step_map, (b, B), dev)
    _int32("num_ref", num_ref, (b,), dev)
    return b, B, V, draft_ids.shape[1], dev


def verify_accept(logits, draft_ids, step_map, num_ref, *, chunks_per_row: int = 0,
                  target_ids=None, confidence=None, draft_prob=None, accept_len=None,
                  workspace=None, stream=None, desc: Optional[AcceptDesc] = None):
    """simsd_verify_accept on torch tensors.
    Returns (target_ids, confidence, draft_prob, accept_len)."""
    b, B, V, L, dev = _check_accept_inputs(logits, draft_ids, step_map, num_ref)
    _out("target_ids", target_ids, (b, B), torch.int32, dev)
    _out("confidence", confidence, (b, B), torch.float32, dev)
    _out("draft_prob", draft_prob, (b, L), torch.float32, dev)
    _out("accept_len", accept_len, (b,), torch.int32, dev)
    if desc is None:
        desc = accept_desc(logits, L, chunks_per_row)
    if target_ids is None:
        target_ids = torch.empty((b, B), dtype=torch.int32, device=dev)
    if confidence is None:
        confidence = torch.empty((b, B), dtype=torch.float32, device=dev)
    if draft_prob is None:
        draft_prob = torch.empty((b, L), dtype=torch.float32, device=dev)
    if accept_len is None:
        accept_len = torch.empty((b,), dtype=torch.int32, device=dev)
    st = _stream_of(stream, dev)
    workspace = _workspace(workspace, dev, st, "accept", accept_workspace_size(desc))
    _check(lib().simsd_verify_accept(
        ctypes.byref(desc), _ptr(logits), _ptr(draft_ids), _ptr(step_map), _ptr(num_ref),
        _ptr(target_ids), _ptr(confidence), _ptr(draft_prob), _ptr(accept_len),
        _ptr(workspace), _nbytes(workspace), ctypes.c_void_p(st.cuda_stream)))
    return target_ids, confidence, draft_prob, accept_len


NOALLOC_SCRATCH_BYTES = 4 << 20      # SIMSD_NOALLOC_SCRATCH_BYTES


def verify_accept_noalloc(logits, draft_ids, step_map, num_ref, *, target_ids=None,
                          confidence=None, draft_prob=None, accept_len=None, stream=None):
    """simsd_verify_accept_noalloc on torch tensors: the greedy accept with the
    library's fixed per-device scratch instead of a workspace (for callers that
    cannot allocate; pass preallocated outputs to allocate nothing at all).
    Calls overlapping on one GPU race on that scratch.
    Returns (target_ids, confidence, draft_prob, accept_len)."""
    b, B, V, L, dev = _check_accept_inputs(logits, draft_ids, step_map, num_ref)
    _out("target_ids", target_ids, (b, B), torch.int32, dev)
    _out("confidence", confidence, (b, B), torch.float32, dev)
    _out("draft_prob", draft_prob, (b, L), torch.float32, dev)
    _out("accept_len", accept_len, (b,), torch.int32, dev)
    desc = accept_desc(logits, L)
    if target_ids is None:
        target_ids = torch.empty((b, B), dtype=torch.int32, device=dev)
    if confidence is None:
        confidence = torch.empty((b, B), dtype=torch.float32, device=dev)
    if draft_prob is None:
        draft_prob = torch.empty((b, L), dtype=torch.float32, device=dev)
    if accept_len is None:
        accept_len = torch.empty((b,), dtype=torch.int32, device=dev)
    st = _stream_of(stream, dev)
    _check(lib().simsd_verify_accept_noalloc(
        ctypes.byref(desc), _ptr(logits), _ptr(draft_ids), _ptr(step_map), _ptr(num_ref),
        _ptr(target_ids), _ptr(confidence), _ptr(draft_prob), _ptr(accept_len),
        ctypes.c_void_p(st.cuda_stream)))
    return target_ids, confidence, draft_prob, accept_len


def accept_sampled_workspace_size(desc: AcceptDesc) -> int:
    return int(lib().simsd_verify_accept_sampled_workspace_size(ctypes.byref(desc)))


def verify_accept_sampled(logits, draft_logits, draft_ids, step_map, num_ref, uniforms, *,
                          temperature: float = 1.0, chunks_per_row: int = 0, p_target=None,
                          p_draft=None, accept_len=None, correction=None, workspace=None,
                          stream=None, desc: Optional[AcceptDesc] = None):
    """simsd_verify_accept_sampled on torch tensors.
    Returns (p_target, p_draft, accept_len, correction)."""
    b, B, V, L, dev = _check_accept_inputs(logits, draft_ids, step_map, num_ref)
    _tensor("draft_logits", draft_logits, (b, L, V), logits.dtype, dev)
    _tensor("uniforms", uniforms, (b, L + 1), torch.float32, dev)
    _out("p_target", p_target, (b, L), torch.float32, dev)
    _out("p_draft", p_draft, (b, L), torch.float32, dev)
    _out("accept_len", accept_len, (b,), torch.int32, dev)
    _out("correction", correction, (b,), torch.int32, dev)
    if desc is None:
        desc = accept_desc(logits, L, chunks_per_row)
    if p_target is None:
        p_target = torch.empty((b, L), dtype=torch.float32, device=dev)
    if p_draft is None:
        p_draft = torch.empty((b, L), dtype=torch.float32, device=dev)
    if accept_len is None:
        accept_len = torch.empty((b,), dtype=torch.int32, device=dev)
    if correction is None:
        correction = torch.empty((b,), dtype=torch.int32, device=dev)
    st = _stream_of(stream, dev)
    workspace = _workspace(workspace, dev, st, "accept_sampled",
                           accept_sampled_workspace_size(desc))
    _check(lib().simsd_verify_accept_sampled(
        ctypes.byref(desc), ctypes.c_float(temperature), _ptr(logits), _ptr(draft_logits),
        _ptr(draft_ids), _ptr(step_map), _ptr(num_ref), _ptr(uniforms), _ptr(p_target),
        _ptr(p_draft), _ptr(accept_len), _ptr(correction), _ptr(workspace),
        _nbytes(workspace), ctypes.c_void_p(st.cuda_stream)))
    return p_target, p_draft, accept_len, correction


def lmhead_desc(hidden: torch.Tensor, weight: torch.Tensor, max_ref: int) -> LmheadDesc:
    b, B, H = hidden.shape
    return LmheadDesc(batch=b, block_size=B, max_ref=max_ref, vocab=weight.shape[0], hidden=H,
                      dtype=_dtype_code(hidden.dtype))


def lmhead_workspace_size(desc: LmheadDesc) -> int:
    return int(lib().simsd_verify_accept_lmhead_workspace_size(ctypes.byref(desc)))


def verify_accept_lmhead(hidden, weight, draft_ids, step_map, num_ref, *, target_ids=None,
                         confidence=None, draft_prob=None, accept_len=None, workspace=None,
                         stream=None, desc: Optional[LmheadDesc] = None):
    """simsd_verify_accept_lmhead on torch tensors (hidden [b, B, H], weight [V, H]).
    Returns (target_ids, confidence, draft_prob, accept_len)."""
    _need(isinstance(hidden, torch.Tensor) and hidden.dim() == 3,
          "hidden must be a 3-D tensor [batch, B, H]")
    b, B, H = hidden.shape
    dev = hidden.device
    _tensor("hidden", hidden, (b, B, H), torch.bfloat16, dev)
    _need(isinstance(weight, torch.Tensor) and weight.dim() == 2, "weight must be a 2-D tensor [V, H]")
    _tensor("weight", weight, (None, H), torch.bfloat16, dev)
    V = weight.shape[0]
    _need(isinstance(draft_ids, torch.Tensor) and draft_ids.dim() == 2,
          "draft_ids must be a 2-D tensor [batch, L]")
    _int32("draft_ids", draft_ids, (b, None), dev)
    _int32("step_map", step_map, (b, B), dev)
    _int32("num_ref", num_ref, (b,), dev)
    L = draft_ids.shape[1]
    _out("target_ids", target_ids, (b, B), torch.int32, dev)
    _out("confidence", confidence, (b, B), torch.float32, dev)
    _out("draft_prob", draft_prob, (b, L), torch.float32, dev)
    _out("accept_len", accept_len, (b,), torch.int32, dev)
    if desc is None:
        desc = lmhead_desc(hidden, weight, L)
    if target_ids is None:
        target_ids = torch.empty((b, B), dtype=torch.int32, device=dev)
    if confidence is None:
        confidence = torch.empty((b, B), dtype=torch.float32, device=dev)
    if draft_prob is None:
        draft_prob = torch.empty((b, L), dtype=torch.float32, device=dev)
    if accept_len is None:
        accept_len = torch.empty((b,), dtype=torch.int32, device=dev)
    st = _stream_of(stream, dev)
    workspace = _workspace(workspace, dev, st, "lmhead", lmhead_workspace_size(desc))
    _check(lib().simsd_verify_accept_lmhead(
        ctypes.byref(desc), _ptr(hidden), _ptr(weight), _ptr(draft_ids), _ptr(step_map),
        _ptr(num_ref), _ptr(target_ids), _ptr(confidence), _ptr(draft_prob), _ptr(accept_len),
        _ptr(workspace), _nbytes(workspace), ctypes.c_void_p(st.cuda_stream)))
    return target_ids, confidence, draft_prob, accept_len


def validate_step_map(step_map, num_ref, max_ref: int):
    """Host-side step-map check (simsd_validate_step_map); raises SimsdError."""
    import numpy as np
    sm = np.ascontiguousarray(step_map, dtype=np.int32)
    nr = np.ascontiguousarray(num_ref, dtype=np.int32)
    _check(lib().simsd_validate_step_map(sm.ctypes.data_as(_I32P), nr.ctypes.data_as(_I32P),
                                         sm.shape[0], sm.shape[1], max_ref))
