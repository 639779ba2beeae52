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


def _stream(stream) -> ctypes.c_void_p:
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


class _Workspaces:
    """Scratch buffers for the workspace argument, one per (device, kind),
    grown on demand.  The library needs no initialised contents."""

    def __init__(self):
        self._bufs = {}

    def get(self, device: torch.device, kind: str, nbytes: int) -> Optional[torch.Tensor]:
        if nbytes == 0:
            return None
        key = (str(device), kind)
        buf = self._bufs.get(key)
        if buf is None or buf.numel() < nbytes:
            buf = torch.empty(nbytes, dtype=torch.uint8, device=device)
            self._bufs[key] = buf
        return buf

    def clear(self):
        self._bufs.clear()


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


def verify_attention(q, k_new, v_new, k_cache, v_cache, block_table, prefix_lens, step_map,
                     num_ref, *, block_size: int, max_ref: int, max_prefix_len: int,
                     page_size: int = 0, kv_chunk: int = 0, scale: float = 0.0,
                     rope_theta: float = 0.0,
                     out: Optional[torch.Tensor] = None, lse: Optional[torch.Tensor] = None,
                     want_lse: bool = True, workspace: Optional[torch.Tensor] = None,
                     stream=None, desc: Optional[AttnDesc] = None):
    """simsd_verify_attention on torch tensors.  Returns (out, lse)."""
    if desc is None:
        desc = attention_desc(q, k_cache, num_kv_heads=k_new.shape[2], block_size=block_size,
                              max_ref=max_ref, max_prefix_len=max_prefix_len,
                              page_size=page_size,
                              max_pages_per_seq=(block_table.shape[1]
                                                 if block_table is not None else 0),
                              kv_chunk=kv_chunk, scale=scale, rope_theta=rope_theta)
    if out is None:
        out = torch.empty_like(q)
    if lse is None and want_lse:
        lse = torch.empty((q.shape[0], q.shape[2], q.shape[1]), dtype=torch.float32,
                          device=q.device)
    if workspace is None:
        workspace = WORKSPACES.get(q.device, "attn", attention_workspace_size(desc))
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib().simsd_verify_attention(
        ctypes.byref(desc), _ptr(q), _ptr(k_new), _ptr(v_new), _ptr(k_cache), _ptr(v_cache),
        _ptr(block_table), _ptr(prefix_lens), _ptr(step_map), _ptr(num_ref), _ptr(out),
        _ptr(lse), _ptr(workspace), ws_bytes, _stream(stream)))
    return out, lse


def accept_desc(logits: torch.Tensor, max_ref: int, chunks_per_row: int = 0) -> AcceptDesc:
    b, B, V = logits.shape
    return AcceptDesc(batch=b, block_size=B, max_ref=max_ref, vocab=V,
                      chunks_per_row=chunks_per_row, logits_dtype=_dtype_code(logits.dtype))


def verify_accept(logits, draft_ids, step_map, num_ref, *, chunks_per_row: int = 0,
                  target_ids=None, confidence=None, draft_prob=None, accept_len=None,
                  workspace=None, stream=None, desc: Optional[AcceptDesc] = None):
    """simsd_verify_accept on torch tensors.
    Returns (target_ids, confidence, draft_prob, accept_len)."""
    b, B, V = logits.shape
    L = draft_ids.shape[1]
    if desc is None:
        desc = accept_desc(logits, L, chunks_per_row)
    dev = logits.device
    if target_ids is None:
        target_ids = torch.empty((b, B), dtype=torch.int32, device=dev)
    if confidence is None:
        confidence = torch.empty((b, B), dtype=torch.float32, device=dev)
    if draft_prob is None:
        draft_prob = torch.empty((b, L), dtype=torch.float32, device=dev)
    if accept_len is None:
        accept_len = torch.empty((b,), dtype=torch.int32, device=dev)
    if workspace is None:
        workspace = WORKSPACES.get(dev, "accept", accept_workspace_size(desc))
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib().simsd_verify_accept(
        ctypes.byref(desc), _ptr(logits), _ptr(draft_ids), _ptr(step_map), _ptr(num_ref),
        _ptr(target_ids), _ptr(confidence), _ptr(draft_prob), _ptr(accept_len),
        _ptr(workspace), ws_bytes, _stream(stream)))
    return target_ids, confidence, draft_prob, accept_len


def accept_sampled_workspace_size(desc: AcceptDesc) -> int:
    return int(lib().simsd_verify_accept_sampled_workspace_size(ctypes.byref(desc)))


def verify_accept_sampled(logits, draft_logits, draft_ids, step_map, num_ref, uniforms, *,
                          temperature: float = 1.0, chunks_per_row: int = 0, p_target=None,
                          p_draft=None, accept_len=None, correction=None, workspace=None,
                          stream=None, desc: Optional[AcceptDesc] = None):
    """simsd_verify_accept_sampled on torch tensors.
    Returns (p_target, p_draft, accept_len, correction)."""
    b, B, V = logits.shape
    L = draft_ids.shape[1]
    if desc is None:
        desc = accept_desc(logits, L, chunks_per_row)
    dev = logits.device
    if p_target is None:
        p_target = torch.empty((b, L), dtype=torch.float32, device=dev)
    if p_draft is None:
        p_draft = torch.empty((b, L), dtype=torch.float32, device=dev)
    if accept_len is None:
        accept_len = torch.empty((b,), dtype=torch.int32, device=dev)
    if correction is None:
        correction = torch.empty((b,), dtype=torch.int32, device=dev)
    if workspace is None:
        workspace = WORKSPACES.get(dev, "accept_sampled", accept_sampled_workspace_size(desc))
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib().simsd_verify_accept_sampled(
        ctypes.byref(desc), ctypes.c_float(temperature), _ptr(logits), _ptr(draft_logits),
        _ptr(draft_ids), _ptr(step_map), _ptr(num_ref), _ptr(uniforms), _ptr(p_target),
        _ptr(p_draft), _ptr(accept_len), _ptr(correction), _ptr(workspace), ws_bytes,
        _stream(stream)))
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
    b, B, H = hidden.shape
    L = draft_ids.shape[1]
    if desc is None:
        desc = lmhead_desc(hidden, weight, L)
    dev = hidden.device
    if target_ids is None:
        target_ids = torch.empty((b, B), dtype=torch.int32, device=dev)
    if confidence is None:
        confidence = torch.empty((b, B), dtype=torch.float32, device=dev)
    if draft_prob is None:
        draft_prob = torch.empty((b, L), dtype=torch.float32, device=dev)
    if accept_len is None:
        accept_len = torch.empty((b,), dtype=torch.int32, device=dev)
    if workspace is None:
        workspace = WORKSPACES.get(dev, "lmhead", lmhead_workspace_size(desc))
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib().simsd_verify_accept_lmhead(
        ctypes.byref(desc), _ptr(hidden), _ptr(weight), _ptr(draft_ids), _ptr(step_map),
        _ptr(num_ref), _ptr(target_ids), _ptr(confidence), _ptr(draft_prob), _ptr(accept_len),
        _ptr(workspace), ws_bytes, _stream(stream)))
    return target_ids, confidence, draft_prob, accept_len


def validate_step_map(step_map, num_ref, max_ref: int):
    """Host-side step-map check (simsd_validate_step_map); raises SimsdError."""
    import numpy as np
    sm = np.ascontiguousarray(step_map, dtype=np.int32)
    nr = np.ascontiguousarray(num_ref, dtype=np.int32)
    _check(lib().simsd_validate_step_map(sm.ctypes.data_as(_I32P), nr.ctypes.data_as(_I32P),
                                         sm.shape[0], sm.shape[1], max_ref))
