"""Helpers shared by the GPU parity tests: move synthetic inputs to the device,
run the two entry points through the binding, and compare with the oracle."""

from __future__ import annotations

import numpy as np
import torch

import oracle


def dev_tensor(a: np.ndarray, dtype: str, device="cuda") -> torch.Tensor:
    """uint16 bf16 bits or float32 -> device tensor of that dtype (bits preserved)."""
    if dtype == "bf16":
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(device)
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(device)


def int_tensor(a: np.ndarray, device="cuda") -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(device)


class DeviceInputs:
    def __init__(self, inp, device="cuda"):
        dt = inp.cfg.dtype
        self.inp = inp
        self.q = dev_tensor(inp.q, dt, device)
        self.k_new = dev_tensor(inp.k_new, dt, device)
        self.v_new = dev_tensor(inp.v_new, dt, device)
        self.k_cache = dev_tensor(inp.k_cache, dt, device)
        self.v_cache = dev_tensor(inp.v_cache, dt, device)
        self.block_table = None if inp.block_table is None else int_tensor(inp.block_table, device)
        self.prefix_lens = int_tensor(inp.prefix_lens, device)
        self.step_map = int_tensor(inp.step_map, device)
        self.num_ref = int_tensor(inp.num_ref, device)
        self.logits = dev_tensor(inp.logits, dt, device)
        self.draft_ids = int_tensor(inp.draft_ids, device)


def run_attention(d: DeviceInputs, kv_chunk: int = 0, rope_theta: float = 0.0):
    from paper_2606_02544_amd import binding
    cfg = d.inp.cfg
    out, lse = binding.verify_attention(
        d.q, d.k_new, d.v_new, d.k_cache, d.v_cache, d.block_table, d.prefix_lens,
        d.step_map, d.num_ref, block_size=cfg.block_size, max_ref=cfg.max_ref,
        max_prefix_len=cfg.max_prefix, page_size=cfg.page_size, kv_chunk=kv_chunk,
        rope_theta=rope_theta)
    torch.cuda.synchronize()
    return out.float().cpu().double().numpy(), lse.cpu().double().numpy()


def run_accept(d: DeviceInputs, chunks_per_row: int = 0):
    from paper_2606_02544_amd import binding
    t, c, p, a = binding.verify_accept(d.logits, d.draft_ids, d.step_map, d.num_ref,
                                       chunks_per_row=chunks_per_row)
    torch.cuda.synchronize()
    return (t.cpu().numpy(), c.cpu().double().numpy(), p.cpu().double().numpy(),
            a.cpu().numpy())


# Tolerances: bf16 outputs within 2e-2 of the row's largest |value| (per
# sequence, head and row); f32 outputs within 1e-5 absolute; LSE within 1e-4
# (scaled by its magnitude above 1); probabilities within 1e-4 relative.
def check_attention(out, lse, ref_out, ref_lse, dtype, rows_mask=None):
    if rows_mask is not None:
        out, lse = out[rows_mask], lse[rows_mask]
        ref_out, ref_lse = ref_out[rows_mask], ref_lse[rows_mask]
    assert np.all(np.isfinite(out)), "non-finite attention output"
    if dtype == "bf16":
        err = np.abs(out - ref_out).max(axis=-1)
        scale = np.abs(ref_out).max(axis=-1)
        bad = err > 2e-2 * scale
        assert not bad.any(), f"{bad.sum()} rows over 2e-2 relative; worst {np.max(err / np.maximum(scale, 1e-30))}"
    else:
        err = np.abs(out - ref_out)
        assert err.max() <= 1e-5, f"max abs error {err.max()}"
    pad = np.isneginf(ref_lse)
    assert np.array_equal(np.isneginf(lse), pad), "padding rows differ"
    d = np.abs(lse[~pad] - ref_lse[~pad])
    tol = 1e-4 * np.maximum(1.0, np.abs(ref_lse[~pad]))
    assert np.all(d <= tol), f"lse error {d.max()}"


def check_accept(got, ref):
    t, c, p, a = got
    rt, rc, rp, ra = ref
    np.testing.assert_array_equal(t, rt)
    np.testing.assert_array_equal(a, ra)
    np.testing.assert_allclose(c, rc, rtol=1e-4, atol=1e-30)
    np.testing.assert_allclose(p, rp, rtol=1e-4, atol=1e-30)


def oracle_accept(inp):
    return oracle.verify_accept(inp.logits, inp.draft_ids, inp.step_map, inp.num_ref,
                                inp.cfg.dtype)


def walk_accept(target_ids, draft_ids, step_map, num_ref):
    """Accepted-prefix length from a given set of target ids (Sec. 3.2, the
    longest accepted prefix of eq. 2 at temperature 0): for each sequence, the
    number of leading drafts r = 1..gamma whose token equals the target id of
    the block slot k_r with step_map = r.  Used where several target ids are
    valid (near-ties of fp32-accumulated logits), so that accept_len is always
    checked against the ids the GPU actually produced."""
    b = len(num_ref)
    out = np.zeros((b,), np.int32)
    for s in range(b):
        for r in range(int(num_ref[s])):
            k = int(np.flatnonzero(step_map[s] == r + 1)[0])
            if int(target_ids[s, k]) != int(draft_ids[s, r]):
                break
            out[s] += 1
    return out
