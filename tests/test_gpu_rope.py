"""GPU parity of the fused rotary embedding at the RoPE-copy positions
(Sec. 3.1-3.2) against the oracle, through the C ABI: q and the new keys
arrive unrotated, the cached prefix keys rotated.  Same tolerances as the
other attention tests (bf16 2e-2 of the row's largest value, fp32 1e-5)."""

import numpy as np
import pytest

import oracle
from gpu_util import DeviceInputs, run_attention, check_attention
from synth import VerifyConfig, generate

pytestmark = pytest.mark.gpu

ROPE_CASES = [
    # dtype, head_dim, Hq, Hkv, B, L, prefix, page, kv_chunk, theta, seed
    ("bf16", 128, 8, 2, 8, 8, (0, 300), 0, 0, 1e6, 1),
    ("bf16", 128, 16, 2, 16, 16, (100, 700), 16, 64, 1e6, 2),
    ("bf16", 64, 8, 2, 16, 16, (0, 3000), 0, -1, 1e4, 3),      # stream decomposition
    ("bf16", 128, 12, 3, 24, 8, (0, 2500), 32, -1, 1e6, 4),    # stream, paged
    ("bf16", 128, 32, 8, 32, 32, (30000, 32800), 0, 0, 1e6, 5),  # positions past 32768
    ("bf16", 128, 8, 2, 16, 16, (100, 700), 16, 64, 1e6, 8),   # 128 rows: 4 whole-tile row waves, paged
    ("bf16", 64, 16, 4, 16, 16, (0, 500), 0, 0, 1e4, 9),       # 128 rows, contiguous, d 64
    ("f32", 64, 4, 2, 8, 6, (0, 200), 0, 64, 1e4, 6),
    ("f32", 128, 8, 2, 4, 4, (1, 90), 5, 0, 1e6, 7),
]


@pytest.mark.parametrize("case", ROPE_CASES, ids=lambda c: "-".join(map(str, c)))
def test_rope_parity(case):
    dt, d, hq, hkv, B, L, prefix, page, kv_chunk, theta, seed = case
    cfg = VerifyConfig(0, "rope", dt, batch=3 if prefix[1] > 10000 else 5, num_q_heads=hq,
                       num_kv_heads=hkv, head_dim=d, prefix=prefix, block_size=B, max_ref=L,
                       vocab=100, page_size=page, qkv_std=0.3 if dt == "bf16" else 1.0,
                       step_mode="mixed")
    inp = generate(cfg, seed=seed, poison=True)
    dev = DeviceInputs(inp)
    out, lse = run_attention(dev, kv_chunk, rope_theta=theta)
    ref_out, ref_lse = oracle.verify_attention(inp, rope_theta=theta)
    check_attention(out, lse, ref_out, ref_lse, dt)
    # the rotation matters: without it the outputs differ from the rotated
    # oracle (with short prefixes, where the new slots carry real weight)
    if prefix[1] < 10000:
        plain, _ = run_attention(dev, kv_chunk)
        valid = np.isfinite(ref_lse.transpose(0, 2, 1))
        assert np.abs(plain - ref_out)[valid].max() > 1e-3
