"""bench.py's host side on the CPU: the algorithmic bytes and flops of one
verification step, pinned to values worked out by hand from the model shapes
(the SDAR-1.7B and SDAR-8B layer shapes and the long-context workload), and
the refusal of more than one GPU before anything touches a device."""

import os
import subprocess
import sys
from types import SimpleNamespace

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from synth import CONFIGS  # noqa: E402


def full_step(cid):
    """Every block slot drafted (step map a permutation of 1..B, gamma = L = B)."""
    cfg = CONFIGS[cid]
    rng = np.random.default_rng(cid)
    step_map = np.stack([rng.permutation(cfg.block_size) + 1 for _ in range(cfg.batch)])
    return SimpleNamespace(cfg=cfg, prefix_lens=np.full(cfg.batch, cfg.prefix, np.int32),
                           step_map=step_map.astype(np.int32),
                           num_ref=np.full(cfg.batch, cfg.max_ref, np.int32))


# By hand, bf16 (2 bytes), V = 151936, d = 128:
#   KV prefix   2 * b * prefix * Hkv * d * 2
#   new slots   b * (B+L) * (2*Hq + 2*Hkv) * d * 2, plus the fp32 LSE b * Hq * (B+L) * 4
#   logits      b * B * V * 2 (every block slot scanned)
#   flops       4 * Hq * d * b * (B+L) * (prefix + B)
EXPECTED = {
    2: dict(attn_bytes=4194304 + 98304 + 512, accept_bytes=1215488,
            attn_flops=67371008, verified=4),
    3: dict(attn_bytes=134217728 + 5242880 + 32768, accept_bytes=38895616,
            attn_flops=17246978048, verified=128),
    4: dict(attn_bytes=1073741824 + 20971520 + 131072, accept_bytes=155582464,
            attn_flops=275414777856, verified=512),
}


@pytest.mark.parametrize("cid", [2, 3, 4])
def test_algorithmic_bytes_and_flops(cid):
    got = bench.workload_numbers(full_step(cid))
    for k, v in EXPECTED[cid].items():
        assert got[k] == v, (k, got[k], v)
    assert got["scanned_rows"] == CONFIGS[cid].batch * CONFIGS[cid].block_size


def test_sampled_rule_reads_verification_and_draft_rows():
    got = bench.workload_numbers(full_step(3), sampled=True)
    assert got["accept_bytes"] == 2 * 128 * 151936 * 2


def test_padding_and_undrafted_slots():
    """A padded block slot is neither a key nor a row; an undrafted slot is
    scanned and attended to but verifies nothing."""
    inp = full_step(2)
    inp.step_map = np.array([[1, 2, 5, -1]], np.int32)     # gamma 2: slot 2 undrafted, 3 padding
    inp.num_ref = np.array([2], np.int32)
    got = bench.workload_numbers(inp)
    assert got["verified"] == 2 and got["scanned_rows"] == 3
    assert got["attn_flops"] == 4 * 16 * 128 * (3 + 2) * (1024 + 3)


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2, r.stderr
    assert "one GPU only" in r.stderr and r.stdout == ""
