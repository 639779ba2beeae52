"""The seeded generator: determinism, planting rate, paging and poisoning."""

import math

import numpy as np

from synth import CONFIGS, VerifyConfig, generate


def test_same_seed_same_inputs():
    a = generate(CONFIGS[1]).checksums()
    b = generate(CONFIGS[1]).checksums()
    c = generate(CONFIGS[1], seed=77).checksums()
    assert a == b and a != c


def test_plant_rate_within_binomial_ci():
    cfg = VerifyConfig(0, "plant", "bf16", batch=64, num_q_heads=2, num_kv_heads=1,
                       head_dim=8, prefix=1, block_size=16, max_ref=16, vocab=257, plant=0.6)
    inp = generate(cfg, seed=9)
    n = inp.planted.size
    rate = inp.planted.mean()
    assert abs(rate - 0.6) < 4 * math.sqrt(0.6 * 0.4 / n)


def test_paged_layout_is_a_permutation_and_poisoned():
    cfg = CONFIGS[5].replace(batch=6, prefix=(1, 70), num_q_heads=4, num_kv_heads=2,
                             head_dim=8, vocab=50)
    inp = generate(cfg, seed=3, poison=True)
    P = cfg.page_size
    used = []
    for s in range(cfg.batch):
        n = int(inp.prefix_lens[s])
        pages = -(-n // P)
        used += list(inp.block_table[s, :pages])
        spare = inp.k_cache.shape[0] - 1
        assert np.all(inp.block_table[s, pages:] == spare)
        tail = n - (pages - 1) * P
        last = inp.block_table[s, pages - 1]
        assert np.all(inp.k_cache[last, tail:] == 0x7FC0)
        assert not np.any(inp.k_cache[last, :tail] == 0x7FC0)
    assert sorted(used) == list(range(inp.k_cache.shape[0] - 1))
    assert np.all(inp.v_cache[-1] == 0x7FC0)


def test_config_shapes():
    inp = generate(CONFIGS[2])
    assert inp.q.shape == (1, 8, 16, 128) and inp.q.dtype == np.uint16
    assert inp.k_cache.shape == (1, 1024, 8, 128)
    assert inp.logits.shape == (1, 4, 151936)
    assert sorted(inp.step_map[0]) == [1, 2, 3, 4] and inp.num_ref[0] == 4
    x = (inp.q.astype(np.uint32) << 16).view(np.float32)
    assert abs(x.std() - 1 / math.sqrt(128)) < 0.01
