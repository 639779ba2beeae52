"""The five verification workloads, as plain data.

Shapes follow the SDAR model family the paper evaluates (Sec. 4.1, "Models"):
a 1.7B-shaped layer (16 query / 8 KV heads) and an 8B-shaped layer (32 / 8),
head_dim 128, vocabulary 151936, block sizes 4 and 8 (Table 1) plus the longer
blocks and prefixes of the long-context and ragged workloads.  Draft length
gamma equals the block length, as in Sec. 4.1 ("Configurations").
"""

from __future__ import annotations

import dataclasses
import math
from dataclasses import dataclass
from typing import Tuple, Union

Range = Tuple[float, float]


@dataclass(frozen=True)
class VerifyConfig:
    """One verification workload.

    prefix      cached prefix length per sequence, or an inclusive (lo, hi) range
                drawn uniformly per sequence (ragged batch).
    block_size  B: block (prediction) slots per sequence.
    max_ref     L: reference (draft data) slots per sequence, L <= B.
    page_size   0 = KV cache contiguous per sequence; >0 = paged cache whose pages
                are laid out in a seeded random order.
    plant       probability that a drafted token is planted as the unique argmax
                of its verification row, or a (lo, hi) range drawn per sequence.
    step_mode   "full": gamma = L drafted slots in a random order (the paper's
                setting is L = B), `committed` slots decoded by earlier steps of
                the block, the rest not drafted.  "mixed": per-sequence gamma,
                committed, undrafted and padding slots (test cases).
    committed   "full" mode: block slots already committed (a later verification
                step inside the block), at most B - L.
    """

    cid: int
    name: str
    dtype: str                 # "f32" or "bf16": q, k, v, out and logits
    batch: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    prefix: Union[int, Tuple[int, int]]
    block_size: int
    max_ref: int
    vocab: int
    page_size: int = 0
    plant: Union[float, Range] = 0.7
    qkv_std: float = 1.0
    logit_std: float = 2.0     # N(0, 4): variance 4
    step_mode: str = "full"
    capacity: int = 0          # contiguous cache rows per sequence; 0 = max prefix
    committed: int = 0

    @property
    def n_new(self) -> int:
        return self.block_size + self.max_ref

    @property
    def group(self) -> int:
        return self.num_q_heads // self.num_kv_heads

    @property
    def max_prefix(self) -> int:
        return self.prefix if isinstance(self.prefix, int) else int(self.prefix[1])

    @property
    def cache_rows(self) -> int:
        return max(self.capacity, self.max_prefix)

    @property
    def elem_bytes(self) -> int:
        return 4 if self.dtype == "f32" else 2

    def replace(self, **kw) -> "VerifyConfig":
        return dataclasses.replace(self, **kw)


_BF16_QKV = 1.0 / math.sqrt(128.0)

CONFIGS = {
    1: VerifyConfig(1, "tiny-f32", "f32", batch=1, num_q_heads=2, num_kv_heads=1,
                    head_dim=64, prefix=64, block_size=4, max_ref=4, vocab=1000,
                    plant=0.7, qkv_std=1.0),
    2: VerifyConfig(2, "sdar-1.7b-layer", "bf16", batch=1, num_q_heads=16, num_kv_heads=8,
                    head_dim=128, prefix=1024, block_size=4, max_ref=4, vocab=151936,
                    plant=0.7, qkv_std=_BF16_QKV),
    3: VerifyConfig(3, "sdar-8b-layer", "bf16", batch=8, num_q_heads=32, num_kv_heads=8,
                    head_dim=128, prefix=4096, block_size=16, max_ref=16, vocab=151936,
                    plant=0.6, qkv_std=_BF16_QKV),
    4: VerifyConfig(4, "long-context", "bf16", batch=16, num_q_heads=32, num_kv_heads=8,
                    head_dim=128, prefix=16384, block_size=32, max_ref=32, vocab=151936,
                    plant=0.5, qkv_std=_BF16_QKV),
    5: VerifyConfig(5, "ragged-paged", "bf16", batch=64, num_q_heads=32, num_kv_heads=8,
                    head_dim=128, prefix=(512, 32768), block_size=8, max_ref=8,
                    vocab=151936, page_size=16, plant=(0.3, 0.9), qkv_std=_BF16_QKV),
}


def config_by_id(cid: int) -> VerifyConfig:
    return CONFIGS[int(cid)]
