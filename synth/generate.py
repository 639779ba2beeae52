"""Seeded generator for verification-step inputs.

Every tensor comes from its own child stream of ``numpy.random.SeedSequence``
(default entropy ``1000 + cid``), spawned in a fixed order, so any subset of the
inputs is reproducible on its own.  Values are drawn in float32 and rounded to
bfloat16 with round-to-nearest-even by integer arithmetic on the bit pattern;
bfloat16 tensors are returned as ``uint16`` bit patterns (numpy has no bf16).

Planting: for a drafted token chosen to match, the generator raises one logit of
its verification row to a level every other logit of the row is clipped below,
so the draft is that row's unique maximum by construction; no maximum is ever
computed here.  Unplanted drafts are uniform vocabulary ids (which may still
match by chance; the oracle decides).
"""

from __future__ import annotations

import concurrent.futures as cf
import os
from dataclasses import dataclass
from typing import Optional

import numpy as np

from .configs import VerifyConfig

BF16_NAN = np.uint16(0x7FC0)


def bf16_bits_from_f32(x: np.ndarray) -> np.ndarray:
    """Round finite float32 values to bfloat16 (nearest, ties to even); uint16 bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    t = u >> np.uint32(16)
    t &= np.uint32(1)
    t += np.uint32(0x7FFF)
    t += u
    t >>= np.uint32(16)
    return t.astype(np.uint16)


@dataclass
class VerifyInputs:
    """Host copies of every argument of the two entry points.

    Layouts (row-major):
      q            [batch, B+L, Hq,  d]   slots [0,B) block, [B,B+L) reference
      k_new, v_new [batch, B+L, Hkv, d]
      k_cache      contiguous [batch, cache_rows, Hkv, d]  or paged
                   [num_pages, page_size, Hkv, d] (v_cache likewise)
      block_table  [batch, max_pages] int32 (paged) or None
      prefix_lens  [batch] int32
      step_map     [batch, B] int32 (0 committed, 1..gamma drafted order,
                   > gamma undrafted, < 0 padding)
      num_ref      [batch] int32 (gamma_b <= L)
      logits       [batch, B, V]   row k is block slot k
      draft_ids    [batch, L] int32 (draft r at index r-1; -1 past gamma_b)
    bf16 tensors are uint16 bit patterns, f32 tensors float32.
    """

    cfg: VerifyConfig
    q: np.ndarray
    k_new: np.ndarray
    v_new: np.ndarray
    k_cache: np.ndarray
    v_cache: np.ndarray
    block_table: Optional[np.ndarray]
    prefix_lens: np.ndarray
    step_map: np.ndarray
    num_ref: np.ndarray
    logits: np.ndarray
    draft_ids: np.ndarray
    planted: np.ndarray          # bool [batch, L]: draft planted as its row's unique max
    seed_entropy: int
    poison: bool

    @property
    def paged(self) -> bool:
        return self.block_table is not None

    def checksums(self) -> dict:
        out = {}
        for name in ("q", "k_new", "v_new", "k_cache", "v_cache", "block_table",
                     "prefix_lens", "step_map", "num_ref", "logits", "draft_ids"):
            a = getattr(self, name)
            if a is None:
                continue
            out[name] = int(np.bitwise_xor.reduce(
                np.ascontiguousarray(a).view(np.uint8).reshape(-1)[: (a.nbytes // 8) * 8]
                .view(np.uint64))) if a.nbytes >= 8 else int(a.view(np.uint8).sum())
        return out


def _normal(rng: np.random.Generator, shape, std: float, dtype: str) -> np.ndarray:
    x = rng.standard_normal(shape, dtype=np.float32)
    if std != 1.0:
        x *= np.float32(std)
    return x if dtype == "f32" else bf16_bits_from_f32(x)


def _poison_value(dtype: str):
    return np.float32(np.nan) if dtype == "f32" else BF16_NAN


def _step_maps(rng, cfg: VerifyConfig):
    B, L, b = cfg.block_size, cfg.max_ref, cfg.batch
    step_map = np.zeros((b, B), np.int32)
    num_ref = np.zeros((b,), np.int32)
    for s in range(b):
        if cfg.step_mode == "full":
            gamma = min(L, B)
            n_pad = 0
            n_com = min(cfg.committed, B - gamma)
        elif cfg.step_mode == "mixed":
            n_pad = int(rng.integers(0, B // 4 + 1))
            n_com = int(rng.integers(0, (B - n_pad) // 2 + 1))
            gamma = int(rng.integers(0, min(L, B - n_pad - n_com) + 1))
        else:
            raise ValueError(f"unknown step_mode {cfg.step_mode!r}")
        slots = rng.permutation(B)
        drafted = slots[:gamma]
        committed = slots[gamma:gamma + n_com]
        padding = slots[gamma + n_com:gamma + n_com + n_pad]
        undrafted = slots[gamma + n_com + n_pad:]
        step_map[s, drafted] = rng.permutation(gamma) + 1
        step_map[s, committed] = 0
        step_map[s, padding] = -1 - rng.integers(0, 3, size=len(padding))
        step_map[s, undrafted] = gamma + 1 + rng.integers(0, B + 1, size=len(undrafted))
        num_ref[s] = gamma
    return step_map, num_ref


def generate(cfg: VerifyConfig, seed: Optional[int] = None, poison: bool = False,
             bad_draft_rate: float = 0.0, threads: Optional[int] = None) -> VerifyInputs:
    """Make every input of one verification step for ``cfg``.

    poison: fill cache rows past each prefix (contiguous tail, last-page tail and a
    spare page that unused block-table entries point to) with NaN, so any read of
    them shows up in the outputs.
    bad_draft_rate: fraction of unplanted drafts replaced by ids outside [0, V).
    """
    entropy = 1000 + cfg.cid if seed is None else int(seed)
    ss = np.random.SeedSequence(entropy)
    (s_q, s_kc, s_vc, s_kn, s_vn, s_len, s_perm, s_step, s_logit,
     s_plant) = ss.spawn(10)
    b, Hq, Hkv, d = cfg.batch, cfg.num_q_heads, cfg.num_kv_heads, cfg.head_dim
    B, L, V, n_new = cfg.block_size, cfg.max_ref, cfg.vocab, cfg.n_new
    if Hq % Hkv or L > B:
        raise ValueError("bad config shape")
    nthreads = threads or min(16, os.cpu_count() or 1)

    q = _normal(np.random.default_rng(s_q), (b, n_new, Hq, d), cfg.qkv_std, cfg.dtype)
    k_new = _normal(np.random.default_rng(s_kn), (b, n_new, Hkv, d), cfg.qkv_std, cfg.dtype)
    v_new = _normal(np.random.default_rng(s_vn), (b, n_new, Hkv, d), cfg.qkv_std, cfg.dtype)

    if isinstance(cfg.prefix, int):
        prefix_lens = np.full((b,), cfg.prefix, np.int32)
    else:
        lo, hi = cfg.prefix
        prefix_lens = np.random.default_rng(s_len).integers(
            lo, hi, endpoint=True, size=b).astype(np.int32)

    # Prefix K/V: one child stream per sequence, so sequences generate in parallel.
    kc_streams, vc_streams = s_kc.spawn(b), s_vc.spawn(b)

    def seq_kv(args):
        s, stream = args
        return _normal(np.random.default_rng(stream), (int(prefix_lens[s]), Hkv, d),
                       cfg.qkv_std, cfg.dtype)

    np_dtype = np.float32 if cfg.dtype == "f32" else np.uint16
    fill = _poison_value(cfg.dtype) if poison else np_dtype(0)
    block_table = None
    if cfg.page_size == 0:
        cap = cfg.cache_rows
        k_cache = np.empty((b, cap, Hkv, d), np_dtype)
        v_cache = np.empty((b, cap, Hkv, d), np_dtype)

        def place(s, kv, dst):
            n = int(prefix_lens[s])
            dst[s, :n] = kv
            dst[s, n:] = fill
    else:
        P = cfg.page_size
        max_pages = -(-cfg.max_prefix // P)
        pages = [-(-int(n) // P) for n in prefix_lens]
        total = int(sum(pages))
        spare = total                      # one extra page: target of unused entries
        perm = np.random.default_rng(s_perm).permutation(total).astype(np.int32)
        block_table = np.full((b, max(max_pages, 1)), spare, np.int32)
        off = 0
        for s in range(b):
            block_table[s, :pages[s]] = perm[off:off + pages[s]]
            off += pages[s]
        k_cache = np.empty((total + 1, P, Hkv, d), np_dtype)
        v_cache = np.empty((total + 1, P, Hkv, d), np_dtype)
        k_cache[spare] = fill
        v_cache[spare] = fill

        def place(s, kv, dst):
            n = int(prefix_lens[s])
            for j in range(pages[s]):
                lo, hi = j * P, min(n, (j + 1) * P)
                pg = dst[block_table[s, j]]
                pg[: hi - lo] = kv[lo:hi]
                pg[hi - lo:] = fill

    def job(s):
        place(s, seq_kv((s, kc_streams[s])), k_cache)
        place(s, seq_kv((s, vc_streams[s])), v_cache)

    with cf.ThreadPoolExecutor(max_workers=nthreads) as ex:
        list(ex.map(job, range(b)))

    step_map, num_ref = _step_maps(np.random.default_rng(s_step), cfg)

    # Logits N(0, logit_std^2), clipped to +-6 sigma so a planted value above the
    # clip level is its row's unique maximum.
    clip = np.float32(6.0 * cfg.logit_std)
    plant_val = np.float32(6.25 * cfg.logit_std)
    logits = np.empty((b, B, V), np_dtype)
    logit_streams = s_logit.spawn(b)

    def logit_job(s):
        x = np.random.default_rng(logit_streams[s]).standard_normal((B, V), dtype=np.float32)
        x *= np.float32(cfg.logit_std)
        np.clip(x, -clip, clip, out=x)
        logits[s] = x if cfg.dtype == "f32" else bf16_bits_from_f32(x)

    with cf.ThreadPoolExecutor(max_workers=nthreads) as ex:
        list(ex.map(logit_job, range(b)))

    rng_p = np.random.default_rng(s_plant)
    draft_ids = np.full((b, L), -1, np.int32)
    planted = np.zeros((b, L), bool)
    plant_bits = (np.float32(plant_val) if cfg.dtype == "f32"
                  else bf16_bits_from_f32(np.array([plant_val], np.float32))[0])
    for s in range(b):
        p = cfg.plant if not isinstance(cfg.plant, tuple) else float(
            rng_p.uniform(cfg.plant[0], cfg.plant[1]))
        for r in range(int(num_ref[s])):
            row = int(np.flatnonzero(step_map[s] == r + 1)[0])
            tok = int(rng_p.integers(0, V))
            if rng_p.random() < p:
                logits[s, row, tok] = plant_bits
                planted[s, r] = True
            elif bad_draft_rate > 0 and rng_p.random() < bad_draft_rate:
                tok = int(rng_p.choice([-7, -1, V, V + 123]))
            draft_ids[s, r] = tok

    return VerifyInputs(cfg=cfg, q=q, k_new=k_new, v_new=v_new, k_cache=k_cache,
                        v_cache=v_cache, block_table=block_table, prefix_lens=prefix_lens,
                        step_map=step_map, num_ref=num_ref, logits=logits,
                        draft_ids=draft_ids, planted=planted, seed_entropy=entropy,
                        poison=poison)


def generate_draft_side(inp: VerifyInputs, corr: float = 0.8,
                        threads: Optional[int] = None):
    """Drafter-side inputs of the stochastic acceptance rule, for `inp`.

    Returns (draft_logits [batch, L, V] in the config's dtype, uniforms
    float32 [batch, L + 1] in [0, 1)).  Draft row r (r < gamma_b) is
    corr * (the target logits of draft r's verification row) + sqrt(1 - corr^2)
    * N(0, logit_std^2), clipped like the target rows, with the draft token's
    own entry raised to the planting value: the drafter rated its proposal
    highly, as it would a sampled token.  Rows past gamma_b are plain noise.
    The uniforms are the random numbers of the rule (u_1..u_L, then the draw).
    From child stream 10 of the sequence's SeedSequence, so the other inputs
    are unchanged.
    """
    cfg = inp.cfg
    b, B, L, V = cfg.batch, cfg.block_size, cfg.max_ref, cfg.vocab
    s_draft = np.random.SeedSequence(inp.seed_entropy).spawn(11)[10]
    s_rows, s_u = s_draft.spawn(2)
    sd = np.float32(cfg.logit_std)
    clip = np.float32(6.0 * cfg.logit_std)
    plant_val = np.float32(6.25 * cfg.logit_std)
    np_dtype = np.float32 if cfg.dtype == "f32" else np.uint16
    draft_logits = np.empty((b, L, V), np_dtype)
    row_streams = s_rows.spawn(b)
    a, c = np.float32(corr), np.float32(np.sqrt(1.0 - corr * corr))

    def as_f32(x):
        return x if cfg.dtype == "f32" else (x.astype(np.uint32) << 16).view(np.float32)

    def job(s):
        rng = np.random.default_rng(row_streams[s])
        gamma = int(inp.num_ref[s])
        for r in range(L):
            x = rng.standard_normal(V, dtype=np.float32) * sd
            if r < gamma:
                k = int(np.flatnonzero(inp.step_map[s] == r + 1)[0])
                x = a * as_f32(inp.logits[s, k]) + c * x
            np.clip(x, -clip, clip, out=x)
            tok = int(inp.draft_ids[s, r])
            if r < gamma and 0 <= tok < V:
                x[tok] = plant_val
            draft_logits[s, r] = x if cfg.dtype == "f32" else bf16_bits_from_f32(x)

    nthreads = threads or min(16, os.cpu_count() or 1)
    with cf.ThreadPoolExecutor(max_workers=nthreads) as ex:
        list(ex.map(job, range(b)))
    u = np.random.default_rng(s_u).random((b, L + 1)).astype(np.float32)
    np.minimum(u, np.nextafter(np.float32(1), np.float32(0)), out=u)
    return draft_logits, u


def generate_lmhead_side(inp: VerifyInputs, hidden_size: int, threads: Optional[int] = None):
    """Final hidden states and LM-head weight for `inp`, in its dtype.

    Returns (hidden [batch, B, H], weight [V, H]).  weight ~ N(0, logit_std^2 / H)
    so that logits = hidden . weight^T have the workload's spread for
    hidden ~ N(0, 1).  For a planted draft (``inp.planted``) the hidden state of
    its verification row is pulled towards the draft's weight row:
    h = 0.5 * noise + (6.25 * logit_std / |w_D|^2) * w_D, which puts the draft's
    logit near 6.25 sigma (no logit or maximum is computed here).  From child
    stream 11 of the sequence's SeedSequence.
    """
    cfg = inp.cfg
    b, B, V, H = cfg.batch, cfg.block_size, cfg.vocab, hidden_size
    s_lm = np.random.default_rng(np.random.SeedSequence(inp.seed_entropy).spawn(12)[11])
    wstd = np.float32(cfg.logit_std / np.sqrt(H))
    bf16 = cfg.dtype != "f32"
    weight = np.empty((V, H), np.uint16 if bf16 else np.float32)
    step = 1 << 13
    streams = s_lm.bit_generator.seed_seq.spawn((V + step - 1) // step + 1)

    def wjob(i):                                  # bounded float32 temporaries
        v0 = i * step
        x = np.random.default_rng(streams[i]).standard_normal((min(step, V - v0), H), dtype=np.float32)
        x *= wstd
        weight[v0:v0 + step] = bf16_bits_from_f32(x) if bf16 else x

    nthreads = threads or min(16, os.cpu_count() or 1)
    with cf.ThreadPoolExecutor(max_workers=nthreads) as ex:
        list(ex.map(wjob, range((V + step - 1) // step)))
    hidden = np.random.default_rng(streams[-1]).standard_normal((b, B, H), dtype=np.float32)
    as_f32 = (lambda a: (a.astype(np.uint32) << 16).view(np.float32)) if bf16 else (lambda a: a)
    for s in range(b):
        for r in range(int(inp.num_ref[s])):
            if not inp.planted[s, r]:
                continue
            k = int(np.flatnonzero(inp.step_map[s] == r + 1)[0])
            w = as_f32(weight[int(inp.draft_ids[s, r])])
            hidden[s, k] = np.float32(0.5) * hidden[s, k] + \
                np.float32(6.25 * cfg.logit_std / float(np.dot(w, w))) * w
    return (bf16_bits_from_f32(hidden) if bf16 else hidden), weight
