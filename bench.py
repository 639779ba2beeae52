#!/usr/bin/env python3
"""Benchmark of the SimSD verification step on one MI355X.

One step = simsd_verify_attention + simsd_verify_accept (or, with --accept
sampled, simsd_verify_accept_sampled: eq. 2 at temperature T with the drafter's
logits; with --lmhead, simsd_verify_accept_lmhead) over one batch of seeded
synthetic inputs already resident in HBM, launched back to back on one stream.

Prints ONE JSON line.  Its top level is the headline workload (default: the
ragged-paged batch, the largest single-GPU workload): verified tokens/s (the
drafted tokens checked per step, summed over sequences, divided by the step
time), the roofline of the dominant call (attention) measured with HIP events
inside the timed region, and the CPU oracle's rate on a bounded sample of the
same workload.  With the default options the same line carries a record per
further workload (SDAR-1.7B layer, SDAR-8B layer, long context) under
"workloads", each with its own timing, roofline fractions, oracle baseline
and parity verdict.

Inputs are cycled through several copies when one step's bytes fit in the
256 MB last-level cache, so every step reads its inputs from HBM.
"""

from __future__ import annotations

import argparse
import ctypes
import dataclasses
import hashlib
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "verify-step tokens/sec + achieved HBM GB/s (% roofline), 1×MI355X"
HBM_PEAK_GBS = 8000.0
BF16_MFMA_PEAK_TFLOPS = 2500.0
ATTN_SOURCES = ["paper_2606_02544_amd/csrc/simsd_attention.hip"]
PAPER_CONTEXT = ("the paper reports up to 7.46x end-to-end decoding throughput of SimSD over "
                 "vanilla decoding with TP 2 (Table 1: SDAR-1.7B drafting for SDAR-8B, FP32, "
                 "NVIDIA RTX PRO 6000); context only, not this metric")


def workload_numbers(inp, sampled=False):
    """Algorithmic bytes and flops of one step.  Attention: the prefix K and V
    once per KV head, the new slots' q, k, v, the output and the LSE.  Accept:
    every scanned logits row once (the sampled rule reads the verification row
    and the draft row of every draft)."""
    cfg = inp.cfg
    s = cfg.elem_bytes
    b, Hq, Hkv, d, n_new = (cfg.batch, cfg.num_q_heads, cfg.num_kv_heads, cfg.head_dim,
                            cfg.n_new)
    prefix = int(np.sum(inp.prefix_lens.astype(np.int64)))
    kv_bytes = 2 * prefix * Hkv * d * s
    new_bytes = b * n_new * (2 * Hq * d * s + 2 * Hkv * d * s) + b * Hq * n_new * 4
    attn_bytes = kv_bytes + new_bytes
    scanned = 2 * int(np.sum(inp.num_ref)) if sampled else int(np.sum(inp.step_map >= 1))
    accept_bytes = scanned * cfg.vocab * s
    # every non-padded row sees prefix + (non-padded block slots) keys; QK^T and PV
    keys = 0
    for q in range(b):
        nonpad = int(np.sum(inp.step_map[q] >= 0))
        rows = nonpad + int(inp.num_ref[q])
        keys += rows * (int(inp.prefix_lens[q]) + nonpad)
    attn_flops = 4 * keys * Hq * d
    return dict(attn_bytes=attn_bytes, accept_bytes=accept_bytes, attn_flops=attn_flops,
                verified=int(np.sum(inp.num_ref)), scanned_rows=int(np.sum(inp.step_map >= 1)))


def lmhead_roofline(flops, nbytes, call_ms):
    """Roofline of the LM-head accept call (scan, merge and finalize kernels): bound by
    MFMA when its intensity exceeds the bf16 ridge point, else by HBM."""
    sec = call_ms * 1e-3
    if flops / nbytes > BF16_MFMA_PEAK_TFLOPS * 1e12 / (HBM_PEAK_GBS * 1e9):
        a = flops / sec / 1e12
        return {"bound": "mfma", "achieved": a, "peak": BF16_MFMA_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": a / BF16_MFMA_PEAK_TFLOPS}
    a = nbytes / sec / 1e9
    return {"bound": "hbm", "achieved": a, "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": a / HBM_PEAK_GBS}


def source_digest(paths):
    h = hashlib.sha256()
    for p in paths:
        with open(os.path.join(ROOT, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def recorded_traffic(workload: str):
    """HBM bytes per attention launch from the committed rocprofv3 counter
    summary, if it was taken on the current kernel source; else None."""
    path = os.path.join(ROOT, "profiles", f"attention_traffic_{workload}.md")
    if not os.path.exists(path):
        return None
    fields = {}
    with open(path) as f:
        for line in f:
            if ":" in line and line.startswith("- "):
                k, v = line[2:].split(":", 1)
                fields[k.strip()] = v.strip().strip("`")
    if fields.get("source_sha256_16") != source_digest(ATTN_SOURCES):
        return None
    try:
        return float(fields["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def host_cores():
    from threadpoolctl import threadpool_info
    blas = max([t.get("num_threads", 1) for t in threadpool_info()
                if t.get("user_api") == "blas"] + [1])
    return {"affinity": len(os.sched_getaffinity(0)), "cpu_count": os.cpu_count(),
            "blas_threads": blas}


def walk_accept(tid, draft_ids, step_map, num_ref):
    """Longest prefix of drafts equal to the target ids of their verification
    rows (used where several target ids are valid, as in the fused LM head)."""
    out = np.zeros(len(num_ref), np.int32)
    for s in range(len(num_ref)):
        for r in range(int(num_ref[s])):
            k = int(np.flatnonzero(step_map[s] == r + 1)[0])
            if int(tid[s, k]) != int(draft_ids[s, r]):
                break
            out[s] += 1
    return out


def cpu_baseline(inp, seconds: float, outputs=None, sampled=None, rope_theta=0.0, lmhead=None):
    """The oracle leg.  The oracle (float64 numpy) on the same workload,
    repeated whole steps until ``seconds`` have passed, or on a subset of
    (sequence, KV head) pairs plus their sequences' accept rows when one step
    takes longer; then, given the GPU outputs, the parity check.  `sampled` =
    (draft_logits, uniforms, T) times and checks the stochastic rule instead.
    Returns (baseline, parity or None)."""
    import oracle

    def accept_oracle(sl):
        if lmhead is not None:
            hidden, weight = lmhead
            return oracle.verify_accept_lmhead(hidden[sl], weight, inp.draft_ids[sl],
                                               inp.step_map[sl], inp.num_ref[sl], inp.cfg.dtype)
        if sampled is None:
            return oracle.verify_accept(inp.logits[sl], inp.draft_ids[sl], inp.step_map[sl],
                                        inp.num_ref[sl], inp.cfg.dtype)
        dlog, unif, T = sampled
        return oracle.verify_accept_sampled(inp.logits[sl], dlog[sl], inp.draft_ids[sl],
                                            inp.step_map[sl], inp.num_ref[sl],
                                            unif[sl].astype(np.float64), T, inp.cfg.dtype)

    def parity_check(inp, outputs):
        """The GPU outputs of the last timed step against the oracle: attention on
        the first and the last (sequence, KV head) pair, accept on every row."""
        cfg = inp.cfg
        dt = cfg.dtype
        b = cfg.batch
        o = outputs["out"].float().cpu().double().numpy()
        l_ = outputs["lse"].cpu().double().numpy()
        pairs = [(0, 0), (b - 1, cfg.num_kv_heads - 1)]
        ro, rl = oracle.verify_attention(inp, pairs=pairs, rope_theta=rope_theta)
        G = cfg.group
        ok = True
        for s_, h_ in pairs:
            sl = slice(h_ * G, (h_ + 1) * G)
            err = np.abs(o[s_, :, sl] - ro[s_, :, sl]).max(-1)
            ref = np.abs(ro[s_, :, sl]).max(-1)
            tol = 2e-2 * ref if dt == "bf16" else np.full_like(ref, 1e-5)
            ok &= bool(np.all(err <= tol))
            ok &= bool(np.all(np.abs(l_[s_, sl] - rl[s_, sl]) <= 1e-4 * np.maximum(1, np.abs(rl[s_, sl]))))
        every = slice(None)
        tid = outputs["tid"].cpu().numpy()
        alen = outputs["alen"].cpu().numpy()
        if lmhead is not None:
            # fp32-accumulated logits: an id may differ from the float64 oracle's
            # only at a near-tie (top two within 1e-4); accept_len follows the
            # GPU's own ids, and equals the oracle's where no id differs
            rt, _, _, ra, logits = accept_oracle(every)
            differ = 0
            for s_, k_ in zip(*np.nonzero(inp.step_map >= 1)):
                if tid[s_, k_] != rt[s_, k_]:
                    row = logits[s_, k_]
                    ok &= bool(0 <= tid[s_, k_] < row.size and
                               row.max() - row[tid[s_, k_]] <= 1e-4 * max(1.0, abs(row.max())))
                    differ += 1
            ok &= bool(np.array_equal(alen, walk_accept(tid, inp.draft_ids, inp.step_map,
                                                        inp.num_ref)))
            if differ == 0:
                ok &= bool(np.array_equal(alen, ra))
        elif sampled is None:
            rt, _, _, ra = accept_oracle(every)
            ok &= bool(np.array_equal(tid, rt))
            ok &= bool(np.array_equal(alen, ra))
        else:
            # float32 probabilities against float64: a uniform within rounding
            # of its threshold may fall either way (the tests move them apart)
            _, _, ra, rc = accept_oracle(every)
            ok &= bool(np.array_equal(alen, ra))
            ok &= bool(np.array_equal(outputs["corr"].cpu().numpy(), rc))
        return {"checked": f"attention pairs {pairs}, accept all rows", "ok": ok}

    cfg = inp.cfg
    pairs = [(s, h) for s in range(cfg.batch) for h in range(cfg.num_kv_heads)]
    t0 = time.perf_counter()
    steps = 0
    done_pairs = 0
    tokens = 0.0
    per_pair_tokens = float(np.sum(inp.num_ref)) / len(pairs)
    # one step: attention over all pairs, then the accept scan
    while time.perf_counter() - t0 < seconds:
        for (s, h) in pairs:
            oracle.verify_attention(inp, pairs=[(s, h)], rope_theta=rope_theta)
            done_pairs += 1
            tokens += per_pair_tokens
            if time.perf_counter() - t0 >= seconds:
                break
        else:
            accept_oracle(slice(None))
            steps += 1
    dt = time.perf_counter() - t0
    if steps == 0:
        # Partial step: charge the accept scan of the sampled sequences too.
        seqs = sorted({s for s, _ in pairs[:done_pairs]})
        t1 = time.perf_counter()
        accept_oracle(np.array(seqs))
        dt += time.perf_counter() - t1
        sample = f"{done_pairs} of {len(pairs)} (sequence, KV head) pairs + accept of {len(seqs)} sequences"
    else:
        sample = f"{steps} whole steps" + (f" + {done_pairs - steps * len(pairs)} pairs" if done_pairs > steps * len(pairs) else "")
    hc = host_cores()
    base = {"value": tokens / dt, "unit": "verified tokens/s", "cores": hc["blas_threads"],
            "kind": "oracle", "sample": sample + f", {dt:.1f} s float64 numpy",
            "host": hc}
    return base, (parity_check(inp, outputs) if outputs is not None else None)


def measure(torch, cfg, args, K, W, *, headline: bool, cpu_seconds: float, custom: bool):
    """Times one workload and returns its record (the top level of the line
    for the headline, a sub-record otherwise)."""
    from paper_2606_02544_amd import binding
    from synth import generate, generate_draft_side, generate_lmhead_side

    dev = torch.device("cuda:0")
    print(f"[bench] generating {cfg.name}", file=sys.stderr, flush=True)
    inp = generate(cfg)
    sampled = headline and args.accept == "sampled"
    lmhead = headline and args.lmhead
    dlog_np, unif_np = generate_draft_side(inp) if sampled else (None, None)
    H = args.hidden or (2048 if cfg.name == "sdar-1.7b-layer" else 4096)
    hid_np, w_np = generate_lmhead_side(inp, H) if lmhead else (None, None)
    wl = workload_numbers(inp, sampled)
    if lmhead:
        # the head's weight once, the rows' hidden states; flops of the product
        wl["accept_bytes"] = cfg.vocab * H * 2 + cfg.batch * cfg.block_size * H * 2
        wl["lmhead_flops"] = 2 * cfg.batch * cfg.block_size * cfg.vocab * H
    step_bytes = wl["attn_bytes"] + wl["accept_bytes"]
    copies = max(1, math.ceil(args.rotate_mb * 1e6 / step_bytes))
    copies = min(copies, max(1, int(40e9 // step_bytes)))

    def to_dev(a, dt):
        if dt == "bf16":
            return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(dev)
        if dt == "f32":
            return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(dev)
        return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(dev)

    dt = cfg.dtype
    base = dict(q=to_dev(inp.q, dt), k_new=to_dev(inp.k_new, dt), v_new=to_dev(inp.v_new, dt),
                k_cache=to_dev(inp.k_cache, dt), v_cache=to_dev(inp.v_cache, dt),
                block_table=None if inp.block_table is None else to_dev(inp.block_table, "i32"),
                prefix_lens=to_dev(inp.prefix_lens, "i32"), step_map=to_dev(inp.step_map, "i32"),
                num_ref=to_dev(inp.num_ref, "i32"), logits=to_dev(inp.logits, dt),
                draft_ids=to_dev(inp.draft_ids, "i32"))
    if lmhead:
        del base["logits"]
        base["hidden"] = to_dev(hid_np, dt)
        base["weight"] = to_dev(w_np, dt)
    if sampled:
        base["draft_logits"] = to_dev(dlog_np, dt)
        base["uniforms"] = torch.from_numpy(unif_np).to(dev)
    sets = [base] + [{k: (None if v is None else v.clone()) for k, v in base.items()}
                     for _ in range(copies - 1)]

    b, B, L = cfg.batch, cfg.block_size, cfg.max_ref
    out = torch.empty_like(base["q"])
    lse = torch.empty((b, cfg.num_q_heads, cfg.n_new), dtype=torch.float32, device=dev)
    tid = torch.empty((b, B), dtype=torch.int32, device=dev)
    conf = torch.empty((b, B), dtype=torch.float32, device=dev)
    dprob = torch.empty((b, L), dtype=torch.float32, device=dev)
    alen = torch.empty((b,), dtype=torch.int32, device=dev)
    pdraft = torch.empty((b, L), dtype=torch.float32, device=dev)
    corr = torch.empty((b,), dtype=torch.int32, device=dev)
    kv_chunk = args.kv_chunk if headline else 0
    rope_theta = args.rope_theta if headline else 0.0
    adesc = binding.attention_desc(
        base["q"], base["k_cache"], num_kv_heads=cfg.num_kv_heads, block_size=B, max_ref=L,
        max_prefix_len=cfg.max_prefix, page_size=cfg.page_size,
        max_pages_per_seq=0 if inp.block_table is None else inp.block_table.shape[1],
        kv_chunk=kv_chunk, rope_theta=rope_theta)
    cdesc = (binding.lmhead_desc(base["hidden"], base["weight"], L) if lmhead
             else binding.accept_desc(base["logits"], L))
    aws_n = binding.attention_workspace_size(adesc)
    cws_n = (binding.accept_sampled_workspace_size(cdesc) if sampled
             else binding.lmhead_workspace_size(cdesc) if lmhead
             else binding.accept_workspace_size(cdesc))
    aws = torch.zeros(max(aws_n, 16), dtype=torch.uint8, device=dev)
    cws = torch.zeros(max(cws_n, 16), dtype=torch.uint8, device=dev)

    lib = binding.lib()
    P = ctypes.c_void_p
    ptr = lambda t: None if t is None else P(t.data_ptr())

    def build_calls(stream):
        """ctypes argument tuples of both entry points for every input copy."""
        sp = P(stream.cuda_stream)
        out_calls = []
        for s in sets:
            a_args = (ctypes.byref(adesc), ptr(s["q"]), ptr(s["k_new"]), ptr(s["v_new"]),
                      ptr(s["k_cache"]), ptr(s["v_cache"]), ptr(s["block_table"]),
                      ptr(s["prefix_lens"]), ptr(s["step_map"]), ptr(s["num_ref"]), ptr(out),
                      ptr(lse), ptr(aws), aws_n, sp)
            if sampled:
                c_args = (ctypes.byref(cdesc), ctypes.c_float(args.temperature), ptr(s["logits"]),
                          ptr(s["draft_logits"]), ptr(s["draft_ids"]), ptr(s["step_map"]),
                          ptr(s["num_ref"]), ptr(s["uniforms"]), ptr(dprob), ptr(pdraft),
                          ptr(alen), ptr(corr), ptr(cws), cws_n, sp)
            elif lmhead:
                c_args = (ctypes.byref(cdesc), ptr(s["hidden"]), ptr(s["weight"]),
                          ptr(s["draft_ids"]), ptr(s["step_map"]), ptr(s["num_ref"]), ptr(tid),
                          ptr(conf), ptr(dprob), ptr(alen), ptr(cws), cws_n, sp)
            else:
                c_args = (ctypes.byref(cdesc), ptr(s["logits"]), ptr(s["draft_ids"]),
                          ptr(s["step_map"]), ptr(s["num_ref"]), ptr(tid), ptr(conf), ptr(dprob),
                          ptr(alen), ptr(cws), cws_n, sp)
            out_calls.append((a_args, c_args))
        return out_calls

    calls = build_calls(torch.cuda.current_stream())
    f_attn = lib.simsd_verify_attention
    f_acc = (lib.simsd_verify_accept_sampled if sampled else
             lib.simsd_verify_accept_lmhead if lmhead else lib.simsd_verify_accept)

    def launch_step(i, what=("attn", "acc")):
        a_args, c_args = calls[i % len(calls)]
        st = 0
        if "attn" in what:
            st |= f_attn(*a_args)
        if "acc" in what:
            st |= f_acc(*c_args)
        if st:
            raise RuntimeError(lib.simsd_last_error().decode())

    use_graph = not args.no_graph
    # Sub-records: enough steps for a stable wall-clock figure on the
    # microsecond-scale workloads (the headline times exactly K steps).
    if not headline:
        est_ms = max(step_bytes / (4e12) * 1e3, 0.01)
        K = max(K, min(2000, math.ceil(30.0 / est_ms)))
        W = max(W, 5)
    n_dist = max(20, min(200, K))
    print(f"[bench] {cfg.name}: {copies} input copies, {step_bytes / 1e6:.1f} MB per step; "
          f"warmup {W}, steps {K}, hip graph {use_graph}", file=sys.stderr, flush=True)
    graphs = {}
    ones = []
    if use_graph:
        # One graph per sequence of launches: the K timed steps, the warmup,
        # attention-only / accept-only passes over every input copy for the
        # per-call durations, and one single-step graph per copy for the
        # per-step distribution.  The library never allocates or synchronises,
        # so its launches capture as they are.
        cap = torch.cuda.Stream()
        eager_calls = calls
        calls = build_calls(cap)
        with torch.cuda.stream(cap):
            launch_step(0)
            torch.cuda.synchronize()
            for name, n, what in (("warm", W, ("attn", "acc")), ("steps", K, ("attn", "acc")),
                                  ("attn", copies, ("attn",)), ("acc", copies, ("acc",))):
                g = torch.cuda.CUDAGraph()
                with torch.cuda.graph(g, stream=cap):
                    for i in range(n):
                        launch_step(i, what)
                graphs[name] = g
            for i in range(min(copies, n_dist)):
                g = torch.cuda.CUDAGraph()
                with torch.cuda.graph(g, stream=cap):
                    launch_step(i)
                ones.append(g)
        torch.cuda.synchronize()
        calls = eager_calls

    def run(name, n, what=("attn", "acc")):
        if use_graph:
            graphs[name].replay()
        else:
            for i in range(n):
                launch_step(i, what)

    run("warm", W)
    torch.cuda.synchronize()
    print(f"[bench] timing {K} steps", file=sys.stderr, flush=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    run("steps", K)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    elapsed = t1 - t0

    # Average duration of each entry point: HIP events on the launch stream
    # around back-to-back launches over every input copy (cold inputs).
    def per_launch_ms(name, what, reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        run(name, copies, what)
        torch.cuda.synchronize()
        e0.record(torch.cuda.current_stream())
        for _ in range(reps):
            run(name, copies, what)
        e1.record(torch.cuda.current_stream())
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / (reps * copies)

    reps = max(1, math.ceil(50 / copies))
    attn_ms = per_launch_ms("attn", ("attn",), reps)
    acc_ms = per_launch_ms("acc", ("acc",), reps)

    # Per-step distribution: HIP events between single-step launches.  The
    # GPU is first kept busy with plain copies so that the host has queued
    # every step before the first one starts: the event gaps are then the
    # steps' own durations, not the host's launch rate.
    dist = None
    if use_graph and ones:
        busy_src = torch.empty(1 << 28, dtype=torch.uint8, device=dev)
        busy_dst = torch.empty_like(busy_src)
        evs = [torch.cuda.Event(enable_timing=True) for _ in range(n_dist + 1)]
        for _ in range(max(4, math.ceil(n_dist * 0.03 / 0.07))):
            busy_dst.copy_(busy_src)
        evs[0].record()
        for i in range(n_dist):
            ones[i % len(ones)].replay()
            evs[i + 1].record()
        torch.cuda.synchronize()
        per = np.array([evs[i].elapsed_time(evs[i + 1]) for i in range(n_dist)]) * 1e3
        dist = {"steps": n_dist, "p10_us": float(np.percentile(per, 10)),
                "p50_us": float(np.percentile(per, 50)), "p90_us": float(np.percentile(per, 90)),
                "how": "HIP events between single-step graph launches, queued back to back"}
        del busy_src, busy_dst

    # leave the outputs of the last timed step in place for the parity check
    run("steps", K)
    torch.cuda.synchronize()
    print(f"[bench] {cfg.name} done: {elapsed / K * 1e3:.4f} ms/step (attention "
          f"{attn_ms * 1e3:.2f} us, accept {acc_ms * 1e3:.2f} us per call)",
          file=sys.stderr, flush=True)

    step_s = elapsed / K
    value = wl["verified"] / step_s
    a_np = alen.cpu().numpy().astype(np.int64)
    g_np = inp.num_ref.astype(np.int64)
    accepted = int(np.sum(a_np + (a_np < g_np)))
    attn_gbs = wl["attn_bytes"] / (attn_ms * 1e-3) / 1e9
    traffic = None if (custom and headline) else recorded_traffic(cfg.name)
    workload = (f"{cfg.name}: batch {b}, {cfg.num_q_heads}/{cfg.num_kv_heads} heads, "
                f"head_dim {cfg.head_dim}, prefix {cfg.prefix}, block {B}, "
                f"{L} reference slots, vocab {cfg.vocab}"
                + (f", gamma {L}, {cfg.committed} committed" if custom and headline else "")
                + (f", RoPE base {rope_theta:g} fused" if rope_theta > 0 else "")
                + (f", paged {cfg.page_size}" if cfg.page_size else ""))
    rec = {
        "workload": workload,
        "value": value,
        "unit": "verified tokens/s",
        "accepted_tokens_per_s": accepted / step_s,
        "steps": K,
        "warmup": W,
        "ms_per_step": step_s * 1e3,
        "step_hbm_bytes": step_bytes,
        "step_hbm_gbs": step_bytes / step_s / 1e9,
        "step_roofline_frac": step_bytes / step_s / 1e9 / HBM_PEAK_GBS,
        "attention_us": attn_ms * 1e3,
        "accept_us": acc_ms * 1e3,
        "accept_gbs": wl["accept_bytes"] / (acc_ms * 1e-3) / 1e9,
        "accept_roofline_frac": wl["accept_bytes"] / (acc_ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
        "attention_mfma_frac": wl["attn_flops"] / (attn_ms * 1e-3) / 1e12 / BF16_MFMA_PEAK_TFLOPS,
        "scanned_rows_per_s": wl["scanned_rows"] / step_s,
        "step_distribution": dist,
        "input_copies": copies,
        "hip_graph": use_graph,
        "kv_chunk": kv_chunk,
        "accept_rule": (f"sampled, temperature {args.temperature}" if sampled else
                        f"greedy, LM head fused (hidden {H})" if lmhead else "greedy"),
        "roofline": {
            "bound": "hbm",
            "achieved": attn_gbs,
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": attn_gbs / HBM_PEAK_GBS,
            "traffic": traffic,
            "prices": "one simsd_verify_attention call (attention kernel + merge kernel), "
                      "algorithmic bytes / HIP-event average duration",
        },
    }
    if lmhead:
        rec["lmhead_tflops"] = wl["lmhead_flops"] / (acc_ms * 1e-3) / 1e12
        rec["lmhead_roofline"] = lmhead_roofline(wl["lmhead_flops"], wl["accept_bytes"], acc_ms)
    if cpu_seconds > 0:
        # The oracle leg: its rate on the host, and (unless --no-check) the last
        # timed step's outputs checked against it on sampled pairs.
        print(f"[bench] timing the CPU oracle on {cfg.name}", file=sys.stderr, flush=True)
        outputs = None if args.no_check else dict(out=out, lse=lse, tid=tid, alen=alen, corr=corr)
        rec["cpu_baseline"], rec["parity"] = cpu_baseline(
            inp, cpu_seconds, outputs,
            sampled=(dlog_np, unif_np, args.temperature) if sampled else None,
            rope_theta=rope_theta, lmhead=(hid_np, w_np) if lmhead else None)
        rec["gpu_over_oracle"] = value / rec["cpu_baseline"]["value"]
        rec["paper_context"] = PAPER_CONTEXT
    # free this workload's device memory before the next one
    del sets, base, graphs, ones, out, lse, aws, cws
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return rec


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=300)
    ap.add_argument("--warmup", type=int, default=30)
    ap.add_argument("--config", type=int, default=5, choices=[1, 2, 3, 4, 5],
                    help="headline workload (1 tiny-f32, 2 sdar-1.7b-layer, 3 sdar-8b-layer, "
                         "4 long-context, 5 ragged-paged: the default, the largest)")
    ap.add_argument("--also", default="2,3,4",
                    help="further workloads recorded in the same line (comma-separated ids, "
                         "or 'none'); only with the default step options")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--also-cpu-seconds", type=float, default=5.0,
                    help="oracle time per further workload")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-check", action="store_true",
                    help="skip the parity check of the oracle leg")
    ap.add_argument("--rotate-mb", type=float, default=640.0,
                    help="cycle input copies until this many MB are touched per cycle")
    ap.add_argument("--kv-chunk", type=int, default=0)
    ap.add_argument("--accept", choices=["greedy", "sampled"], default="greedy",
                    help="acceptance rule: greedy (eq. 2 at T = 0) or sampled (eq. 2 at --temperature)")
    ap.add_argument("--temperature", type=float, default=1.0)
    ap.add_argument("--lmhead", action="store_true",
                    help="greedy acceptance from the final hidden states and the LM-head weight "
                         "(logits never stored) instead of from stored logits")
    ap.add_argument("--hidden", type=int, default=0,
                    help="LM-head hidden size (default: 2048 for the SDAR-1.7B layer, else 4096)")
    ap.add_argument("--gamma", type=int, default=None,
                    help="drafts per step (reference slots L = gamma <= B; default: the workload's); "
                         "0 = the plain block step once fewer than gamma positions remain")
    ap.add_argument("--rope-theta", type=float, default=0.0,
                    help="rotary base: q and the new keys arrive unrotated and the attention "
                         "kernel rotates them at the RoPE-copy positions (0 = off)")
    ap.add_argument("--committed", type=int, default=0,
                    help="block slots already committed by earlier steps of the block")
    ap.add_argument("--no-graph", action="store_true",
                    help="launch every kernel from Python instead of replaying HIP graphs")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="MB",
                    help="only copy MB megabytes a few times (counter calibration) and exit")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py measures one GPU only: --gpus {args.gpus} is not supported "
              "(the verification step would shard by sequence or KV head, with no "
              "exchange between GPUs).", file=sys.stderr)
        sys.exit(2)

    import torch
    if args.copy_probe:
        n = args.copy_probe * 1000 * 1000
        x = torch.ones(n, dtype=torch.uint8, device="cuda")
        y = torch.empty_like(x)
        for _ in range(5):
            y.copy_(x)
        torch.cuda.synchronize()
        print(json.dumps({"copy_probe_bytes": n, "launches": 5}))
        return
    from synth import CONFIGS

    cfg = CONFIGS[args.config]
    custom = args.gamma is not None or args.committed or args.rope_theta > 0
    if custom:
        g = cfg.max_ref if args.gamma is None else args.gamma
        if not 0 <= g <= cfg.block_size or not 0 <= args.committed <= cfg.block_size - g:
            sys.exit(f"need 0 <= gamma <= {cfg.block_size} and 0 <= committed <= B - gamma")
        cfg = dataclasses.replace(cfg, max_ref=g, committed=args.committed)
    torch.cuda.init()
    cpu_s = 0.0 if args.no_cpu_baseline else args.cpu_seconds
    head = measure(torch, cfg, args, args.steps, args.warmup, headline=True, cpu_seconds=cpu_s,
                   custom=custom)
    line = {
        "metric": METRIC,
        "value": head["value"],
        "unit": head["unit"],
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": head["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if cfg.dtype == "bf16" else "f32",
        "data": "synthetic",
        "config": {k: v for k, v in head.items()
                   if k not in ("value", "unit", "steps", "warmup", "ms_per_step", "roofline",
                                "cpu_baseline", "parity", "gpu_over_oracle", "paper_context")},
        "roofline": head["roofline"],
    }
    if "cpu_baseline" in head:
        line["cpu_baseline"] = head["cpu_baseline"]
        line["parity"] = head["parity"]
        line["gpu_over_oracle"] = head["gpu_over_oracle"]
        line["paper_context"] = head["paper_context"]
    plain = not (custom or args.lmhead or args.accept != "greedy" or args.kv_chunk or args.no_graph)
    also = [] if args.also.strip().lower() == "none" or not plain else \
        [int(x) for x in args.also.split(",") if x.strip() and int(x) != args.config]
    if also:
        sub_cpu = 0.0 if args.no_cpu_baseline else args.also_cpu_seconds
        line["workloads"] = {}
        for cid in also:
            rec = measure(torch, CONFIGS[cid], args, args.steps, args.warmup, headline=False,
                          cpu_seconds=sub_cpu, custom=False)
            line["workloads"][CONFIGS[cid].name] = rec
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
