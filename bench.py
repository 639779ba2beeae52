#!/usr/bin/env python3
"""Benchmark of the SimSD verification step on one MI355X.

One step = simsd_verify_attention + simsd_verify_accept (or, with --accept
sampled, simsd_verify_accept_sampled: eq. 2 at temperature T with the drafter's
logits) over one batch of seeded synthetic inputs already resident in HBM,
launched back to back on one stream.  Prints ONE JSON line: verified tokens/s (sum over sequences of the
drafted tokens checked per step, divided by the step time), the roofline of the
dominant kernel (attention) measured with HIP events inside the timed region,
and the CPU oracle's rate on a bounded sample of the same workload.

Inputs are cycled through several copies when one step's bytes fit in the
256 MB last-level cache, so every step reads its inputs from HBM.
"""

from __future__ import annotations

import argparse
import ctypes
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


def workload_numbers(inp, sampled=False):
    """Algorithmic bytes and flops of one step (see the design notes).  The
    sampled rule reads the verification row and the draft row of every draft."""
    cfg = inp.cfg
    s = cfg.elem_bytes
    b, Hq, Hkv, d, n_new, B = (cfg.batch, cfg.num_q_heads, cfg.num_kv_heads, cfg.head_dim,
                               cfg.n_new, cfg.block_size)
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
                                               inp.step_map[sl], inp.num_ref[sl], inp.cfg.dtype)[:4]
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
        if sampled is None:
            rt, _, _, ra = accept_oracle(every)
            ok &= bool(np.array_equal(outputs["tid"].cpu().numpy(), rt))
            ok &= bool(np.array_equal(outputs["alen"].cpu().numpy(), ra))
        else:
            # float32 probabilities against float64: a uniform within rounding
            # of its threshold may fall either way (the tests move them apart)
            _, _, ra, rc = accept_oracle(every)
            ok &= bool(np.array_equal(outputs["alen"].cpu().numpy(), ra))
            ok &= bool(np.array_equal(outputs["corr"].cpu().numpy(), rc))
        return {"checked": f"attention pairs {pairs}, accept all rows", "ok": ok}

    from threadpoolctl import threadpool_info
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
    threads = max([t.get("num_threads", 1) for t in threadpool_info()] + [1])
    base = {"value": tokens / dt, "unit": "verified tokens/s", "cores": threads,
            "kind": "oracle", "sample": sample + f", {dt:.1f} s float64 numpy"}
    return base, (parity_check(inp, outputs) if outputs is not None else None)


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=300)
    ap.add_argument("--warmup", type=int, default=30)
    ap.add_argument("--config", type=int, default=2, choices=[1, 2, 3, 4, 5],
                    help="workload (1 tiny-f32, 2 sdar-1.7b-layer, 3 sdar-8b-layer, "
                         "4 long-context, 5 ragged-paged)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
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
              "(the verification step shards by sequence / KV head with no exchange; "
              "see the design notes).", file=sys.stderr)
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
    from paper_2606_02544_amd import binding
    from synth import CONFIGS, generate, generate_draft_side, generate_lmhead_side

    cfg = CONFIGS[args.config]
    custom = args.gamma is not None or args.committed or args.rope_theta > 0
    if custom:
        import dataclasses
        g = cfg.max_ref if args.gamma is None else args.gamma
        if not 0 <= g <= cfg.block_size or not 0 <= args.committed <= cfg.block_size - g:
            sys.exit(f"need 0 <= gamma <= {cfg.block_size} and 0 <= committed <= B - gamma")
        cfg = dataclasses.replace(cfg, max_ref=g, committed=args.committed)
    torch.cuda.init()
    dev = torch.device("cuda:0")
    print(f"[bench] generating {cfg.name}", file=sys.stderr, flush=True)
    inp = generate(cfg)
    sampled = args.accept == "sampled"
    if sampled and args.lmhead:
        sys.exit("--lmhead computes the greedy rule; it does not combine with --accept sampled")
    dlog_np, unif_np = generate_draft_side(inp) if sampled else (None, None)
    H = args.hidden or (2048 if cfg.name == "sdar-1.7b-layer" else 4096)
    hid_np, w_np = generate_lmhead_side(inp, H) if args.lmhead else (None, None)
    wl = workload_numbers(inp, sampled)
    if args.lmhead:
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
    if args.lmhead:
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
    adesc = binding.attention_desc(
        base["q"], base["k_cache"], num_kv_heads=cfg.num_kv_heads, block_size=B, max_ref=L,
        max_prefix_len=cfg.max_prefix, page_size=cfg.page_size,
        max_pages_per_seq=0 if inp.block_table is None else inp.block_table.shape[1],
        kv_chunk=args.kv_chunk, rope_theta=args.rope_theta)
    cdesc = (binding.lmhead_desc(base["hidden"], base["weight"], L) if args.lmhead
             else binding.accept_desc(base["logits"], L))
    aws_n = binding.attention_workspace_size(adesc)
    cws_n = (binding.accept_sampled_workspace_size(cdesc) if sampled
             else binding.lmhead_workspace_size(cdesc) if args.lmhead
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
            elif args.lmhead:
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
             lib.simsd_verify_accept_lmhead if args.lmhead else lib.simsd_verify_accept)

    def launch_step(i, what=("attn", "acc")):
        a_args, c_args = calls[i % len(calls)]
        st = 0
        if "attn" in what:
            st |= f_attn(*a_args)
        if "acc" in what:
            st |= f_acc(*c_args)
        if st:
            raise RuntimeError(lib.simsd_last_error().decode())

    K, W = args.steps, args.warmup
    print(f"[bench] {cfg.name}: {copies} input copies, {step_bytes / 1e6:.1f} MB per step; "
          f"warmup {W}, steps {K}, hip graph {not args.no_graph}", file=sys.stderr, flush=True)
    graphs = {}
    use_graph = not args.no_graph
    if use_graph:
        # One graph per sequence of launches: the K timed steps, the warmup, and
        # attention-only / accept-only passes over every input copy for the
        # per-kernel durations.  The library never allocates or synchronises,
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
    # leave the outputs of the last timed step in place for the parity check
    run("steps", K)
    torch.cuda.synchronize()
    print(f"[bench] done: {elapsed / K * 1e3:.4f} ms/step (attention {attn_ms * 1e3:.2f} us, "
          f"accept {acc_ms * 1e3:.2f} us per launch)", file=sys.stderr, flush=True)

    value = wl["verified"] * K / elapsed
    attn_gbs = wl["attn_bytes"] / (attn_ms * 1e-3) / 1e9
    traffic = None if custom else recorded_traffic(cfg.name)
    line = {
        "metric": METRIC,
        "value": value,
        "unit": "verified tokens/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": elapsed / K * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if dt == "bf16" else "f32",
        "data": "synthetic",
        "config": {
            "workload": f"{cfg.name}: batch {b}, {cfg.num_q_heads}/{cfg.num_kv_heads} heads, "
                        f"head_dim {cfg.head_dim}, prefix {cfg.prefix}, block {B}, "
                        f"{L} reference slots, vocab {cfg.vocab}"
                        + (f", gamma {L}, {cfg.committed} committed" if custom else "")
                        + (f", RoPE base {args.rope_theta:g} fused" if args.rope_theta > 0 else "")
                        + (f", paged {cfg.page_size}" if cfg.page_size else ""),
            "step_hbm_bytes": step_bytes,
            "step_hbm_gbs": step_bytes / (elapsed / K) / 1e9,
            "step_roofline_frac": step_bytes / (elapsed / K) / 1e9 / HBM_PEAK_GBS,
            "attention_us": attn_ms * 1e3,
            "accept_us": acc_ms * 1e3,
            "accept_gbs": wl["accept_bytes"] / (acc_ms * 1e-3) / 1e9,
            **({"lmhead_tflops": wl["lmhead_flops"] / (acc_ms * 1e-3) / 1e12,
                "lmhead_mfma_frac": wl["lmhead_flops"] / (acc_ms * 1e-3) / 1e12 / BF16_MFMA_PEAK_TFLOPS,
                "lmhead_roofline": lmhead_roofline(wl["lmhead_flops"], wl["accept_bytes"], acc_ms)}
               if args.lmhead else {}),
            "scanned_rows_per_s": wl["scanned_rows"] * K / elapsed,
            "attention_mfma_frac": wl["attn_flops"] / (attn_ms * 1e-3) / 1e12 / BF16_MFMA_PEAK_TFLOPS,
            "input_copies": copies,
            "hip_graph": use_graph,
            "kv_chunk": args.kv_chunk,
            "accept_rule": (f"sampled, temperature {args.temperature}" if sampled else
                            f"greedy, LM head fused (hidden {H})" if args.lmhead else "greedy"),
        },
        "roofline": {
            "bound": "hbm",
            "achieved": attn_gbs,
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": attn_gbs / HBM_PEAK_GBS,
            "traffic": traffic,
        },
    }
    if not args.no_cpu_baseline:
        # The oracle leg: its rate on the host, and (unless --no-check) the last
        # timed step's outputs checked against it on sampled pairs.
        print("[bench] timing the CPU oracle", file=sys.stderr, flush=True)
        outputs = None if args.no_check else dict(out=out, lse=lse, tid=tid, alen=alen, corr=corr)
        line["cpu_baseline"], line["parity"] = cpu_baseline(
            inp, args.cpu_seconds, outputs,
            sampled=(dlog_np, unif_np, args.temperature) if sampled else None,
            rope_theta=args.rope_theta, lmhead=(hid_np, w_np) if args.lmhead else None)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
