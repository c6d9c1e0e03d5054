#!/usr/bin/env python3
"""Decode-step benchmark of the SpotAttention hot path on one MI355X.

One step = selector scoring of every KV block + dual top-p/top-K selection +
block-sparse GQA decode attention, for all sequences of one layer, on the
Qwen3-8B-shaped 128K-token workload (batch 4, 32 query / 8 KV heads, d = 128,
2048 blocks of 64 tokens, p = 0.95, K_max = 128, 1 sink + 2 recent blocks).
The headline value times spot_decode_step (all three stages in one launch):
the median of --repeats (5) runs of K back-to-back steps, each timed with HIP
events on the launch stream.  The three separate calls are timed too, with
their per-stage times.

Inputs are resident in HBM before timing starts.  The timed loop rotates
over NCOPY distinct copies of the KV cache and selector cache so that the
256 MB last-level cache cannot serve repeated steps.  Prints one JSON line.

    python bench.py [--steps K] [--warmup W] [--repeats R] [--gpus 1] [--no-cpu-baseline]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import platform
import re
import sys
import time

import numpy as np

HBM_PEAK_GBS = 8000.0
MFMA_BF16_PEAK_TFLOPS = 2500.0
METRIC = "decode steps/s at L=128K (selector+sparse attn), % of HBM peak GB/s"


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--copies", type=int, default=4)
    ap.add_argument("--repeats", type=int, default=5,
                    help="timed repeats of --steps steps; the headline is their median")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--no-dense", action="store_true", help="skip the dense decode baseline")
    ap.add_argument("--dense", action="store_true", help=argparse.SUPPRESS)   # the default
    ap.add_argument("--no-extra", action="store_true",
                    help="skip the quantized-selector and smaller-workload decode timings")
    ap.add_argument("--tokens", action="store_true",
                    help="run the per-token selector leg even with --no-extra")
    ap.add_argument("--fmt", default="bf16", choices=["bf16", "int4", "mxfp4", "int8", "mxfp8"])
    ap.add_argument("--no-prefill", action="store_true",
                    help="skip the block-sparse prefill leg (32K-token layer)")
    ap.add_argument("--prefill-iters", type=int, default=10)
    return ap.parse_args()


def log(msg):
    print(msg, file=sys.stderr, flush=True)


ROOT = os.path.dirname(os.path.abspath(__file__))
STEP_PROFILE = os.path.join(ROOT, "profiles", "decode_step_L131072_B4.md")
# Sources whose code the fused step kernel is built from.
STEP_SOURCES = ("step.hip", "decode_core.h", "score_core.h", "select_core.h", "spot_internal.h")
TOKENS_PROFILE = os.path.join(ROOT, "profiles", "score_tokens_L131072_B4.md")
TOKENS_SOURCES = ("score_tokens.hip", "score_core.h", "spot_internal.h")
SEED_TOKENS = 20260611
QUANT_TOKENS = 2048      # tokens per sequence quantized for the per-token format timings


def source_hash(files=STEP_SOURCES) -> str:
    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(ROOT, "paper_2606_22874_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic(path=STEP_PROFILE, files=STEP_SOURCES):
    """HBM bytes per launch from the committed rocprofv3 counter runs, or
    None when the kernel's sources changed since they were taken."""
    try:
        text = open(path).read()
    except OSError:
        return None
    m = re.search(r"traffic_bytes_per_launch: (\d+)\s*\(source: .*? sha256 prefix (\w+)\)",
                  text, re.S)
    if not m or m.group(2) != source_hash(files):
        return None
    return int(m.group(1))


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}): it measures the "
              "kernels on a single device's share of the work (a multi-GPU layout would "
              "shard by sequence and KV head, with no exchange on the decode path).",
              file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2606_22874_amd import spot, synth

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    dev = torch.device("cuda:0")
    spot.load()

    log("[bench] generating the 128K-token decode workload")
    t0 = time.time()
    wl = synth.decode_config(3)
    log(f"[bench] generated in {time.time() - t0:.1f}s")
    B, Hq, Hkv, d, L = wl.B, wl.Hq, wl.Hkv, wl.d, wl.L
    nblk, rule = wl.nblk, wl.rule

    def bf(a):
        return spot.to_device_bf16(a, dev)

    # Selector cache in the requested storage format.
    if args.fmt == "bf16":
        ksel_host, kscale_host = wl.k_sel, None
        sel_bytes = wl.k_sel.nbytes
    else:
        ksel_host, kscale_host = synth.QUANTIZERS[args.fmt](wl.k_sel)
        sel_bytes = ksel_host.nbytes + kscale_host.nbytes

    def dev_sel():
        if args.fmt == "bf16":
            return bf(ksel_host), None
        ks = torch.from_numpy(np.ascontiguousarray(ksel_host)).to(dev)
        sc = kscale_host.view(np.int16) if args.fmt in ("int4", "int8") else kscale_host
        return ks, torch.from_numpy(np.ascontiguousarray(sc)).to(dev)

    q = bf(wl.q)
    q_sel = bf(wl.q_sel)
    w = torch.from_numpy(wl.w).to(dev)
    seq_len = torch.from_numpy(wl.seq_len).to(dev)
    n_valid = torch.from_numpy(wl.n_valid).to(dev)
    k0, v0 = bf(wl.k), bf(wl.v)
    copies = []
    for c in range(args.copies):
        ks, sc = dev_sel()
        copies.append((k0 if c == 0 else k0.clone(), v0 if c == 0 else v0.clone(), ks, sc))
    torch.cuda.synchronize()

    scores = torch.empty((B, nblk), dtype=torch.float32, device=dev)
    idx = torch.empty((B, rule.k_max), dtype=torch.int32, device=dev)
    cnt = torch.empty(B, dtype=torch.int32, device=dev)
    mass = torch.empty(B, dtype=torch.float32, device=dev)
    out = torch.empty((B, Hq, d), dtype=torch.bfloat16, device=dev)
    lse = torch.empty((B, Hq), dtype=torch.float32, device=dev)
    ws = spot.decode_workspace(B, Hq, Hkv, d, rule.k_max, dev)
    ws_step = spot.step_workspace(B, Hq, Hkv, d, rule.k_max, dev)
    stream = torch.cuda.current_stream()

    def score(c):
        _, _, ks, sc = copies[c % len(copies)]
        spot.spot_selector_score(q_sel, w, ks, sc, args.fmt, B, 1, nblk, wl.Hs, wl.ds, n_valid,
                                 scores, stream)

    def select(c):
        spot.spot_select_blocks(scores, B, nblk, n_valid, rule.top_p, rule.k_max, rule.k_min,
                                rule.n_sink, rule.n_recent, idx, cnt, mass, stream)

    def attend(c):
        k, v, _, _ = copies[c % len(copies)]
        spot.spot_sparse_decode(q, k, v, seq_len, idx, cnt, rule.k_max, B, Hq, Hkv, d, L,
                                wl.sm_scale, out, lse, ws, stream)

    def separate_step(c):
        score(c)
        select(c)
        attend(c)

    def step(c):
        k, v, ks, sc = copies[c % len(copies)]
        spot.spot_decode_step(q_sel, w, ks, sc, args.fmt, wl.Hs, wl.ds, n_valid, rule.top_p,
                              rule.k_max, rule.k_min, rule.n_sink, rule.n_recent, q, k, v,
                              seq_len, B, Hq, Hkv, d, L, wl.sm_scale, scores, idx, cnt, mass,
                              out, lse, ws_step, stream)

    def timed(fn, n):
        """Average time of n back-to-back calls, HIP events on the launch stream."""
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        a.record(stream)
        for i in range(n):
            fn(i)
        b.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(b) / n

    log(f"[bench] warmup {args.warmup} steps")
    for i in range(args.warmup):
        separate_step(i)
        step(i)
    torch.cuda.synchronize()
    counts = cnt.cpu().numpy()

    log(f"[bench] timing {args.repeats} x {args.steps} steps")
    rep_ms = [timed(step, args.steps) for _ in range(max(1, args.repeats))]
    ms = float(np.median(rep_ms))
    sep_ms = timed(separate_step, args.steps)
    # Per-stage averages (same launch stream, back to back, rotating copies).
    attn_ms = timed(attend, args.steps)
    score_ms = timed(score, args.steps)
    select_ms = timed(select, args.steps)
    log(f"[bench] fused {ms * 1e3:.1f} us/step, separate {sep_ms * 1e3:.1f} us/step; score "
        f"{score_ms * 1e3:.1f} us, select {select_ms * 1e3:.1f} us, attention "
        f"{attn_ms * 1e3:.1f} us")

    # Reference point, not a bound: one plain kernel reading the same byte
    # count as one contiguous buffer (no gather, no dependency chain).
    kv_block_bytes = 64 * Hkv * d * 2 * 2          # K and V of one 64-token block
    attn_bytes = int(counts.sum()) * kv_block_bytes
    step_bytes = sel_bytes + attn_bytes
    sink = torch.empty(spot.load().spot_probe_sink_words(), dtype=torch.float32, device=dev)
    n_el = step_bytes // 2
    bufs = [copies[c][0].view(-1)[:n_el] for c in range(len(copies))]
    stream_ms = timed(lambda i: spot.spot_probe_stream_read(bufs[i % len(bufs)], sink, stream),
                      args.steps)
    stream_gbs = step_bytes / (stream_ms * 1e-3) / 1e9
    # Known-size write (64 MiB fill) for calibrating the WRITE_SIZE counter.
    calib = torch.empty(64 << 20, dtype=torch.uint8, device=dev)
    calib.fill_(1)
    torch.cuda.synchronize()
    del calib

    steps_per_s = 1e3 / ms
    step_gbs = step_bytes / (ms * 1e-3) / 1e9
    attn_gbs = attn_bytes / (attn_ms * 1e-3) / 1e9

    result = {
        "metric": METRIC,
        "value": round(steps_per_s, 1),
        "unit": "steps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": "decode L=131072 B=4 (Qwen3-8B-shaped layer: 32 q / 8 kv heads, d=128; "
                        "selector 8x64 pooled per 64-token block; p=0.95 K_max=128 sink 1 recent 2)",
            "selector_cache": args.fmt,
            "copies_rotated": args.copies,
            "repeats": len(rep_ms),
            "repeat_us_per_step": [round(r * 1e3, 2) for r in rep_ms],
            "mean_selected_blocks": float(counts.mean()),
            "bytes_per_step": step_bytes,
            "step_hbm_gbs": round(step_gbs, 1),
            "step_hbm_frac": round(step_gbs / HBM_PEAK_GBS, 4),
            "path": "spot_decode_step (score + select + attention in one launch)",
            "separate_calls_us_per_step": round(sep_ms * 1e3, 2),
            "stage_us": {"score": round(score_ms * 1e3, 2), "select": round(select_ms * 1e3, 2),
                         "attention": round(attn_ms * 1e3, 2)},
            "plain_contiguous_read_gbs": round(stream_gbs, 1),
            "attention_kernel": {
                "kernel": "decode_split_kernel (spot_sparse_decode)",
                "achieved_gbs": round(attn_gbs, 1),
                "frac": round(attn_gbs / HBM_PEAK_GBS, 4),
                "bytes_per_launch": attn_bytes,
                "avg_launch_us": round(attn_ms * 1e3, 2),
            },
        },
        "roofline": {
            "bound": "hbm",
            "kernel": "step_kernel (spot_decode_step: scoring, selection, attention)",
            "achieved": round(step_gbs, 1),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(step_gbs / HBM_PEAK_GBS, 4),
            "traffic": measured_traffic() if args.fmt == "bf16" else None,
            "bytes_per_launch": step_bytes,
            "avg_launch_us": round(ms * 1e3, 2),
            "avg_launch_timing": "HIP events around back-to-back launches on the launch "
                                 "stream (the time per launch includes the gap between launches)",
        },
    }

    if not args.no_extra and args.fmt == "bf16":
        # The same step with quantized selector caches (INT4-g32 / MXFP4-g32 /
        # INT8-g32 / MXFP8-g32, quantized from the BF16 cache): fewer selector
        # bytes, same K/V; then with the queries quantized to the same format
        # as well (spot_decode_step_q).
        quant = {}
        for fmt in ("int4", "mxfp4", "int8", "mxfp8"):
            codes, scales = synth.QUANTIZERS[fmt](wl.k_sel)
            sc = scales.view(np.int16) if fmt in ("int4", "int8") else scales
            qsel = [(torch.from_numpy(np.ascontiguousarray(codes)).to(dev),
                     torch.from_numpy(np.ascontiguousarray(sc)).to(dev))
                    for _ in range(args.copies)]

            def qstep(c, fmt=fmt, qsel=qsel):
                k, v, _, _ = copies[c % len(copies)]
                ks, sc_ = qsel[c % len(qsel)]
                spot.spot_decode_step(q_sel, w, ks, sc_, fmt, wl.Hs, wl.ds, n_valid, rule.top_p,
                                      rule.k_max, rule.k_min, rule.n_sink, rule.n_recent, q, k,
                                      v, seq_len, B, Hq, Hkv, d, L, wl.sm_scale, scores, idx,
                                      cnt, mass, out, lse, ws_step, stream)

            for i in range(args.warmup):
                qstep(i)
            qms = timed(qstep, args.steps)
            qbytes = codes.nbytes + scales.nbytes + attn_bytes
            quant[fmt] = {"us_per_step": round(qms * 1e3, 2), "steps_per_s": round(1e3 / qms, 1),
                          "bytes_per_step": int(qbytes),
                          "hbm_frac": round(qbytes / (qms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)}
            log(f"[bench] {fmt} selector cache: {qms * 1e3:.1f} us/step")

            qc, qsc = synth.QUANTIZERS[fmt](wl.q_sel)
            qsc = qsc.view(np.int16) if fmt in ("int4", "int8") else qsc
            q_codes = torch.from_numpy(np.ascontiguousarray(qc)).to(dev)
            q_scale = torch.from_numpy(np.ascontiguousarray(qsc)).to(dev)

            def qqstep(c, fmt=fmt, qsel=qsel, q_codes=q_codes, q_scale=q_scale):
                k, v, _, _ = copies[c % len(copies)]
                ks, sc_ = qsel[c % len(qsel)]
                spot.spot_decode_step(q_codes, w, ks, sc_, fmt, wl.Hs, wl.ds, n_valid,
                                      rule.top_p, rule.k_max, rule.k_min, rule.n_sink,
                                      rule.n_recent, q, k, v, seq_len, B, Hq, Hkv, d, L,
                                      wl.sm_scale, scores, idx, cnt, mass, out, lse, ws_step,
                                      stream, q_scale=q_scale, qfmt=fmt)

            for i in range(args.warmup):
                qqstep(i)
            qqms = timed(qqstep, args.steps)
            quant[fmt]["quantized_queries"] = {
                "us_per_step": round(qqms * 1e3, 2), "steps_per_s": round(1e3 / qqms, 1),
                "hbm_frac": round(qbytes / (qqms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)}
            log(f"[bench] {fmt} selector cache and queries: {qqms * 1e3:.1f} us/step")
        result["config"]["quantized_selector"] = quant

    if not args.no_extra and args.fmt == "bf16":
        # The same layer with 64 query heads over the 8 KV heads (GQA group 8,
        # the Qwen3-32B shape): the fused step compiled for groups of 8.
        hq8 = 8 * Hkv
        q8 = bf(synth.normal_bf16(SEED_TOKENS + 8, 1, (B, hq8, d)))
        out8 = torch.empty((B, hq8, d), dtype=torch.bfloat16, device=dev)
        lse8 = torch.empty((B, hq8), dtype=torch.float32, device=dev)
        ws8 = spot.step_workspace(B, hq8, Hkv, d, rule.k_max, dev)

        def step8(c):
            k, v, ks, sc = copies[c % len(copies)]
            spot.spot_decode_step(q_sel, w, ks, sc, args.fmt, wl.Hs, wl.ds, n_valid, rule.top_p,
                                  rule.k_max, rule.k_min, rule.n_sink, rule.n_recent, q8, k, v,
                                  seq_len, B, hq8, Hkv, d, L, wl.sm_scale, scores, idx, cnt, mass,
                                  out8, lse8, ws8, stream)

        for i in range(args.warmup):
            step8(i)
        g8ms = timed(step8, args.steps)
        result["config"]["group8_step"] = {
            "workload": f"decode L={L} B={B}, 64 q / 8 kv heads (GQA group 8), selector and "
                        "rule as above; spot_decode_step, one launch",
            "us_per_step": round(g8ms * 1e3, 2), "steps_per_s": round(1e3 / g8ms, 1),
            "bytes_per_step": step_bytes,
            "hbm_frac": round(step_bytes / (g8ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)}
        log(f"[bench] group-8 step (64 q heads): {g8ms * 1e3:.1f} us/step")

    if not args.no_dense:
        wsd = spot.decode_workspace(B, Hq, Hkv, d, nblk, dev)

        def dense(i):
            k, v, _, _ = copies[i % len(copies)]
            spot.spot_dense_decode(q, k, v, seq_len, B, Hq, Hkv, d, L, wl.sm_scale, out, lse,
                                   wsd, stream)

        for i in range(3):
            dense(i)
        dms = timed(dense, 20)
        dbytes = B * Hkv * L * d * 2 * 2
        result["dense_baseline"] = {
            "value": round(1e3 / dms, 1), "unit": "steps/s", "ms_per_step": round(dms, 4),
            "hbm_gbs": round(dbytes / (dms * 1e-3) / 1e9, 1),
            "hbm_frac": round(dbytes / (dms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
        }

    if not args.no_extra and args.fmt == "bf16":
        result["static_topk"] = static_topk_leg(args, torch, spot, dev, timed, wl, copies, q,
                                                q_sel, w, seq_len, n_valid, out, lse, stream)

    if (args.tokens or not args.no_extra) and args.fmt == "bf16":
        result["per_token_selector"] = per_token_leg(args, torch, spot, synth, dev, timed, wl,
                                                     copies, q, seq_len, n_valid, idx, cnt,
                                                     mass, out, lse, ws, stream)

    if not args.no_extra:
        result["selector_front_end"] = front_end_leg(args, torch, spot, synth, dev, timed, wl)

    if not args.no_extra:
        del copies, bufs
        torch.cuda.empty_cache()
        result["config"]["smaller_workloads"] = small_decode_legs(args, torch, spot, synth, dev,
                                                                  timed)

    if not args.no_prefill:
        copies = bufs = None
        torch.cuda.empty_cache()
        result["prefill"] = prefill_leg(args, torch, spot, synth, dev, timed)
        if not args.no_extra:
            result["prefill"]["selector_formats"] = selector_format_leg(torch, spot, synth, dev)

    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(wl, args.cpu_seconds)

    print(json.dumps(result), flush=True)


def static_topk_leg(args, torch, spot, dev, timed, wl, copies, q, q_sel, w, seq_len, n_valid,
                    out, lse, stream):
    """Static top-K (Eq. select-topk) at large budgets on the 128K-token,
    batch-4 workload: K = 0.25, 0.5 and 0.75 of the 2048 blocks, no reserved
    blocks, through spot_decode_step (fused for K <= 512, three stages
    above)."""
    B, L, nblk = wl.B, wl.L, wl.nblk
    res = {}
    for frac in (0.25, 0.5, 0.75):
        K = int(frac * nblk)
        ws_k = spot.step_workspace(B, wl.Hq, wl.Hkv, wl.d, K, dev)
        scores = torch.empty((B, nblk), dtype=torch.float32, device=dev)
        idx = torch.empty((B, K), dtype=torch.int32, device=dev)
        cnt = torch.empty(B, dtype=torch.int32, device=dev)

        def step(c, K=K, ws_k=ws_k, scores=scores, idx=idx, cnt=cnt):
            k, v, ks, sc = copies[c % len(copies)]
            spot.spot_decode_step(q_sel, w, ks, sc, "bf16", wl.Hs, wl.ds, n_valid, 1.0, K, 0,
                                  0, 0, q, k, v, seq_len, B, wl.Hq, wl.Hkv, wl.d, L,
                                  wl.sm_scale, scores, idx, cnt, None, out, lse, ws_k, stream)

        for i in range(3):
            step(i)
        n = max(5, args.steps // 10)
        ms = timed(step, n)
        counts = cnt.cpu().numpy()
        nbytes = wl.k_sel.nbytes + int(counts.sum()) * 64 * wl.Hkv * wl.d * 4
        res[f"K={K}"] = {"fraction_of_blocks": frac, "us_per_step": round(ms * 1e3, 2),
                         "steps_per_s": round(1e3 / ms, 1), "bytes_per_step": int(nbytes),
                         "hbm_frac": round(nbytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                         "path": "fused" if K <= 512 else "three launches"}
        log(f"[bench] static top-K K={K}: {ms * 1e3:.1f} us/step")
        del ws_k
    return {"workload": f"decode L={L} B={B}, static top-K (p >= 1, no reserved blocks)",
            "budgets": res}


def graph_ms(torch, fn, n=50, reps=5):
    """Average time of fn(stream) captured n times in a HIP graph (no host
    work between the kernels), over reps replays, in ms."""
    for _ in range(3):
        fn(torch.cuda.current_stream())
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        st = torch.cuda.current_stream()
        for _ in range(n):
            fn(st)
    g.replay()
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(reps):
        g.replay()
    b.record()
    torch.cuda.synchronize()
    return a.elapsed_time(b) / (n * reps)


def selector_format_leg(torch, spot, synth, dev):
    """Prefill selector tiles (one 32K-token sequence: 512 x 512 query-block x
    key-block scores, causal) with the paper's 4 x 128 selector, BF16 and with
    queries and keys both MXFP4 or MXFP8 on the block-scaled matrix cores."""
    nqb, Hs, ds = 512, 4, 128
    rng = np.random.default_rng(SEED_TOKENS)
    q_sel, w, k_sel = synth.selector_prefill(rng, 1, nqb, nqb, Hs, ds)
    q_sel = q_sel.reshape(nqb, Hs, ds)
    w = torch.from_numpy(np.ascontiguousarray(w.reshape(nqb, Hs))).to(dev)
    n_valid = torch.from_numpy(np.arange(1, nqb + 1, dtype=np.int32)).to(dev)
    out = torch.empty((nqb, nqb), dtype=torch.float32, device=dev)
    res = {}
    qb, kb = spot.to_device_bf16(q_sel, dev), spot.to_device_bf16(k_sel, dev)
    res["bf16"] = graph_ms(torch, lambda st: spot.spot_selector_score(
        qb, w, kb, None, "bf16", 1, nqb, nqb, Hs, ds, n_valid, out, st)) * 1e3
    for fmt in ("mxfp4", "mxfp8"):
        qc, qs = synth.QUANTIZERS[fmt](q_sel)
        kc, ks = synth.QUANTIZERS[fmt](k_sel)
        t = [torch.from_numpy(np.ascontiguousarray(x)).to(dev) for x in (qc, qs, kc, ks)]
        res[fmt] = graph_ms(torch, lambda st, t=t, fmt=fmt: spot.spot_selector_score_q(
            t[0], t[1], fmt, w, t[2], t[3], fmt, 1, nqb, nqb, Hs, ds, n_valid, out, st)) * 1e3
    log("[bench] prefill selector 4x128: " + ", ".join(f"{k} {v:.1f} us" for k, v in res.items()))
    return {"workload": "512 x 512 query-block x key-block selector tiles, 4 x 128 heads, causal",
            "us": {k: round(v, 2) for k, v in res.items()}}


def front_end_leg(args, torch, spot, synth, dev, timed, wl):
    """The selector front end of one decode step for the 4 sequences:
    projections of the new token's hidden state (Qwen3-8B width 4096, 4 x 128
    selector heads, rotary on 64 dims) with the key appended to the per-token
    cache, then the pooled key of the block it landed in re-computed."""
    B, L, Hs, ds, d_model = wl.B, wl.L, 4, 128, 4096
    h, wq, wk, ww = synth.selector_frontend(SEED_TOKENS, B, d_model, Hs, ds)

    def bf(a):
        return spot.to_device_bf16(a, dev)

    hd, wqd, wkd, wwd = bf(h), bf(wq), bf(wk), bf(ww)
    pos = torch.from_numpy(wl.seq_len - 1).to(dev)
    first = torch.from_numpy((wl.seq_len - 1) // 64).to(dev)
    seq_len = torch.from_numpy(wl.seq_len).to(dev)
    q_out = torch.empty((B, Hs, ds), dtype=torch.bfloat16, device=dev)
    w_out = torch.empty((B, Hs), dtype=torch.float32, device=dev)
    cache = torch.zeros((B, L, Hs, ds), dtype=torch.bfloat16, device=dev)
    pooled = torch.zeros((B, L // 64, Hs, ds), dtype=torch.bfloat16, device=dev)
    def project(st):
        spot.spot_selector_project(hd, wqd, wkd, wwd, pos, B, d_model, Hs, ds, 64, 1.0e6, q_out,
                                   w_out, cache, 1, L, st)

    def pool(st):
        spot.spot_selector_pool(cache, pooled, B, L, Hs, ds, seq_len, first, 1, st)

    def both(st):
        project(st)
        pool(st)

    def fused(st):
        spot.spot_selector_project_pooled(hd, wqd, wkd, wwd, pos, seq_len, B, d_model, Hs, ds, 64,
                                          1.0e6, q_out, w_out, cache, pooled, L, st)

    # These launches last a few microseconds, less than the binding's host
    # overhead per call, so they are timed as replayed HIP graphs.
    pms = graph_ms(torch, project)
    qms = graph_ms(torch, pool)
    two_ms = graph_ms(torch, both)
    ms = graph_ms(torch, fused)
    wbytes = wq.nbytes + wk.nbytes + ww.nbytes
    log(f"[bench] selector front end: one launch {ms * 1e3:.1f} us; project "
        f"{pms * 1e3:.1f} us + pool {qms * 1e3:.1f} us = {two_ms * 1e3:.1f} us")
    del cache, pooled
    return {
        "workload": f"decode B={B}: hidden {d_model} -> selector {Hs}x{ds} (RoPE 64 dims), "
                    "key appended to the per-token cache, its block re-pooled",
        "path": "spot_selector_project_pooled (projection and pooling in one launch)",
        "us_per_step": round(ms * 1e3, 2),
        "two_launch_us": round(two_ms * 1e3, 2),
        "project_us": round(pms * 1e3, 2),
        "pool_us": round(qms * 1e3, 2),
        "project_weight_bytes": int(wbytes),
        "weight_gbs": round(wbytes / (ms * 1e-3) / 1e9, 1),
        "timing": "replayed HIP graph of the launch(es), per step",
    }


def per_token_leg(args, torch, spot, synth, dev, timed, wl, copies, q, seq_len, n_valid, idx,
                  cnt, mass, out, lse, ws, stream):
    """The decode step with the paper's own selector cache -- one 4 x 128
    selector key per token, block value = maximum of its tokens' scores --
    on the same 128K-token, batch-4 layer: spot_selector_score_tokens, then
    selection and sparse attention as separate launches."""
    B, L, rule = wl.B, wl.L, wl.rule
    Hs, ds = 4, 128
    log("[bench] per-token selector: generating the 4 x 128 per-token cache")
    q_tok, w_tok, k_tok = synth.selector_tokens(SEED_TOKENS, B, L, Hs, ds, wl.seq_len)
    qs = spot.to_device_bf16(q_tok, dev)
    ws_ = torch.from_numpy(w_tok).to(dev)
    ktoks = [spot.to_device_bf16(k_tok, dev) for _ in range(2)]
    tok_bytes = k_tok.nbytes
    k_head = np.ascontiguousarray(k_tok[:, :QUANT_TOKENS])
    del k_tok
    nblk = L // 64
    scores = torch.empty((B, nblk), dtype=torch.float32, device=dev)

    def score(c):
        spot.spot_selector_score_tokens(qs, ws_, ktoks[c % 2], None, "bf16", B, 1, L, Hs, ds,
                                        seq_len, scores, stream)

    def step(c):
        score(c)
        k, v, _, _ = copies[c % len(copies)]
        spot.spot_select_blocks(scores, B, nblk, n_valid, rule.top_p, rule.k_max, rule.k_min,
                                rule.n_sink, rule.n_recent, idx, cnt, mass, stream)
        spot.spot_sparse_decode(q, k, v, seq_len, idx, cnt, rule.k_max, B, wl.Hq, wl.Hkv, wl.d,
                                L, wl.sm_scale, out, lse, ws, stream)

    for i in range(args.warmup):
        step(i)
    sms = timed(score, args.steps)
    ms = timed(step, args.steps)
    counts = cnt.cpu().numpy()
    attn_bytes = int(counts.sum()) * 64 * wl.Hkv * wl.d * 4
    gbs = tok_bytes / (sms * 1e-3) / 1e9
    log(f"[bench] per-token selector: score {sms * 1e3:.1f} us ({gbs:.0f} GB/s), "
        f"step {ms * 1e3:.1f} us")
    del ktoks
    torch.cuda.empty_cache()
    block16 = block16_leg(args, torch, spot, synth, dev, timed, wl, copies, q, seq_len, out, lse,
                          stream)

    # The scorer alone over quantized per-token caches: the first QUANT_TOKENS
    # tokens of each sequence quantized and repeated to L tokens (the encoders
    # run on the host and would take minutes over all 512 Mi elements); four
    # copies rotated, 0.6-1.1 GB in all, so the last-level cache cannot serve
    # repeated launches.
    fmts = {}
    for fmt in ("int4", "mxfp4", "int8", "mxfp8"):
        c, sc = synth.QUANTIZERS[fmt](k_head)
        reps = L // QUANT_TOKENS
        c = np.tile(c, (1, reps, 1, 1))
        sc = np.tile(sc.view(np.int16) if fmt in ("int4", "int8") else sc, (1, reps, 1, 1))
        nbytes = c.nbytes + sc.nbytes
        c0 = torch.from_numpy(c).to(dev)
        s0 = torch.from_numpy(sc).to(dev)
        del c, sc
        qcopies = [(c0, s0)] + [(c0.clone(), s0.clone()) for _ in range(3)]

        def qscore(i, fmt=fmt, qcopies=qcopies):
            kc, kscale = qcopies[i % len(qcopies)]
            spot.spot_selector_score_tokens(qs, ws_, kc, kscale, fmt, B, 1, L, Hs, ds, seq_len,
                                            scores, stream)

        for i in range(args.warmup):
            qscore(i)
        qms = timed(qscore, args.steps)
        qgbs = nbytes / (qms * 1e-3) / 1e9
        kern = "score_tokens4_kernel" if fmt in ("int4", "mxfp4") else "score_tokens_kernel"
        fmts[fmt] = {"kernel": kern, "us": round(qms * 1e3, 2), "bytes_per_launch": int(nbytes),
                     "achieved_gbs": round(qgbs, 1), "frac": round(qgbs / HBM_PEAK_GBS, 4)}
        log(f"[bench] per-token {fmt} scorer: {qms * 1e3:.1f} us ({qgbs:.0f} GB/s)")
        del qcopies, c0, s0
        torch.cuda.empty_cache()
    return {
        "workload": f"decode L={L} B={B}, per-token selector cache {Hs}x{ds} BF16 "
                    f"({tok_bytes >> 20} MiB), block value = max over its 64 tokens; "
                    f"p={rule.top_p} K_max={rule.k_max}",
        "us_per_step": round(ms * 1e3, 2),
        "steps_per_s": round(1e3 / ms, 1),
        "mean_selected_blocks": float(counts.mean()),
        "bytes_per_step": int(tok_bytes + attn_bytes),
        "hbm_frac": round((tok_bytes + attn_bytes) / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
        "scorer_roofline": {
            "bound": "hbm", "kernel": "score_tokens_kernel (spot_selector_score_tokens)",
            "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(gbs / HBM_PEAK_GBS, 4), "bytes_per_launch": int(tok_bytes),
            "avg_launch_us": round(sms * 1e3, 2),
            "traffic": measured_traffic(TOKENS_PROFILE, TOKENS_SOURCES),
        },
        "quantized_scorer": fmts,
        "block16": block16,
    }


def block16_leg(args, torch, spot, synth, dev, timed, wl, copies, q, seq_len, out, lse, stream):
    """The per-token decode step with the paper's 16-token selector block
    (Appendix A): the same 4 x 128 per-token cache and KV layer, block value =
    maximum over 16 tokens, dual top-p / top-K over L / 16 blocks with the
    same token budget as the 64-token workload (K_max = 512 blocks = 8192
    tokens, 4 sink + 8 recent blocks = 64 + 128 tokens), attention over the
    selected 16-token blocks; three launches."""
    B, L = wl.B, wl.L
    Hs, ds, blk = 4, 128, 16
    rule = synth.Rule(wl.rule.top_p, 512, 0, 4, 8)
    log("[bench] 16-token blocks: generating the per-token cache (one lead token per block)")
    q_tok, w_tok, k_tok = synth.selector_tokens(SEED_TOKENS + 1, B, L, Hs, ds, wl.seq_len,
                                                rule=rule, blk=blk)
    qs = spot.to_device_bf16(q_tok, dev)
    ws_ = torch.from_numpy(w_tok).to(dev)
    ktoks = [spot.to_device_bf16(k_tok, dev) for _ in range(2)]
    tok_bytes = k_tok.nbytes
    del k_tok
    nb = L // blk
    nv = torch.from_numpy(((wl.seq_len + blk - 1) // blk).astype(np.int32)).to(dev)
    scores = torch.empty((B, nb), dtype=torch.float32, device=dev)
    idx = torch.empty((B, rule.k_max), dtype=torch.int32, device=dev)
    cnt = torch.empty(B, dtype=torch.int32, device=dev)
    mass = torch.empty(B, dtype=torch.float32, device=dev)
    ws = spot.decode_workspace(B, wl.Hq, wl.Hkv, wl.d, rule.k_max, dev)

    def score(c):
        spot.spot_selector_score_tokens_blk(qs, ws_, ktoks[c % 2], None, "bf16", B, 1, L, blk,
                                            Hs, ds, seq_len, scores, stream)

    def select(c):
        spot.spot_select_blocks(scores, B, nb, nv, rule.top_p, rule.k_max, rule.k_min,
                                rule.n_sink, rule.n_recent, idx, cnt, mass, stream)

    def attend(c):
        k, v, _, _ = copies[c % len(copies)]
        spot.spot_sparse_decode_blk(q, k, v, seq_len, idx, cnt, rule.k_max, blk, B, wl.Hq,
                                    wl.Hkv, wl.d, L, wl.sm_scale, out, lse, ws, stream)

    def step(c):
        score(c)
        select(c)
        attend(c)

    for i in range(args.warmup):
        step(i)
    ms = timed(step, args.steps)
    s_ms, sel_ms, att_ms = timed(score, args.steps), timed(select, args.steps), \
        timed(attend, args.steps)
    counts = cnt.cpu().numpy()
    attn_bytes = int(counts.sum()) * blk * wl.Hkv * wl.d * 4
    log(f"[bench] 16-token blocks: step {ms * 1e3:.1f} us (score {s_ms * 1e3:.1f}, select "
        f"{sel_ms * 1e3:.1f}, attention {att_ms * 1e3:.1f}), {counts.mean():.0f} blocks")
    del ktoks
    torch.cuda.empty_cache()
    return {
        "workload": f"decode L={L} B={B}, per-token selector cache {Hs}x{ds} BF16 "
                    f"({tok_bytes >> 20} MiB), block of {blk} tokens = max over its tokens; "
                    f"p={rule.top_p} K_max={rule.k_max} blocks, {rule.n_sink} sink + "
                    f"{rule.n_recent} recent blocks",
        "us_per_step": round(ms * 1e3, 2),
        "steps_per_s": round(1e3 / ms, 1),
        "stage_us": {"score": round(s_ms * 1e3, 2), "select": round(sel_ms * 1e3, 2),
                     "attention": round(att_ms * 1e3, 2)},
        "mean_selected_blocks": float(counts.mean()),
        "bytes_per_step": int(tok_bytes + attn_bytes),
        "hbm_frac": round((tok_bytes + attn_bytes) / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
        "attention_gbs": round(attn_bytes / (att_ms * 1e-3) / 1e9, 1),
    }


def small_decode_legs(args, torch, spot, synth, dev, timed):
    """The fused decode step on the two smaller decode workloads (4K tokens,
    batch 1, K_max 16; 32K tokens, batch 8, K_max 64): launch-bound sizes,
    reported for context.  A call from Python costs ~15 us of host time, more
    than the step itself at 4K tokens, so each step is timed as a replayed
    HIP graph of 50 launches (the way a serving loop issues launch-bound
    steps); the back-to-back Python launches are reported beside it."""
    res = {}
    for i, name in ((1, "decode L=4096 B=1 p=0.9 K_max=16"),
                    (2, "decode L=32768 B=8 p=0.9 K_max=64")):
        wl = synth.decode_config(i)
        rule = wl.rule

        def bf(a):
            return spot.to_device_bf16(a, dev)

        q, q_sel, ks = bf(wl.q), bf(wl.q_sel), bf(wl.k_sel)
        w = torch.from_numpy(wl.w).to(dev)
        seq_len = torch.from_numpy(wl.seq_len).to(dev)
        n_valid = torch.from_numpy(wl.n_valid).to(dev)
        k0, v0 = bf(wl.k), bf(wl.v)
        kv = [(k0, v0)] + [(k0.clone(), v0.clone()) for _ in range(args.copies - 1)]
        scores = torch.empty((wl.B, wl.nblk), dtype=torch.float32, device=dev)
        idx = torch.empty((wl.B, rule.k_max), dtype=torch.int32, device=dev)
        cnt = torch.empty(wl.B, dtype=torch.int32, device=dev)
        out = torch.empty((wl.B, wl.Hq, wl.d), dtype=torch.bfloat16, device=dev)
        ws = spot.step_workspace(wl.B, wl.Hq, wl.Hkv, wl.d, rule.k_max, dev)
        stream = torch.cuda.current_stream()

        def step(c, st=stream):
            k, v = kv[c % len(kv)]
            spot.spot_decode_step(q_sel, w, ks, None, "bf16", wl.Hs, wl.ds, n_valid, rule.top_p,
                                  rule.k_max, rule.k_min, rule.n_sink, rule.n_recent, q, k, v,
                                  seq_len, wl.B, wl.Hq, wl.Hkv, wl.d, wl.L, wl.sm_scale, scores,
                                  idx, cnt, None, out, None, ws, st)

        for c in range(args.warmup):
            step(c)
        launch_ms = timed(step, args.steps)
        calls = iter(range(1 << 30))
        ms = graph_ms(torch, lambda st: step(next(calls), st))
        counts = cnt.cpu().numpy()
        nbytes = wl.k_sel.nbytes + int(counts.sum()) * 64 * wl.Hkv * wl.d * 4
        res[f"decode{i}"] = {"workload": name, "us_per_step": round(ms * 1e3, 2),
                             "steps_per_s": round(1e3 / ms, 1),
                             "timing": "replayed HIP graph of 50 launches",
                             "python_launch_us_per_step": round(launch_ms * 1e3, 2),
                             "mean_selected_blocks": float(counts.mean()),
                             "bytes_per_step": int(nbytes),
                             "hbm_frac": round(nbytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)}
        log(f"[bench] {name}: {ms * 1e3:.1f} us/step (graph; {launch_ms * 1e3:.1f} us from "
            "Python launches)")
        del kv, k0, v0
        torch.cuda.empty_cache()
    return res


def prefill_leg(args, torch, spot, synth, dev, timed):
    """Block-sparse causal prefill of one 32K-token Qwen3-32B-shaped layer
    (64 query / 8 KV heads, d = 128): query-block selector scores, selection
    (p = 0.9, K_max = 64) and the MFMA block-sparse attention."""
    log("[bench] prefill: generating the 32K-token layer")
    pw = synth.prefill_config()
    nqb, rule = pw.nblk, pw.rule

    def bf(a):
        return spot.to_device_bf16(a, dev)

    q, k, v = bf(pw.q), bf(pw.k), bf(pw.v)
    q_sel, k_sel = bf(pw.q_sel), bf(pw.k_sel)
    w = torch.from_numpy(pw.w).to(dev)
    n_valid = torch.from_numpy(pw.n_valid).to(dev)
    rows = pw.B * nqb
    scores = torch.empty((rows, nqb), dtype=torch.float32, device=dev)
    idx = torch.empty((rows, rule.k_max), dtype=torch.int32, device=dev)
    cnt = torch.empty(rows, dtype=torch.int32, device=dev)
    out = torch.empty_like(q)
    lse = torch.empty((pw.B, pw.Hq, pw.L), dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream()

    def score(i):
        spot.spot_selector_score(q_sel, w, k_sel, None, "bf16", pw.B, nqb, nqb, pw.Hs, pw.ds,
                                 n_valid, scores, stream)

    def select(i):
        spot.spot_select_blocks(scores, rows, nqb, n_valid, rule.top_p, rule.k_max, rule.k_min,
                                rule.n_sink, rule.n_recent, idx, cnt, None, stream)

    def attend(i):
        spot.spot_sparse_prefill(q, k, v, pw.L, idx, cnt, rule.k_max, pw.B, pw.Hq, pw.Hkv, pw.d,
                                 pw.sm_scale, out, lse, stream)

    for i in range(2):
        score(i), select(i), attend(i)
    torch.cuda.synchronize()
    # The layer and its stages are timed in three interleaved rounds and each
    # figure is the median of its rounds (the ~3 ms prefill launches vary by
    # several percent from one loop to the next).
    n = args.prefill_iters
    rounds = {"attn": [], "score": [], "select": [], "step": []}
    for _ in range(3):
        rounds["step"].append(timed(lambda i: (score(i), select(i), attend(i)), n))
        rounds["attn"].append(timed(attend, n))
        rounds["score"].append(timed(score, n))
        rounds["select"].append(timed(select, n))
    med = {k: float(np.median(v)) for k, v in rounds.items()}
    attn_ms, score_ms, select_ms, step_ms = med["attn"], med["score"], med["select"], med["step"]

    ids = idx.cpu().numpy()
    c = cnt.cpu().numpy()
    qb = np.arange(rows) % nqb
    take = np.arange(rule.k_max)[None, :] < c[:, None]
    n_tiles = int(take.sum())
    n_diag = int((take & (ids == qb[:, None])).sum())
    tile_flops = 4.0 * 64 * 64 * pw.d * pw.Hq          # QK^T and PV, all query heads
    mfma_flops = n_tiles * tile_flops
    useful_flops = (n_tiles - n_diag + n_diag * (64 * 65 / 2) / (64 * 64)) * tile_flops
    # Algorithmic FLOPs: a diagonal tile counts only its causal half (64 * 65
    # / 2 of its 64 * 64 query-key pairs); the kernel issues the whole tile.
    tflops = useful_flops / (attn_ms * 1e-3) / 1e12
    issued_tflops = mfma_flops / (attn_ms * 1e-3) / 1e12
    log(f"[bench] prefill: {step_ms:.3f} ms/layer; attention {attn_ms:.3f} ms "
        f"({tflops:.0f} TFLOP/s useful, {issued_tflops:.0f} issued), score "
        f"{score_ms * 1e3:.1f} us, select {select_ms * 1e3:.1f} us")
    res = {
        "workload": "prefill L=32768 B=1 (Qwen3-32B-shaped layer: 64 q / 8 kv heads, d=128; "
                    "selector 8x64 pooled per 64-token block; p=0.9 K_max=64 sink 1 recent 2)",
        "value": round(pw.L / (step_ms * 1e-3), 1), "unit": "tokens/s",
        "ms_per_layer": round(step_ms, 4),
        "stage_us": {"score": round(score_ms * 1e3, 2), "select": round(select_ms * 1e3, 2),
                     "attention": round(attn_ms * 1e3, 2)},
        "selected_tiles": n_tiles, "diagonal_tiles": n_diag,
        "roofline": {
            "bound": "mfma", "kernel": "prefill_kernel (spot_sparse_prefill)",
            "achieved": round(tflops, 1), "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
            "frac": round(tflops / MFMA_BF16_PEAK_TFLOPS, 4),
            "flops_per_launch": useful_flops,
            "issued_flops_per_launch": mfma_flops,
            "issued_tflops": round(issued_tflops, 1),
            "avg_launch_us": round(attn_ms * 1e3, 1),
            "avg_launch_timing": "HIP events around back-to-back launches on the launch "
                                 "stream; median of three interleaved rounds",
        },
        "round_ms": {"layer": [round(x, 4) for x in rounds["step"]],
                     "attention": [round(x, 4) for x in rounds["attn"]]},
    }
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = prefill_cpu_baseline(pw)
    return res


# Query blocks of the 512-block prefill layer on which the oracle is timed:
# the first blocks (almost no history), powers of two minus one and plus
# zero across the range, and the last blocks (the K_max cap binds).
PREFILL_SAMPLE_QB = (0, 1, 2, 3, 31, 63, 64, 127, 191, 255, 256, 319, 383, 447, 510, 511)


def prefill_cpu_baseline(pw):
    """The FP64 oracle's prefill layer on the host cores: selector scores and
    selection for all query blocks, attention on a fixed sample of query
    blocks (all 64 heads), extrapolated to the layer."""
    import oracle
    try:
        cores = len(os.sched_getaffinity(0))
    except AttributeError:
        cores = os.cpu_count() or 1
    oracle.set_threads(cores)
    t0 = time.time()
    s = oracle.selector_score(pw.q_sel, pw.w, pw.k_sel, rows_per_seq=pw.nblk,
                              n_valid=pw.n_valid).astype(np.float32)
    idx, cnt, _ = oracle.select_blocks(s.astype(np.float64), pw.rule, pw.n_valid)
    sel_s = time.time() - t0
    rows = np.asarray([r for r in PREFILL_SAMPLE_QB if r < pw.nblk], np.int32)
    log(f"[bench] prefill cpu baseline: oracle attention on {rows.size} query blocks, "
        f"{cores} threads")
    t0 = time.time()
    oracle.sparse_prefill(pw.q, pw.k, pw.v, idx, cnt, pw.sm_scale, rows)
    attn_s = time.time() - t0
    per_qb = attn_s / rows.size
    per_tile = attn_s / max(1, int(cnt[rows].sum()))
    layer_s = sel_s + per_tile * int(cnt.sum())
    return {"value": round(pw.L / layer_s, 2), "unit": "tokens/s", "cores": oracle.get_threads(),
            "kind": "oracle", "cpu_model": cpu_model(),
            "sample": f"selector scores + selection of all {pw.nblk} query blocks, then "
                      f"attention (64 heads, FP64 C with OpenMP) on query blocks "
                      f"{rows.tolist()}; the layer time extrapolates the sample's time per "
                      f"selected tile to the layer's {int(cnt.sum())} tiles",
            "selection_s": round(sel_s, 3),
            "attention_s_per_qblock": round(per_qb, 4),
            "attention_s_x512": round(per_qb * 512, 1),
            "layer_s_extrapolated": round(layer_s, 1)}


def cpu_model():
    """The host processor's model name, as /proc/cpuinfo (and lscpu) give it."""
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or "unknown"


def cpu_baseline(wl, budget_s):
    """The FP64 oracle timed on the host cores over whole decode steps."""
    import oracle
    try:
        cores = len(os.sched_getaffinity(0))
    except AttributeError:
        cores = os.cpu_count() or 1
    oracle.set_threads(cores)
    log(f"[bench] cpu baseline: oracle on {cores} threads for ~{budget_s:.0f}s")
    n, t0 = 0, time.time()
    while True:
        s = oracle.selector_score(wl.q_sel, wl.w, wl.k_sel, n_valid=wl.n_valid)
        idx, cnt, _ = oracle.select_blocks(s.astype(np.float32), wl.rule, wl.n_valid)
        oracle.sparse_decode(wl.q, wl.k, wl.v, wl.seq_len, idx, cnt, wl.sm_scale)
        n += 1
        el = time.time() - t0
        if el >= budget_s or (n >= 1 and el * (n + 1) / n > 30.0):
            break
    used = oracle.get_threads()
    # The same steps on one thread, over a shorter sample.
    oracle.set_threads(1)
    n1, t1 = 0, time.time()
    while True:
        s = oracle.selector_score(wl.q_sel, wl.w, wl.k_sel, n_valid=wl.n_valid)
        idx, cnt, _ = oracle.select_blocks(s.astype(np.float32), wl.rule, wl.n_valid)
        oracle.sparse_decode(wl.q, wl.k, wl.v, wl.seq_len, idx, cnt, wl.sm_scale)
        n1 += 1
        el1 = time.time() - t1
        if el1 >= budget_s / 4 or (n1 >= 1 and el1 * (n1 + 1) / n1 > 10.0):
            break
    oracle.set_threads(cores)
    return {"value": round(n / el, 4), "unit": "steps/s", "cores": used,
            "kind": "oracle", "cpu_model": cpu_model(),
            "sample": f"{n} full decode steps (score + select + sparse attention, all 4 "
                      f"sequences) of the same workload, FP64 C with OpenMP",
            "single_thread_value": round(n1 / el1, 4),
            "single_thread_sample": f"{n1} of the same steps on 1 thread"}


if __name__ == "__main__":
    main()
