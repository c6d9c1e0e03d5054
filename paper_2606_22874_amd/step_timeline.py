"""Per-phase timeline of the fused decode step (measurement tool).

    python -m paper_2606_22874_amd.step_timeline [--cfg 3] [--trials 6] [--burst 1]

Builds ``libspot_timeline.so`` (next to libspot.so) -- the library with the step kernel
compiled from ``csrc/step_timeline.hip`` (step.hip with its phase hooks
stamping the device's 100 MHz real-time counter) -- then runs the decode
workload (default: 131072 tokens, batch 4), times 200 back-to-back fused
steps, and stamps ``--trials`` launches: with ``--burst 1`` each one starts
on an idle device, with ``--burst N`` it is the last of N back-to-back
launches (the regime bench.py times; every launch overwrites the stamps).
It prints, as markdown, the median over the trials of each phase's time in
microseconds since the first workgroup of the launch started.  Needs an
MI355X.
"""
from __future__ import annotations

import argparse
import ctypes
import os
import subprocess

import numpy as np

from . import build as B

TIMELINE_SO = os.path.join(B.PKG, "libspot_timeline.so")
SCORERS_PER_ROW = 64   # the step kernel's scoring workgroups per row
TIMELINE_SRC = "step_timeline.hip"


def build() -> str:
    """Compiles the timeline object and links it with the library's other objects."""
    B.build()
    obj = os.path.join(B.BUILD, "step_timeline.o")
    r = subprocess.run([B.hipcc(), *B.HIPCC_FLAGS, "-c", os.path.join(B.CSRC, TIMELINE_SRC),
                        "-o", obj], capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {TIMELINE_SRC}:\n{r.stderr}")
    objs = [os.path.join(B.BUILD, os.path.splitext(s)[0] + ".o") for s in B.SOURCES
            if s != "step.hip"]
    tmp = TIMELINE_SO + f".tmp{os.getpid()}"
    r = subprocess.run([B.hipcc(), f"--offload-arch={B.ARCH}", "-shared", "-fPIC", "-o", tmp,
                        *objs, obj], capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stderr}")
    os.replace(tmp, TIMELINE_SO)
    return TIMELINE_SO


def _pct(x, q):
    return float(np.percentile(x, q)) if len(x) else float("nan")


def run(cfg: int = 3, trials: int = 6, burst: int = 1) -> dict:
    import torch

    from . import spot, synth

    lib = spot.load(TIMELINE_SO)
    spot._lib = lib
    lib.spot_timeline_read.argtypes = [ctypes.c_void_p] * 3
    cap = lib.spot_timeline_capacity()
    dev = torch.device("cuda:0")
    wl = synth.decode_config(cfg)
    bf = lambda a: spot.to_device_bf16(a, dev)   # noqa: E731
    q, q_sel = bf(wl.q), bf(wl.q_sel)
    w = torch.from_numpy(wl.w).to(dev)
    seq_len = torch.from_numpy(wl.seq_len).to(dev)
    n_valid = torch.from_numpy(wl.n_valid).to(dev)
    k0, v0, ks0 = bf(wl.k), bf(wl.v), bf(wl.k_sel)
    # four copies of the caches, rotated so that repeated steps miss the caches
    copies = [(k0, v0, ks0)] + [(k0.clone(), v0.clone(), ks0.clone()) for _ in range(3)]
    rule, nblk = wl.rule, wl.nblk
    B_, Hq, Hkv, d, L = wl.B, wl.Hq, wl.Hkv, wl.d, wl.L
    scores = torch.empty((B_, nblk), device=dev)
    idx = torch.empty((B_, rule.k_max), dtype=torch.int32, device=dev)
    cnt = torch.empty(B_, dtype=torch.int32, device=dev)
    mass = torch.empty(B_, device=dev)
    out = torch.empty((B_, Hq, d), dtype=torch.bfloat16, device=dev)
    lse = torch.empty((B_, Hq), device=dev)
    ws = spot.step_workspace(B_, Hq, Hkv, d, rule.k_max, dev)
    st = torch.cuda.current_stream()

    def step(i):
        k, v, ks = copies[i % len(copies)]
        spot.spot_decode_step(q_sel, w, ks, None, 0, wl.Hs, wl.ds, n_valid, rule.top_p,
                              rule.k_max, rule.k_min, rule.n_sink, rule.n_recent, q, k, v,
                              seq_len, B_, Hq, Hkv, d, L, wl.sm_scale, scores, idx, cnt, mass,
                              out, lse, ws, st)

    for i in range(30):
        step(i)
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record(st)
    for i in range(200):
        step(i)
    b.record(st)
    torch.cuda.synchronize()
    us_per_step = a.elapsed_time(b) / 200 * 1e3

    ts = np.zeros((cap, 8), np.uint64)
    sel = np.zeros((cap, 10), np.uint64)
    xcc = np.zeros(cap, np.uint32)
    rows = []
    for t in range(trials):
        if lib.spot_timeline_clear() != 0:
            raise RuntimeError("spot_timeline_clear failed")
        torch.cuda.synchronize()
        for i in range(burst):
            step(t + 1 + i)
        torch.cuda.synchronize()
        if lib.spot_timeline_read(ts.ctypes.data, sel.ctypes.data, xcc.ctypes.data) != 0:
            raise RuntimeError("spot_timeline_read failed")
        n = int((ts[:, 0] > 0).sum())
        t_ = ts[:n].astype(np.int64)
        s_ = sel[:n].astype(np.int64)
        x_ = xcc[:n]
        g0 = t_[:, 0].min()
        us = lambda v: (np.asarray(v, np.int64) - g0) * 0.01   # noqa: E731
        # workgroup i scores for row i % B when i / B is below the per-row count
        # (every workgroup stamps phase 1; only these did scoring before it)
        scorer = np.arange(n) // B_ < min(SCORERS_PER_ROW, n // B_)
        selector = np.arange(n) < B_
        merged = t_[:, 7] > t_[:, 6]   # stamped by this launch's merge
        end = np.where(merged, t_[:, 7], t_[:, 6])
        r = {
            "workgroups": n,
            "xcd_first_start": [float(us(t_[x_ == c, 0]).min()) for c in range(8)
                                if (x_ == c).any()],
            "start_max": float(us(t_[:, 0]).max()),
            "scoring_done_p50": float(np.median(us(t_[scorer, 1]))),
            "scoring_done_max": float(us(t_[scorer, 1]).max()),
            "sel_first_wave_scores_in": float(us(s_[selector, 1]).max()),
            "sel_all_scores_in": float(us(s_[selector, 2]).max()),
            "sel_core_done": float(us(t_[selector, 2]).max()),
            "sel_written": float(us(t_[selector, 3]).max()),
            "attn_start_p10": _pct(us(t_[:, 4]), 10),
            "attn_start_p50": _pct(us(t_[:, 4]), 50),
            "attn_start_max": float(us(t_[:, 4]).max()),
            "attn_done_p50": _pct(us(t_[:, 5]), 50),
            "attn_done_max": float(us(t_[:, 5]).max()),
            "attn_us_p50": float(np.median((t_[:, 5] - t_[:, 4]) * 0.01)),
            "attn_us_max": float(((t_[:, 5] - t_[:, 4]) * 0.01).max()),
            "merge_us_p50": float(np.median((t_[merged, 7] - t_[merged, 6]) * 0.01)),
            "end_p50": _pct(us(end), 50),
            "end_max": float(us(end).max()),
        }
        rows.append(r)
    med = {k: (float(np.median([r[k] for r in rows])) if not isinstance(rows[0][k], list)
               else [float(np.median([r[k][i] for r in rows])) for i in range(len(rows[0][k]))])
           for k in rows[0]}
    med["us_per_step_untraced"] = us_per_step
    med["trials"] = trials
    med["burst"] = burst
    return med


def table(m: dict) -> str:
    f = lambda x: f"{x:.2f}"   # noqa: E731
    lines = [
        "| phase | time since the first workgroup started (us, median of trials) |",
        "|---|---|",
        f"| first workgroup on each XCD (dispatch ramp) | {' / '.join(f(x) for x in m['xcd_first_start'])} |",
        f"| last workgroup started | {f(m['start_max'])} |",
        f"| scoring done (scoring workgroups, p50 / max) | {f(m['scoring_done_p50'])} / {f(m['scoring_done_max'])} |",
        f"| selection: first wave's scores in (latest row) | {f(m['sel_first_wave_scores_in'])} |",
        f"| selection: all scores in (latest row) | {f(m['sel_all_scores_in'])} |",
        f"| selection core done, bitmap out (latest row) | {f(m['sel_core_done'])} |",
        f"| attention start (p10 / p50 / max) | {f(m['attn_start_p10'])} / {f(m['attn_start_p50'])} / {f(m['attn_start_max'])} |",
        f"| attention done (p50 / max) | {f(m['attn_done_p50'])} / {f(m['attn_done_max'])} |",
        f"| per-workgroup attention (p50 / max) | {f(m['attn_us_p50'])} / {f(m['attn_us_max'])} |",
        f"| merge after the last partial (p50) | {f(m['merge_us_p50'])} |",
        f"| workgroup end (p50 / max) | {f(m['end_p50'])} / {f(m['end_max'])} |",
    ]
    return "\n".join(lines)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--cfg", type=int, default=3)
    ap.add_argument("--trials", type=int, default=6)
    ap.add_argument("--burst", type=int, default=1,
                    help="stamp the last of this many back-to-back launches")
    ap.add_argument("--no-build", action="store_true")
    args = ap.parse_args()
    if not args.no_build or not os.path.exists(TIMELINE_SO):
        build()
    m = run(args.cfg, args.trials, max(args.burst, 1))
    start = ("the launch starts on an idle device" if m["burst"] == 1 else
             f"the last of {m['burst']} back-to-back launches")
    print(f"decode workload {args.cfg}: {m['workgroups']:.0f} workgroups; "
          f"{m['us_per_step_untraced']:.2f} us per step (timeline build, 200 steps, "
          f"HIP events); stamped: {start}\n")
    print(table(m))


if __name__ == "__main__":
    main()
