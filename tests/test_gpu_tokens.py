"""Parity of the per-token selector (block value = maximum of the per-token
scores, Section 2.3) with the FP64 oracle (needs an MI355X).

Calls go through the C ABI (spot_selector_score_tokens); the oracle runs on
the same seeded inputs.  Tolerance as for the pooled scores:
|gpu - oracle| <= 1e-4 |oracle| + 1e-6 (FP32 dot products of 512 terms
against FP64), and exactly the same -inf entries.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_22874_amd import spot, synth
from paper_2606_22874_amd.synth import Rule

from selcheck import check_all

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

DEV = "cuda:0"


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def bf(a):
    return spot.to_device_bf16(a, DEV)


def assert_scores_close(g, o):
    fin = np.isfinite(o)
    assert np.array_equal(np.isfinite(g), fin)
    assert np.all(g[~fin] == -np.inf)
    err = np.abs(g[fin] - o[fin])
    bound = 1e-4 * np.abs(o[fin]) + 1e-6
    assert np.all(err <= bound), f"max excess {np.max(err - bound)}"


def inputs(seed, n_seq, rows_per_seq, L, Hs, ds, lens, fmt):
    """Per-token keys for n_seq sequences and rows_per_seq query rows each."""
    lens = np.asarray(lens, dtype=np.int32)
    seq_vis = lens.reshape(n_seq, rows_per_seq).max(axis=1)
    q, w, k = synth.selector_tokens(seed, n_seq, L, Hs, ds, seq_vis)
    rng = np.random.default_rng([seed, 5])
    if rows_per_seq > 1:   # further query rows of each sequence
        q = np.concatenate([q[:, None], synth.bf16_bits(rng.standard_normal(
            (n_seq, rows_per_seq - 1, Hs, ds), dtype=np.float32))], axis=1)
        w = np.concatenate([w[:, None], rng.uniform(0, 1, (n_seq, rows_per_seq - 1, Hs))
                            .astype(np.float32)], axis=1)
    q = q.reshape(n_seq * rows_per_seq, Hs, ds)
    w = w.reshape(n_seq * rows_per_seq, Hs)
    if fmt == "bf16":
        return q, w, k, None
    c, s = synth.QUANTIZERS[fmt](k)
    return q, w, c, (s.view(np.uint16) if fmt in ("int4", "int8") else s)


def run_both(q, w, k, sc, fmt, rows_per_seq, L, lens):
    Hs, ds = q.shape[-2:]
    sl_o = None if lens is None else np.asarray(lens, np.int32)
    s_o = oracle.selector_score_tokens(q, w, k, sc, fmt, rows_per_seq=rows_per_seq,
                                       seq_len=sl_o, l_cap=L, h_s=Hs, d_s=ds)
    k_d = bf(k) if fmt == "bf16" else dev(k)
    sc_d = None if sc is None else (dev(sc.view(np.int16)) if fmt in ("int4", "int8")
                                    else dev(sc))
    sl_d = None if lens is None else dev(np.asarray(lens, np.int32))
    s_g = spot.selector_score_tokens(bf(q), dev(w), k_d, sc_d, fmt,
                                     rows_per_seq=rows_per_seq, seq_len=sl_d, l_cap=L)
    torch.cuda.synchronize()
    return s_g.cpu().numpy(), s_o


CASES = [
    # n_seq, rows_per_seq, L, Hs, ds, lens (per row), fmt
    (2, 1, 4096, 8, 64, [4096, 4096], "bf16"),
    (3, 1, 8192, 4, 128, [8192, 5000, 1], "bf16"),      # ragged, one-token sequence
    (9, 1, 448, 4, 128, [448, 447, 65, 64, 63, 0, 1, 300, 5000], "bf16"),  # 7 blocks, empty,
                                                         # clamped, units not a multiple of 8
    (2, 1, 4096, 8, 64, [4096, 3001], "int4"),
    (2, 1, 4096, 4, 128, [2500, 4096], "int4"),
    (2, 1, 4096, 8, 64, [4096, 129], "mxfp4"),
    (2, 1, 4096, 4, 128, [4096, 4000], "mxfp4"),
    (2, 3, 2048, 4, 128, [2048, 1000, 64, 1500, 1501, 2047], "bf16"),  # rows share keys
    (3, 2, 1024, 8, 64, [1024, 700, 1, 2, 900, 1024], "int4"),
    (2, 1, 4096, 4, 128, [4096, 2049], "int8"),
    (2, 1, 4096, 8, 64, [3000, 4096], "mxfp8"),
    (3, 2, 1024, 4, 128, [1024, 1, 700, 64, 1000, 65], "mxfp8"),
    # quantized keys run one wave per block, four blocks per workgroup: block
    # counts that leave a workgroup's run partly empty (7 and 1 blocks)
    (3, 1, 448, 4, 128, [448, 300, 0], "int4"),
    (3, 1, 448, 8, 64, [447, 65, 448], "mxfp4"),
    (2, 1, 448, 4, 128, [448, 129], "int8"),
    (2, 1, 448, 8, 64, [63, 448], "mxfp8"),
    (2, 1, 64, 4, 128, [64, 5], "mxfp4"),
    (2, 3, 2048, 4, 128, [2048, 1000, 64, 1500, 1501, 2047], "mxfp4"),
    (2, 3, 2048, 8, 64, [2048, 999, 1, 2000, 1501, 2048], "int8"),
]


@pytest.mark.parametrize("n_seq,rps,L,Hs,ds,lens,fmt", CASES)
def test_score_tokens_parity(n_seq, rps, L, Hs, ds, lens, fmt):
    print(f"[tokens] n_seq={n_seq} rps={rps} L={L} Hs={Hs} ds={ds} {fmt}", flush=True)
    q, w, k, sc = inputs(n_seq * 100 + L, n_seq, rps, L, Hs, ds, lens, fmt)
    s_g, s_o = run_both(q, w, k, sc, fmt, rps, L, lens)
    assert_scores_close(s_g, s_o)


def test_score_tokens_without_seq_len():
    q, w, k, _ = inputs(3, 2, 1, 2048, 4, 128, [2048, 2048], "bf16")
    s_g, s_o = run_both(q, w, k, None, "bf16", 1, 2048, None)
    assert np.all(np.isfinite(s_o))
    assert_scores_close(s_g, s_o)


def test_score_tokens_full_size_and_selection():
    """Four sequences of 131072 tokens with the paper's selector geometry
    (4 heads x 128): every block value, then the dual top-p / top-K set of
    the GPU scores against the oracle's set of its own scores."""
    B, L, Hs, ds = 4, 131072, 4, 128
    lens = [131072, 131072, 100000, 70001]
    print("[tokens] full size", flush=True)
    q, w, k, _ = inputs(11, B, 1, L, Hs, ds, lens, "bf16")
    s_g, s_o = run_both(q, w, k, None, "bf16", 1, L, lens)
    assert_scores_close(s_g, s_o)
    rule = Rule(0.95, 128, 0, 1, 2)
    nv = (np.asarray(lens, np.int32) + 63) // 64
    s_o32 = s_o.astype(np.float32)
    idx_o, cnt_o, _ = oracle.select_blocks(s_o32.astype(np.float64), rule, nv)
    idx_g, cnt_g, _ = spot.select_blocks(dev(s_g), rule, dev(nv))
    torch.cuda.synchronize()
    print("[tokens] selection", check_all(s_o32, nv, rule, idx_o, cnt_o, idx_g.cpu().numpy(),
                                          cnt_g.cpu().numpy()))


def test_score_tokens_repeated_key_equals_pooled_kernel():
    """Tokens of a block all holding the pooled key kbar: the per-token kernel
    agrees with the pooled kernel on kbar, to the scores' tolerance (the two
    sum the dot products in different orders)."""
    rng = np.random.default_rng(41)
    B, nblk, Hs, ds = 2, 40, 8, 64
    q = synth.bf16_bits(rng.standard_normal((B, Hs, ds), dtype=np.float32))
    w = rng.uniform(0, 1, (B, Hs)).astype(np.float32)
    kbar = synth.bf16_bits(rng.standard_normal((B, nblk, Hs, ds), dtype=np.float32))
    k_tok = np.repeat(kbar, 64, axis=1)
    pooled = spot.selector_score(bf(q), dev(w), bf(kbar), nblk=nblk)
    per_tok = spot.selector_score_tokens(bf(q), dev(w), bf(k_tok),
                                         l_cap=nblk * 64)
    torch.cuda.synchronize()
    assert_scores_close(per_tok.cpu().numpy(), pooled.cpu().numpy().astype(np.float64))
