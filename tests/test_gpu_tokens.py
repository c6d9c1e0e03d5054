"""Parity of the per-token selector (block value = maximum of the per-token
scores, Section 2.3) with the FP64 oracle (needs an MI355X), for 64-token
blocks and for the paper's 16-token selector block (Appendix A), the latter
through selection and attention as well.

Calls go through the C ABI (spot_selector_score_tokens,
spot_selector_score_tokens_blk, spot_sparse_decode_blk); the oracle runs on
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


def assert_out_close(out_g, lse_g, out_o, lse_o):
    """Decode outputs as in the 64-token decode tests: max-abs 2e-2 and
    relative L2 1e-2 on the BF16 outputs, 2e-3 on the log-sum-exps."""
    g = out_g.float().cpu().numpy().astype(np.float64)
    diff = g - out_o
    assert np.max(np.abs(diff)) <= 2e-2, np.max(np.abs(diff))
    rel = np.linalg.norm(diff) / max(np.linalg.norm(out_o), 1e-30)
    assert rel <= 1e-2, rel
    lg = lse_g.cpu().numpy().astype(np.float64)
    fin = np.isfinite(lse_o)
    assert np.array_equal(np.isfinite(lg), fin)
    assert np.all(np.abs(lg[fin] - lse_o[fin]) <= 2e-3)


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


def device_keys(k, sc, fmt):
    k_d = bf(k) if fmt == "bf16" else dev(k)
    sc_d = None if sc is None else (dev(sc.view(np.int16)) if fmt in ("int4", "int8")
                                    else dev(sc))
    return k_d, sc_d


def run_both(q, w, k, sc, fmt, rows_per_seq, L, lens, blk=64):
    Hs, ds = q.shape[-2:]
    sl_o = None if lens is None else np.asarray(lens, np.int32)
    s_o = oracle.selector_score_tokens(q, w, k, sc, fmt, rows_per_seq=rows_per_seq,
                                       seq_len=sl_o, l_cap=L, blk=blk, h_s=Hs, d_s=ds)
    k_d, sc_d = device_keys(k, sc, fmt)
    sl_d = None if lens is None else dev(np.asarray(lens, np.int32))
    s_g = spot.selector_score_tokens(bf(q), dev(w), k_d, sc_d, fmt,
                                     rows_per_seq=rows_per_seq, seq_len=sl_d, l_cap=L, blk=blk)
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


# ----------------------------------------------- the paper's 16-token block
# Appendix A's hyper-parameter table sets the selector block to 16 tokens:
# spot_selector_score_tokens_blk takes each 16-token block's maximum, the
# selection runs over l_cap / 16 blocks, and spot_sparse_decode_blk attends to
# the selected 16-token blocks.
CASES16 = [
    # n_seq, rows_per_seq, L, Hs, ds, lens (per row), fmt
    (2, 1, 4096, 8, 64, [4096, 4000], "bf16"),
    (3, 1, 448, 4, 128, [448, 447, 17], "bf16"),
    (9, 1, 448, 4, 128, [448, 16, 15, 1, 0, 65, 300, 5000, 33], "bf16"),  # empty, clamped
    (2, 3, 2048, 4, 128, [2048, 1000, 16, 1500, 1501, 2047], "bf16"),     # rows share keys
    (2, 1, 4096, 8, 64, [4096, 3001], "int4"),
    (3, 1, 448, 4, 128, [448, 300, 17], "int4"),
    (2, 1, 4096, 4, 128, [4096, 4000], "mxfp4"),
    (3, 2, 1024, 8, 64, [1024, 1, 700, 64, 1000, 65], "mxfp4"),
    (2, 1, 4096, 4, 128, [4096, 2049], "int8"),
    (2, 1, 448, 8, 64, [447, 31], "int8"),
    (2, 1, 4096, 8, 64, [3000, 4096], "mxfp8"),
    (3, 2, 1024, 4, 128, [1024, 1, 700, 64, 1000, 65], "mxfp8"),
]


@pytest.mark.parametrize("n_seq,rps,L,Hs,ds,lens,fmt", CASES16)
def test_score_tokens16_parity(n_seq, rps, L, Hs, ds, lens, fmt):
    print(f"[tokens16] n_seq={n_seq} rps={rps} L={L} Hs={Hs} ds={ds} {fmt}", flush=True)
    q, w, k, sc = inputs(n_seq * 100 + L + 1, n_seq, rps, L, Hs, ds, lens, fmt)
    s_g, s_o = run_both(q, w, k, sc, fmt, rps, L, lens, blk=16)
    assert s_g.shape == (n_seq * rps, L // 16)
    assert_scores_close(s_g, s_o)


@pytest.mark.parametrize("fmt,Hs,ds", [("bf16", 8, 64), ("bf16", 4, 128), ("int4", 4, 128),
                                       ("mxfp4", 8, 64), ("int8", 8, 64), ("mxfp8", 4, 128)])
def test_score_tokens16_nest_in_64_bitwise(fmt, Hs, ds):
    """Both block sizes take maxima of the same per-token FP32 scores, so a
    64-token value is the largest of its four 16-token values exactly."""
    n_seq, L, lens = 3, 1024, [1024, 531, 16]
    print(f"[tokens16] nesting {fmt} {Hs}x{ds}", flush=True)
    q, w, k, sc = inputs(77, n_seq, 1, L, Hs, ds, lens, fmt)
    k_d, sc_d = device_keys(k, sc, fmt)
    sl = dev(np.asarray(lens, np.int32))
    s16 = spot.selector_score_tokens(bf(q), dev(w), k_d, sc_d, fmt, seq_len=sl, l_cap=L, blk=16)
    s64 = spot.selector_score_tokens(bf(q), dev(w), k_d, sc_d, fmt, seq_len=sl, l_cap=L)
    torch.cuda.synchronize()
    s16 = s16.cpu().numpy()
    np.testing.assert_array_equal(s64.cpu().numpy(), s16.reshape(n_seq, L // 64, 4).max(axis=2))


def _rand_sets(rng, B, nb, n_per, extra_bad):
    """Distinct random 16-token block ids per sequence (unsorted), plus bad
    ids (negative, past the visible blocks) when extra_bad."""
    k_max = max(n_per) + 2
    idx = np.full((B, k_max), -1, np.int32)
    cnt = np.zeros(B, np.int32)
    for b in range(B):
        row = list(rng.permutation(nb[b])[: min(nb[b], n_per[b])])
        if extra_bad and b % 2:
            row += [-3, nb[b] + 1]
        idx[b, :len(row)] = row
        cnt[b] = len(row)
    return idx, cnt


@pytest.mark.parametrize("Hq,Hkv", [(32, 8), (8, 8), (16, 8), (64, 8)])
def test_sparse_decode16_parity(Hq, Hkv):
    """16-token blocks at every GQA group: ragged lengths (not multiples of
    16), list lengths that leave a workgroup's last four-entry step partly
    empty, unsorted ids and bad ids."""
    B, L, d = 4, 4096, 128
    print(f"[decode16] Hq={Hq} Hkv={Hkv}", flush=True)
    q, k, v = synth._backbone_decode(901 + Hq, B, L, Hq, Hkv, d)
    seq_len = np.array([4096, 3001, 17, 1], np.int32)
    nb = (seq_len + 15) // 16
    rng = np.random.default_rng(Hq)
    idx, cnt = _rand_sets(rng, B, nb, [131, 77, 2, 1], True)
    scale = 1 / np.sqrt(d)
    out_o, lse_o = oracle.sparse_decode(q, k, v, seq_len, idx, cnt, scale, blk=16)
    out_g, lse_g = spot.sparse_decode(bf(q), bf(k), bf(v), dev(seq_len), dev(idx), dev(cnt),
                                      scale, blk=16)
    torch.cuda.synchronize()
    assert_out_close(out_g, lse_g, out_o, lse_o)
    # An empty set gives zeros and lse = -inf.
    out_g, lse_g = spot.sparse_decode(bf(q), bf(k), bf(v), dev(seq_len), dev(idx),
                                      dev(np.zeros(B, np.int32)), scale, blk=16)
    torch.cuda.synchronize()
    assert torch.all(out_g.float() == 0) and torch.all(torch.isinf(lse_g))


def test_sparse_decode16_long_lists():
    """2048 entries per sequence (a quarter of a 128K cache): several hundred
    per workgroup."""
    B, Hq, Hkv, L, d = 2, 32, 8, 32768, 128
    q, k, v = synth._backbone_decode(917, B, L, Hq, Hkv, d)
    seq_len = np.array([32768, 30001], np.int32)
    idx, cnt = _rand_sets(np.random.default_rng(5), B, (seq_len + 15) // 16, [2048, 1999],
                          False)
    scale = 1 / np.sqrt(d)
    print("[decode16] long lists", flush=True)
    out_o, lse_o = oracle.sparse_decode(q, k, v, seq_len, idx, cnt, scale, blk=16)
    out_g, lse_g = spot.sparse_decode(bf(q), bf(k), bf(v), dev(seq_len), dev(idx), dev(cnt),
                                      scale, blk=16)
    torch.cuda.synchronize()
    assert_out_close(out_g, lse_g, out_o, lse_o)


def test_sparse_decode16_quarters_equal_64():
    """Selecting the four 16-token quarters of some 64-token blocks attends to
    the same tokens as selecting those blocks (summation orders differ)."""
    B, Hq, Hkv, L, d = 3, 32, 8, 8192, 128
    q, k, v = synth._backbone_decode(923, B, L, Hq, Hkv, d)
    seq_len = np.array([8192, 5000, 100], np.int32)
    rng = np.random.default_rng(9)
    idx64, cnt64 = _rand_sets(rng, B, (seq_len + 63) // 64, [40, 33, 2], False)
    idx16 = np.full((B, 4 * idx64.shape[1]), -1, np.int32)
    for b in range(B):
        ids = idx64[b, :cnt64[b]]
        idx16[b, :4 * len(ids)] = (4 * ids[:, None] + np.arange(4)).reshape(-1)
    scale = 1 / np.sqrt(d)
    a, la = spot.sparse_decode(bf(q), bf(k), bf(v), dev(seq_len), dev(idx64), dev(cnt64), scale)
    b_, lb = spot.sparse_decode(bf(q), bf(k), bf(v), dev(seq_len), dev(idx16), dev(4 * cnt64),
                                scale, blk=16)
    torch.cuda.synchronize()
    assert torch.max(torch.abs(a.float() - b_.float())).item() <= 1e-2
    assert torch.max(torch.abs(la - lb)).item() <= 1e-4


def test_block16_full_size_pipeline():
    """The paper's selector geometry (4 heads x 128) and block (16 tokens) at
    128K tokens, batch 4: every 16-token block value against the oracle, the
    dual top-p / top-K set over 8192 blocks against the oracle's set of its
    own scores, then attention over the GPU's set against the oracle on that
    set (32 query / 8 KV heads)."""
    B, L, Hs, ds, Hq, Hkv, d = 4, 131072, 4, 128, 32, 8, 128
    lens = np.array([131072, 131072, 100000, 70001], np.int32)
    rule = Rule(0.95, 512, 0, 4, 8)
    print("[block16] full size: generating", flush=True)
    q_s, w, k_tok = synth.selector_tokens(13, B, L, Hs, ds, lens, rule=rule, blk=16)
    s_g, s_o = run_both(q_s, w, k_tok, None, "bf16", 1, L, lens, blk=16)
    assert_scores_close(s_g, s_o)
    del k_tok
    nv = (lens + 15) // 16
    s_o32 = s_o.astype(np.float32)
    idx_o, cnt_o, _ = oracle.select_blocks(s_o32.astype(np.float64), rule, nv)
    idx_g, cnt_g, _ = spot.select_blocks(dev(s_g), rule, dev(nv))
    torch.cuda.synchronize()
    idx_g, cnt_g = idx_g.cpu().numpy(), cnt_g.cpu().numpy()
    print("[block16] selection", check_all(s_o32, nv, rule, idx_o, cnt_o, idx_g, cnt_g),
          flush=True)
    q, k, v = synth._backbone_decode(929, B, L, Hq, Hkv, d)
    scale = 1 / np.sqrt(d)
    out_g, lse_g = spot.sparse_decode(bf(q), bf(k), bf(v), dev(lens), dev(idx_g), dev(cnt_g),
                                      scale, blk=16)
    torch.cuda.synchronize()
    out_o, lse_o = oracle.sparse_decode(q, k, v, lens, idx_g, cnt_g, scale, blk=16)
    assert_out_close(out_g, lse_g, out_o, lse_o)


def test_block_size_errors_leave_outputs_untouched():
    """Blocks other than 16 or 64 tokens are refused before any launch."""
    q = bf(np.zeros((1, 4, 128), np.uint16))
    w = dev(np.zeros((1, 4), np.float32))
    k_tok = bf(np.zeros((1, 128, 4, 128), np.uint16))
    scores = torch.full((1, 4), 7.0, device=DEV)
    with pytest.raises(spot.SpotError) as e:
        spot.spot_selector_score_tokens_blk(q, w, k_tok, None, "bf16", 1, 1, 128, 32, 4, 128,
                                            None, scores)
    assert e.value.status == 3
    qd = bf(np.zeros((1, 8, 128), np.uint16))
    kv = bf(np.zeros((1, 8, 128, 128), np.uint16))
    out = torch.full((1, 8, 128), 3.0, dtype=torch.bfloat16, device=DEV)
    ws = spot.decode_workspace(1, 8, 8, 128, 4, DEV)
    with pytest.raises(spot.SpotError) as e:
        spot.spot_sparse_decode_blk(qd, kv, kv, dev(np.array([128], np.int32)),
                                    dev(np.zeros((1, 4), np.int32)), dev(np.array([1], np.int32)),
                                    4, 32, 1, 8, 8, 128, 128, 0.1, out, None, ws)
    assert e.value.status == 3
    torch.cuda.synchronize()
    assert torch.all(scores == 7.0) and torch.all(out.float() == 3.0)
