"""Parity of the selector front end (projections with rotary embedding and
the cache append; block pooling) with the FP64 oracle (needs an MI355X).

Tolerances: a projected value g (FP32 products of BF16, rounded to BF16)
against the oracle o: |g - o| <= 2^-8 |o| + 1e-5 S, with S the sum of
|W_ji h_i| over the terms that make it up (the FP32 summation bound for
4096-term dots, with margin); the weights w_out (FP32) to 1e-5 S.  Pooled
keys: within one BF16 step (2^-8 relative) of the FP64 block mean, and
bitwise equal to the documented FP32 summation order.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_22874_amd import spot, synth
from paper_2606_22874_amd.synth import bf16_bits, bf16_value

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

DEV = "cuda:0"


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def bf(a):
    return spot.to_device_bf16(a, DEV)


def host_bf16(t):
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


def abs_sums(h, w):
    """S[r, j] = sum_i |W[j, i] h[r, i]|."""
    return np.abs(bf16_value(h).astype(np.float64)) @ np.abs(bf16_value(w).astype(np.float64)).T


def rot_sums(S, Hs, ds, rope_dim):
    """Bound terms after the rotation: a rotated value mixes its pair."""
    S = S.reshape(S.shape[0], Hs, ds).copy()
    half = rope_dim // 2
    both = S[..., :half] + S[..., half:rope_dim]
    S[..., :half] = both
    S[..., half:rope_dim] = both
    return S


def run_project(rows, d_model, Hs, ds, rope_dim, base, pos, rows_per_seq, l_cap, seed=1):
    h, wq, wk, ww = synth.selector_frontend(seed, rows, d_model, Hs, ds)
    n_seq = rows // rows_per_seq
    q_out = torch.empty((rows, Hs, ds), dtype=torch.bfloat16, device=DEV)
    w_out = torch.empty((rows, Hs), dtype=torch.float32, device=DEV)
    cache = torch.zeros((n_seq, l_cap, Hs, ds), dtype=torch.bfloat16, device=DEV)
    spot.spot_selector_project(bf(h), bf(wq), bf(wk), bf(ww), dev(np.asarray(pos, np.int32)),
                               rows, d_model, Hs, ds, rope_dim, base, q_out, w_out, cache,
                               rows_per_seq, l_cap)
    torch.cuda.synchronize()
    q_o, k_o, w_o = oracle.selector_project(h, wq, wk, ww, np.asarray(pos, np.int32), Hs, ds,
                                            rope_dim=rope_dim, rope_base=base)
    return (h, wq, wk, ww), (q_out, w_out, cache), (q_o, k_o, w_o)


def check_bf16(g_bits, o, S):
    g = bf16_value(g_bits).astype(np.float64)
    err = np.abs(g - o)
    bound = 2.0 ** -8 * np.abs(o) + 1e-5 * S
    assert np.all(err <= bound), f"max excess {np.max(err - bound)}"


CASES = [
    # rows, d_model, Hs, ds, rope_dim, base, rows_per_seq, l_cap
    (4, 4096, 4, 128, 64, 1.0e6, 1, 131072),     # decode, Qwen3-8B hidden size
    (4, 4096, 8, 64, 32, 1.0e6, 1, 8192),
    (3, 5120, 4, 128, 64, 1.0e6, 1, 4096),       # Qwen3-32B hidden size: two chunk passes
    (20, 2560, 4, 128, 64, 1.0e4, 20, 64),       # prefill rows, two row passes
    (6, 1000, 8, 64, 64, 500.0, 3, 128),         # d_model not a multiple of 512, all dims rotated
    (2, 512, 4, 128, 0, 1.0e6, 1, 64),           # no rotary dims
]


@pytest.mark.parametrize("rows,d_model,Hs,ds,rope_dim,base,rps,l_cap", CASES)
def test_project_parity(rows, d_model, Hs, ds, rope_dim, base, rps, l_cap):
    print(f"[frontend] project rows={rows} d_model={d_model} {Hs}x{ds} rope {rope_dim}",
          flush=True)
    rng = np.random.default_rng(rows * d_model)
    if rps == 1:
        pos = rng.integers(0, l_cap, rows)
        pos[0] = l_cap - 1
    else:
        pos = np.tile(np.arange(rps), rows // rps)
    (h, wq, wk, ww), (q_out, w_out, cache), (q_o, k_o, w_o) = run_project(
        rows, d_model, Hs, ds, rope_dim, base, pos, rps, l_cap)
    Sq = rot_sums(abs_sums(h, wq), Hs, ds, rope_dim)
    Sk = rot_sums(abs_sums(h, wk), Hs, ds, rope_dim)
    check_bf16(host_bf16(q_out), q_o, Sq)
    cache_h = host_bf16(cache)
    k_g = np.stack([cache_h[r // rps, pos[r]] for r in range(rows)])
    check_bf16(k_g, k_o, Sk)
    Sw = abs_sums(h, ww)
    assert np.all(np.abs(w_out.cpu().numpy() - w_o) <= 1e-5 * Sw)
    # nothing else of the cache was written
    mask = np.ones(cache_h.shape[:2], bool)
    for r in range(rows):
        mask[r // rps, pos[r]] = False
    assert np.all(cache_h[mask] == 0)


def test_project_skips_keys_outside_the_cache():
    rows, l_cap = 4, 128
    pos = np.array([5, -1, 128, 127], np.int32)
    (h, wq, wk, ww), (q_out, w_out, cache), (q_o, k_o, w_o) = run_project(
        rows, 1024, 4, 128, 64, 1.0e6, pos, 1, l_cap)
    cache_h = host_bf16(cache)
    assert np.all(cache_h[1] == 0) and np.all(cache_h[2] == 0)
    assert np.any(cache_h[0, 5] != 0) and np.any(cache_h[3, 127] != 0)
    # the queries are still produced at the given (even out-of-range) positions
    check_bf16(host_bf16(q_out), q_o, rot_sums(abs_sums(h, wq), 4, 128, 64))


def fp32_quarter_mean(k_tok, b, lo, hi):
    """The documented FP32 order: each 16-token quarter of the block summed
    as a pairwise tree ((t0 + t1) + (t2 + t3), then groups of 4 and 8; absent
    tokens -0.0), the quarters added in order, one division."""
    zero = np.full(k_tok.shape[2:], -0.0, np.float32)
    parts = []
    for q in range(4):
        vals = [bf16_value(k_tok[b, t]).astype(np.float32) if t < hi else zero
                for t in range(lo + 16 * q, lo + 16 * q + 16)]
        while len(vals) > 1:
            vals = [vals[2 * i] + vals[2 * i + 1] for i in range(len(vals) // 2)]
        parts.append(vals[0])
    tot = ((parts[0] + parts[1]) + parts[2]) + parts[3]
    return bf16_bits(tot / np.float32(hi - lo))


@pytest.mark.parametrize("n_seq,L,Hs,ds", [(3, 1024, 4, 128), (2, 4096, 8, 64)])
def test_pool_parity(n_seq, L, Hs, ds):
    rng = np.random.default_rng(L + n_seq)
    k_tok = bf16_bits(rng.standard_normal((n_seq, L, Hs, ds), dtype=np.float32))
    seq_len = np.array([L, L - 100, 1][:n_seq], np.int32)
    pooled = torch.zeros((n_seq, L // 64, Hs, ds), dtype=torch.bfloat16, device=DEV)
    spot.spot_selector_pool(bf(k_tok), pooled, n_seq, L, Hs, ds, dev(seq_len))
    torch.cuda.synchronize()
    g = host_bf16(pooled)
    o = oracle.selector_pool(k_tok, seq_len)
    gv = bf16_value(g).astype(np.float64)
    nv = (seq_len + 63) // 64
    for b in range(n_seq):
        assert np.all(np.abs(gv[b, :nv[b]] - o[b, :nv[b]]) <= 2.0 ** -8 * np.abs(o[b, :nv[b]]))
        assert np.all(g[b, nv[b]:] == 0)                      # blocks without tokens untouched
        for j in (0, nv[b] - 1):
            lo, hi = j * 64, min(j * 64 + 64, int(seq_len[b]))
            np.testing.assert_array_equal(g[b, j], fp32_quarter_mean(k_tok, b, lo, hi))


def test_decode_front_end_step():
    """One decode step's front end: project the new token (append its key),
    re-pool only its block, then score; against the oracle run on the same
    cache contents."""
    B, L, Hs, ds, d_model = 4, 8192, 8, 64, 4096
    rng = np.random.default_rng(99)
    k_tok = bf16_bits(rng.standard_normal((B, L, Hs, ds), dtype=np.float32))
    seq_len = np.array([8192, 5000, 65, 64], np.int32)
    pos = seq_len - 1
    h, wq, wk, ww = synth.selector_frontend(7, B, d_model, Hs, ds)
    cache = bf(k_tok)
    pooled = torch.zeros((B, L // 64, Hs, ds), dtype=torch.bfloat16, device=DEV)
    spot.spot_selector_pool(cache, pooled, B, L, Hs, ds, dev(seq_len))      # the prefill pooling
    q_out = torch.empty((B, Hs, ds), dtype=torch.bfloat16, device=DEV)
    w_out = torch.empty((B, Hs), dtype=torch.float32, device=DEV)
    spot.spot_selector_project(bf(h), bf(wq), bf(wk), bf(ww), dev(pos), B, d_model, Hs, ds, 32,
                               1.0e6, q_out, w_out, cache, 1, L)
    spot.spot_selector_pool(cache, pooled, B, L, Hs, ds, dev(seq_len), dev(pos // 64), 1)
    nv = (seq_len + 63) // 64
    scores = spot.selector_score(q_out, w_out, pooled, n_valid=dev(nv), nblk=L // 64)
    torch.cuda.synchronize()
    cache_h = host_bf16(cache)
    # the appended keys are the GPU's; everything downstream is checked on them
    q_o, k_o, w_o = oracle.selector_project(h, wq, wk, ww, pos, Hs, ds, rope_dim=32,
                                            rope_base=1.0e6)
    check_bf16(np.stack([cache_h[b, pos[b]] for b in range(B)]), k_o,
               rot_sums(abs_sums(h, wk), Hs, ds, 32))
    pooled_o = oracle.selector_pool(cache_h, seq_len)
    pv = bf16_value(host_bf16(pooled)).astype(np.float64)
    for b in range(B):
        assert np.all(np.abs(pv[b, :nv[b]] - pooled_o[b, :nv[b]]) <=
                      2.0 ** -8 * np.abs(pooled_o[b, :nv[b]]))
    s_o = oracle.selector_score(host_bf16(q_out), w_out.cpu().numpy(), host_bf16(pooled),
                                n_valid=nv)
    s_g = scores.cpu().numpy()
    fin = np.isfinite(s_o)
    assert np.array_equal(np.isfinite(s_g), fin)
    assert np.all(np.abs(s_g[fin] - s_o[fin]) <= 1e-4 * np.abs(s_o[fin]) + 1e-6)


@pytest.mark.parametrize("B,L,Hs,ds,rope_dim,with_len", [
    (4, 8192, 8, 64, 32, True),       # decode, Qwen3-8B hidden size
    (4, 32768, 4, 128, 64, False),    # seq_len = pos + 1
    (9, 4096, 4, 128, 0, True),       # more rows than one pass (RP = 16 path)
])
def test_fused_front_end_equals_project_then_pool(B, L, Hs, ds, rope_dim, with_len):
    """spot_selector_project_pooled gives exactly what spot_selector_project
    followed by spot_selector_pool of the new token's block gives: queries,
    weights, the cache and the whole pooled cache, bit for bit.  Positions
    cover the first token of a block, the last, the middle, position 0, a
    seq_len past pos (later tokens of the block count) and a position
    outside the cache (nothing stored or pooled)."""
    d_model = 4096
    rng = np.random.default_rng([B, L, Hs])
    k_tok = bf16_bits(rng.standard_normal((B, L, Hs, ds), dtype=np.float32))
    pos = np.array([L - 1, 64, 127, 0, 5000 % L, 200, 63, L, 1000][:B], np.int32)
    seq_len = np.minimum(pos + 1 + np.array([0, 0, 0, 0, 7, 0, 0, 0, 30][:B]), L).astype(np.int32)
    h, wq, wk, ww = synth.selector_frontend(11, B, d_model, Hs, ds)
    args = (bf(h), bf(wq), bf(wk), bf(ww))
    pool0 = torch.zeros((B, L // 64, Hs, ds), dtype=torch.bfloat16, device=DEV)
    spot.spot_selector_pool(bf(k_tok), pool0, B, L, Hs, ds, dev(np.minimum(pos, L)))
    outs = []
    for fused in (False, True):
        q_out = torch.empty((B, Hs, ds), dtype=torch.bfloat16, device=DEV)
        w_out = torch.empty((B, Hs), dtype=torch.float32, device=DEV)
        cache, pooled = bf(k_tok), pool0.clone()
        sl = dev(seq_len) if with_len else None
        if fused:
            spot.spot_selector_project_pooled(*args, dev(pos), sl, B, d_model, Hs, ds, rope_dim,
                                              1.0e6, q_out, w_out, cache, pooled, L)
        else:
            spot.spot_selector_project(*args, dev(pos), B, d_model, Hs, ds, rope_dim, 1.0e6,
                                       q_out, w_out, cache, 1, L)
            spot.spot_selector_pool(cache, pooled, B, L, Hs, ds,
                                    sl if with_len else dev(pos + 1), dev(pos // 64), 1)
        outs.append((q_out, w_out, cache, pooled))
    torch.cuda.synchronize()
    for name, a, b in zip(("q_out", "w_out", "k_cache", "k_pool"), *outs):
        if a.dtype == torch.bfloat16:
            a, b = a.view(torch.int16), b.view(torch.int16)
        assert torch.equal(a, b), name
    assert not torch.equal(outs[1][3].view(torch.int16), pool0.view(torch.int16))


def test_front_end_in_a_graph_matches_eager():
    """Projection and pooling captured in a HIP graph: every replay (with
    eager work and synchronisations between replays) gives the eager result."""
    B, L, Hs, ds, d_model = 4, 4096, 4, 128, 4096
    h, wq, wk, ww = synth.selector_frontend(5, B, d_model, Hs, ds)
    hd, wqd, wkd, wwd = bf(h), bf(wq), bf(wk), bf(ww)
    seq_len = np.array([4096, 3000, 64, 1], np.int32)
    pos, first, sl = dev(seq_len - 1), dev((seq_len - 1) // 64), dev(seq_len)
    outs = []
    for _ in range(2):
        outs.append((torch.empty((B, Hs, ds), dtype=torch.bfloat16, device=DEV),
                     torch.empty((B, Hs), dtype=torch.float32, device=DEV),
                     torch.zeros((B, L, Hs, ds), dtype=torch.bfloat16, device=DEV),
                     torch.zeros((B, L // 64, Hs, ds), dtype=torch.bfloat16, device=DEV)))

    def run(o, st):
        spot.spot_selector_project(hd, wqd, wkd, wwd, pos, B, d_model, Hs, ds, 64, 1.0e6, o[0],
                                   o[1], o[2], 1, L, st)
        spot.spot_selector_pool(o[2], o[3], B, L, Hs, ds, sl, first, 1, st)

    run(outs[0], torch.cuda.current_stream())
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        run(outs[1], torch.cuda.current_stream())
    for rep in range(3):
        for t in outs[1]:
            t.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for a, b in zip(outs[0], outs[1]):
            assert torch.equal(a.view(torch.int16) if a.dtype == torch.bfloat16 else a,
                               b.view(torch.int16) if b.dtype == torch.bfloat16 else b), rep
