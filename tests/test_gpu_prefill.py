"""Parity of the HIP block-sparse causal prefill with the FP64 oracle (MI355X).

The kernel is fed the oracle's own block selection (or a hand-built one) and
every compared output must satisfy the decode tolerances:
  max |gpu - oracle| <= 2e-2, ||gpu - oracle|| / ||oracle|| <= 1e-2,
  |lse_gpu - lse_oracle| <= 2e-3, and the same -inf pattern in lse.
The probabilities enter the P.V product in BF16 (relative error <= 2^-9 per
weight), which with FP32 accumulation and a BF16 output stays well inside
these bounds for unit-variance inputs.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_22874_amd import spot, synth

from selcheck import check_all

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

DEV = "cuda:0"


def bf(a):
    return spot.to_device_bf16(a, DEV)


def i32(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(DEV)


def qkv(seed, B, h_q, h_kv, L, d=128):
    return (synth.normal_bf16(seed, 1, (B, h_q, L, d)), synth.normal_bf16(seed, 2, (B, h_kv, L, d)),
            synth.normal_bf16(seed, 3, (B, h_kv, L, d)))


def rows_of(out, lse, B, L, rows):
    """GPU [B, h, L, d] outputs regrouped as the oracle's [n, h, 64, d] rows."""
    nqb = L // 64
    o = out.float().cpu().numpy().astype(np.float64)
    s = lse.cpu().numpy().astype(np.float64)
    og = np.stack([o[r // nqb, :, (r % nqb) * 64:(r % nqb + 1) * 64] for r in rows])
    sg = np.stack([s[r // nqb, :, (r % nqb) * 64:(r % nqb + 1) * 64] for r in rows])
    return og, sg


def assert_close(og, sg, oo, so):
    diff = og - oo
    max_abs = np.max(np.abs(diff)) if diff.size else 0.0
    rel = np.linalg.norm(diff) / max(np.linalg.norm(oo), 1e-30)
    assert max_abs <= 2e-2, max_abs
    assert rel <= 1e-2, rel
    fin = np.isfinite(so)
    assert np.array_equal(np.isfinite(sg), fin)
    assert np.all(sg[~fin] == -np.inf)
    assert np.all(np.abs(sg[fin] - so[fin]) <= 2e-3), np.max(np.abs(sg[fin] - so[fin]))


def random_selection(rng, B, nqb, k_max, junk=True):
    """Random id lists per (sequence, query block) row, with skipped ids mixed in."""
    rows = B * nqb
    idx = np.full((rows, k_max), -1, np.int32)
    cnt = np.zeros(rows, np.int32)
    for r in range(rows):
        qb = r % nqb
        n = int(rng.integers(0, min(qb + 1, k_max) + 1))
        ids = np.sort(rng.choice(qb + 1, size=n, replace=False)).astype(np.int32)
        row = list(ids)
        if junk and r % 3 == 1 and len(row) + 2 <= k_max:
            row += [qb + 1 + int(rng.integers(0, 4)), -7]     # future block, negative id
        if r % 5 == 2:
            rng.shuffle(row)                                   # any list order
        idx[r, :len(row)] = row
        cnt[r] = len(row)
        if r % 7 == 3:
            cnt[r] = k_max + 5                                 # count past k_max is clipped
            idx[r, len(row):] = -1
    return idx, cnt


@pytest.mark.parametrize("h_q,h_kv,B,L", [(8, 1, 2, 512), (4, 1, 1, 512), (2, 1, 2, 256),
                                          (1, 1, 1, 640), (16, 2, 1, 384)])
def test_prefill_random_selection_all_rows(h_q, h_kv, B, L):
    """Every output row of small problems, every supported GQA group size."""
    rng = np.random.default_rng([h_q, h_kv, B, L])
    nqb = L // 64
    q, k, v = qkv(11 + h_q, B, h_q, h_kv, L)
    idx, cnt = random_selection(rng, B, nqb, k_max=6)
    scale = 1.0 / np.sqrt(128)
    print(f"[prefill] h_q={h_q} h_kv={h_kv} B={B} L={L}", flush=True)
    out_g, lse_g = spot.sparse_prefill(bf(q), bf(k), bf(v), i32(idx), i32(cnt), scale)
    torch.cuda.synchronize()
    rows = np.arange(B * nqb, dtype=np.int32)
    out_o, lse_o = oracle.sparse_prefill(q, k, v, idx, cnt, scale, rows)
    og, sg = rows_of(out_g, lse_g, B, L, rows)
    assert_close(og, sg, out_o, lse_o)


def test_prefill_all_blocks_selected_is_causal_attention():
    """Every block <= qb selected: dense causal attention, all rows."""
    B, h_q, h_kv, L = 1, 8, 1, 1024
    nqb = L // 64
    q, k, v = qkv(5, B, h_q, h_kv, L)
    idx = np.tile(np.arange(nqb, dtype=np.int32), (nqb, 1))
    cnt = np.arange(1, nqb + 1, dtype=np.int32)
    scale = 0.0883
    out_g, lse_g = spot.sparse_prefill(bf(q), bf(k), bf(v), i32(idx), i32(cnt), scale)
    torch.cuda.synchronize()
    rows = np.arange(nqb, dtype=np.int32)
    out_o, lse_o = oracle.sparse_prefill(q, k, v, idx, cnt, scale, rows)
    og, sg = rows_of(out_g, lse_g, B, L, rows)
    assert_close(og, sg, out_o, lse_o)


_c5 = {}


def c5():
    if not _c5:
        print("[gen] prefill workload L=32768 Hq=64 Hkv=8", flush=True)
        wl = synth.prefill_config()
        s = oracle.selector_score(wl.q_sel, wl.w, wl.k_sel, rows_per_seq=wl.nblk,
                                  n_valid=wl.n_valid).astype(np.float32)
        idx, cnt, _ = oracle.select_blocks(s.astype(np.float64), wl.rule, wl.n_valid)
        _c5.update(wl=wl, idx=idx, cnt=cnt)
    return _c5["wl"], _c5["idx"], _c5["cnt"]


def test_prefill_full_size_selection_all_rows():
    """Selector scores (the query-block x key-block matrix-core kernel) and
    the dual top-p / top-K selection of every one of the 512 query blocks of
    the 32K-token layer, on the GPU, against the oracle: all 512 x 512
    scores element by element (1e-4 relative), then the selection."""
    wl, idx_o, cnt_o = c5()
    nqb, rule = wl.nblk, wl.rule
    s64 = oracle.selector_score(wl.q_sel, wl.w, wl.k_sel, rows_per_seq=nqb, n_valid=wl.n_valid)
    s_o = s64.astype(np.float32)
    s_g = spot.selector_score(bf(wl.q_sel), torch.from_numpy(wl.w).to(DEV), bf(wl.k_sel),
                              rows_per_seq=nqb, n_valid=i32(wl.n_valid), nblk=nqb)
    idx_g, cnt_g, _ = spot.select_blocks(s_g, rule, i32(wl.n_valid))
    torch.cuda.synchronize()
    g = s_g.cpu().numpy().astype(np.float64)
    assert g.shape == (nqb, nqb)
    fin = np.isfinite(s64)
    assert np.array_equal(np.isfinite(g), fin) and np.all(g[~fin] == -np.inf)
    assert fin.sum() == nqb * (nqb + 1) // 2          # causal: row qb has qb + 1 blocks
    err = np.abs(g[fin] - s64[fin])
    bound = 1e-4 * np.abs(s64[fin]) + 1e-6
    assert np.all(err <= bound), f"max excess {np.max(err - bound)}"
    print("[prefill] selection of all rows", check_all(
        s_o, wl.n_valid, rule, idx_o, cnt_o, idx_g.cpu().numpy(), cnt_g.cpu().numpy()),
        flush=True)


def test_prefill_full_size_sampled_rows():
    """The 32K-token, 64/8-head layer with the oracle's selection; sampled rows
    are a fixed stratified set over the layer (first query blocks, powers of
    two, the K_max-capped end), capped rows and a few random ones."""
    wl, idx, cnt = c5()
    assert cnt.max() == wl.rule.k_max          # the cap binds on some rows
    out_g, lse_g = spot.sparse_prefill(bf(wl.q), bf(wl.k), bf(wl.v), i32(idx), i32(cnt),
                                       wl.sm_scale)
    torch.cuda.synchronize()
    nqb = wl.nblk
    capped = np.flatnonzero(cnt == wl.rule.k_max)
    rng = np.random.default_rng(9)
    stratified = [0, 1, 2, 3, 31, 63, 64, 127, 191, 255, 256, 319, 383, 447, 510, 511]
    rows = np.unique(np.concatenate([stratified, [nqb - 1], capped[:2],
                                     rng.choice(nqb, 4, replace=False)])).astype(np.int32)
    print(f"[prefill] full size, rows {rows.tolist()}", flush=True)
    out_o, lse_o = oracle.sparse_prefill(wl.q, wl.k, wl.v, idx, cnt, wl.sm_scale, rows)
    og, sg = rows_of(out_g, lse_g, wl.B, wl.L, rows)
    assert_close(og, sg, out_o, lse_o)


def test_prefill_edge_cases():
    """Single block, empty rows (zeros, lse = -inf), only skipped ids, NULL lse."""
    scale = 1.0 / np.sqrt(128)
    q, k, v = qkv(21, 1, 8, 1, 64)
    idx = np.array([[0]], np.int32)
    out_g, lse_g = spot.sparse_prefill(bf(q), bf(k), bf(v), i32(idx), i32([1]), scale)
    torch.cuda.synchronize()
    out_o, lse_o = oracle.sparse_prefill(q, k, v, idx, np.array([1], np.int32), scale,
                                         np.array([0], np.int32))
    og, sg = rows_of(out_g, lse_g, 1, 64, [0])
    assert_close(og, sg, out_o, lse_o)

    q, k, v = qkv(22, 2, 8, 2, 256)
    nqb = 4
    idx = np.array([[5, -1, 9], [0, 1, 2], [2, 3, 0], [7, 8, 9]] * 2, np.int32)
    cnt = np.array([3, 0, 3, 3, 2, 3, -4, 1], np.int32)
    out_g, lse_g = spot.sparse_prefill(bf(q), bf(k), bf(v), i32(idx), i32(cnt), scale)
    torch.cuda.synchronize()
    rows = np.arange(2 * nqb, dtype=np.int32)
    out_o, lse_o = oracle.sparse_prefill(q, k, v, idx, cnt, scale, rows)
    og, sg = rows_of(out_g, lse_g, 2, 256, rows)
    assert_close(og, sg, out_o, lse_o)
    empty = [0, 1, 3, 4, 6, 7]
    assert np.all(og[empty] == 0) and np.all(sg[empty] == -np.inf)

    # lse = NULL writes the same outputs.
    out2 = torch.empty_like(out_g)
    spot.spot_sparse_prefill(bf(q), bf(k), bf(v), 256, i32(idx), i32(cnt), 3, 2, 8, 2, 128, scale,
                             out2, None)
    torch.cuda.synchronize()
    assert torch.equal(out2, out_g)


def test_prefill_deterministic():
    wl, idx, cnt = c5()
    q, k, v, di, dc = bf(wl.q), bf(wl.k), bf(wl.v), i32(idx), i32(cnt)
    res = [spot.sparse_prefill(q, k, v, di, dc, wl.sm_scale) for _ in range(2)]
    torch.cuda.synchronize()
    assert torch.equal(res[0][0], res[1][0]) and torch.equal(res[0][1], res[1][1])


def test_prefill_rejects_before_launch():
    q, k, v = qkv(23, 1, 8, 1, 128)
    q, k, v = bf(q), bf(k), bf(v)
    out = torch.full((1, 8, 128, 128), 7.0, dtype=torch.bfloat16, device=DEV)
    lse = torch.full((1, 8, 128), 7.0, device=DEV)
    cases = [dict(sm_scale=-0.1, status=3), dict(sm_scale=0.0, status=3),
             dict(sm_scale=float("nan"), status=3), dict(sm_scale=float("inf"), status=3),
             dict(k_max=5000, status=3), dict(h_q=6, status=3), dict(L=100, status=2)]
    for c in cases:
        k_max = c.get("k_max", 4)
        idx, cnt = i32(np.zeros((2, k_max), np.int32)), i32([1, 1])
        with pytest.raises(spot.SpotError) as e:
            spot.spot_sparse_prefill(q, k, v, c.get("L", 128), idx, cnt, k_max, 1,
                                     c.get("h_q", 8), 1, 128, c.get("sm_scale", 0.1), out, lse)
        assert e.value.status == c["status"], c
    torch.cuda.synchronize()
    assert torch.all(out.float() == 7.0) and torch.all(lse == 7.0)
