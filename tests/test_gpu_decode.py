"""Parity of the HIP decode path with the FP64 oracle (needs an MI355X).

Every call goes through the C ABI (libspot.so via the ctypes binding); the
oracle runs on the host on the very same seeded inputs.  Tolerances:
  scores   |gpu - oracle| <= 1e-4 |oracle| + 1e-6          (FP32 vs FP64)
  sets     equal, up to near-ties (1e-4 relative) and mass-boundary rows
  outputs  with the oracle's block set fed to the kernel:
           max |gpu - oracle| <= 2e-2 and ||gpu - oracle|| / ||oracle|| <= 1e-2,
           |lse_gpu - lse_oracle| <= 2e-3
"""
import math

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


def bf(a):
    return spot.to_device_bf16(a, DEV)


def t32(a, dtype):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV).to(dtype)


def i32(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(DEV)


def f32(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(DEV)


_cache = {}


def workload(i, **kw):
    key = (i, tuple(sorted(kw.items())))
    if key not in _cache:
        print(f"[gen] decode workload {i} {kw}", flush=True)
        _cache[key] = synth.decode_config(i, **kw)
    return _cache[key]


def quantized(wl, fmt):
    codes, scales = synth.QUANTIZERS[fmt](wl.k_sel)
    return codes, (scales.view(np.uint16) if fmt in ("int4", "int8") else scales)


def gpu_scores(wl, fmt="bf16"):
    if fmt == "bf16":
        k_sel, k_scale = bf(wl.k_sel), None
    else:
        c, s = quantized(wl, fmt)
        k_sel = torch.from_numpy(c).to(DEV)
        k_scale = (torch.from_numpy(s.view(np.int16)).to(DEV) if fmt in ("int4", "int8")
                   else torch.from_numpy(s).to(DEV))
    out = spot.selector_score(bf(wl.q_sel), f32(wl.w), k_sel, k_scale, fmt,
                              n_valid=i32(wl.n_valid), nblk=wl.nblk)
    torch.cuda.synchronize()
    return out.cpu().numpy()


def oracle_scores(wl, fmt="bf16"):
    if fmt == "bf16":
        return oracle.selector_score(wl.q_sel, wl.w, wl.k_sel, n_valid=wl.n_valid)
    c, s = quantized(wl, fmt)
    return oracle.selector_score(wl.q_sel, wl.w, c, s, fmt, n_valid=wl.n_valid, nblk=wl.nblk,
                                 h_s=wl.Hs, d_s=wl.ds)


def assert_scores_close(g, o):
    fin = np.isfinite(o)
    assert np.array_equal(np.isfinite(g), fin)
    assert np.all(g[~fin] == -np.inf)
    err = np.abs(g[fin] - o[fin])
    bound = 1e-4 * np.abs(o[fin]) + 1e-6
    assert np.all(err <= bound), f"max excess {np.max(err - bound)}"


def assert_out_close(out_g, lse_g, out_o, lse_o):
    g = out_g.float().cpu().numpy().astype(np.float64)
    diff = g - out_o
    max_abs = np.max(np.abs(diff))
    rel = np.linalg.norm(diff) / max(np.linalg.norm(out_o), 1e-30)
    assert max_abs <= 2e-2, max_abs
    assert rel <= 1e-2, rel
    lg = lse_g.cpu().numpy().astype(np.float64)
    fin = np.isfinite(lse_o)
    assert np.array_equal(np.isfinite(lg), fin)
    assert np.all(np.abs(lg[fin] - lse_o[fin]) <= 2e-3)


# ------------------------------------------------------------------ scoring
@pytest.mark.parametrize("cfg,fmt", [(1, "bf16"), (2, "bf16"), (3, "bf16"), (3, "int4"),
                                     (3, "mxfp4"), (1, "int4"), (1, "mxfp4"), (3, "int8"),
                                     (3, "mxfp8"), (1, "int8"), (1, "mxfp8")])
def test_selector_score_parity(cfg, fmt):
    wl = workload(cfg, backbone=False)
    assert_scores_close(gpu_scores(wl, fmt), oracle_scores(wl, fmt))


def test_selector_score_ragged():
    # ragged seq_len (n_valid not a multiple of the 32-block workgroup chunk)
    wl = workload(2, B=5, L=8192, seq_len=(8192, 5000, 64, 1, 4097), backbone=False)
    for fmt in ("bf16", "int4", "mxfp4", "int8", "mxfp8"):
        assert_scores_close(gpu_scores(wl, fmt), oracle_scores(wl, fmt))


def test_selector_score_prefill_rows():
    """rows_per_seq > 1: query-block x key-block scores with a causal n_valid."""
    wl = synth.prefill_config(L=4096, backbone=False)
    nqb = wl.nblk
    s_o = oracle.selector_score(wl.q_sel, wl.w, wl.k_sel, rows_per_seq=nqb, n_valid=wl.n_valid)
    s_g = spot.selector_score(bf(wl.q_sel), f32(wl.w), bf(wl.k_sel), rows_per_seq=nqb,
                              n_valid=i32(wl.n_valid), nblk=nqb)
    assert_scores_close(s_g.cpu().numpy(), s_o)


@pytest.mark.parametrize("B,nqb,Hs,ds", [(2, 48, 8, 64), (3, 32, 4, 128), (1, 20, 8, 64)])
def test_selector_score_prefill_tiles(B, nqb, Hs, ds):
    """Query-block x key-block scores on the matrix cores (rows_per_seq a
    multiple of 16) and on the row kernel otherwise: several sequences,
    a block count that is not a multiple of the 32-block workgroup tile,
    both head splits of the 512-wide pooled key, a causal n_valid."""
    rng = np.random.default_rng([B, nqb, Hs, ds])
    q_sel, w, k_sel = synth.selector_prefill(rng, B, nqb, nqb, Hs, ds)
    q_sel = q_sel.reshape(B * nqb, Hs, ds)
    w = w.reshape(B * nqb, Hs)
    n_valid = np.tile(np.arange(1, nqb + 1, dtype=np.int32), B)
    s_o = oracle.selector_score(q_sel, w, k_sel, rows_per_seq=nqb, n_valid=n_valid)
    s_g = spot.selector_score(bf(q_sel), f32(w), bf(k_sel), rows_per_seq=nqb,
                              n_valid=i32(n_valid), nblk=nqb)
    assert_scores_close(s_g.cpu().numpy(), s_o)


# ---------------------------------------------------------------- selection
SELECT_CASES = [
    # rows, nblk, rule, n_valid spec
    (64, 64, Rule(0.9, 16, 0, 1, 2), None),
    (16, 512, Rule(0.9, 64, 0, 1, 2), "ragged"),
    (8, 2048, Rule(0.95, 128, 0, 1, 2), None),
    (8, 2048, Rule(0.5, 128, 40, 1, 2), None),
    (8, 1000, Rule(1.0, 300, 0, 0, 0), None),           # static top-K
    (8, 300, Rule(0.0, 32, 0, 2, 3), "ragged"),          # p = 0: reserved only
    (8, 100, Rule(0.9, 200, 0, 1, 2), None),            # k_max > nblk
    (16, 5, Rule(0.7, 4, 0, 1, 2), "tiny"),              # nblk <= sink + recent
    (4, 16384, Rule(0.99, 4096, 0, 4, 4), None),         # largest supported sizes
    (8, 2048, Rule(1.0, 1536, 0, 1, 2), None),          # static top-K, cap above 512
    (8, 4096, Rule(1.0, 3000, 0, 0, 0), "ragged"),      # static top-K, cap above 2048
    (8, 2048, Rule(0.999, 1000, 0, 1, 2), None),        # nucleus under a 1000-block cap
    (4, 2048, Rule(0.0, 900, 600, 1, 2), None),         # k_min floor of 600 blocks
    # long rows, small caps: the cut inside at most 64 survivors is ranked by
    # counting, above 64 by the sort
    (8, 2048, Rule(0.9, 64, 0, 1, 2), None),            # cap 61
    (8, 1024, Rule(0.5, 67, 0, 1, 2), "ragged"),        # cap 64: the last counted
    (8, 1024, Rule(0.5, 68, 0, 1, 2), "ragged"),        # cap 65: the first sorted
    (8, 2048, Rule(0.3, 40, 30, 1, 2), None),           # k_min floor under a cap of 37
    (8, 600, Rule(0.2, 20, 0, 2, 3), None),             # short nucleus, cap 15
    # rows of 16-token blocks (128K tokens: 8192 blocks) on the workgroup kernel
    (4, 8192, Rule(0.95, 512, 0, 4, 8), None),          # the paper's block, 8192-token budget
    (8, 8192, Rule(0.9, 64, 0, 4, 8), "ragged"),        # counted cut
    (4, 8192, Rule(1.0, 2048, 0, 0, 0), None),          # static top-K
    (4, 6000, Rule(0.5, 1000, 0, 1, 2), "ragged"),      # 1000-block cap
]


@pytest.mark.parametrize("case", range(len(SELECT_CASES)))
def test_select_parity_same_scores(case):
    rows, nblk, rule, nv_spec = SELECT_CASES[case]
    rng = np.random.default_rng(case)
    if nv_spec == "ragged":
        nv = rng.integers(0, nblk + 1, rows).astype(np.int32)
        nv[0] = nblk
    elif nv_spec == "tiny":
        nv = rng.integers(0, nblk + 1, rows).astype(np.int32)
    else:
        nv = np.full(rows, nblk, np.int32)
    s = synth.random_scores(100 + case, rows, nblk, nv)
    idx_o, cnt_o, mass_o = oracle.select_blocks(s.astype(np.float64), rule, nv)
    idx_g, cnt_g, mass_g = spot.select_blocks(f32(s), rule, i32(nv))
    torch.cuda.synchronize()
    idx_g, cnt_g = idx_g.cpu().numpy(), cnt_g.cpu().numpy()
    # Same FP32 scores on both sides: the order is identical, only a row whose
    # cumulative mass sits within 1e-5 of p may legitimately differ.
    stats = check_all(s, nv, rule, idx_o, cnt_o, idx_g, cnt_g, rel_tie=0.0)
    assert stats["tie"] == 0
    assert stats["mass"] <= max(1, rows // 50), stats
    exact = cnt_g == cnt_o
    np.testing.assert_allclose(mass_g.cpu().numpy()[exact], mass_o[exact], atol=2e-5)


@pytest.mark.parametrize("rule", [Rule(0.9, 100, 0, 1, 2), Rule(0.02, 40, 0, 1, 2)])
def test_select_deterministic_and_ties(rule):
    """Exact ties break toward the lower block id; repeated runs are bitwise
    equal (a cap of 97 that binds; a cut inside 37 tied survivors)."""
    rows, nblk = 32, 2048
    s = np.zeros((rows, nblk), np.float32)
    s[:, ::7] = 1.0                       # many exactly equal maxima
    idx_o, cnt_o, _ = oracle.select_blocks(s.astype(np.float64), rule)
    a = spot.select_blocks(f32(s), rule)
    b = spot.select_blocks(f32(s), rule)
    torch.cuda.synchronize()
    for x, y in zip(a, b):
        assert torch.equal(x, y)
    np.testing.assert_array_equal(a[0].cpu().numpy(), idx_o)
    np.testing.assert_array_equal(a[1].cpu().numpy(), cnt_o)


@pytest.mark.parametrize("nblk,k_max", [(300, 100), (2048, 100), (2048, 40), (2048, 1500),
                                        (8192, 700), (16384, 700)])
def test_select_negative_zero_ties_positive_zero(nblk, k_max):
    """-0.0 and +0.0 are the same score: a cut through a run of zeros of
    both signs takes the lower ids, whatever their sign (every selection
    kernel: one wave, one workgroup, the sort-based kernel)."""
    rng = np.random.default_rng(nblk + k_max)
    rows = 8
    s = np.where(rng.random((rows, nblk)) < 0.5, np.float32(0.0), np.float32(-0.0))
    s[:, rng.choice(nblk, size=k_max // 3, replace=False)] = 1.0   # the cut falls in the zeros
    s = s.astype(np.float32)
    for rule in (Rule(1.0, k_max, 0, 1, 2), Rule(0.5, k_max, 0, 1, 2)):
        idx_o, cnt_o, _ = oracle.select_blocks(s.astype(np.float64), rule)
        idx_g, cnt_g, _ = spot.select_blocks(f32(s), rule)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(cnt_g.cpu().numpy(), cnt_o)
        np.testing.assert_array_equal(idx_g.cpu().numpy(), idx_o)


@pytest.mark.parametrize("cfg,fmt", [(1, "bf16"), (2, "bf16"), (3, "bf16"), (3, "int4"),
                                     (3, "mxfp4"), (3, "int8"), (3, "mxfp8")])
def test_score_and_select_end_to_end(cfg, fmt):
    """GPU scores -> GPU selection vs oracle scores -> oracle selection."""
    wl = workload(cfg, backbone=False)
    s_o = oracle_scores(wl, fmt).astype(np.float32)
    idx_o, cnt_o, _ = oracle.select_blocks(s_o.astype(np.float64), wl.rule, wl.n_valid)
    s_g = torch.from_numpy(gpu_scores(wl, fmt)).to(DEV)
    idx_g, cnt_g, _ = spot.select_blocks(s_g, wl.rule, i32(wl.n_valid))
    torch.cuda.synchronize()
    stats = check_all(s_o, wl.n_valid, wl.rule, idx_o, cnt_o, idx_g.cpu().numpy(),
                      cnt_g.cpu().numpy())
    print(f"[select] cfg {cfg} {fmt}: {stats}")


# ---------------------------------------------------------------- attention
def oracle_selection(wl):
    s = oracle.selector_score(wl.q_sel, wl.w, wl.k_sel, n_valid=wl.n_valid).astype(np.float32)
    return oracle.select_blocks(s.astype(np.float64), wl.rule, wl.n_valid)


@pytest.mark.parametrize("cfg", [1, 2, 3])
def test_sparse_decode_parity(cfg):
    wl = workload(cfg)
    idx, cnt, _ = oracle_selection(wl)
    out_o, lse_o = oracle.sparse_decode(wl.q, wl.k, wl.v, wl.seq_len, idx, cnt, wl.sm_scale)
    out_g, lse_g = spot.sparse_decode(bf(wl.q), bf(wl.k), bf(wl.v), i32(wl.seq_len), i32(idx),
                                      i32(cnt), wl.sm_scale)
    torch.cuda.synchronize()
    assert_out_close(out_g, lse_g, out_o, lse_o)


def test_sparse_decode_ragged_and_bad_ids():
    """Partial last blocks, unsorted ids, ids past seq_len and negative ids."""
    B, L = 4, 2048
    wl = workload(2, B=B, L=L, seq_len=(2048, 1000, 65, 1))
    rng = np.random.default_rng(3)
    k_max = 12
    idx = np.full((B, k_max), -1, np.int32)
    cnt = np.zeros(B, np.int32)
    for b in range(B):
        nv = int(wl.n_valid[b])
        ids = rng.permutation(nv)[: min(nv, 9)]
        extra = [-5, nv + 3] if b % 2 else []
        row = list(ids) + extra
        idx[b, :len(row)] = row
        cnt[b] = len(row)
    out_o, lse_o = oracle.sparse_decode(wl.q, wl.k, wl.v, wl.seq_len, idx, cnt, wl.sm_scale)
    out_g, lse_g = spot.sparse_decode(bf(wl.q), bf(wl.k), bf(wl.v), i32(wl.seq_len), i32(idx),
                                      i32(cnt), wl.sm_scale)
    torch.cuda.synchronize()
    assert_out_close(out_g, lse_g, out_o, lse_o)
    # An empty set gives zeros and lse = -inf.
    cnt0 = np.zeros(B, np.int32)
    out_g, lse_g = spot.sparse_decode(bf(wl.q), bf(wl.k), bf(wl.v), i32(wl.seq_len), i32(idx),
                                      i32(cnt0), wl.sm_scale)
    torch.cuda.synchronize()
    assert torch.all(out_g.float() == 0) and torch.all(torch.isinf(lse_g))


@pytest.mark.parametrize("Hq,Hkv", [(6, 2), (10, 2), (24, 4), (32, 2), (48, 4)])
def test_sparse_decode_group_sizes(Hq, Hkv):
    """Groups other than 1, 2, 4, 8 query heads per KV head (3, 5, 6, 16, 12):
    the group's heads are the columns of the 16-wide matrix tiles."""
    B, L, d = 3, 4096, 128
    print(f"[decode] Hq={Hq} Hkv={Hkv}", flush=True)
    q, k, v = synth._backbone_decode(960 + Hq, B, L, Hq, Hkv, d)
    seq_len = np.array([4096, 2500, 65], np.int32)
    rng = np.random.default_rng(Hq)
    k_max = 40
    idx = np.full((B, k_max), -1, np.int32)
    cnt = np.zeros(B, np.int32)
    for b in range(B):
        nv = int((seq_len[b] + 63) // 64)
        row = rng.permutation(nv)[: min(nv, 37)]
        idx[b, :len(row)] = row
        cnt[b] = len(row)
    scale = 1 / np.sqrt(d)
    out_o, lse_o = oracle.sparse_decode(q, k, v, seq_len, idx, cnt, scale)
    out_g, lse_g = spot.sparse_decode(bf(q), bf(k), bf(v), i32(seq_len), i32(idx), i32(cnt),
                                      scale)
    torch.cuda.synchronize()
    assert_out_close(out_g, lse_g, out_o, lse_o)
    out_o, lse_o = oracle.dense_decode(q, k, v, seq_len, scale)
    out_g, lse_g = spot.dense_decode(bf(q), bf(k), bf(v), i32(seq_len), scale)
    torch.cuda.synchronize()
    assert_out_close(out_g, lse_g, out_o, lse_o)


@pytest.mark.parametrize("cfg,B,L", [(1, None, None), (2, 2, 8192), (2, 3, 4160)])
def test_dense_decode_parity(cfg, B, L):
    kw = {} if B is None else {"B": B, "L": L, "seq_len": tuple([L, L - 37, 64][:B])}
    wl = workload(cfg, **kw)
    out_o, lse_o = oracle.dense_decode(wl.q, wl.k, wl.v, wl.seq_len, wl.sm_scale)
    out_g, lse_g = spot.dense_decode(bf(wl.q), bf(wl.k), bf(wl.v), i32(wl.seq_len), wl.sm_scale)
    torch.cuda.synchronize()
    assert_out_close(out_g, lse_g, out_o, lse_o)


def test_dense_decode_full_size_sampled():
    """128K-token dense decode: every output of two sequences vs the oracle."""
    wl = workload(3)
    out_g, lse_g = spot.dense_decode(bf(wl.q), bf(wl.k), bf(wl.v), i32(wl.seq_len), wl.sm_scale)
    torch.cuda.synchronize()
    pick = [0, 3]
    out_o, lse_o = oracle.dense_decode(wl.q[pick], wl.k[pick], wl.v[pick], wl.seq_len[pick],
                                       wl.sm_scale)
    assert_out_close(out_g[pick], lse_g[pick], out_o, lse_o)


def test_sparse_equals_dense_when_all_selected():
    wl = workload(2, B=2, L=4096)
    nb = wl.nblk
    idx = np.tile(np.arange(nb, dtype=np.int32), (2, 1))
    cnt = np.full(2, nb, np.int32)
    a, la = spot.sparse_decode(bf(wl.q), bf(wl.k), bf(wl.v), i32(wl.seq_len), i32(idx), i32(cnt),
                               wl.sm_scale)
    b, lb = spot.dense_decode(bf(wl.q), bf(wl.k), bf(wl.v), i32(wl.seq_len), wl.sm_scale)
    torch.cuda.synchronize()
    assert torch.max(torch.abs(a.float() - b.float())).item() <= 1e-2
    assert torch.max(torch.abs(la - lb)).item() <= 1e-4


def test_full_step_deterministic():
    """Scores, selection and attention outputs are bitwise repeatable."""
    wl = workload(3)
    q_sel, w, k_sel, nv = bf(wl.q_sel), f32(wl.w), bf(wl.k_sel), i32(wl.n_valid)
    q, k, v, sl = bf(wl.q), bf(wl.k), bf(wl.v), i32(wl.seq_len)
    res = []
    for _ in range(3):
        s = spot.selector_score(q_sel, w, k_sel, n_valid=nv, nblk=wl.nblk)
        idx, cnt, mass = spot.select_blocks(s, wl.rule, nv)
        out, lse = spot.sparse_decode(q, k, v, sl, idx, cnt, wl.sm_scale)
        res.append((s, idx, cnt, mass, out, lse))
    torch.cuda.synchronize()
    for r in res[1:]:
        for x, y in zip(res[0], r):
            assert torch.equal(x, y)


def test_error_paths_leave_outputs_untouched():
    wl = workload(1)
    out = torch.full((1, 32, 128), 7.0, dtype=torch.bfloat16, device=DEV)
    lse = torch.full((1, 32), 7.0, device=DEV)
    ws = spot.decode_workspace(1, 32, 8, 128, 16, DEV)
    idx = i32(np.zeros((1, 16)))
    with pytest.raises(spot.SpotError) as e:
        spot.spot_sparse_decode(bf(wl.q), bf(wl.k), bf(wl.v), i32(wl.seq_len), idx,
                                i32(np.ones(1)), 16, 1, 32, 8, 128, 4000, 0.1, out, lse, ws)
    assert e.value.status == 2
    with pytest.raises(spot.SpotError) as e:
        spot.spot_sparse_decode(bf(wl.q), bf(wl.k), bf(wl.v), i32(wl.seq_len), idx,
                                i32(np.ones(1)), 16, 1, 32, 8, 128, 4096, 0.1, out, lse, ws[:8])
    assert e.value.status == 5
    scores = torch.full((1, 64), 3.0, device=DEV)
    cnt = torch.full((1,), 99, dtype=torch.int32, device=DEV)
    with pytest.raises(spot.SpotError) as e:
        spot.spot_select_blocks(scores, 1, 64, None, float("nan"), 16, 0, 1, 2, idx, cnt)
    assert e.value.status == 4
    torch.cuda.synchronize()
    assert torch.all(out.float() == 7.0) and torch.all(lse == 7.0)
    assert torch.all(idx == 0) and int(cnt.item()) == 99


# ------------------------------------------------------- quantized queries
def _dev_scale(s, fmt):
    return torch.from_numpy(np.ascontiguousarray(
        s.view(np.uint16).view(np.int16) if fmt in ("int4", "int8") else s)).to(DEV)


@pytest.mark.parametrize("B,nqb,Hs,ds,qfmt,kfmt", [
    (2, 48, 4, 128, "mxfp4", "mxfp4"),     # block-scaled matrix cores
    (1, 64, 4, 128, "mxfp8", "mxfp8"),     # block-scaled matrix cores
    (2, 20, 4, 128, "mxfp4", "mxfp4"),     # 20 rows per sequence: row kernel
    (2, 32, 8, 64, "mxfp8", "mxfp8"),      # d_s = 64: row kernel
    (2, 32, 4, 128, "mxfp4", "bf16"),
    (2, 32, 8, 64, "mxfp8", "int4"),
    (1, 16, 4, 128, "mxfp4", "int8"),
    (1, 16, 8, 64, "mxfp8", "mxfp4"),
    (2, 32, 8, 64, "int4", "int4"),       # integer queries: row kernel, any key format
    (2, 32, 4, 128, "int8", "int8"),
    (2, 20, 8, 64, "int8", "bf16"),
    (1, 16, 4, 128, "int4", "bf16"),
    (2, 32, 8, 64, "int4", "mxfp4"),
    (1, 16, 4, 128, "int8", "mxfp8"),
    (1, 16, 8, 64, "int8", "int4"),
])
def test_selector_score_quantized_queries(B, nqb, Hs, ds, qfmt, kfmt):
    """Query-block x key-block scores with coded queries (MX or integer),
    against the oracle decoding the same codes (causal n_valid, several
    sequences)."""
    print(f"[qscore] B={B} nqb={nqb} {Hs}x{ds} q={qfmt} k={kfmt}", flush=True)
    rng = np.random.default_rng([B, nqb, Hs, ds])
    q_sel, w, k_sel = synth.selector_prefill(rng, B, nqb, nqb, Hs, ds)
    q_sel = q_sel.reshape(B * nqb, Hs, ds)
    w = w.reshape(B * nqb, Hs)
    n_valid = np.tile(np.arange(1, nqb + 1, dtype=np.int32), B)
    qc, qs = synth.QUANTIZERS[qfmt](q_sel)
    if kfmt == "bf16":
        kc, ks = k_sel, None
        kd, ksd = bf(k_sel), None
    else:
        kc, ks = synth.QUANTIZERS[kfmt](k_sel)
        kd, ksd = torch.from_numpy(kc).to(DEV), _dev_scale(ks, kfmt)
    s_o = oracle.selector_score_qk(qc, qs, qfmt, w, kc, ks, kfmt, B * nqb, nqb, Hs, ds,
                                   rows_per_seq=nqb, n_valid=n_valid)
    out = torch.empty((B * nqb, nqb), dtype=torch.float32, device=DEV)
    spot.spot_selector_score_q(torch.from_numpy(qc).to(DEV), _dev_scale(qs, qfmt), qfmt,
                               f32(w), kd, ksd, kfmt, B, nqb, nqb, Hs, ds, i32(n_valid), out)
    torch.cuda.synchronize()
    assert_scores_close(out.cpu().numpy(), s_o)


@pytest.mark.parametrize("qfmt", ["mxfp4", "mxfp8", "int4", "int8"])
def test_decode_scores_quantized_queries(qfmt):
    """Decode rows (one query per sequence) with coded queries and the
    128K-token workload's BF16 pooled keys."""
    wl = workload(3, backbone=False)
    qc, qs = synth.QUANTIZERS[qfmt](wl.q_sel)
    s_o = oracle.selector_score_qk(qc, qs, qfmt, wl.w, wl.k_sel, None, "bf16", wl.B, wl.nblk,
                                   wl.Hs, wl.ds, n_valid=wl.n_valid)
    out = torch.empty((wl.B, wl.nblk), dtype=torch.float32, device=DEV)
    spot.spot_selector_score_q(torch.from_numpy(qc).to(DEV), _dev_scale(qs, qfmt), qfmt,
                               f32(wl.w), bf(wl.k_sel), None, "bf16", wl.B, 1, wl.nblk, wl.Hs,
                               wl.ds, i32(wl.n_valid), out)
    torch.cuda.synchronize()
    assert_scores_close(out.cpu().numpy(), s_o)
