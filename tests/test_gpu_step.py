"""The fused decode step (spot_decode_step) against the three separate calls
and against the FP64 oracle (needs an MI355X).

The fused launch runs the same scoring, selection and attention cores as the
separate kernels, so scores and block sets must match them exactly; the
attention outputs must match to the decode tolerances (they are bitwise equal
whenever both paths split the attention the same way).  End to end, the block
sets are checked against the oracle's with the near-tie / mass-boundary
exemptions of selcheck, and the outputs against the oracle run on the fused
path's own block sets.
"""
import copy

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


def selector(wl, fmt):
    if fmt == "bf16":
        return bf(wl.k_sel), None
    c, s = synth.QUANTIZERS[fmt](wl.k_sel)
    if fmt in ("int4", "int8"):
        s = s.view(np.uint16).view(np.int16)
    return torch.from_numpy(c).to(DEV), torch.from_numpy(s).to(DEV)


def inputs(wl, fmt):
    k_sel, k_scale = selector(wl, fmt)
    return dict(q_sel=bf(wl.q_sel), w=f32(wl.w), k_sel=k_sel, k_scale=k_scale, kfmt=fmt,
                q=bf(wl.q), k=bf(wl.k), v=bf(wl.v), seq_len=i32(wl.seq_len),
                n_valid=i32(wl.n_valid))


def separate(x, wl):
    s = spot.selector_score(x["q_sel"], x["w"], x["k_sel"], x["k_scale"], x["kfmt"],
                            n_valid=x["n_valid"], nblk=wl.nblk)
    idx, cnt, mass = spot.select_blocks(s, wl.rule, x["n_valid"])
    out, lse = spot.sparse_decode(x["q"], x["k"], x["v"], x["seq_len"], idx, cnt, wl.sm_scale)
    return s, idx, cnt, mass, out, lse


def fused(x, wl, ws=None):
    return spot.decode_step(x["q_sel"], x["w"], x["k_sel"], x["q"], x["k"], x["v"],
                            x["seq_len"], wl.rule, k_scale=x["k_scale"], kfmt=x["kfmt"],
                            n_valid=x["n_valid"], sm_scale=wl.sm_scale, ws=ws)


def assert_same(sep, fus, bitwise=False):
    """Scores and block sets equal; with bitwise=True (same selection kernel
    and the same attention split on both paths) every output bit for bit."""
    s0, i0, c0, m0, o0, l0 = sep
    s1, i1, c1, m1, o1, l1 = fus
    assert torch.equal(s0, s1), "scores differ"
    assert torch.equal(c0, c1), "counts differ"
    assert torch.equal(i0, i1), "block sets differ"
    if bitwise:
        assert torch.equal(m0, m1), "nucleus mass differs"
        assert torch.equal(o0, o1), "outputs differ"
        assert torch.equal(l0, l1), "lse differs"
        return
    assert torch.allclose(m0, m1, rtol=1e-5, atol=1e-7), "nucleus mass differs"
    assert torch.max(torch.abs(o0.float() - o1.float())).item() <= 1e-2
    assert torch.max(torch.abs(l0 - l1)).item() <= 1e-4


@pytest.mark.parametrize("cfg,fmt", [(1, "bf16"), (2, "bf16"), (3, "bf16"), (3, "int4"),
                                     (3, "mxfp4"), (3, "int8"), (3, "mxfp8")])
def test_step_matches_separate_calls(cfg, fmt):
    wl = workload(cfg)
    x = inputs(wl, fmt)
    print(f"[step] cfg {cfg} {fmt}", flush=True)
    sep = separate(x, wl)
    fus = fused(x, wl)
    torch.cuda.synchronize()
    # 2048 blocks: both paths select with the workgroup core and split the
    # attention 16 ways, so every output matches bit for bit.
    assert_same(sep, fus, bitwise=(cfg == 3))


@pytest.mark.parametrize("fmt", ["int4", "int8", "mxfp4", "mxfp8"])
@pytest.mark.parametrize("cfg", [3, 1])
def test_step_quantized_queries(fmt, cfg):
    """spot_decode_step_q: queries and the selector key cache in one quantized
    format (the 128K-token workload; and 4K tokens, batch 1, on the short-row
    kernel).  The fused launch equals the separate calls
    (spot_selector_score_q, selection, decode) bit for bit (at 4K tokens the
    nucleus mass to FP32 rounding: the separate selection of short rows is
    the one-wave kernel), and its scores and selection match the oracle on
    the same codes."""
    wl = workload(cfg)
    x = inputs(wl, fmt)
    qc, qs = synth.QUANTIZERS[fmt](wl.q_sel)
    qs_dev = qs.view(np.uint16).view(np.int16) if fmt in ("int4", "int8") else qs
    q_codes = torch.from_numpy(np.ascontiguousarray(qc)).to(DEV)
    q_scale = torch.from_numpy(np.ascontiguousarray(qs_dev)).to(DEV)
    print(f"[step] quantized queries {fmt}", flush=True)
    s0 = torch.empty((wl.B, wl.nblk), dtype=torch.float32, device=DEV)
    spot.spot_selector_score_q(q_codes, q_scale, fmt, x["w"], x["k_sel"], x["k_scale"], fmt,
                               wl.B, 1, wl.nblk, wl.Hs, wl.ds, x["n_valid"], s0)
    i0, c0, m0 = spot.select_blocks(s0, wl.rule, x["n_valid"])
    o0, l0 = spot.sparse_decode(x["q"], x["k"], x["v"], x["seq_len"], i0, c0, wl.sm_scale)
    fus = spot.decode_step(q_codes, x["w"], x["k_sel"], x["q"], x["k"], x["v"], x["seq_len"],
                           wl.rule, k_scale=x["k_scale"], kfmt=fmt, n_valid=x["n_valid"],
                           sm_scale=wl.sm_scale, q_scale=q_scale, qfmt=fmt)
    torch.cuda.synchronize()
    assert_same((s0, i0, c0, m0, o0, l0), fus, bitwise=(cfg == 3))
    assert torch.equal(o0, fus[4]) and torch.equal(l0, fus[5])
    kc, ks = synth.QUANTIZERS[fmt](wl.k_sel)
    s_o = oracle.selector_score_qk(qc, qs, fmt, wl.w, kc, ks, fmt, wl.B, wl.nblk, wl.Hs, wl.ds,
                                   n_valid=wl.n_valid)
    s = fus[0].cpu().numpy()
    fin = np.isfinite(s_o)
    assert np.array_equal(np.isfinite(s), fin)
    assert np.all(np.abs(s[fin] - s_o[fin]) <= 1e-4 * np.abs(s_o[fin]) + 1e-6)
    idx_o, cnt_o, _ = oracle.select_blocks(s_o.astype(np.float32).astype(np.float64), wl.rule,
                                           wl.n_valid)
    print("[step] selection vs oracle:",
          check_all(s_o.astype(np.float32), wl.n_valid, wl.rule, idx_o, cnt_o,
                    fus[1].cpu().numpy(), fus[2].cpu().numpy()))


def test_step_end_to_end_vs_oracle():
    wl = workload(3)
    x = inputs(wl, "bf16")
    s, idx, cnt, mass, out, lse = fused(x, wl)
    torch.cuda.synchronize()
    s_o = oracle.selector_score(wl.q_sel, wl.w, wl.k_sel, n_valid=wl.n_valid)
    err = np.abs(s.cpu().numpy() - s_o)
    fin = np.isfinite(s_o)
    assert np.all(err[fin] <= 1e-4 * np.abs(s_o[fin]) + 1e-6)
    idx_o, cnt_o, _ = oracle.select_blocks(s_o.astype(np.float32).astype(np.float64), wl.rule,
                                           wl.n_valid)
    idx_g, cnt_g = idx.cpu().numpy(), cnt.cpu().numpy()
    print("[step] selection vs oracle:",
          check_all(s_o.astype(np.float32), wl.n_valid, wl.rule, idx_o, cnt_o, idx_g, cnt_g))
    out_o, lse_o = oracle.sparse_decode(wl.q, wl.k, wl.v, wl.seq_len, idx_g, cnt_g, wl.sm_scale)
    g = out.float().cpu().numpy().astype(np.float64)
    assert np.max(np.abs(g - out_o)) <= 2e-2
    assert np.linalg.norm(g - out_o) / np.linalg.norm(out_o) <= 1e-2
    assert np.max(np.abs(lse.cpu().numpy() - lse_o)) <= 2e-3


@pytest.mark.parametrize("frac", [0.25, 0.5, 0.75])
def test_static_topk_large_budgets(frac):
    """Static top-K (Eq. select-topk: p >= 1 keeps every block, no reserved
    blocks, the cap K_max = K picks the top K) at a quarter, half and three
    quarters of the 2048 blocks of the 128K-token workload.  K = 512 runs in
    the fused launch, 1024 and 1536 as three stages.  The sets must equal the
    oracle's top-K of the same FP32 scores (unique: ties go to the lower id);
    the outputs are checked against the oracle on two sequences."""
    wl = copy.copy(workload(3))
    K = int(frac * wl.nblk)
    wl.rule = Rule(1.0, K, 0, 0, 0)
    print(f"[step] static top-K K={K}", flush=True)
    x = inputs(wl, "bf16")
    s, idx, cnt, mass, out, lse = fused(x, wl)
    torch.cuda.synchronize()
    s_g = s.cpu().numpy().astype(np.float64)
    idx_o, cnt_o, _ = oracle.select_blocks(s_g, wl.rule, wl.n_valid)
    idx_g, cnt_g = idx.cpu().numpy(), cnt.cpu().numpy()
    assert np.all(cnt_g == K)
    np.testing.assert_array_equal(cnt_g, cnt_o)
    np.testing.assert_array_equal(idx_g, idx_o)
    pick = [0, 3]
    out_o, lse_o = oracle.sparse_decode(wl.q[pick], wl.k[pick], wl.v[pick], wl.seq_len[pick],
                                        idx_g[pick], cnt_g[pick], wl.sm_scale)
    g = out.float().cpu().numpy().astype(np.float64)[pick]
    assert np.max(np.abs(g - out_o)) <= 2e-2
    assert np.linalg.norm(g - out_o) / np.linalg.norm(out_o) <= 1e-2
    assert np.max(np.abs(lse.cpu().numpy()[pick] - lse_o)) <= 2e-3


def test_step_repeated_calls_reset_workspace():
    """Back-to-back steps on one workspace: every call right, counters zero after."""
    wl = workload(3)
    x = inputs(wl, "bf16")
    ws = spot.step_workspace(wl.B, wl.Hq, wl.Hkv, wl.d, wl.rule.k_max, DEV)
    qs = [x["q"], x["q"].flip(-1).contiguous(), (x["q"].float() * 0.5).to(torch.bfloat16)]
    results = []
    for qv in qs:
        y = dict(x, q=qv)
        results.append((separate(y, wl), fused(y, wl, ws)))
    torch.cuda.synchronize()
    for sep, fus in results:
        assert_same(sep, fus)
    # The control region at the start of the workspace (completion counters,
    # expiry word, score records, bitmap copies) is back to zero; the
    # partials (16 splits per head here) follow it.
    n_bytes = spot.spot_decode_step_workspace_bytes(wl.B, wl.Hq, wl.Hkv, wl.d, wl.rule.k_max)
    ctrl = (wl.B * wl.Hkv * 4 + 15) // 16 * 16 + 16 + wl.B * 4096 * 4 + wl.B * wl.Hkv * 256 * 4
    ctrl = (ctrl + 255) // 256 * 256
    assert n_bytes == ctrl + wl.B * wl.Hq * 16 * 130 * 4
    assert int(torch.count_nonzero(ws[:ctrl]).item()) == 0
    assert spot.spot_decode_step_status(ws, wl.B, wl.Hq, wl.Hkv, wl.d, wl.rule.k_max) == 0


@pytest.mark.parametrize("cfg", [3, 1])
def test_step_expired_wait_is_reported(cfg):
    """A fused step whose waits expire (forced from the host: every
    workgroup's wait for its sequence's scores gives up at once, so every
    kernel still exits normally) attends to nothing, reports count = -1 and
    sets the workspace's expiry word; later calls on that workspace do the
    same without waiting until spot_decode_step_status reports the expiry and
    restores the workspace, after which a call equals the three separate
    calls bit for bit.  Workload 1 (64 blocks per row) runs the short-row
    kernel, which waits for nothing but honours the forced expiry and the
    expiry word the same way."""
    wl = workload(cfg)
    x = inputs(wl, "bf16")
    args = (wl.B, wl.Hq, wl.Hkv, wl.d, wl.rule.k_max)
    ws = spot.step_workspace(*args, DEV)
    sep = separate(x, wl)
    print("[step] forced expiry", flush=True)
    spot.spot_test_force_expiry(True)
    try:
        s1, _, c1, _, o1, l1 = fused(x, wl, ws)
        torch.cuda.synchronize()
    finally:
        spot.spot_test_force_expiry(False)
    assert torch.equal(s1, sep[0])                    # scoring never waits
    assert torch.all(c1 == -1)
    assert torch.all(o1.float() == 0) and torch.all(torch.isinf(l1))
    # the word is sticky: a normal call on the same workspace does not wait
    print("[step] call after the expiry", flush=True)
    _, _, c2, _, o2, _ = fused(x, wl, ws)
    torch.cuda.synchronize()
    assert torch.all(c2 == -1) and torch.all(o2.float() == 0)
    assert spot.spot_decode_step_status(ws, *args) == spot.SPOT_ERR_EXPIRED
    assert int(torch.count_nonzero(ws).item()) == 0   # zero-filled again
    assert spot.spot_decode_step_status(ws, *args) == 0
    print("[step] normal call after the reset", flush=True)
    fus = fused(x, wl, ws)
    torch.cuda.synchronize()
    assert_same(sep, fus, bitwise=(cfg == 3))


SHORT_ROWS = [
    dict(i=1),                                            # 4096 tokens, batch 1: 64 blocks
    dict(i=2, B=3, L=8192, seq_len=(8192, 100, 4097)),    # 128 blocks, ragged
    dict(i=2, B=2, L=2048, seq_len=(2048, 1)),            # 32 blocks, fewer than k_max
    dict(i=2, B=2, L=6400, seq_len=(6400, 3001)),         # 100 blocks: a partial scoring run
]


@pytest.mark.parametrize("case", range(len(SHORT_ROWS)))
@pytest.mark.parametrize("fmt", ["bf16", "int4", "mxfp8"])
def test_step_short_rows(case, fmt):
    """Rows of at most 128 blocks take the short-row kernel: every workgroup
    of a sequence scores and selects the sequence itself.  Scores, block sets
    and counts equal the separate calls bit for bit (the same scoring code;
    the selection rule decides the same set), the outputs too where both
    paths split the attention alike (batch 1), the nucleus mass to FP32
    rounding; and the outputs match the oracle's attention on that set."""
    kw = dict(SHORT_ROWS[case])
    wl = workload(kw.pop("i"), **kw)
    assert wl.nblk <= 128
    x = inputs(wl, fmt)
    print(f"[step] short rows {SHORT_ROWS[case]} {fmt}", flush=True)
    sep = separate(x, wl)
    fus = fused(x, wl)
    torch.cuda.synchronize()
    assert_same(sep, fus)
    if wl.B == 1:
        assert torch.equal(sep[4], fus[4]) and torch.equal(sep[5], fus[5])
    idx, cnt = fus[1].cpu().numpy(), fus[2].cpu().numpy()
    out_o, lse_o = oracle.sparse_decode(wl.q, wl.k, wl.v, wl.seq_len, idx, cnt, wl.sm_scale)
    g = fus[4].float().cpu().numpy().astype(np.float64)
    assert np.max(np.abs(g - out_o)) <= 2e-2
    assert np.linalg.norm(g - out_o) / max(np.linalg.norm(out_o), 1e-30) <= 1e-2


def test_step_ragged_sequences():
    wl = workload(2, B=5, L=8192, seq_len=(8192, 5000, 64, 1, 4097))
    x = inputs(wl, "bf16")
    sep = separate(x, wl)
    fus = fused(x, wl)
    torch.cuda.synchronize()
    assert_same(sep, fus)


@pytest.mark.parametrize("G", [1, 2, 5, 8, 16])
def test_step_group_sizes(G):
    """spot_decode_step at other GQA group sizes (G query heads per KV head,
    up to the 16 columns of a matrix tile): G = 8 (64 / 8 heads) runs fused,
    the others as three launches; the separate calls' results, and the
    attention outputs against the oracle on the selected set."""
    wl = workload(2, B=2, L=8192, seq_len=(8192, 5001))
    x = inputs(wl, "bf16")
    q = synth.normal_bf16(70 + G, 1, (wl.B, 8 * G, wl.d))
    xg = dict(x, q=bf(q))
    print(f"[step] group {G}", flush=True)
    sep = separate(xg, wl)
    fus = fused(xg, wl)
    torch.cuda.synchronize()
    assert_same(sep, fus)
    idx, cnt = fus[1].cpu().numpy(), fus[2].cpu().numpy()
    out_o, lse_o = oracle.sparse_decode(q, wl.k, wl.v, wl.seq_len, idx, cnt, wl.sm_scale)
    g = fus[4].float().cpu().numpy().astype(np.float64)
    assert np.max(np.abs(g - out_o)) <= 2e-2
    assert np.linalg.norm(g - out_o) / np.linalg.norm(out_o) <= 1e-2
    assert np.max(np.abs(fus[5].cpu().numpy() - lse_o)) <= 2e-3


def test_step_fallback_shapes():
    """Shapes outside the fused path (8192 blocks) run the three stages one
    after the other and give the separate calls' results."""
    # 8192 blocks (L = 524288) exceed the fused selection core: k_max 256.
    wl_long = synth.decode_config(3, B=1, L=524288, backbone=False)
    rule = Rule(0.95, 256, 0, 1, 2)
    wl_long.rule = rule
    nb = wl_long.nblk
    q_sel, w, k_sel = bf(wl_long.q_sel), f32(wl_long.w), bf(wl_long.k_sel)
    seq = i32(wl_long.seq_len)
    nv = i32(wl_long.n_valid)
    qq = bf(synth.normal_bf16(78, 1, (1, 32, 128)))
    kk = torch.zeros((1, 8, 524288, 128), dtype=torch.bfloat16, device=DEV)
    vv = torch.zeros_like(kk)
    s0 = spot.selector_score(q_sel, w, k_sel, n_valid=nv, nblk=nb)
    i0, c0, _ = spot.select_blocks(s0, rule, nv)
    s1, i1, c1, _, o1, l1 = spot.decode_step(q_sel, w, k_sel, qq, kk, vv, seq, rule, n_valid=nv)
    torch.cuda.synchronize()
    assert torch.equal(s0, s1) and torch.equal(i0, i1) and torch.equal(c0, c1)
    assert torch.all(o1.float() == 0)   # zero values give zero outputs
