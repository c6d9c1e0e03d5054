"""spot_decode_step_static -- the fused decode step on the device's static
scratch, for callers that cannot allocate -- against spot_decode_step with a
caller workspace, through the C ABI (needs an MI355X).

Both calls run the same kernels with the same work split, so every output
must match bit for bit; this is checked on two calls in a row, the second with
a smaller input, and the scratch must be left clean (status query).  A shape
that runs the three stages as separate launches (k_max above the fused
limit) leaves its partials in the scratch; a fused call after it must not be
disturbed by them."""
import dataclasses

import numpy as np
import pytest
import torch

from paper_2606_22874_amd import spot, synth

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

DEV = "cuda:0"


def bf(a):
    return spot.to_device_bf16(a, DEV)


def i32(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(DEV)


def both(wl):
    q_sel, w, k_sel = bf(wl.q_sel), torch.from_numpy(wl.w).to(DEV), bf(wl.k_sel)
    q, k, v = bf(wl.q), bf(wl.k), bf(wl.v)
    seq, nv = i32(wl.seq_len), i32(wl.n_valid)
    ref = spot.decode_step(q_sel, w, k_sel, q, k, v, seq, wl.rule, n_valid=nv,
                           sm_scale=wl.sm_scale)
    B, Hq, Hkv, d, L, r = wl.B, wl.Hq, wl.Hkv, wl.d, wl.L, wl.rule
    nblk = L // 64
    out = (torch.full((B, nblk), -7.0, device=DEV),
           torch.full((B, r.k_max), -7, dtype=torch.int32, device=DEV),
           torch.full((B,), -7, dtype=torch.int32, device=DEV),
           torch.full((B,), -7.0, device=DEV),
           torch.zeros((B, Hq, d), dtype=torch.bfloat16, device=DEV),
           torch.full((B, Hq), -7.0, device=DEV))
    spot.spot_decode_step_static(q_sel, w, k_sel, None, 0, wl.Hs, wl.ds, nv, r.top_p, r.k_max,
                                 r.k_min, r.n_sink, r.n_recent, q, k, v, seq, B, Hq, Hkv, d, L,
                                 wl.sm_scale, *out)
    torch.cuda.synchronize()
    for name, a, b in zip(("scores", "idx", "count", "nuc_mass", "out", "lse"), ref, out):
        assert torch.equal(a, b), name
    assert spot.spot_decode_step_status(None, B, Hq, Hkv, d, r.k_max) == 0


def test_static_scratch_matches_workspace_twice():
    print("[no-alloc] 128K-token workload, batch 4", flush=True)
    both(synth.decode_config(3))
    print("[no-alloc] 8K-token workload, batch 2 (smaller)", flush=True)
    both(synth.decode_config(2, B=2, L=8192))


def test_static_scratch_after_separate_launches():
    wl = synth.decode_config(2, B=1, L=65536)
    wl = dataclasses.replace(wl, rule=dataclasses.replace(wl.rule, k_max=600))
    print("[no-alloc] 64K-token workload, k_max 600 (separate launches)", flush=True)
    both(wl)
    print("[no-alloc] 8K-token workload, batch 2 (fused) after it", flush=True)
    both(synth.decode_config(2, B=2, L=8192))
