"""Acceptance of a selected block set against the oracle's.

Selection is an integer decision taken from floating-point scores, so two
implementations can legitimately differ where the decision sits on a
rounding boundary.  A set from the HIP path is accepted for a row when it
equals the oracle's, or when every difference is explained by one of:

  (i)  near-ties: the two sets differ only in blocks whose score lies within
       ``rel_tie`` (relative) of the cutoff score between chosen and unchosen
       residual blocks -- both orders are then correct;
  (ii) mass boundary: the oracle's cumulative residual mass after n-1 or n
       blocks is within ``mass_tol`` of p, so a nucleus one block shorter or
       longer is equally correct.

Whatever the exemption, the set must still contain every reserved block,
respect k_max, and be a top-n set of the residual scores up to ``rel_tie``.
Exempted rows must stay rare: check_all allows at most max(1, rows // 50)
of them per call (2 %), so a systematic difference cannot hide behind the
exemptions.

Why these tolerances: the HIP path sums the exponentials in FP32 along a
reduction tree of depth about 11 (8 per thread, 64 per wave, 4 waves), so
the nucleus mass it compares with p carries a relative error of at most
about 2 * 11 * 2^-24 = 1.3e-6 of Z (plus one ulp per v_exp_f32 term);
mass_tol = 1e-5 leaves a factor of about 8 over that.  Scores are compared
at 1e-4 relative, so two blocks closer than that may rank either way.
"""
from __future__ import annotations

import numpy as np


def reserved_ids(nv, n_sink, n_recent):
    return set(range(min(n_sink, nv))) | set(range(max(0, nv - n_recent), nv))


def nucleus_len_candidates(res_sorted_scores, rule, n_reserved, mass_tol):
    s = np.asarray(res_sorted_scores, dtype=np.float64)
    n_res = len(s)
    cap = min(rule.k_max - n_reserved, n_res)
    if n_res == 0:
        return {0}
    e = np.exp(s - s.max())
    cum = np.cumsum(e / e.sum())
    p = rule.top_p
    if p >= 1:
        raw = {n_res}
    elif p <= 0:
        raw = {0}
    else:
        n0 = int(np.searchsorted(cum, p, side="left")) + 1  # first cum >= p
        n0 = min(n0, n_res)
        raw = {n0}
        if n0 - 1 >= 1 and cum[n0 - 2] >= p - mass_tol:
            raw.add(n0 - 1)
        if n0 < n_res and cum[n0 - 1] < p + mass_tol:
            raw.add(n0 + 1)
    out = set()
    for n in raw:
        n = min(n, cap)
        if n_reserved + n < rule.k_min:
            n = min(rule.k_min - n_reserved, cap)
        out.add(n)
    return out


def check_row(scores, nv, rule, S_oracle, S_gpu, rel_tie=1e-4, mass_tol=1e-5):
    """Return 'exact', 'tie', 'mass' or raise AssertionError with a reason."""
    S_o, S_g = set(int(x) for x in S_oracle), set(int(x) for x in S_gpu)
    if S_o == S_g:
        return "exact"
    R = reserved_ids(nv, rule.n_sink, rule.n_recent)
    assert R <= S_g, f"reserved {sorted(R - S_g)} missing"
    assert len(S_g) <= rule.k_max, "k_max exceeded"
    assert all(0 <= j < nv for j in S_g), "id out of range"
    res = [j for j in range(nv) if j not in R]
    s = np.asarray(scores, dtype=np.float64)
    order = sorted(res, key=lambda j: (-s[j], j))
    n_allowed = nucleus_len_candidates(s[order], rule, len(R), mass_tol)
    n_g = len(S_g) - len(R)
    assert n_g in n_allowed, f"nucleus size {n_g} not in {sorted(n_allowed)}"
    nuc = S_g - R
    rest = [j for j in res if j not in nuc]
    if nuc and rest:
        lo = min(s[j] for j in nuc)
        hi = max(s[j] for j in rest)
        tol = rel_tie * max(abs(lo), abs(hi)) + 1e-30
        assert lo >= hi - tol, f"not a top-n set: chosen min {lo} < unchosen max {hi}"
    n_o = len(S_o) - len(R)
    return "tie" if n_g == n_o else "mass"


def check_all(scores, n_valid, rule, idx_o, cnt_o, idx_g, cnt_g, max_exempt=None, **kw):
    stats = {"exact": 0, "tie": 0, "mass": 0}
    for r in range(len(cnt_o)):
        g = idx_g[r, :cnt_g[r]]
        assert np.all(idx_g[r, cnt_g[r]:] == -1), f"row {r}: padding"
        assert np.all(np.diff(g) > 0), f"row {r}: not ascending"
        try:
            kind = check_row(scores[r], int(n_valid[r]), rule, idx_o[r, :cnt_o[r]], g, **kw)
        except AssertionError as e:
            raise AssertionError(f"row {r}: {e}") from None
        stats[kind] += 1
    if max_exempt is None:
        max_exempt = max(1, len(cnt_o) // 50)
    assert stats["tie"] + stats["mass"] <= max_exempt, f"too many exempted rows: {stats}"
    return stats
