"""Seeded synthetic workloads for the SpotAttention decode/prefill hot path.

This module only *creates inputs*: random draws, BF16 rounding of the draws,
the planted/Zipf structure of the selector keys, and the two microscale
encoders that turn a BF16 selector key cache into the INT4 and MXFP4 byte
formats a caller would store (the encoders sit on the cache-append side; the
hot path only ever decodes those bytes).  It holds none of the hot path's
arithmetic (no block score, no softmax, no selection, no attention) and
imports neither the HIP binding nor the oracle, so the tests can feed the very
same arrays to both.

Shapes follow the paper's setting (Section 2.1 selector, Section 2.3 selection,
Section 3 Qwen3 backbones): a Qwen3-shaped layer with H_q query heads, H_kv KV
heads, head dim d = 128, and a block-pooled selector key cache with H_s = 8
heads of width d_s = 64, one key per 64-token block.

Layouts (all C-contiguous, BF16 stored as uint16 bit patterns):
  decode  q      [B, H_q, d]            k, v   [B, H_kv, L, d]
          q_sel  [B, H_s, d_s]          w      [B, H_s] float32
          k_sel  [B, nblk, H_s, d_s]
  prefill q      [B, H_q, L, d]         q_sel  [B, nqb, H_s, d_s]   w [B, nqb, H_s]
  INT4    codes  [..., d_s/2] uint8 (element 2i in the low nibble), scales
          [..., d_s/32] float16 bit patterns (uint16)
  MXFP4   codes  [..., d_s/2] uint8 (E2M1, element 2i low), scales [..., d_s/32]
          uint8 E8M0
"""
from __future__ import annotations

import dataclasses
import math
import os
from concurrent.futures import ThreadPoolExecutor
from typing import Optional

import numpy as np

BLK = 64            # tokens per KV block (one selector key per block)
SEED_BASE = 20260   # seed of config i is SEED_BASE + i


# --------------------------------------------------------------------------
# BF16 / FP16 storage helpers (bit-pattern conversion of the *inputs*)
# --------------------------------------------------------------------------
def bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> BF16 bit patterns, round to nearest even (finite inputs)."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32)
    r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_value(b: np.ndarray) -> np.ndarray:
    """BF16 bit patterns -> float32 (exact)."""
    b = np.ascontiguousarray(b, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


def _threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def normal_bf16(seed: int, tag: int, shape: tuple, lead: int = 2) -> np.ndarray:
    """N(0,1) draws rounded to BF16, filled in parallel.

    The first ``lead`` axes index independent sub-streams, each seeded from
    (seed, tag, i0, i1, ...), so the result does not depend on the number of
    threads used to fill it.
    """
    out = np.empty(shape, dtype=np.uint16)
    lead_shape = shape[:lead]
    inner = shape[lead:]
    jobs = list(np.ndindex(*lead_shape))

    def fill(ix):
        rng = np.random.default_rng([seed, tag, *ix])
        out[ix] = bf16_bits(rng.standard_normal(inner, dtype=np.float32))

    with ThreadPoolExecutor(_threads()) as ex:
        list(ex.map(fill, jobs))
    return out


# --------------------------------------------------------------------------
# Workload description
# --------------------------------------------------------------------------
@dataclasses.dataclass
class Rule:
    """Dual top-p / top-K rule (Section 2.3) plus the total-budget cap k_max."""
    top_p: float
    k_max: int
    k_min: int = 0
    n_sink: int = 1
    n_recent: int = 2


@dataclasses.dataclass
class Decode:
    name: str
    B: int
    L: int          # cache capacity in tokens (multiple of 64)
    Hq: int
    Hkv: int
    d: int
    Hs: int
    ds: int
    rule: Rule
    seq_len: np.ndarray   # int32 [B]
    q_sel: np.ndarray     # bf16 [B, Hs, ds]
    w: np.ndarray         # f32  [B, Hs]
    k_sel: np.ndarray     # bf16 [B, nblk, Hs, ds]
    q: Optional[np.ndarray] = None  # bf16 [B, Hq, d]
    k: Optional[np.ndarray] = None  # bf16 [B, Hkv, L, d]
    v: Optional[np.ndarray] = None

    @property
    def nblk(self) -> int:
        return self.L // BLK

    @property
    def n_valid(self) -> np.ndarray:
        return ((self.seq_len + BLK - 1) // BLK).astype(np.int32)

    @property
    def sm_scale(self) -> float:
        return 1.0 / math.sqrt(self.d)


@dataclasses.dataclass
class Prefill:
    name: str
    B: int
    L: int
    Hq: int
    Hkv: int
    d: int
    Hs: int
    ds: int
    rule: Rule
    q_sel: np.ndarray     # bf16 [B, nqb, Hs, ds]   (query-block pooled)
    w: np.ndarray         # f32  [B, nqb, Hs]
    k_sel: np.ndarray     # bf16 [B, nkb, Hs, ds]   (key-block pooled)
    q: Optional[np.ndarray] = None  # bf16 [B, Hq, L, d]
    k: Optional[np.ndarray] = None  # bf16 [B, Hkv, L, d]
    v: Optional[np.ndarray] = None

    @property
    def nblk(self) -> int:
        return self.L // BLK

    @property
    def n_valid(self) -> np.ndarray:
        """Causal block limit per (sequence, query block) row: qb + 1."""
        nqb = self.nblk
        return np.tile(np.arange(1, nqb + 1, dtype=np.int32), self.B)

    @property
    def sm_scale(self) -> float:
        return 1.0 / math.sqrt(self.d)


# --------------------------------------------------------------------------
# Selector-key structure generators
# --------------------------------------------------------------------------
def _unit(x: np.ndarray, axis=-1) -> np.ndarray:
    return x / np.linalg.norm(x, axis=axis, keepdims=True)


def _reserved_mask(nv: int, n_sink: int, n_recent: int) -> np.ndarray:
    m = np.zeros(nv, dtype=bool)
    m[: min(n_sink, nv)] = True
    m[max(0, nv - n_recent): nv] = True
    return m


def selector_planted(rng, B, L, Hs, ds, seq_len, n_planted=4, cosine=0.8):
    """Per-token selector keys ~ N(0,1), mean-pooled over 64-token blocks.

    ``n_planted`` blocks per sequence, drawn from the residual range
    [1, nv-4], get every token shifted along the selector query direction of
    each head so that the pooled key makes angle acos(cosine) with the query.
    Pooling: float32 sum of the BF16 token keys in token order over the valid
    tokens of the block, divided by their count, rounded to BF16.
    """
    nblk = L // BLK
    q_sel = bf16_bits(rng.standard_normal((B, Hs, ds), dtype=np.float32))
    w = rng.uniform(0.0, 1.0, (B, Hs)).astype(np.float32)
    qf = bf16_value(q_sel).astype(np.float64)
    qhat = _unit(qf)
    k_sel = np.zeros((B, nblk, Hs, ds), dtype=np.uint16)
    ratio = cosine / math.sqrt(1.0 - cosine * cosine)
    for b in range(B):
        tok = rng.standard_normal((L, Hs, ds), dtype=np.float32)
        seqlen = int(seq_len[b])
        nv = (seqlen + BLK - 1) // BLK
        hi = max(1, nv - 4)
        planted = rng.choice(np.arange(1, hi + 1), size=min(n_planted, hi), replace=False)
        for j in planted:
            seg = tok[j * BLK:(j + 1) * BLK].astype(np.float64)
            m = seg.mean(axis=0)                              # [Hs, ds]
            a = np.sum(m * qhat[b], axis=-1)                  # along q
            perp = np.linalg.norm(m - a[:, None] * qhat[b], axis=-1)
            delta = ratio * perp - a
            tok[j * BLK:(j + 1) * BLK] = (seg + delta[None, :, None] * qhat[b][None]).astype(np.float32)
        tokb = bf16_value(bf16_bits(tok))
        for j in range(nblk):
            lo, hi_t = j * BLK, min((j + 1) * BLK, seqlen)
            if hi_t <= lo:
                continue
            acc = np.zeros((Hs, ds), dtype=np.float32)
            for t in range(lo, hi_t):
                acc += tokb[t]
            k_sel[b, j] = bf16_bits(acc / np.float32(hi_t - lo))
    return q_sel, w, k_sel


def selector_tokens(seed, B, L, Hs, ds, seq_len, rule=None, zipf_a=1.1, t0=16.0,
                    noise=0.06, blk=BLK):
    """Per-token selector inputs with the Zipf relevance profile of
    ``selector_zipf`` carried by one token per block of ``blk`` tokens (64,
    the KV block, or 16, the paper's selector block).

    Returns q_sel [B, Hs, ds] (N(0, I/ds) draws, so |q_h| is about 1),
    w [B, Hs] ~ U(0, 1) and k_tok [B, L, Hs, ds] (BF16 bits).  Every token key
    is N(0, I) (filled in parallel in runs of up to 4096 tokens), which gives
    background token scores of order sum_h w_h.  In each residual block (not
    a sink or recency block of ``rule``, counted in blocks of ``blk``) one
    visible "lead" token, at a random
    position, is replaced by a key whose dot product with each head's query is
    T_j / sum_h w_h + N(0, noise^2), with T_j = t0 - zipf_a * ln(rank_j) for a
    random permutation rank of 1..n_res; its other directions are N(0, I).
    The lead token's score is then T_j, so block values follow a Zipf law
    under the residual softmax, as in the pooled-key workloads.
    """
    rule = Rule(0.95, 128, 0, 1, 2) if rule is None else rule
    rng = np.random.default_rng([seed, 91])
    q = rng.standard_normal((B, Hs, ds)) / math.sqrt(ds)
    q_sel = bf16_bits(q.astype(np.float32))
    w = rng.uniform(0.0, 1.0, (B, Hs)).astype(np.float32)
    qf = bf16_value(q_sel).astype(np.float64)
    qn = np.linalg.norm(qf, axis=-1)                          # [B, Hs]
    qhat = qf / qn[..., None]
    run = min(L, 4096)
    assert L % run == 0
    k_tok = normal_bf16(seed, 4, (B, L // run, run * Hs * ds)).reshape(B, L, Hs, ds)
    for b in range(B):
        n = int(min(max(int(seq_len[b]), 0), L))
        nv = (n + blk - 1) // blk
        res = np.flatnonzero(~_reserved_mask(nv, rule.n_sink, rule.n_recent))
        if len(res) == 0:
            continue
        T = t0 - zipf_a * np.log(rng.permutation(len(res)) + 1.0)
        lo = res * blk
        pos = lo + (rng.random(len(res)) * (np.minimum(lo + blk, n) - lo)).astype(np.int64)
        z = rng.standard_normal((len(res), Hs, ds))
        along = np.sum(z * qhat[b][None], axis=-1)
        perp = z - along[..., None] * qhat[b][None]
        t = T[:, None] / float(np.sum(w[b], dtype=np.float64)) + \
            rng.standard_normal((len(res), Hs)) * noise
        lead = perp + (t / qn[b][None])[..., None] * qhat[b][None]
        k_tok[b, pos] = bf16_bits(lead.astype(np.float32))
    return q_sel, w, k_tok


def selector_frontend(seed, rows, d_model, Hs, ds):
    """Hidden states and synthetic selector weights for the front end:
    h [rows, d_model] ~ N(0, 1); W_q, W_k [Hs*ds, d_model] and W_w
    [Hs, d_model] ~ N(0, 1/d_model) (so projections are of order 1); all BF16
    bits.  Trained weights are not available; only the shapes matter to the
    kernels."""
    rng = np.random.default_rng([seed, 57])
    sd = 1.0 / math.sqrt(d_model)
    h = bf16_bits(rng.standard_normal((rows, d_model), dtype=np.float32))
    wq = bf16_bits(rng.standard_normal((Hs * ds, d_model), dtype=np.float32) * np.float32(sd))
    wk = bf16_bits(rng.standard_normal((Hs * ds, d_model), dtype=np.float32) * np.float32(sd))
    ww = bf16_bits(rng.standard_normal((Hs, d_model), dtype=np.float32) * np.float32(sd))
    return h, wq, wk, ww


def selector_zipf(rng, B, nblk, Hs, ds, n_valid, rule: Rule, n_spikes=0,
                  zipf_a=1.1, t0=16.0, noise=0.06):
    """Pooled selector keys with a Zipf(zipf_a) relevance profile over blocks.

    For each residual block j (not a sink or recency block) a target score
    T_j = t0 - zipf_a * ln(rank_j), rank a random permutation of 1..n_res, so
    that exp(T_j) follows a Zipf law.  ``n_spikes`` random residual blocks get
    T = t0 + ln 2.  Each head's key is noise ~ N(0, I/ds) orthogonal to that
    head's (BF16-rounded) selector query, plus a component along the query
    whose dot product with it is T_j / sum_h w_h + N(0, noise^2).  Reserved
    blocks and blocks past n_valid get plain N(0, I/ds) keys.
    """
    q_sel = bf16_bits(rng.standard_normal((B, Hs, ds), dtype=np.float32))
    w = rng.uniform(0.0, 1.0, (B, Hs)).astype(np.float32)
    qf = bf16_value(q_sel).astype(np.float64)
    qn = np.linalg.norm(qf, axis=-1)                          # [B, Hs]
    qhat = qf / qn[..., None]
    k = np.empty((B, nblk, Hs, ds), dtype=np.float64)
    for b in range(B):
        nv = int(n_valid[b])
        res = np.flatnonzero(~_reserved_mask(nv, rule.n_sink, rule.n_recent))
        T = np.zeros(nblk)
        rank = rng.permutation(len(res)) + 1
        T[res] = t0 - zipf_a * np.log(rank)
        if n_spikes and len(res):
            sp = rng.choice(res, size=min(n_spikes, len(res)), replace=False)
            T[sp] = t0 + math.log(2.0)
        z = rng.standard_normal((nblk, Hs, ds)) / math.sqrt(ds)
        eps = rng.standard_normal((nblk, Hs)) * noise
        along = np.sum(z * qhat[b][None], axis=-1)
        perp = z - along[..., None] * qhat[b][None]
        t = T[:, None] / float(np.sum(w[b], dtype=np.float64)) + eps
        planted = perp + (t / qn[b][None])[..., None] * qhat[b][None]
        is_res = np.zeros(nblk, dtype=bool)
        is_res[res] = True
        k[b] = np.where(is_res[:, None, None], planted, z)
    return q_sel, w, bf16_bits(k.astype(np.float32))


def selector_prefill(rng, B, nqb, nkb, Hs, ds, zipf_a=1.1, t0=16.0):
    """Query-block x key-block selector inputs for block-sparse prefill.

    Per head a unit direction u_h.  Key block kb: (T_kb/32) u_h + noise
    N(0, I/ds) orthogonal to u_h, with T_kb = t0 - zipf_a ln(rank_kb) over one
    random ranking of all key blocks.  Query block qb: 8 u_h + noise
    N(0, 0.25^2 I) orthogonal to u_h.  Mixing weights w ~ U(0,1).
    """
    u = _unit(rng.standard_normal((Hs, ds)))
    qs, ws, ks = [], [], []
    for _ in range(B):
        rank = rng.permutation(nkb) + 1
        T = t0 - zipf_a * np.log(rank)
        zk = rng.standard_normal((nkb, Hs, ds)) / math.sqrt(ds)
        zk -= np.sum(zk * u[None], axis=-1, keepdims=True) * u[None]
        kk = zk + (T / 32.0)[:, None, None] * u[None]
        zq = rng.standard_normal((nqb, Hs, ds)) * 0.25
        zq -= np.sum(zq * u[None], axis=-1, keepdims=True) * u[None]
        qq = zq + 8.0 * u[None]
        qs.append(bf16_bits(qq.astype(np.float32)))
        ks.append(bf16_bits(kk.astype(np.float32)))
        ws.append(rng.uniform(0.0, 1.0, (nqb, Hs)).astype(np.float32))
    return np.stack(qs), np.stack(ws), np.stack(ks)


# --------------------------------------------------------------------------
# Microscale encoders for the selector key cache (cache-append side)
# --------------------------------------------------------------------------
E2M1_GRID = np.array([0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0])


def quantize_int4_g32(k_bits: np.ndarray):
    """Symmetric INT4 with one FP16 scale per 32 consecutive elements.

    scale = fp16_rne(amax / 7); code = clamp(rne(x / scale), -7, 7), stored
    as a two's-complement nibble; an all-zero group gets scale 0 and codes 0.
    Returns (codes uint8 [..., n/2], scales float16-bits uint16 [..., n/32]).
    """
    x = bf16_value(k_bits).astype(np.float64)
    *lead, n = x.shape
    assert n % 32 == 0
    g = x.reshape(*lead, n // 32, 32)
    amax = np.max(np.abs(g), axis=-1)
    scale = (amax / 7.0).astype(np.float32).astype(np.float16)
    sf = scale.astype(np.float64)
    with np.errstate(divide="ignore", invalid="ignore"):
        c = np.where(sf[..., None] > 0, np.rint(g / sf[..., None]), 0.0)
    c = np.clip(c, -7, 7).astype(np.int8).reshape(*lead, n)
    nib = (c.astype(np.int16) & 0xF).astype(np.uint8)
    codes = (nib[..., 0::2] | (nib[..., 1::2] << 4)).astype(np.uint8)
    return codes, scale.view(np.uint16)


def _e2m1_rne(y: np.ndarray) -> np.ndarray:
    """|y| -> E2M1 magnitude code (0..7), round to nearest, ties to even code."""
    a = np.minimum(np.abs(y), 6.0)
    # distance to each grid point; choose nearest, ties -> even code index
    dist = np.abs(a[..., None] - E2M1_GRID)
    best = np.min(dist, axis=-1, keepdims=True)
    cand = dist == best
    idx = np.arange(8)
    # prefer even codes among ties: score = tie ? (idx odd) : big
    pick = np.where(cand, (idx % 2) * 8 + idx, 99)
    code = np.argmin(pick, axis=-1)
    return code.astype(np.uint8)


def quantize_mxfp4_g32(k_bits: np.ndarray):
    """OCP MX v1.0 MXFP4: E2M1 elements, one E8M0 scale per 32 elements.

    X = floor(log2(amax)) - 2 (2 = E2M1's max exponent), clamped to
    [-127, 127]; E8M0 = X + 127; element code = E2M1_rne(x / 2^X) saturating
    to +-6; amax = 0 gives E8M0 = 0 and zero codes.
    Returns (codes uint8 [..., n/2], e8m0 uint8 [..., n/32]).
    """
    x = bf16_value(k_bits).astype(np.float64)
    *lead, n = x.shape
    assert n % 32 == 0
    g = x.reshape(*lead, n // 32, 32)
    amax = np.max(np.abs(g), axis=-1)
    with np.errstate(divide="ignore"):
        X = np.where(amax > 0, np.floor(np.log2(np.where(amax > 0, amax, 1.0))) - 2, -127)
    X = np.clip(X, -127, 127).astype(np.int32)
    e8 = (X + 127).astype(np.uint8)
    y = g / np.ldexp(1.0, X)[..., None]
    mag = _e2m1_rne(y)
    sign = ((y < 0) & (mag > 0)).astype(np.uint8) << 3
    c = (mag | sign).reshape(*lead, n)
    codes = (c[..., 0::2] | (c[..., 1::2] << 4)).astype(np.uint8)
    return codes, e8


def quantize_int8_g32(k_bits: np.ndarray):
    """Symmetric INT8 with one FP16 scale per 32 consecutive elements.

    scale = fp16_rne(amax / 127); code = clamp(rne(x / scale), -127, 127),
    two's complement in a byte; an all-zero group gets scale 0 and codes 0.
    Returns (codes uint8 [..., n], scales float16-bits uint16 [..., n/32]).
    """
    x = bf16_value(k_bits).astype(np.float64)
    *lead, n = x.shape
    assert n % 32 == 0
    g = x.reshape(*lead, n // 32, 32)
    amax = np.max(np.abs(g), axis=-1)
    scale = (amax / 127.0).astype(np.float32).astype(np.float16)
    sf = scale.astype(np.float64)
    with np.errstate(divide="ignore", invalid="ignore"):
        c = np.where(sf[..., None] > 0, np.rint(g / sf[..., None]), 0.0)
    c = np.clip(c, -127, 127).astype(np.int8).reshape(*lead, n)
    return c.view(np.uint8), scale.view(np.uint16)


def _e4m3_values() -> np.ndarray:
    """Values of the non-negative finite OCP E4M3 codes 0 .. 126 (ascending)."""
    v = []
    for code in range(127):
        e, m = code >> 3, code & 7
        v.append(m / 8.0 * 2.0 ** -6 if e == 0 else (1.0 + m / 8.0) * 2.0 ** (e - 7))
    return np.array(v)


E4M3_GRID = _e4m3_values()


def _e4m3_rne(y: np.ndarray) -> np.ndarray:
    """|y| -> E4M3 magnitude code (0 .. 126), nearest, ties to the even code,
    saturating at 448."""
    a = np.minimum(np.abs(y), 448.0)
    hi = np.clip(np.searchsorted(E4M3_GRID, a), 1, 126)
    lo = hi - 1
    d_lo = a - E4M3_GRID[lo]
    d_hi = E4M3_GRID[hi] - a
    pick_hi = (d_hi < d_lo) | ((d_hi == d_lo) & (hi % 2 == 0))
    return np.where(pick_hi, hi, lo).astype(np.uint8)


def quantize_mxfp8_g32(k_bits: np.ndarray):
    """OCP MX v1.0 MXFP8 (E4M3): one E8M0 scale per 32 elements.

    X = floor(log2(amax)) - 8 (8 = E4M3's max exponent), clamped to
    [-127, 127]; E8M0 = X + 127; element code = E4M3_rne(x / 2^X) saturating
    to +-448; amax = 0 gives E8M0 = 0 and zero codes.
    Returns (codes uint8 [..., n], e8m0 uint8 [..., n/32]).
    """
    x = bf16_value(k_bits).astype(np.float64)
    *lead, n = x.shape
    assert n % 32 == 0
    g = x.reshape(*lead, n // 32, 32)
    amax = np.max(np.abs(g), axis=-1)
    with np.errstate(divide="ignore"):
        X = np.where(amax > 0, np.floor(np.log2(np.where(amax > 0, amax, 1.0))) - 8, -127)
    X = np.clip(X, -127, 127).astype(np.int32)
    e8 = (X + 127).astype(np.uint8)
    y = g / np.ldexp(1.0, X)[..., None]
    mag = _e4m3_rne(y)
    sign = ((y < 0) & (mag > 0)).astype(np.uint8) << 7
    return (mag | sign).reshape(*lead, n).astype(np.uint8), e8


QUANTIZERS = {"int4": quantize_int4_g32, "mxfp4": quantize_mxfp4_g32,
              "int8": quantize_int8_g32, "mxfp8": quantize_mxfp8_g32}


# --------------------------------------------------------------------------
# The five workloads
# --------------------------------------------------------------------------
def _backbone_decode(seed, B, L, Hq, Hkv, d):
    q = normal_bf16(seed, 1, (B, Hq, d), lead=1)
    k = normal_bf16(seed, 2, (B, Hkv, L, d))
    v = normal_bf16(seed, 3, (B, Hkv, L, d))
    return q, k, v


def decode_config(i: int, *, B=None, L=None, seq_len=None, backbone=True,
                  seed=None) -> Decode:
    """Decode workloads 1-3 (4 = 3 with a quantized selector cache).

    Overrides (B, L, seq_len, seed) shrink a workload for tests while keeping
    its structure; seq_len may be ragged (each sequence's n_valid follows it).
    """
    if i == 1:
        B0, L0, rule, kind = 1, 4096, Rule(0.9, 16, 0, 1, 2), "planted"
    elif i == 2:
        B0, L0, rule, kind = 8, 32768, Rule(0.9, 64, 0, 1, 2), "zipf16"
    elif i in (3, 4):
        B0, L0, rule, kind = 4, 131072, Rule(0.95, 128, 0, 1, 2), "zipf"
    else:
        raise ValueError(i)
    B = B0 if B is None else B
    L = L0 if L is None else L
    assert L % BLK == 0
    seed = SEED_BASE + i if seed is None else seed
    rng = np.random.default_rng(seed)
    if seq_len is None:
        seq_len = np.full(B, L, dtype=np.int32)
    seq_len = np.asarray(seq_len, dtype=np.int32)
    n_valid = (seq_len + BLK - 1) // BLK
    Hq, Hkv, d, Hs, ds = 32, 8, 128, 8, 64
    if kind == "planted":
        q_sel, w, k_sel = selector_planted(rng, B, L, Hs, ds, seq_len)
    else:
        q_sel, w, k_sel = selector_zipf(rng, B, L // BLK, Hs, ds, n_valid, rule,
                                        n_spikes=16 if kind == "zipf16" else 0)
    wl = Decode(f"decode{i}", B, L, Hq, Hkv, d, Hs, ds, rule, seq_len, q_sel, w, k_sel)
    if backbone:
        wl.q, wl.k, wl.v = _backbone_decode(seed, B, L, Hq, Hkv, d)
    return wl


def prefill_config(*, L=None, Hq=None, backbone=True, seed=None) -> Prefill:
    """Workload 5: block-sparse causal prefill, Qwen3-32B-shaped layer."""
    L = 32768 if L is None else L
    Hq = 64 if Hq is None else Hq
    B, Hkv, d, Hs, ds = 1, 8, 128, 8, 64
    seed = SEED_BASE + 5 if seed is None else seed
    rng = np.random.default_rng(seed)
    nb = L // BLK
    q_sel, w, k_sel = selector_prefill(rng, B, nb, nb, Hs, ds)
    wl = Prefill("prefill5", B, L, Hq, Hkv, d, Hs, ds, Rule(0.9, 64, 0, 1, 2), q_sel, w, k_sel)
    if backbone:
        wl.q = normal_bf16(seed, 1, (B, Hq, L, d))
        wl.k = normal_bf16(seed, 2, (B, Hkv, L, d))
        wl.v = normal_bf16(seed, 3, (B, Hkv, L, d))
    return wl


def random_scores(seed: int, rows: int, nblk: int, n_valid=None, scale=3.0) -> np.ndarray:
    """Float32 block-score matrices for exercising the selection rule alone.

    Mixes continuous draws with deliberate exact ties (values snapped to a
    coarse grid on a random third of the rows); entries past n_valid are -inf.
    """
    rng = np.random.default_rng([seed, 77])
    s = (rng.standard_normal((rows, nblk)) * scale).astype(np.float32)
    snap = rng.random(rows) < 0.33
    s[snap] = np.round(s[snap] * 2.0) / 2.0
    if n_valid is not None:
        cols = np.arange(nblk)[None, :]
        s = np.where(cols < np.asarray(n_valid)[:, None], s, -np.inf).astype(np.float32)
    return s
