"""Python face of the FP64 CPU oracle (``oracle/spot_oracle.c``).

TEST INFRASTRUCTURE: only the tests, the smoke check and the CPU-baseline leg
of the benchmark may import this package.  It never touches the HIP library,
and the HIP library never touches it.

``build()`` compiles the C file with gcc (OpenMP) into ``liboracle.so`` next
to it; ``lib()`` builds on first use when the library is missing or older
than its source.  ``SPOT_ORACLE_SO`` names another build of the same source
to load instead (the sanitizer test uses it).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "spot_oracle.c")
HDR = os.path.join(HERE, "spot_oracle.h")
SO = os.path.join(HERE, "liboracle.so")

KFMT = {"bf16": 0, "int4": 1, "mxfp4": 2, "int8": 3, "mxfp8": 4}

_lock = threading.Lock()
_lib = None


def build(force: bool = True) -> str:
    tmp = SO + f".tmp{os.getpid()}"
    cmd = ["gcc", "-O2", "-fopenmp", "-std=c11", "-Wall", "-Wextra", "-shared", "-fPIC",
           "-o", tmp, SRC, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, SO)
    return SO


def _stale() -> bool:
    if not os.path.exists(SO):
        return True
    t = os.path.getmtime(SO)
    return t < os.path.getmtime(SRC) or t < os.path.getmtime(HDR)


def lib():
    global _lib
    with _lock:
        if _lib is None:
            path = os.environ.get("SPOT_ORACLE_SO")
            if not path:
                path = SO
                if _stale():
                    build()
            L = ctypes.CDLL(path)
            P, I, D = ctypes.c_void_p, ctypes.c_int, ctypes.c_double
            L.oracle_set_threads.argtypes = [I]
            L.oracle_get_threads.restype = I
            L.oracle_key_value.argtypes = [P, P, I, ctypes.c_int64]
            L.oracle_key_value.restype = D
            L.oracle_selector_score.argtypes = [P, P, P, P, I, I, I, I, I, I, P, P]
            L.oracle_selector_score_qk.argtypes = [P, P, I, P, P, P, I, I, I, I, I, I, P, P]
            L.oracle_selector_score_tokens.argtypes = [P, P, P, P, I, I, I, I, I, I, I, P, P]
            L.oracle_selector_project.argtypes = [P, P, P, P, P, I, I, I, I, I, D, P, P, P]
            L.oracle_selector_pool.argtypes = [P, I, I, I, I, P, P]
            L.oracle_select_blocks.argtypes = [P, I, I, P, D, I, I, I, I, P, P, P]
            L.oracle_select_blocks.restype = I
            L.oracle_sparse_decode.argtypes = [P, P, P, P, P, P, I, I, I, I, I, I, I, D, P, P]
            L.oracle_dense_decode.argtypes = [P, P, P, P, I, I, I, I, I, D, P, P]
            L.oracle_sparse_prefill.argtypes = [P, P, P, I, P, P, I, I, I, I, I, I, D, P, I, P, P]
            _lib = L
    return _lib


def _p(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dt):
    return np.ascontiguousarray(a, dtype=dt)


def set_threads(n: int) -> None:
    lib().oracle_set_threads(int(n))


def get_threads() -> int:
    return int(lib().oracle_get_threads())


def key_values(k_sel, k_scale=None, kfmt="bf16", n=None) -> np.ndarray:
    """Decoded float64 values of the first n stored key elements."""
    L = lib()
    f = KFMT[kfmt] if isinstance(kfmt, str) else int(kfmt)
    ks = np.ascontiguousarray(k_sel)
    sc = None if k_scale is None else np.ascontiguousarray(k_scale)
    if n is None:
        n = ks.size if f in (0, 3, 4) else ks.size * 2
    return np.array([L.oracle_key_value(_p(ks), _p(sc), f, i) for i in range(n)])


def selector_score(q_sel, w, k_sel, k_scale=None, kfmt="bf16", rows_per_seq=1,
                   n_valid=None, nblk=None, h_s=None, d_s=None) -> np.ndarray:
    """Block scores [rows, nblk] in float64 (Section 2.1)."""
    f = KFMT[kfmt] if isinstance(kfmt, str) else int(kfmt)
    q_sel = _c(q_sel, np.uint16)
    w = _c(w, np.float32)
    h_s = q_sel.shape[-2] if h_s is None else h_s
    d_s = q_sel.shape[-1] if d_s is None else d_s
    rows = q_sel.size // (h_s * d_s)
    n_seq = rows // rows_per_seq
    k_sel = np.ascontiguousarray(k_sel)
    if nblk is None:
        per = h_s * d_s if f in (0, 3, 4) else h_s * d_s // 2
        nblk = k_sel.size // (n_seq * per)
    sc = None if k_scale is None else np.ascontiguousarray(k_scale)
    nv = None if n_valid is None else _c(n_valid, np.int32)
    out = np.empty((rows, nblk), dtype=np.float64)
    lib().oracle_selector_score(_p(q_sel), _p(w), _p(k_sel), _p(sc), f, n_seq, rows_per_seq,
                                nblk, h_s, d_s, _p(nv), _p(out))
    return out


def selector_score_qk(q_sel, q_scale, qfmt, w, k_sel, k_scale, kfmt, rows, nblk, h_s, d_s,
                      rows_per_seq=1, n_valid=None) -> np.ndarray:
    """Block scores [rows, nblk] in float64 with quantized queries and keys."""
    qf = KFMT[qfmt] if isinstance(qfmt, str) else int(qfmt)
    kf = KFMT[kfmt] if isinstance(kfmt, str) else int(kfmt)
    q = np.ascontiguousarray(q_sel)
    qs = None if q_scale is None else np.ascontiguousarray(q_scale)
    k = np.ascontiguousarray(k_sel)
    ks = None if k_scale is None else np.ascontiguousarray(k_scale)
    w = _c(w, np.float32)
    nv = None if n_valid is None else _c(n_valid, np.int32)
    out = np.empty((rows, nblk), dtype=np.float64)
    lib().oracle_selector_score_qk(_p(q), _p(qs), qf, _p(w), _p(k), _p(ks), kf,
                                   rows // rows_per_seq, rows_per_seq, nblk, h_s, d_s, _p(nv),
                                   _p(out))
    return out


def selector_score_tokens(q_sel, w, k_tok, k_scale=None, kfmt="bf16", rows_per_seq=1,
                          seq_len=None, l_cap=None, blk=64, h_s=None, d_s=None) -> np.ndarray:
    """Per-block maximum of per-token scores [rows, l_cap // blk] in float64
    (Section 2.3 over the score of Section 2.1)."""
    f = KFMT[kfmt] if isinstance(kfmt, str) else int(kfmt)
    q_sel = _c(q_sel, np.uint16)
    w = _c(w, np.float32)
    h_s = q_sel.shape[-2] if h_s is None else h_s
    d_s = q_sel.shape[-1] if d_s is None else d_s
    rows = q_sel.size // (h_s * d_s)
    n_seq = rows // rows_per_seq
    k_tok = np.ascontiguousarray(k_tok)
    if l_cap is None:
        per = h_s * d_s if f in (0, 3, 4) else h_s * d_s // 2
        l_cap = k_tok.size // (n_seq * per)
    sc = None if k_scale is None else np.ascontiguousarray(k_scale)
    sl = None if seq_len is None else _c(seq_len, np.int32)
    out = np.empty((rows, l_cap // blk), dtype=np.float64)
    lib().oracle_selector_score_tokens(_p(q_sel), _p(w), _p(k_tok), _p(sc), f, n_seq,
                                       rows_per_seq, l_cap, blk, h_s, d_s, _p(sl), _p(out))
    return out


def selector_project(h, w_q, w_k, w_w, pos, h_s, d_s, rope_dim=64, rope_base=1.0e6):
    """(q [rows, h_s, d_s], k [rows, h_s, d_s], w [rows, h_s]) in float64:
    the selector projections of hidden states h [rows, d_model] with rotary
    embedding at positions pos (Section 2.1, Appendix A)."""
    h = _c(h, np.uint16)
    rows, d_model = h.shape
    w_q, w_k, w_w = _c(w_q, np.uint16), _c(w_k, np.uint16), _c(w_w, np.uint16)
    pos = _c(pos, np.int32)
    q = np.empty((rows, h_s, d_s))
    k = np.empty((rows, h_s, d_s))
    w = np.empty((rows, h_s))
    lib().oracle_selector_project(_p(h), _p(w_q), _p(w_k), _p(w_w), _p(pos), rows, d_model,
                                  h_s, d_s, rope_dim, float(rope_base), _p(q), _p(k), _p(w))
    return q, k, w


def selector_pool(k_tok, seq_len=None, blk=64):
    """Pooled keys [n_seq, l_cap // blk, ...] in float64: the mean of each
    block's existing tokens (0 where there are none)."""
    k_tok = _c(k_tok, np.uint16)
    n_seq, l_cap = k_tok.shape[:2]
    width = k_tok.size // (n_seq * l_cap)
    sl = None if seq_len is None else _c(seq_len, np.int32)
    out = np.empty((n_seq, l_cap // blk) + k_tok.shape[2:])
    lib().oracle_selector_pool(_p(k_tok), n_seq, l_cap, blk, width, _p(sl), _p(out))
    return out


def select_blocks(scores, rule, n_valid=None):
    """(idx [rows, k_max] int32 ascending -1 padded, count [rows], nuc_mass [rows])."""
    s = _c(scores, np.float64)
    rows, nblk = s.shape
    nv = None if n_valid is None else _c(n_valid, np.int32)
    idx = np.empty((rows, rule.k_max), dtype=np.int32)
    cnt = np.empty(rows, dtype=np.int32)
    mass = np.empty(rows, dtype=np.float64)
    rc = lib().oracle_select_blocks(_p(s), rows, nblk, _p(nv), float(rule.top_p), rule.k_max,
                                    rule.k_min, rule.n_sink, rule.n_recent, _p(idx), _p(cnt),
                                    _p(mass))
    if rc != 0:
        raise ValueError("oracle_select_blocks: invalid rule")
    return idx, cnt, mass


def sparse_decode(q, k, v, seq_len, idx, count, sm_scale, blk=64):
    """Attention over the tokens of the selected blocks of blk tokens each
    (Section 2): [B, h_q, d] outputs and [B, h_q] log-sum-exps in float64."""
    q, k, v = _c(q, np.uint16), _c(k, np.uint16), _c(v, np.uint16)
    B, h_q, d = q.shape
    _, h_kv, l_cap, _ = k.shape
    idx = _c(idx, np.int32)
    cnt = _c(count, np.int32)
    sl = _c(seq_len, np.int32)
    out = np.empty((B, h_q, d), dtype=np.float64)
    lse = np.empty((B, h_q), dtype=np.float64)
    lib().oracle_sparse_decode(_p(q), _p(k), _p(v), _p(sl), _p(idx), _p(cnt), idx.shape[1], B,
                               h_q, h_kv, d, l_cap, int(blk), float(sm_scale), _p(out), _p(lse))
    return out, lse


def dense_decode(q, k, v, seq_len, sm_scale):
    q, k, v = _c(q, np.uint16), _c(k, np.uint16), _c(v, np.uint16)
    B, h_q, d = q.shape
    _, h_kv, l_cap, _ = k.shape
    sl = _c(seq_len, np.int32)
    out = np.empty((B, h_q, d), dtype=np.float64)
    lse = np.empty((B, h_q), dtype=np.float64)
    lib().oracle_dense_decode(_p(q), _p(k), _p(v), _p(sl), B, h_q, h_kv, d, l_cap,
                              float(sm_scale), _p(out), _p(lse))
    return out, lse


def sparse_prefill(q, k, v, idx, count, sm_scale, qrows):
    """Outputs for the listed (sequence, query-block) rows: [n, h_q, 64, d], [n, h_q, 64]."""
    q, k, v = _c(q, np.uint16), _c(k, np.uint16), _c(v, np.uint16)
    B, h_q, L, d = q.shape
    h_kv = k.shape[1]
    idx = _c(idx, np.int32)
    cnt = _c(count, np.int32)
    rows = _c(qrows, np.int32)
    n = rows.size
    out = np.empty((n, h_q, 64, d), dtype=np.float64)
    lse = np.empty((n, h_q, 64), dtype=np.float64)
    lib().oracle_sparse_prefill(_p(q), _p(k), _p(v), L, _p(idx), _p(cnt), idx.shape[1], B, h_q,
                                h_kv, d, 64, float(sm_scale), _p(rows), n, _p(out), _p(lse))
    return out, lse
