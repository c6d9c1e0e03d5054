"""ctypes binding of libspot (include/spot.h).

The functions ``spot_*`` mirror the C ABI one to one: they take torch tensors
(device memory), check dtype / device / contiguity / size, and pass raw
pointers plus the current HIP stream.  Every step of the path runs in the HIP
kernels of libspot.so; there is no fallback: if the library cannot be loaded
on a machine with a GPU, the first call raises.

Convenience wrappers without the ``spot_`` prefix allocate outputs with torch.
"""
from __future__ import annotations

import ctypes
import math
import os
import sys
import threading
from typing import Optional

import torch

from . import build as _build

SPOT_OK = 0
STATUS = {0: "ok", 1: "null pointer", 2: "invalid shape", 3: "unsupported", 4: "invalid rule",
          5: "workspace", 6: "HIP launch error", 7: "fused-step wait expired"}
SPOT_ERR_EXPIRED = 7
KFMT = {"bf16": 0, "int4": 1, "mxfp4": 2, "int8": 3, "mxfp8": 4}
BLK = 64

SYMBOLS = ["spot_status_str", "spot_version", "spot_selector_score",
           "spot_selector_score_q", "spot_selector_score_tokens",
           "spot_selector_score_tokens_blk", "spot_selector_project",
           "spot_selector_project_pooled", "spot_selector_pool",
           "spot_select_blocks",
           "spot_decode_workspace_bytes", "spot_sparse_decode", "spot_sparse_decode_blk",
           "spot_dense_decode",
           "spot_sparse_prefill", "spot_decode_step_workspace_bytes", "spot_decode_step",
           "spot_decode_step_q", "spot_decode_step_static", "spot_decode_step_status",
           "spot_test_force_expiry",
           "spot_probe_stream_read", "spot_probe_sink_words"]


class SpotError(RuntimeError):
    def __init__(self, fn: str, status: int):
        super().__init__(f"{fn} failed: status {status} ({STATUS.get(status, '?')})")
        self.status = status


_lock = threading.Lock()
_lib = None


def load(path: Optional[str] = None):
    """Load libspot.so, building it first only if it does not exist."""
    global _lib
    with _lock:
        if _lib is not None and path is None:
            return _lib
        so = path or _build.SO
        if not os.path.exists(so):
            _build.build()
        elif path is None and _build.stale():
            print(f"warning: {so} is older than its sources; rebuild with "
                  "`python -m paper_2606_22874_amd.build`", file=sys.stderr)
        L = ctypes.CDLL(so)
        P, I, F, Z = ctypes.c_void_p, ctypes.c_int, ctypes.c_float, ctypes.c_size_t
        L.spot_status_str.argtypes = [I]
        L.spot_status_str.restype = ctypes.c_char_p
        L.spot_version.restype = ctypes.c_char_p
        L.spot_selector_score.argtypes = [P, P, P, P, I, I, I, I, I, I, P, P, P]
        L.spot_selector_score_tokens.argtypes = [P, P, P, P, I, I, I, I, I, I, P, P, P]
        L.spot_selector_score_tokens_blk.argtypes = [P, P, P, P, I, I, I, I, I, I, I, P, P, P]
        L.spot_selector_score_q.argtypes = [P, P, I, P, P, P, I, I, I, I, I, I, P, P, P]
        L.spot_selector_project.argtypes = [P, P, P, P, P, I, I, I, I, I, F, P, P, P, I, I, P]
        L.spot_selector_pool.argtypes = [P, P, I, I, I, I, P, P, I, P]
        L.spot_selector_project_pooled.argtypes = [P, P, P, P, P, P, I, I, I, I, I, F, P, P, P,
                                                   P, I, P]
        L.spot_select_blocks.argtypes = [P, I, I, P, F, I, I, I, I, P, P, P, P]
        L.spot_decode_workspace_bytes.argtypes = [I, I, I, I, I]
        L.spot_decode_workspace_bytes.restype = Z
        L.spot_sparse_decode.argtypes = [P, P, P, P, P, P, I, I, I, I, I, I, F, P, P, P, Z, P]
        L.spot_sparse_decode_blk.argtypes = [P, P, P, P, P, P, I, I, I, I, I, I, I, F, P, P, P,
                                             Z, P]
        L.spot_dense_decode.argtypes = [P, P, P, P, I, I, I, I, I, F, P, P, P, Z, P]
        L.spot_sparse_prefill.argtypes = [P, P, P, I, P, P, I, I, I, I, I, F, P, P, P]
        L.spot_decode_step_workspace_bytes.argtypes = [I, I, I, I, I]
        L.spot_decode_step_workspace_bytes.restype = Z
        L.spot_decode_step.argtypes = [P, P, P, P, I, I, I, P, F, I, I, I, I, P, P, P, P, I, I,
                                       I, I, I, F, P, P, P, P, P, P, P, Z, P]
        L.spot_decode_step_q.argtypes = [P, P, I, P, P, P, I, I, I, P, F, I, I, I, I, P, P, P, P,
                                         I, I, I, I, I, F, P, P, P, P, P, P, P, Z, P]
        L.spot_decode_step_static.argtypes = [P, P, P, P, I, I, I, P, F, I, I, I, I, P, P, P, P,
                                              I, I, I, I, I, F, P, P, P, P, P, P, P]
        L.spot_decode_step_status.argtypes = [P, Z, I, I, I, I, I, P]
        L.spot_test_force_expiry.argtypes = [I]
        L.spot_test_force_expiry.restype = None
        L.spot_probe_stream_read.argtypes = [P, Z, P, P]
        L.spot_probe_stream_read.restype = ctypes.c_int32
        L.spot_probe_sink_words.restype = I
        for name in ("spot_selector_score", "spot_selector_score_q", "spot_selector_score_tokens",
                     "spot_selector_score_tokens_blk",
                     "spot_selector_project", "spot_selector_project_pooled",
                     "spot_selector_pool", "spot_select_blocks", "spot_sparse_decode",
                     "spot_sparse_decode_blk",
                     "spot_dense_decode", "spot_sparse_prefill", "spot_decode_step",
                     "spot_decode_step_q", "spot_decode_step_static", "spot_decode_step_status"):
            getattr(L, name).restype = ctypes.c_int32
        if path is None:
            _lib = L
        return L


# ------------------------------------------------------------- marshalling
def _ptr(t: Optional[torch.Tensor]):
    if t is None:
        return None
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream) -> ctypes.c_void_p:
    if stream is None:
        stream = torch.cuda.current_stream()
    if isinstance(stream, torch.cuda.Stream):
        return ctypes.c_void_p(stream.cuda_stream)
    return ctypes.c_void_p(int(stream))


def _dev(t: torch.Tensor, name: str, dtypes, numel: Optional[int] = None):
    if t is None:
        raise ValueError(f"{name} is required")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if t.data_ptr() % 16:
        raise ValueError(f"{name} must start on a 16-byte boundary")
    if dtypes is not None and t.dtype not in dtypes:
        raise ValueError(f"{name}: dtype {t.dtype} not in {dtypes}")
    if numel is not None and t.numel() < numel:
        raise ValueError(f"{name}: {t.numel()} elements, need {numel}")
    return t


BF16 = (torch.bfloat16, torch.int16)
I32 = (torch.int32,)
F32 = (torch.float32,)
U8 = (torch.uint8,)


def _check(fn: str, st: int):
    if st != SPOT_OK:
        raise SpotError(fn, st)


def _sel_cache(k, k_scale, f, n_keys, h_s, d_s, name, scale_name="k_scale"):
    """Checks n_keys selector keys (or queries) of h_s * d_s elements in format f."""
    if f == 0:
        _dev(k, name, BF16, n_keys * h_s * d_s)
        return
    per = h_s * d_s if f in (3, 4) else h_s * d_s // 2      # 8-bit or 4-bit codes
    _dev(k, name, U8 + (torch.int8,), n_keys * per)
    _dev(k_scale, scale_name, (torch.float16, torch.int16) if f in (1, 3) else U8,
         n_keys * h_s * d_s // 32)


# ------------------------------------------------------------- C ABI calls
def spot_selector_score(q_sel, w, k_sel, k_scale, kfmt, n_seq, rows_per_seq, nblk, h_s, d_s,
                        n_valid, scores, stream=None):
    rows = n_seq * rows_per_seq
    f = KFMT[kfmt] if isinstance(kfmt, str) else int(kfmt)
    _dev(q_sel, "q_sel", BF16, rows * h_s * d_s)
    _dev(w, "w", F32, rows * h_s)
    _sel_cache(k_sel, k_scale, f, n_seq * nblk, h_s, d_s, "k_sel")
    if n_valid is not None:
        _dev(n_valid, "n_valid", I32, rows)
    _dev(scores, "scores", F32, rows * nblk)
    _check("spot_selector_score", load().spot_selector_score(
        _ptr(q_sel), _ptr(w), _ptr(k_sel), _ptr(k_scale), f, n_seq, rows_per_seq, nblk, h_s,
        d_s, _ptr(n_valid), _ptr(scores), _stream(stream)))


def spot_selector_score_q(q_sel, q_scale, qfmt, w, k_sel, k_scale, kfmt, n_seq, rows_per_seq,
                          nblk, h_s, d_s, n_valid, scores, stream=None):
    rows = n_seq * rows_per_seq
    qf = KFMT[qfmt] if isinstance(qfmt, str) else int(qfmt)
    f = KFMT[kfmt] if isinstance(kfmt, str) else int(kfmt)
    _sel_cache(q_sel, q_scale, qf, rows, h_s, d_s, "q_sel", "q_scale")
    _dev(w, "w", F32, rows * h_s)
    _sel_cache(k_sel, k_scale, f, n_seq * nblk, h_s, d_s, "k_sel")
    if n_valid is not None:
        _dev(n_valid, "n_valid", I32, rows)
    _dev(scores, "scores", F32, rows * nblk)
    _check("spot_selector_score_q", load().spot_selector_score_q(
        _ptr(q_sel), _ptr(q_scale), qf, _ptr(w), _ptr(k_sel), _ptr(k_scale), f, n_seq,
        rows_per_seq, nblk, h_s, d_s, _ptr(n_valid), _ptr(scores), _stream(stream)))


def _tokens_args(q_sel, w, k_tok, k_scale, kfmt, n_seq, rows_per_seq, l_cap, blk, h_s, d_s,
                 seq_len, scores):
    rows = n_seq * rows_per_seq
    f = KFMT[kfmt] if isinstance(kfmt, str) else int(kfmt)
    _dev(q_sel, "q_sel", BF16, rows * h_s * d_s)
    _dev(w, "w", F32, rows * h_s)
    _sel_cache(k_tok, k_scale, f, n_seq * l_cap, h_s, d_s, "k_tok")
    if seq_len is not None:
        _dev(seq_len, "seq_len", I32, rows)
    _dev(scores, "scores", F32, rows * (l_cap // blk))
    return f


def spot_selector_score_tokens(q_sel, w, k_tok, k_scale, kfmt, n_seq, rows_per_seq, l_cap, h_s,
                               d_s, seq_len, scores, stream=None):
    f = _tokens_args(q_sel, w, k_tok, k_scale, kfmt, n_seq, rows_per_seq, l_cap, 64, h_s, d_s,
                     seq_len, scores)
    _check("spot_selector_score_tokens", load().spot_selector_score_tokens(
        _ptr(q_sel), _ptr(w), _ptr(k_tok), _ptr(k_scale), f, n_seq, rows_per_seq, l_cap, h_s,
        d_s, _ptr(seq_len), _ptr(scores), _stream(stream)))


def spot_selector_score_tokens_blk(q_sel, w, k_tok, k_scale, kfmt, n_seq, rows_per_seq, l_cap,
                                   blk, h_s, d_s, seq_len, scores, stream=None):
    f = _tokens_args(q_sel, w, k_tok, k_scale, kfmt, n_seq, rows_per_seq, l_cap, blk, h_s, d_s,
                     seq_len, scores)
    _check("spot_selector_score_tokens_blk", load().spot_selector_score_tokens_blk(
        _ptr(q_sel), _ptr(w), _ptr(k_tok), _ptr(k_scale), f, n_seq, rows_per_seq, l_cap, blk,
        h_s, d_s, _ptr(seq_len), _ptr(scores), _stream(stream)))


def spot_selector_project(h, w_q, w_k, w_w, pos, rows, d_model, h_s, d_s, rope_dim, rope_base,
                          q_out, w_out, k_cache, rows_per_seq, l_cap, stream=None):
    n_out = h_s * d_s
    _dev(h, "h", BF16, rows * d_model)
    _dev(w_q, "w_q", BF16, n_out * d_model)
    _dev(w_k, "w_k", BF16, n_out * d_model)
    _dev(w_w, "w_w", BF16, h_s * d_model)
    _dev(pos, "pos", I32, rows)
    _dev(q_out, "q_out", BF16, rows * n_out)
    _dev(w_out, "w_out", F32, rows * h_s)
    _dev(k_cache, "k_cache", BF16, (rows // max(rows_per_seq, 1)) * l_cap * n_out)
    _check("spot_selector_project", load().spot_selector_project(
        _ptr(h), _ptr(w_q), _ptr(w_k), _ptr(w_w), _ptr(pos), rows, d_model, h_s, d_s, rope_dim,
        rope_base, _ptr(q_out), _ptr(w_out), _ptr(k_cache), rows_per_seq, l_cap,
        _stream(stream)))


def spot_selector_project_pooled(h, w_q, w_k, w_w, pos, seq_len, n_seq, d_model, h_s, d_s,
                                 rope_dim, rope_base, q_out, w_out, k_cache, k_pool, l_cap,
                                 stream=None):
    n_out = h_s * d_s
    _dev(h, "h", BF16, n_seq * d_model)
    _dev(w_q, "w_q", BF16, n_out * d_model)
    _dev(w_k, "w_k", BF16, n_out * d_model)
    _dev(w_w, "w_w", BF16, h_s * d_model)
    _dev(pos, "pos", I32, n_seq)
    if seq_len is not None:
        _dev(seq_len, "seq_len", I32, n_seq)
    _dev(q_out, "q_out", BF16, n_seq * n_out)
    _dev(w_out, "w_out", F32, n_seq * h_s)
    _dev(k_cache, "k_cache", BF16, n_seq * l_cap * n_out)
    _dev(k_pool, "k_pool", BF16, n_seq * (l_cap // BLK) * n_out)
    _check("spot_selector_project_pooled", load().spot_selector_project_pooled(
        _ptr(h), _ptr(w_q), _ptr(w_k), _ptr(w_w), _ptr(pos), _ptr(seq_len), n_seq, d_model, h_s,
        d_s, rope_dim, rope_base, _ptr(q_out), _ptr(w_out), _ptr(k_cache), _ptr(k_pool), l_cap,
        _stream(stream)))


def spot_selector_pool(k_tok, k_pool, n_seq, l_cap, h_s, d_s, seq_len=None, first_block=None,
                       max_blocks=None, stream=None):
    _dev(k_tok, "k_tok", BF16, n_seq * l_cap * h_s * d_s)
    _dev(k_pool, "k_pool", BF16, n_seq * (l_cap // 64) * h_s * d_s)
    if seq_len is not None:
        _dev(seq_len, "seq_len", I32, n_seq)
    if first_block is not None:
        _dev(first_block, "first_block", I32, n_seq)
    if max_blocks is None:
        max_blocks = l_cap // 64
    _check("spot_selector_pool", load().spot_selector_pool(
        _ptr(k_tok), _ptr(k_pool), n_seq, l_cap, h_s, d_s, _ptr(seq_len), _ptr(first_block),
        max_blocks, _stream(stream)))


def spot_select_blocks(scores, rows, nblk, n_valid, top_p, k_max, k_min, n_sink, n_recent, idx,
                       count, nuc_mass=None, stream=None):
    _dev(scores, "scores", F32, rows * nblk)
    if n_valid is not None:
        _dev(n_valid, "n_valid", I32, rows)
    _dev(idx, "idx", I32, rows * k_max)
    _dev(count, "count", I32, rows)
    if nuc_mass is not None:
        _dev(nuc_mass, "nuc_mass", F32, rows)
    _check("spot_select_blocks", load().spot_select_blocks(
        _ptr(scores), rows, nblk, _ptr(n_valid), float(top_p), k_max, k_min, n_sink, n_recent,
        _ptr(idx), _ptr(count), _ptr(nuc_mass), _stream(stream)))


def spot_decode_workspace_bytes(batch, h_q, h_kv, d, max_blocks) -> int:
    return int(load().spot_decode_workspace_bytes(batch, h_q, h_kv, d, max_blocks))


def spot_sparse_decode(q, k, v, seq_len, idx, count, k_max, batch, h_q, h_kv, d, l_cap,
                       sm_scale, out, lse, ws, stream=None):
    _decode_args(q, k, v, seq_len, idx, count, k_max, batch, h_q, h_kv, d, l_cap, out, lse, ws)
    _check("spot_sparse_decode", load().spot_sparse_decode(
        _ptr(q), _ptr(k), _ptr(v), _ptr(seq_len), _ptr(idx), _ptr(count), k_max, batch, h_q,
        h_kv, d, l_cap, float(sm_scale), _ptr(out), _ptr(lse), _ptr(ws),
        ws.numel() * ws.element_size(), _stream(stream)))


def spot_sparse_decode_blk(q, k, v, seq_len, idx, count, k_max, blk, batch, h_q, h_kv, d, l_cap,
                           sm_scale, out, lse, ws, stream=None):
    _decode_args(q, k, v, seq_len, idx, count, k_max, batch, h_q, h_kv, d, l_cap, out, lse, ws)
    _check("spot_sparse_decode_blk", load().spot_sparse_decode_blk(
        _ptr(q), _ptr(k), _ptr(v), _ptr(seq_len), _ptr(idx), _ptr(count), k_max, blk, batch,
        h_q, h_kv, d, l_cap, float(sm_scale), _ptr(out), _ptr(lse), _ptr(ws),
        ws.numel() * ws.element_size(), _stream(stream)))


def _decode_args(q, k, v, seq_len, idx, count, k_max, batch, h_q, h_kv, d, l_cap, out, lse, ws):
    _dev(q, "q", BF16, batch * h_q * d)
    _dev(k, "k", BF16, batch * h_kv * l_cap * d)
    _dev(v, "v", BF16, batch * h_kv * l_cap * d)
    _dev(seq_len, "seq_len", I32, batch)
    _dev(idx, "idx", I32, batch * k_max)
    _dev(count, "count", I32, batch)
    _dev(out, "out", BF16, batch * h_q * d)
    if lse is not None:
        _dev(lse, "lse", F32, batch * h_q)
    _dev(ws, "ws", None)


def spot_dense_decode(q, k, v, seq_len, batch, h_q, h_kv, d, l_cap, sm_scale, out, lse, ws,
                      stream=None):
    _dev(q, "q", BF16, batch * h_q * d)
    _dev(k, "k", BF16, batch * h_kv * l_cap * d)
    _dev(v, "v", BF16, batch * h_kv * l_cap * d)
    _dev(seq_len, "seq_len", I32, batch)
    _dev(out, "out", BF16, batch * h_q * d)
    if lse is not None:
        _dev(lse, "lse", F32, batch * h_q)
    _dev(ws, "ws", None)
    _check("spot_dense_decode", load().spot_dense_decode(
        _ptr(q), _ptr(k), _ptr(v), _ptr(seq_len), batch, h_q, h_kv, d, l_cap, float(sm_scale),
        _ptr(out), _ptr(lse), _ptr(ws), ws.numel() * ws.element_size(), _stream(stream)))


def spot_sparse_prefill(q, k, v, L, idx, count, k_max, batch, h_q, h_kv, d, sm_scale, out, lse,
                        stream=None):
    nqb = L // BLK
    _dev(q, "q", BF16, batch * h_q * L * d)
    _dev(k, "k", BF16, batch * h_kv * L * d)
    _dev(v, "v", BF16, batch * h_kv * L * d)
    _dev(idx, "idx", I32, batch * nqb * k_max)
    _dev(count, "count", I32, batch * nqb)
    _dev(out, "out", BF16, batch * h_q * L * d)
    if lse is not None:
        _dev(lse, "lse", F32, batch * h_q * L)
    _check("spot_sparse_prefill", load().spot_sparse_prefill(
        _ptr(q), _ptr(k), _ptr(v), L, _ptr(idx), _ptr(count), k_max, batch, h_q, h_kv, d,
        float(sm_scale), _ptr(out), _ptr(lse), _stream(stream)))


def spot_decode_step_workspace_bytes(batch, h_q, h_kv, d, k_max) -> int:
    return int(load().spot_decode_step_workspace_bytes(batch, h_q, h_kv, d, k_max))


def spot_decode_step(q_sel, w, k_sel, k_scale, kfmt, h_s, d_s, n_valid, top_p, k_max, k_min,
                     n_sink, n_recent, q, k, v, seq_len, batch, h_q, h_kv, d, l_cap, sm_scale,
                     scores, idx, count, nuc_mass, out, lse, ws, stream=None, q_scale=None,
                     qfmt="bf16"):
    """spot_decode_step, or spot_decode_step_q when qfmt is not BF16."""
    nblk = l_cap // BLK
    f = KFMT[kfmt] if isinstance(kfmt, str) else int(kfmt)
    qf = KFMT[qfmt] if isinstance(qfmt, str) else int(qfmt)
    _sel_cache(q_sel, q_scale, qf, batch, h_s, d_s, "q_sel", "q_scale")
    _dev(w, "w", F32, batch * h_s)
    _sel_cache(k_sel, k_scale, f, batch * nblk, h_s, d_s, "k_sel")
    if n_valid is not None:
        _dev(n_valid, "n_valid", I32, batch)
    _dev(q, "q", BF16, batch * h_q * d)
    _dev(k, "k", BF16, batch * h_kv * l_cap * d)
    _dev(v, "v", BF16, batch * h_kv * l_cap * d)
    _dev(seq_len, "seq_len", I32, batch)
    _dev(scores, "scores", F32, batch * nblk)
    _dev(idx, "idx", I32, batch * k_max)
    _dev(count, "count", I32, batch)
    if nuc_mass is not None:
        _dev(nuc_mass, "nuc_mass", F32, batch)
    _dev(out, "out", BF16, batch * h_q * d)
    if lse is not None:
        _dev(lse, "lse", F32, batch * h_q)
    _dev(ws, "ws", None)
    rest = (f, h_s, d_s, _ptr(n_valid), float(top_p), k_max, k_min, n_sink, n_recent, _ptr(q),
            _ptr(k), _ptr(v), _ptr(seq_len), batch, h_q, h_kv, d, l_cap, float(sm_scale),
            _ptr(scores), _ptr(idx), _ptr(count), _ptr(nuc_mass), _ptr(out), _ptr(lse), _ptr(ws),
            ws.numel() * ws.element_size(), _stream(stream))
    if qf == 0:
        _check("spot_decode_step", load().spot_decode_step(
            _ptr(q_sel), _ptr(w), _ptr(k_sel), _ptr(k_scale), *rest))
    else:
        _check("spot_decode_step_q", load().spot_decode_step_q(
            _ptr(q_sel), _ptr(q_scale), qf, _ptr(w), _ptr(k_sel), _ptr(k_scale), *rest))


def spot_decode_step_static(q_sel, w, k_sel, k_scale, kfmt, h_s, d_s, n_valid, top_p, k_max,
                            k_min, n_sink, n_recent, q, k, v, seq_len, batch, h_q, h_kv, d, l_cap,
                            sm_scale, scores, idx, count, nuc_mass, out, lse, stream=None):
    """spot_decode_step on the device's static scratch (no workspace argument)."""
    nblk = l_cap // BLK
    f = KFMT[kfmt] if isinstance(kfmt, str) else int(kfmt)
    _dev(q_sel, "q_sel", BF16, batch * h_s * d_s)
    _dev(w, "w", F32, batch * h_s)
    _sel_cache(k_sel, k_scale, f, batch * nblk, h_s, d_s, "k_sel")
    if n_valid is not None:
        _dev(n_valid, "n_valid", I32, batch)
    _dev(q, "q", BF16, batch * h_q * d)
    _dev(k, "k", BF16, batch * h_kv * l_cap * d)
    _dev(v, "v", BF16, batch * h_kv * l_cap * d)
    _dev(seq_len, "seq_len", I32, batch)
    _dev(scores, "scores", F32, batch * nblk)
    _dev(idx, "idx", I32, batch * k_max)
    _dev(count, "count", I32, batch)
    if nuc_mass is not None:
        _dev(nuc_mass, "nuc_mass", F32, batch)
    _dev(out, "out", BF16, batch * h_q * d)
    if lse is not None:
        _dev(lse, "lse", F32, batch * h_q)
    _check("spot_decode_step_static", load().spot_decode_step_static(
        _ptr(q_sel), _ptr(w), _ptr(k_sel), _ptr(k_scale), f, h_s, d_s, _ptr(n_valid),
        float(top_p), k_max, k_min, n_sink, n_recent, _ptr(q), _ptr(k), _ptr(v), _ptr(seq_len),
        batch, h_q, h_kv, d, l_cap, float(sm_scale), _ptr(scores), _ptr(idx), _ptr(count),
        _ptr(nuc_mass), _ptr(out), _ptr(lse), _stream(stream)))


def spot_decode_step_status(ws, batch, h_q, h_kv, d, k_max, stream=None) -> int:
    """Status of a fused-step workspace (ws None: the device's static scratch
    of spot_decode_step_static): SPOT_OK, or SPOT_ERR_EXPIRED after a bounded
    wait expired (the workspace is then zero-filled again).  Any other status
    raises."""
    if ws is not None:
        _dev(ws, "ws", None)
    st = load().spot_decode_step_status(_ptr(ws), 0 if ws is None else ws.numel() * ws.element_size(),
                                        batch, h_q, h_kv, d, k_max, _stream(stream))
    if st not in (SPOT_OK, SPOT_ERR_EXPIRED):
        raise SpotError("spot_decode_step_status", st)
    return int(st)


def spot_test_force_expiry(on: bool):
    load().spot_test_force_expiry(1 if on else 0)


def spot_probe_stream_read(buf, sink, stream=None):
    _dev(buf, "buf", None)
    _dev(sink, "sink", F32, int(load().spot_probe_sink_words()))
    _check("spot_probe_stream_read", load().spot_probe_stream_read(
        _ptr(buf), buf.numel() * buf.element_size(), _ptr(sink), _stream(stream)))


# --------------------------------------------------- allocating wrappers
def selector_score(q_sel, w, k_sel, k_scale=None, kfmt="bf16", rows_per_seq=1, n_valid=None,
                   nblk=None, out=None, stream=None):
    """Block scores [rows, nblk] float32 for q_sel [rows, h_s, d_s]."""
    h_s, d_s = q_sel.shape[-2], q_sel.shape[-1]
    rows = q_sel.numel() // (h_s * d_s)
    n_seq = rows // rows_per_seq
    if nblk is None:
        f = KFMT.get(kfmt, kfmt)
        per = h_s * d_s if f in (0, 3, 4) else h_s * d_s // 2
        nblk = k_sel.numel() // (n_seq * per)
    if out is None:
        out = torch.empty((rows, nblk), dtype=torch.float32, device=q_sel.device)
    spot_selector_score(q_sel, w, k_sel, k_scale, kfmt, n_seq, rows_per_seq, nblk, h_s, d_s,
                        n_valid, out, stream)
    return out


def selector_score_tokens(q_sel, w, k_tok, k_scale=None, kfmt="bf16", rows_per_seq=1,
                          seq_len=None, l_cap=None, out=None, stream=None, blk=64):
    """Per-block maximum of per-token scores [rows, l_cap // blk] float32
    (blocks of 64 tokens, or 16: the paper's selector block)."""
    h_s, d_s = q_sel.shape[-2], q_sel.shape[-1]
    rows = q_sel.numel() // (h_s * d_s)
    n_seq = rows // rows_per_seq
    if l_cap is None:
        f = KFMT.get(kfmt, kfmt)
        per = h_s * d_s if f in (0, 3, 4) else h_s * d_s // 2
        l_cap = k_tok.numel() // (n_seq * per)
    if out is None:
        out = torch.empty((rows, l_cap // blk), dtype=torch.float32, device=q_sel.device)
    if blk == 64:
        spot_selector_score_tokens(q_sel, w, k_tok, k_scale, kfmt, n_seq, rows_per_seq, l_cap,
                                   h_s, d_s, seq_len, out, stream)
    else:
        spot_selector_score_tokens_blk(q_sel, w, k_tok, k_scale, kfmt, n_seq, rows_per_seq,
                                       l_cap, blk, h_s, d_s, seq_len, out, stream)
    return out


def select_blocks(scores, rule, n_valid=None, idx=None, count=None, nuc_mass=None, stream=None):
    rows, nblk = scores.shape
    dev = scores.device
    if idx is None:
        idx = torch.empty((rows, rule.k_max), dtype=torch.int32, device=dev)
    if count is None:
        count = torch.empty(rows, dtype=torch.int32, device=dev)
    if nuc_mass is None:
        nuc_mass = torch.empty(rows, dtype=torch.float32, device=dev)
    spot_select_blocks(scores, rows, nblk, n_valid, rule.top_p, rule.k_max, rule.k_min,
                       rule.n_sink, rule.n_recent, idx, count, nuc_mass, stream)
    return idx, count, nuc_mass


def decode_workspace(batch, h_q, h_kv, d, max_blocks, device="cuda"):
    """Zero-filled decode workspace (the library keeps it zeroed between calls)."""
    n = spot_decode_workspace_bytes(batch, h_q, h_kv, d, max_blocks)
    return torch.zeros(max(n, 16), dtype=torch.uint8, device=device)


def sparse_decode(q, k, v, seq_len, idx, count, sm_scale=None, out=None, lse=None, ws=None,
                  stream=None, blk=64):
    """Attention over the selected blocks of blk tokens (64, or 16: the
    paper's selector block); returns (out [batch, h_q, d] BF16, lse)."""
    batch, h_q, d = q.shape
    _, h_kv, l_cap, _ = k.shape
    k_max = idx.shape[-1]
    sm_scale = 1.0 / math.sqrt(d) if sm_scale is None else sm_scale
    if out is None:
        out = torch.empty((batch, h_q, d), dtype=torch.bfloat16, device=q.device)
    if lse is None:
        lse = torch.empty((batch, h_q), dtype=torch.float32, device=q.device)
    if ws is None:
        ws = decode_workspace(batch, h_q, h_kv, d, k_max, q.device)
    if blk == 64:
        spot_sparse_decode(q, k, v, seq_len, idx, count, k_max, batch, h_q, h_kv, d, l_cap,
                           sm_scale, out, lse, ws, stream)
    else:
        spot_sparse_decode_blk(q, k, v, seq_len, idx, count, k_max, blk, batch, h_q, h_kv, d,
                               l_cap, sm_scale, out, lse, ws, stream)
    return out, lse


def dense_decode(q, k, v, seq_len, sm_scale=None, out=None, lse=None, ws=None, stream=None):
    batch, h_q, d = q.shape
    _, h_kv, l_cap, _ = k.shape
    sm_scale = 1.0 / math.sqrt(d) if sm_scale is None else sm_scale
    if out is None:
        out = torch.empty((batch, h_q, d), dtype=torch.bfloat16, device=q.device)
    if lse is None:
        lse = torch.empty((batch, h_q), dtype=torch.float32, device=q.device)
    if ws is None:
        ws = decode_workspace(batch, h_q, h_kv, d, l_cap // BLK, q.device)
    spot_dense_decode(q, k, v, seq_len, batch, h_q, h_kv, d, l_cap, sm_scale, out, lse, ws,
                      stream)
    return out, lse


def sparse_prefill(q, k, v, idx, count, sm_scale=None, out=None, lse=None, stream=None):
    batch, h_q, L, d = q.shape
    h_kv = k.shape[1]
    k_max = idx.shape[-1]
    sm_scale = 1.0 / math.sqrt(d) if sm_scale is None else sm_scale
    if out is None:
        out = torch.empty_like(q, dtype=torch.bfloat16)
    if lse is None:
        lse = torch.empty((batch, h_q, L), dtype=torch.float32, device=q.device)
    spot_sparse_prefill(q, k, v, L, idx, count, k_max, batch, h_q, h_kv, d, sm_scale, out, lse,
                        stream)
    return out, lse


def step_workspace(batch, h_q, h_kv, d, k_max, device="cuda"):
    """Zero-filled workspace of spot_decode_step (kept zeroed between calls)."""
    n = spot_decode_step_workspace_bytes(batch, h_q, h_kv, d, k_max)
    return torch.zeros(max(n, 16), dtype=torch.uint8, device=device)


def decode_step(q_sel, w, k_sel, q, k, v, seq_len, rule, k_scale=None, kfmt="bf16",
                n_valid=None, sm_scale=None, ws=None, stream=None, q_scale=None, qfmt="bf16"):
    """One fused decode step: (scores, idx, count, nuc_mass, out, lse).
    Quantized queries (qfmt = kfmt, codes in q_sel) go through spot_decode_step_q."""
    batch, h_q, d = q.shape
    _, h_kv, l_cap, _ = k.shape
    qf = KFMT[qfmt] if isinstance(qfmt, str) else int(qfmt)
    h_s, d_s = q_sel.shape[-2], q_sel.shape[-1] * (2 if qf in (1, 2) else 1)   # 4-bit codes
    nblk = l_cap // BLK
    dev = q.device
    sm_scale = 1.0 / math.sqrt(d) if sm_scale is None else sm_scale
    scores = torch.empty((batch, nblk), dtype=torch.float32, device=dev)
    idx = torch.empty((batch, rule.k_max), dtype=torch.int32, device=dev)
    count = torch.empty(batch, dtype=torch.int32, device=dev)
    mass = torch.empty(batch, dtype=torch.float32, device=dev)
    out = torch.empty((batch, h_q, d), dtype=torch.bfloat16, device=dev)
    lse = torch.empty((batch, h_q), dtype=torch.float32, device=dev)
    if ws is None:
        ws = step_workspace(batch, h_q, h_kv, d, rule.k_max, dev)
    spot_decode_step(q_sel, w, k_sel, k_scale, kfmt, h_s, d_s, n_valid, rule.top_p, rule.k_max,
                     rule.k_min, rule.n_sink, rule.n_recent, q, k, v, seq_len, batch, h_q, h_kv,
                     d, l_cap, sm_scale, scores, idx, count, mass, out, lse, ws, stream,
                     q_scale=q_scale, qfmt=qfmt)
    return scores, idx, count, mass, out, lse


# ------------------------------------------------------- host helpers
def to_device_bf16(a, device="cuda") -> torch.Tensor:
    """uint16 BF16 bit patterns (numpy) -> torch.bfloat16 device tensor."""
    import numpy as np
    t = torch.from_numpy(np.ascontiguousarray(a).view(np.int16))
    return t.to(device).view(torch.bfloat16)


def bf16_to_float_host(t: torch.Tensor):
    return t.detach().float().cpu().numpy()
