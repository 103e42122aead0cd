"""Python front-end of the CPU oracle for Reformer LSH attention.

TEST INFRASTRUCTURE ONLY.  The oracle exists to check the GPU library.  Only
the test suite, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import it.  The product package never imports it and it
never imports the product package.

Every function takes and returns NumPy arrays.  Floating-point inputs are
converted to float64 (exact for bf16 and fp32 values) and the arithmetic is
done in float64 by ``lsh_oracle.c``; see that file for layouts and for the
paper passages each step follows.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "lsh_oracle.c")
# LSH_ORACLE_LIB points at another build of the same source (the sanitizer
# test loads an instrumented one); it is never built here
_LIB = os.environ.get("LSH_ORACLE_LIB") or os.path.join(_HERE, "liblsh_oracle.so")
_FIXED = "LSH_ORACLE_LIB" in os.environ
_lib = None

_i64 = ctypes.c_int64
_f64 = ctypes.c_double
_ptr = ctypes.c_void_p


def build(force: bool = False) -> str:
    """Compile lsh_oracle.c into liblsh_oracle.so with gcc and OpenMP."""
    if _FIXED:
        return _LIB
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + f".tmp{os.getpid()}"
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared",
                               "-Wall", "-Wextra", _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        build()
        lib = ctypes.CDLL(_LIB)
        lib.lsh_ref_hash.argtypes = [_i64, _i64, _i64, _i64, _i64, _i64, _ptr, _ptr, _ptr, _ptr]
        lib.lsh_ref_sort_permute.argtypes = [_i64, _i64, _i64, _ptr, _ptr, _ptr]
        lib.lsh_ref_chunk_attn_fwd.argtypes = [_i64, _i64, _i64, _i64, _i64, _i64, ctypes.c_int,
                                               ctypes.c_int, _f64, _f64, _ptr, _ptr, _ptr, _ptr,
                                               _ptr, _ptr]
        lib.lsh_ref_combine_rounds.argtypes = [_i64, _i64, _i64, _i64, _ptr, _ptr, _ptr, _ptr, _ptr]
        lib.lsh_ref_chunk_attn_bwd.argtypes = [_i64, _i64, _i64, _i64, _i64, _i64, ctypes.c_int,
                                               ctypes.c_int, _f64, _f64, _ptr, _ptr, _ptr, _ptr,
                                               _ptr, _ptr, _ptr, _ptr, _ptr]
        lib.lsh_ref_dense_attn_fwd.argtypes = [_i64, _i64, _i64, ctypes.c_int, _f64, _f64, _ptr,
                                               _ptr, _i64, _ptr, _ptr, _ptr]
        lib.lsh_ref_num_threads.argtypes = []
        for name in ("lsh_ref_num_threads", "lsh_ref_hash", "lsh_ref_sort_permute", "lsh_ref_chunk_attn_fwd",
                     "lsh_ref_combine_rounds", "lsh_ref_chunk_attn_bwd", "lsh_ref_dense_attn_fwd"):
            getattr(lib, name).restype = ctypes.c_int
        _lib = lib
    return _lib


def num_threads() -> int:
    """Threads the oracle's OpenMP loops use."""
    return int(_load().lsh_ref_num_threads())


def _f(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.float64)


def _i(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.int32)


def _p(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def _check(rc: int, what: str) -> None:
    if rc != 0:
        raise RuntimeError(f"oracle {what} failed with status {rc}")


def lsh_hash(q, R):
    """Bucket ids [B,H,L,n_rounds] and near-tie flags for q [B,H,L,d] and
    R [n_r,d,n_b/2] (shared by every head) or [H,n_r,d,n_b/2] (one per head)."""
    q, R = _f(q), _f(R)
    B, H, L, d = q.shape
    if R.ndim == 4:
        assert R.shape[0] == H, "one R per head"
        H_R = H
    else:
        H_R = 1
    n_rounds, dR, half = R.shape[-3:]
    assert dR == d
    buckets = np.empty((B, H, L, n_rounds), np.int32)
    near_tie = np.empty((B, H, L, n_rounds), np.uint8)
    _check(_load().lsh_ref_hash(B * H, L, d, 2 * half, n_rounds, H_R, _p(q), _p(R),
                                _p(buckets), _p(near_tie)), "hash")
    return buckets, near_tie.astype(bool)


def lsh_sort_permute(buckets):
    """perm, undo [B,H,n_rounds,L] for bucket ids [B,H,L,n_rounds]."""
    buckets = _i(buckets)
    B, H, L, n_rounds = buckets.shape
    perm = np.empty((B, H, n_rounds, L), np.int32)
    undo = np.empty((B, H, n_rounds, L), np.int32)
    _check(_load().lsh_ref_sort_permute(B * H, L, n_rounds, _p(buckets), _p(perm), _p(undo)),
           "sort_permute")
    return perm, undo


def lsh_chunk_attn_fwd(q, v, buckets, perm, chunk, causal, scale=None, self_mask=1e5,
                       after=0, across=False):
    """Per-round outputs o_rounds [B,H,n_r,L,d] and lse_rounds [B,H,n_r,L], sorted order.
    after: look-ahead chunks in the window; across: attend across buckets."""
    q, v, buckets, perm = _f(q), _f(v), _i(buckets), _i(perm)
    B, H, L, d = q.shape
    n_rounds = buckets.shape[-1]
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    o_rounds = np.empty((B, H, n_rounds, L, d), np.float64)
    lse_rounds = np.empty((B, H, n_rounds, L), np.float64)
    _check(_load().lsh_ref_chunk_attn_fwd(B * H, L, d, n_rounds, chunk, int(after),
                                          int(bool(across)), int(bool(causal)),
                                          float(scale), float(self_mask), _p(q), _p(v),
                                          _p(buckets), _p(perm), _p(o_rounds), _p(lse_rounds)),
           "chunk_attn_fwd")
    return o_rounds, lse_rounds


def dense_attn_fwd(q, v, causal, scale=None, self_mask=1e5, rows=None):
    """Full shared-QK attention (the memory-efficient baseline of Sec. 2):
    out [B,H,L,d] and lse [B,H,L]; or, for `rows` (flat indices b*H*L + h*L + i),
    out [len(rows), d] and lse [len(rows)] of those rows only."""
    q, v = _f(q), _f(v)
    B, H, L, d = q.shape
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    if rows is None:
        sel, n_sel = None, B * H * L
        out = np.empty((B, H, L, d), np.float64)
        lse = np.empty((B, H, L), np.float64)
    else:
        sel = np.ascontiguousarray(rows, dtype=np.int64)
        n_sel = len(sel)
        out = np.empty((n_sel, d), np.float64)
        lse = np.empty((n_sel,), np.float64)
    _check(_load().lsh_ref_dense_attn_fwd(B * H, L, d, int(bool(causal)), float(scale),
                                          float(self_mask), _p(q), _p(v), n_sel,
                                          None if sel is None else _p(sel), _p(out), _p(lse)),
           "dense_attn_fwd")
    return out, lse


def lsh_combine_rounds(o_rounds, lse_rounds, undo):
    """Unsorted output [B,H,L,d] and total log-partition [B,H,L]."""
    o_rounds, lse_rounds, undo = _f(o_rounds), _f(lse_rounds), _i(undo)
    B, H, n_rounds, L, d = o_rounds.shape
    out = np.empty((B, H, L, d), np.float64)
    lse = np.empty((B, H, L), np.float64)
    _check(_load().lsh_ref_combine_rounds(B * H, L, d, n_rounds, _p(o_rounds), _p(lse_rounds),
                                          _p(undo), _p(out), _p(lse)), "combine_rounds")
    return out, lse


def lsh_chunk_attn_bwd(q, v, out, dout, lse_total, buckets, perm, chunk, causal,
                       scale=None, self_mask=1e5, after=0, across=False):
    """dq, dv [B,H,L,d] for upstream gradient dout, buckets held fixed."""
    q, v, out, dout, lse_total = _f(q), _f(v), _f(out), _f(dout), _f(lse_total)
    buckets, perm = _i(buckets), _i(perm)
    B, H, L, d = q.shape
    n_rounds = buckets.shape[-1]
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    dq = np.empty((B, H, L, d), np.float64)
    dv = np.empty((B, H, L, d), np.float64)
    _check(_load().lsh_ref_chunk_attn_bwd(B * H, L, d, n_rounds, chunk, int(after),
                                          int(bool(across)), int(bool(causal)),
                                          float(scale), float(self_mask), _p(q), _p(v), _p(out),
                                          _p(dout), _p(lse_total), _p(buckets), _p(perm),
                                          _p(dq), _p(dv)), "chunk_attn_bwd")
    return dq, dv


def lsh_attention_fwd(q, v, R, chunk, causal, scale=None, self_mask=1e5, after=0,
                      across=False):
    """The whole forward: hash, sort, chunked attention per round, combine.
    R: [n_r,d,n_b/2] shared, or [H,n_r,d,n_b/2] one per head.

    Returns a dict with every intermediate so tests can compare stage by stage.
    """
    buckets, near_tie = lsh_hash(q, R)
    perm, undo = lsh_sort_permute(buckets)
    o_rounds, lse_rounds = lsh_chunk_attn_fwd(q, v, buckets, perm, chunk, causal, scale, self_mask,
                                              after, across)
    out, lse = lsh_combine_rounds(o_rounds, lse_rounds, undo)
    return dict(buckets=buckets, near_tie=near_tie, perm=perm, undo=undo, o_rounds=o_rounds,
                lse_rounds=lse_rounds, out=out, lse=lse)
