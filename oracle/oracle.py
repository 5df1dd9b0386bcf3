"""ctypes binding of the fp64 CPU attention oracle (``oracle_attn.c``).

TEST INFRASTRUCTURE ONLY: the test suite, the smoke check and the
benchmark's CPU-baseline leg may import this module; the product path must
not.  It shares no code with the HIP library.

Inputs are raw bf16 bit patterns (``numpy.uint16``), exactly the bits the
GPU receives; outputs are ``numpy.float64``.  See ``oracle_attn.c`` for the
definition (plain softmax(Q K^T * scale + mask) V with a natural-log LSE,
grouped heads, bottom-right causal alignment, clamped lengths).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle_attn.c")
_LIB = os.path.join(_HERE, "liboracle_attn.so")

_u16p = ctypes.POINTER(ctypes.c_uint16)
_i32p = ctypes.POINTER(ctypes.c_int32)
_f64p = ctypes.POINTER(ctypes.c_double)

_lib = None


def build(src: str = _SRC, out: str = _LIB) -> str:
    """Compile the oracle with plain gcc (no -ffast-math, libm only)."""
    cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-pthread",
           "-fno-fast-math", "-ffp-contract=off", src, "-o", out, "-lm"]
    subprocess.run(cmd, check=True)
    return out


def load(path: str | None = None):
    """Load (building first if absent) and return the ctypes handle."""
    global _lib
    if path is not None:
        return _declare(ctypes.CDLL(path))
    if _lib is None:
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
            build()
        _lib = _declare(ctypes.CDLL(_LIB))
    return _lib


def _declare(lib):
    i, d = ctypes.c_int, ctypes.c_double
    lib.oracle_attn_fwd.argtypes = [_u16p, _u16p, _u16p, i, i, i, i, i, i, i, d,
                                    _i32p, _i32p, i, _f64p, _f64p, i]
    lib.oracle_attn_fwd.restype = i
    lib.oracle_attn_probs.argtypes = [_u16p, _u16p, i, i, i, i, i, i, i, d, _i32p, _f64p]
    lib.oracle_attn_probs.restype = i
    lib.oracle_decode.argtypes = [_u16p, _u16p, _u16p, i, i, i, i, i, d, _i32p,
                                  _f64p, _f64p, i]
    lib.oracle_decode.restype = i
    lib.oracle_lse_combine.argtypes = [_f64p, _f64p, i, i, i, _f64p, _f64p]
    lib.oracle_lse_combine.restype = i
    lib.oracle_decode_split.argtypes = [_u16p, _u16p, _u16p, i, i, i, i, i, d,
                                        _i32p, i, _f64p, _f64p, _f64p, _f64p]
    lib.oracle_decode_split.restype = i
    lib.oracle_decode_paged.argtypes = [_u16p, _u16p, _u16p, _i32p, i, i, i, i, i, i, i, d,
                                        _i32p, _f64p, _f64p]
    lib.oracle_decode_paged.restype = i
    lib.oracle_attn_fwd_varlen.argtypes = [_u16p, _u16p, _u16p, _i32p, _i32p, i, i, i, i, i, i,
                                           i, d, _f64p, _f64p]
    lib.oracle_attn_fwd_varlen.restype = i
    lib.oracle_attn_fwd_ragged_paged.argtypes = [_u16p, _u16p, _u16p, _i32p, _i32p, _i32p, i, i,
                                                 i, i, i, i, i, i, i, d, _f64p, _f64p]
    lib.oracle_attn_fwd_ragged_paged.restype = i
    lib.oracle_attn_bwd.argtypes = [_u16p, _u16p, _u16p, _u16p, i, i, i, i, i, i, i, d, _i32p,
                                    _f64p, _f64p, _f64p]
    lib.oracle_attn_bwd.restype = i
    lib.oracle_mla_decode.argtypes = [_u16p, _u16p, i, i, i, i, i, d, _i32p, _f64p, _f64p]
    lib.oracle_mla_decode.restype = i
    lib.oracle_version.restype = i
    return lib


def default_threads() -> int:
    # the GPU machine gives one GPU a share of 16 host cores
    return max(1, min(16, os.cpu_count() or 1))


def _u16(a) -> np.ndarray:
    a = np.ascontiguousarray(a)
    if a.dtype != np.uint16:
        raise TypeError("oracle inputs are bf16 bit patterns (uint16)")
    return a


def _ptr(a, t):
    return a.ctypes.data_as(t)


def _seqlens(kv_seqlens, B):
    if kv_seqlens is None:
        return None
    s = np.ascontiguousarray(np.asarray(kv_seqlens, dtype=np.int32))
    if s.shape != (B,):
        raise ValueError("kv_seqlens must have shape [B]")
    return s


def attn_fwd(q, k, v, *, causal: bool, scale: float, kv_seqlens=None,
             rows=None, threads: int | None = None, lib=None):
    """Plain-definition attention.  q [B,Hq,Sq,D], k/v [B,Hkv,Skv,D] uint16.

    rows: optional int array [B,Hq,R] of query rows to evaluate.
    Returns (o [B,Hq,R,D] float64, lse [B,Hq,R] float64).
    """
    lib = lib or load()
    q, k, v = _u16(q), _u16(k), _u16(v)
    B, Hq, Sq, D = q.shape
    Bk, Hkv, Skv, Dk = k.shape
    if v.shape != k.shape or Bk != B or Dk != D:
        raise ValueError("shape mismatch")
    sl = _seqlens(kv_seqlens, B)
    if rows is not None:
        rows = np.ascontiguousarray(np.asarray(rows, dtype=np.int32))
        if rows.ndim != 3 or rows.shape[:2] != (B, Hq):
            raise ValueError("rows must have shape [B,Hq,R]")
        R = rows.shape[2]
    else:
        R = Sq
    o = np.empty((B, Hq, R, D), np.float64)
    lse = np.empty((B, Hq, R), np.float64)
    rc = lib.oracle_attn_fwd(_ptr(q, _u16p), _ptr(k, _u16p), _ptr(v, _u16p),
                             B, Hq, Hkv, Sq, Skv, D, int(bool(causal)), float(scale),
                             _ptr(sl, _i32p) if sl is not None else None,
                             _ptr(rows, _i32p) if rows is not None else None, R,
                             _ptr(o, _f64p), _ptr(lse, _f64p),
                             threads or default_threads())
    if rc != 0:
        raise ValueError(f"oracle_attn_fwd failed ({rc})")
    return o, lse


def attn_probs(q, k, *, causal: bool, scale: float, kv_seqlens=None, lib=None):
    """Normalised attention weights P [B,Hq,Sq,Skv] (0 where masked)."""
    lib = lib or load()
    q, k = _u16(q), _u16(k)
    B, Hq, Sq, D = q.shape
    _, Hkv, Skv, _ = k.shape
    sl = _seqlens(kv_seqlens, B)
    p = np.empty((B, Hq, Sq, Skv), np.float64)
    rc = lib.oracle_attn_probs(_ptr(q, _u16p), _ptr(k, _u16p), B, Hq, Hkv, Sq, Skv, D,
                               int(bool(causal)), float(scale),
                               _ptr(sl, _i32p) if sl is not None else None,
                               _ptr(p, _f64p))
    if rc != 0:
        raise ValueError(f"oracle_attn_probs failed ({rc})")
    return p


def decode(q, k_cache, v_cache, kv_seqlens, *, scale: float,
           threads: int | None = None, lib=None):
    """Decode step.  q [B,Hq,D], caches [B,Hkv,Smax,D] -> (o [B,Hq,D], lse [B,Hq])."""
    lib = lib or load()
    q, kc, vc = _u16(q), _u16(k_cache), _u16(v_cache)
    B, Hq, D = q.shape
    _, Hkv, Smax, _ = kc.shape
    sl = _seqlens(kv_seqlens, B)
    o = np.empty((B, Hq, D), np.float64)
    lse = np.empty((B, Hq), np.float64)
    rc = lib.oracle_decode(_ptr(q, _u16p), _ptr(kc, _u16p), _ptr(vc, _u16p),
                           B, Hq, Hkv, Smax, D, float(scale), _ptr(sl, _i32p),
                           _ptr(o, _f64p), _ptr(lse, _f64p), threads or default_threads())
    if rc != 0:
        raise ValueError(f"oracle_decode failed ({rc})")
    return o, lse


def attn_bwd(q, k, v, dout, *, causal: bool, scale: float, kv_seqlens=None, lib=None):
    """Gradients of L = <dout, O> for q [B,Hq,Sq,D], k/v [B,Hkv,Skv,D] (bf16 bits)
    -> (dq, dk, dv) float64, same shapes."""
    lib = lib or load()
    q, k, v, do = _u16(q), _u16(k), _u16(v), _u16(dout)
    B, Hq, Sq, D = q.shape
    _, Hkv, Skv, _ = k.shape
    if do.shape != q.shape:
        raise ValueError("dout must have q's shape")
    sl = None if kv_seqlens is None else _seqlens(kv_seqlens, B)
    dq = np.empty(q.shape, np.float64)
    dk = np.empty(k.shape, np.float64)
    dv = np.empty(v.shape, np.float64)
    rc = lib.oracle_attn_bwd(_ptr(q, _u16p), _ptr(k, _u16p), _ptr(v, _u16p), _ptr(do, _u16p),
                             B, Hq, Hkv, Sq, Skv, D, int(bool(causal)), float(scale),
                             None if sl is None else _ptr(sl, _i32p), _ptr(dq, _f64p),
                             _ptr(dk, _f64p), _ptr(dv, _f64p))
    if rc != 0:
        raise ValueError(f"oracle_attn_bwd failed ({rc})")
    return dq, dk, dv


def attn_fwd_varlen(q, k, v, cu_seqlens_q, cu_seqlens_k, *, causal: bool, scale: float,
                    lib=None):
    """Packed ragged forward.  q [total_q,Hq,D], k/v [total_k,Hkv,D], cu_seqlens int32
    [B+1] -> (o [total_q,Hq,D], lse [Hq,total_q]); rows no sequence owns stay NaN."""
    lib = lib or load()
    q, k, v = _u16(q), _u16(k), _u16(v)
    total_q, Hq, D = q.shape
    total_k, Hkv, _ = k.shape
    cq = np.ascontiguousarray(cu_seqlens_q, dtype=np.int32)
    ck = np.ascontiguousarray(cu_seqlens_k, dtype=np.int32)
    if cq.shape != ck.shape or cq.ndim != 1 or cq.shape[0] < 2:
        raise ValueError("cu_seqlens_q / cu_seqlens_k must both be [B+1]")
    B = cq.shape[0] - 1
    o = np.full((total_q, Hq, D), np.nan, np.float64)
    lse = np.full((Hq, total_q), np.nan, np.float64)
    rc = lib.oracle_attn_fwd_varlen(_ptr(q, _u16p), _ptr(k, _u16p), _ptr(v, _u16p),
                                    _ptr(cq, _i32p), _ptr(ck, _i32p), B, Hq, Hkv, total_q,
                                    total_k, D, int(bool(causal)), float(scale), _ptr(o, _f64p),
                                    _ptr(lse, _f64p))
    if rc != 0:
        raise ValueError(f"oracle_attn_fwd_varlen failed ({rc})")
    return o, lse


def attn_fwd_ragged_paged(q, k_pages, v_pages, cu_seqlens_q, kv_seqlens, block_table, *,
                          causal: bool, scale: float, lib=None):
    """Ragged paged forward.  q [total_q,Hq,D] packed, pages [n_pages,Hkv,page_size,D],
    cu_seqlens_q int32 [B+1], kv_seqlens int32 [B], block_table int32 [B,max_pages]
    -> (o [total_q,Hq,D], lse [Hq,total_q]); rows no sequence owns stay NaN."""
    lib = lib or load()
    q, kp, vp = _u16(q), _u16(k_pages), _u16(v_pages)
    total_q, Hq, D = q.shape
    n_pages, Hkv, page_size, _ = kp.shape
    cq = np.ascontiguousarray(cu_seqlens_q, dtype=np.int32)
    if cq.ndim != 1 or cq.shape[0] < 2:
        raise ValueError("cu_seqlens_q must be [B+1]")
    B = cq.shape[0] - 1
    sl = _seqlens(kv_seqlens, B)
    if sl is None:
        raise ValueError("kv_seqlens is required")
    bt = np.ascontiguousarray(block_table, dtype=np.int32)
    if bt.ndim != 2 or bt.shape[0] != B:
        raise ValueError("block_table must be [B, max_pages]")
    o = np.full((total_q, Hq, D), np.nan, np.float64)
    lse = np.full((Hq, total_q), np.nan, np.float64)
    rc = lib.oracle_attn_fwd_ragged_paged(_ptr(q, _u16p), _ptr(kp, _u16p), _ptr(vp, _u16p),
                                          _ptr(cq, _i32p), _ptr(sl, _i32p), _ptr(bt, _i32p), B,
                                          Hq, Hkv, total_q, page_size, bt.shape[1], n_pages, D,
                                          int(bool(causal)), float(scale), _ptr(o, _f64p),
                                          _ptr(lse, _f64p))
    if rc != 0:
        raise ValueError(f"oracle_attn_fwd_ragged_paged failed ({rc})")
    return o, lse


def decode_paged(q, k_pages, v_pages, block_table, kv_seqlens, *, scale: float, lib=None):
    """Paged decode step.  q [B,Hq,D], pages [n_pages,Hkv,page_size,D], block_table
    [B,max_pages] int32 -> (o [B,Hq,D], lse [B,Hq])."""
    lib = lib or load()
    q, kp, vp = _u16(q), _u16(k_pages), _u16(v_pages)
    B, Hq, D = q.shape
    n_pages, Hkv, page_size, _ = kp.shape
    bt = np.ascontiguousarray(block_table, dtype=np.int32)
    if bt.ndim != 2 or bt.shape[0] != B:
        raise ValueError("block_table must be [B, max_pages]")
    sl = _seqlens(kv_seqlens, B)
    o = np.empty((B, Hq, D), np.float64)
    lse = np.empty((B, Hq), np.float64)
    rc = lib.oracle_decode_paged(_ptr(q, _u16p), _ptr(kp, _u16p), _ptr(vp, _u16p),
                                 _ptr(bt, _i32p), B, Hq, Hkv, page_size, bt.shape[1], n_pages,
                                 D, float(scale), _ptr(sl, _i32p), _ptr(o, _f64p),
                                 _ptr(lse, _f64p))
    if rc != 0:
        raise ValueError(f"oracle_decode_paged failed ({rc})")
    return o, lse


def decode_split(q, k_cache, v_cache, kv_seqlens, *, scale: float, split: int, lib=None):
    """Split-KV decode step by step.  Returns (o, lse, o_part, lse_part)."""
    lib = lib or load()
    q, kc, vc = _u16(q), _u16(k_cache), _u16(v_cache)
    B, Hq, D = q.shape
    _, Hkv, Smax, _ = kc.shape
    sl = _seqlens(kv_seqlens, B)
    nsplit = -(-Smax // split)
    o_part = np.empty((B, Hq, nsplit, D), np.float64)
    lse_part = np.empty((B, Hq, nsplit), np.float64)
    o = np.empty((B, Hq, D), np.float64)
    lse = np.empty((B, Hq), np.float64)
    rc = lib.oracle_decode_split(_ptr(q, _u16p), _ptr(kc, _u16p), _ptr(vc, _u16p),
                                 B, Hq, Hkv, Smax, D, float(scale), _ptr(sl, _i32p), split,
                                 _ptr(o_part, _f64p), _ptr(lse_part, _f64p),
                                 _ptr(o, _f64p), _ptr(lse, _f64p))
    if rc != 0:
        raise ValueError(f"oracle_decode_split failed ({rc})")
    return o, lse, o_part, lse_part


def lse_combine(o_part, lse_part, lib=None):
    """Merge partials o_part [R,nsplit,D], lse_part [R,nsplit] -> (o [R,D], lse [R])."""
    lib = lib or load()
    o_part = np.ascontiguousarray(o_part, dtype=np.float64)
    lse_part = np.ascontiguousarray(lse_part, dtype=np.float64)
    R, nsplit, D = o_part.shape
    o = np.empty((R, D), np.float64)
    lse = np.empty((R,), np.float64)
    rc = lib.oracle_lse_combine(_ptr(o_part, _f64p), _ptr(lse_part, _f64p), R, nsplit, D,
                                _ptr(o, _f64p), _ptr(lse, _f64p))
    if rc != 0:
        raise ValueError(f"oracle_lse_combine failed ({rc})")
    return o, lse


def mla_decode(q, ckv, kv_seqlens, *, Dc: int, scale: float, lib=None):
    """MLA decode.  q [B,H,Dc+Dr], ckv [B,Smax,Dc+Dr] (bf16 bits), lengths [B]
    -> (o [B,H,Dc], lse [B,H]) float64."""
    lib = lib or load()
    q, ckv = _u16(q), _u16(ckv)
    B, H, Dk = q.shape
    _, Smax, Dk2 = ckv.shape
    if Dk2 != Dk or not 0 < Dc <= Dk:
        raise ValueError("q and ckv must share the last dim, Dc within it")
    sl = _seqlens(kv_seqlens, B)
    o = np.empty((B, H, Dc), np.float64)
    lse = np.empty((B, H), np.float64)
    rc = lib.oracle_mla_decode(_ptr(q, _u16p), _ptr(ckv, _u16p), B, H, Dc, Dk - Dc, Smax,
                               float(scale), _ptr(sl, _i32p), _ptr(o, _f64p), _ptr(lse, _f64p))
    if rc != 0:
        raise ValueError(f"oracle_mla_decode failed ({rc})")
    return o, lse
