"""Fused causal grouped-query attention for MI355X (gfx950).

Thin ctypes binding of ``libmk_attn.so`` (C ABI in ``include/mk_attn.h``).
The functions named like the C entry points take torch tensors where the C
call takes device pointers and otherwise mirror its argument list; they do
argument marshalling only -- every step of the computation runs in the HIP
kernels.  ``fwd`` and ``decode`` are conveniences that allocate the outputs
with torch and call those entry points.

There is no fallback: when the library is missing, every call raises.
"""
from __future__ import annotations

import ctypes
import os

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libmk_attn.so")

DECODE_MAX_PARTS = 1 << 20  # largest n_parts

MK_STATUS = {0: "MK_OK", 1: "MK_ERR_NULL", 2: "MK_ERR_SHAPE", 3: "MK_ERR_UNSUPPORTED",
             4: "MK_ERR_ALIGN", 5: "MK_ERR_WORKSPACE", 6: "MK_ERR_HIP", 7: "MK_ERR_ARG",
             8: "MK_ERR_SCRATCH"}

# every symbol include/mk_attn.h declares
EXPORTS = ("mk_attn_fwd", "mk_attn_fwd_ws", "mk_attn_fwd_workspace_bytes", "mk_attn_fwd_o32",
           "mk_attn_fwd_varlen", "mk_attn_fwd_ragged_paged",
           "mk_attn_decode_workspace_bytes", "mk_attn_decode", "mk_attn_decode_paged",
           "mk_attn_decode_noalloc", "mk_attn_decode_noalloc_max_bytes",
           "mk_attn_decode_default_parts", "mk_attn_bwd", "mk_attn_bwd_workspace_bytes",
           "mk_attn_mla_decode", "mk_attn_mla_decode_workspace_bytes",
           "mk_status_str", "mk_attn_version")


class MkAttnError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(msg)
        self.status = status


_lib = None


def lib():
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                f"{LIB_PATH} is missing: the HIP library has not been built "
                "(run __graft_entry__.build() or python paper_2609_04523_amd/build.py)")
        h = ctypes.CDLL(LIB_PATH)
        vp, i, f, sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_float, ctypes.c_size_t
        h.mk_attn_fwd.argtypes = [vp, vp, vp, vp, vp, i, i, i, i, i, i, i, f, vp, vp]
        h.mk_attn_fwd.restype = i
        h.mk_attn_fwd_ws.argtypes = [vp, vp, vp, vp, vp, i, i, i, i, i, i, i, f, vp, vp, sz, vp]
        h.mk_attn_fwd_ws.restype = i
        h.mk_attn_fwd_workspace_bytes.argtypes = [i, i, i, i]
        h.mk_attn_fwd_workspace_bytes.restype = sz
        h.mk_attn_fwd_o32.argtypes = [vp, vp, vp, vp, vp, i, i, i, i, i, i, i, f, vp, vp]
        h.mk_attn_fwd_o32.restype = i
        h.mk_attn_fwd_varlen.argtypes = [vp, vp, vp, vp, vp, vp, vp, i, i, i, i, i, i, i, i, f, vp]
        h.mk_attn_fwd_varlen.restype = i
        h.mk_attn_fwd_ragged_paged.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, i, i, i, i, i, i,
                                               i, i, i, i, f, vp]
        h.mk_attn_fwd_ragged_paged.restype = i
        h.mk_attn_decode_workspace_bytes.argtypes = [i, i, i, i]
        h.mk_attn_decode_workspace_bytes.restype = sz
        h.mk_attn_decode.argtypes = [vp, vp, vp, vp, vp, i, i, i, i, i, f, vp, i, vp, sz, vp]
        h.mk_attn_decode.restype = i
        h.mk_attn_decode_noalloc.argtypes = [vp, vp, vp, vp, vp, i, i, i, i, i, f, vp, i, vp]
        h.mk_attn_decode_noalloc.restype = i
        h.mk_attn_decode_noalloc_max_bytes.argtypes = []
        h.mk_attn_decode_noalloc_max_bytes.restype = sz
        h.mk_attn_decode_paged.argtypes = [vp, vp, vp, vp, vp, vp, i, i, i, i, i, i, i, f, vp, i,
                                           vp, sz, vp]
        h.mk_attn_decode_paged.restype = i
        h.mk_attn_decode_default_parts.argtypes = [i, i, i]
        h.mk_attn_decode_default_parts.restype = i
        h.mk_attn_bwd.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp, i, i, i, i, i, i, i, f,
                                  vp, vp, sz, vp]
        h.mk_attn_bwd.restype = i
        h.mk_attn_bwd_workspace_bytes.argtypes = [i, i, i]
        h.mk_attn_bwd_workspace_bytes.restype = sz
        h.mk_attn_mla_decode.argtypes = [vp, vp, vp, vp, i, i, i, i, i, f, vp, i, vp, sz, vp]
        h.mk_attn_mla_decode.restype = i
        h.mk_attn_mla_decode_workspace_bytes.argtypes = [i, i, i]
        h.mk_attn_mla_decode_workspace_bytes.restype = sz
        h.mk_status_str.argtypes = [i]
        h.mk_status_str.restype = ctypes.c_char_p
        h.mk_attn_version.argtypes = []
        h.mk_attn_version.restype = i
        _lib = h
    return _lib


def mk_status_str(status: int) -> str:
    return lib().mk_status_str(int(status)).decode()


def mk_attn_version() -> int:
    return lib().mk_attn_version()


def mk_attn_decode_default_parts(Hq: int, Hkv: int, D: int) -> int:
    return lib().mk_attn_decode_default_parts(Hq, Hkv, D)


def mk_attn_decode_workspace_bytes(Hq: int, Hkv: int, D: int, n_parts: int = 0) -> int:
    return lib().mk_attn_decode_workspace_bytes(Hq, Hkv, D, n_parts)


def mk_attn_fwd_workspace_bytes(B: int, Hkv: int, Skv: int, D: int) -> int:
    return int(lib().mk_attn_fwd_workspace_bytes(B, Hkv, Skv, D))


def mk_attn_bwd_workspace_bytes(B: int, Hq: int, Sq: int) -> int:
    return int(lib().mk_attn_bwd_workspace_bytes(B, Hq, Sq))


def mk_attn_mla_decode_workspace_bytes(H: int, Dc: int, n_parts: int = 0) -> int:
    return int(lib().mk_attn_mla_decode_workspace_bytes(H, Dc, n_parts))


def _check(rc: int):
    if rc != 0:
        raise MkAttnError(rc, mk_status_str(rc))


def _ptr(t):
    """Device pointer of a tensor (None -> NULL).  Plain ints pass through."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def mk_attn_fwd(q, k, v, o, lse, B, Hq, Hkv, Sq, Skv, D, causal, scale, kv_seqlens=None,
                stream=None):
    _check(lib().mk_attn_fwd(_ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(lse), B, Hq, Hkv, Sq,
                             Skv, D, int(causal), float(scale), _ptr(kv_seqlens),
                             _stream(stream)))


def mk_attn_fwd_ws(q, k, v, o, lse, B, Hq, Hkv, Sq, Skv, D, causal, scale, kv_seqlens,
                   workspace, workspace_bytes, stream=None):
    _check(lib().mk_attn_fwd_ws(_ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(lse), B, Hq, Hkv, Sq,
                                Skv, D, int(causal), float(scale), _ptr(kv_seqlens),
                                _ptr(workspace), int(workspace_bytes), _stream(stream)))


def mk_attn_fwd_o32(q, k, v, o, lse, B, Hq, Hkv, Sq, Skv, D, causal, scale, kv_seqlens=None,
                    stream=None):
    _check(lib().mk_attn_fwd_o32(_ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(lse), B, Hq, Hkv,
                                 Sq, Skv, D, int(causal), float(scale), _ptr(kv_seqlens),
                                 _stream(stream)))


def mk_attn_fwd_varlen(q, k, v, o, lse, cu_seqlens_q, cu_seqlens_k, B, Hq, Hkv, max_seqlen_q,
                       total_q, total_k, D, causal, scale, stream=None):
    _check(lib().mk_attn_fwd_varlen(_ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(lse),
                                    _ptr(cu_seqlens_q), _ptr(cu_seqlens_k), B, Hq, Hkv,
                                    max_seqlen_q, total_q, total_k, D, int(causal), float(scale),
                                    _stream(stream)))


def mk_attn_fwd_ragged_paged(q, k_pages, v_pages, block_table, o, lse, cu_seqlens_q, kv_seqlens,
                             B, Hq, Hkv, max_seqlen_q, total_q, page_size, max_pages, n_pages, D,
                             causal, scale, stream=None):
    _check(lib().mk_attn_fwd_ragged_paged(_ptr(q), _ptr(k_pages), _ptr(v_pages),
                                          _ptr(block_table), _ptr(o), _ptr(lse),
                                          _ptr(cu_seqlens_q), _ptr(kv_seqlens), B, Hq, Hkv,
                                          max_seqlen_q, total_q, page_size, max_pages, n_pages,
                                          D, int(causal), float(scale), _stream(stream)))


def mk_attn_decode(q, k_cache, v_cache, o, lse, B, Hq, Hkv, Smax, D, scale, kv_seqlens,
                   n_parts, workspace, workspace_bytes, stream=None):
    _check(lib().mk_attn_decode(_ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(o), _ptr(lse), B,
                                Hq, Hkv, Smax, D, float(scale), _ptr(kv_seqlens), int(n_parts),
                                _ptr(workspace), int(workspace_bytes), _stream(stream)))


def mk_attn_decode_noalloc(q, k_cache, v_cache, o, lse, B, Hq, Hkv, Smax, D, scale, kv_seqlens,
                           n_parts, stream=None):
    _check(lib().mk_attn_decode_noalloc(_ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(o),
                                        _ptr(lse), B, Hq, Hkv, Smax, D, float(scale),
                                        _ptr(kv_seqlens), int(n_parts), _stream(stream)))


def mk_attn_decode_noalloc_max_bytes() -> int:
    return int(lib().mk_attn_decode_noalloc_max_bytes())


def mk_attn_decode_paged(q, k_pages, v_pages, block_table, o, lse, B, Hq, Hkv, page_size,
                         max_pages, n_pages, D, scale, kv_seqlens, n_parts, workspace,
                         workspace_bytes, stream=None):
    _check(lib().mk_attn_decode_paged(_ptr(q), _ptr(k_pages), _ptr(v_pages), _ptr(block_table),
                                      _ptr(o), _ptr(lse), B, Hq, Hkv, page_size, max_pages,
                                      n_pages, D, float(scale), _ptr(kv_seqlens), int(n_parts),
                                      _ptr(workspace), int(workspace_bytes), _stream(stream)))


def mk_attn_bwd(q, k, v, o, dout, lse, dq, dk, dv, B, Hq, Hkv, Sq, Skv, D, causal, scale,
                kv_seqlens, workspace, workspace_bytes, stream=None):
    _check(lib().mk_attn_bwd(_ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(dout), _ptr(lse),
                             _ptr(dq), _ptr(dk), _ptr(dv), B, Hq, Hkv, Sq, Skv, D, int(causal),
                             float(scale), _ptr(kv_seqlens), _ptr(workspace),
                             int(workspace_bytes), _stream(stream)))


def mk_attn_mla_decode(q, ckv, o, lse, B, H, Dc, Dr, Smax, scale, kv_seqlens, n_parts,
                       workspace, workspace_bytes, stream=None):
    _check(lib().mk_attn_mla_decode(_ptr(q), _ptr(ckv), _ptr(o), _ptr(lse), B, H, Dc, Dr, Smax,
                                    float(scale), _ptr(kv_seqlens), int(n_parts),
                                    _ptr(workspace), int(workspace_bytes), _stream(stream)))


# ---------------------------------------------------------------------------
# conveniences: allocate outputs with torch, then call the entry points above
# ---------------------------------------------------------------------------
def _require(t, name, dtype, ndim):
    import torch
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a device tensor")
    if t.dtype != dtype or t.dim() != ndim or not t.is_contiguous():
        raise TypeError(f"{name} must be a contiguous {ndim}-d {dtype} tensor")


def fwd(q, k, v, *, causal: bool = True, scale: float | None = None, kv_seqlens=None,
        out_fp32: bool = False, with_lse: bool = True, workspace=None, stream=None):
    """q [B,Hq,Sq,D], k/v [B,Hkv,Skv,D] bf16 -> (o [B,Hq,Sq,D], lse [B,Hq,Sq] or None).
    With a workspace (a uint8 tensor of at least mk_attn_fwd_workspace_bytes)
    the bf16 forward goes through mk_attn_fwd_ws (V^T tiles in the
    workspace; the same result)."""
    import torch
    _require(q, "q", torch.bfloat16, 4)
    _require(k, "k", torch.bfloat16, 4)
    _require(v, "v", torch.bfloat16, 4)
    B, Hq, Sq, D = q.shape
    _, Hkv, Skv, _ = k.shape
    if scale is None:
        scale = D ** -0.5
    if kv_seqlens is not None:
        _require(kv_seqlens, "kv_seqlens", torch.int32, 1)
    o = torch.empty((B, Hq, Sq, D), device=q.device,
                    dtype=torch.float32 if out_fp32 else torch.bfloat16)
    lse = torch.empty((B, Hq, Sq), device=q.device, dtype=torch.float32) if with_lse else None
    if workspace is not None:
        if out_fp32:
            raise ValueError("the workspace forward writes bf16 O")
        mk_attn_fwd_ws(q, k, v, o, lse, B, Hq, Hkv, Sq, Skv, D, causal, scale, kv_seqlens,
                       workspace, workspace.numel() * workspace.element_size(), stream)
        return o, lse
    entry = mk_attn_fwd_o32 if out_fp32 else mk_attn_fwd
    entry(q, k, v, o, lse, B, Hq, Hkv, Sq, Skv, D, causal, scale, kv_seqlens, stream)
    return o, lse


def bwd(q, k, v, o, lse, dout, *, causal: bool = True, scale: float | None = None,
        kv_seqlens=None, workspace=None, stream=None):
    """Gradients of the forward fwd(q, k, v) -> (o, lse) given dout = dL/dO:
    -> (dq [B,Hq,Sq,D], dk, dv [B,Hkv,Skv,D]) bf16.  The LSE is not
    differentiated."""
    import torch
    for t, nm in ((q, "q"), (k, "k"), (v, "v"), (o, "o"), (dout, "dout")):
        _require(t, nm, torch.bfloat16, 4)
    _require(lse, "lse", torch.float32, 3)
    B, Hq, Sq, D = q.shape
    _, Hkv, Skv, _ = k.shape
    if o.shape != q.shape or dout.shape != q.shape or tuple(lse.shape) != (B, Hq, Sq):
        raise ValueError("o and dout must have q's shape, lse [B, Hq, Sq]")
    if scale is None:
        scale = D ** -0.5
    if kv_seqlens is not None:
        _require(kv_seqlens, "kv_seqlens", torch.int32, 1)
    need = mk_attn_bwd_workspace_bytes(B, Hq, Sq)
    if workspace is None:
        workspace = torch.empty(need, device=q.device, dtype=torch.uint8)
    dq = torch.empty_like(q)
    dk = torch.empty_like(k)
    dv = torch.empty_like(v)
    mk_attn_bwd(q, k, v, o, dout, lse, dq, dk, dv, B, Hq, Hkv, Sq, Skv, D, causal, scale,
                kv_seqlens, workspace, workspace.numel() * workspace.element_size(), stream)
    return dq, dk, dv


def mla_decode(q, ckv, kv_seqlens, *, Dc: int = 512, scale: float | None = None,
               n_parts: int = 0, workspace=None, stream=None):
    """MLA decode.  q [B,H,Dc+Dr], ckv [B,Smax,Dc+Dr] bf16, kv_seqlens int32 [B]
    -> (o [B,H,Dc] bf16, lse [B,H] fp32)."""
    import torch
    _require(q, "q", torch.bfloat16, 3)
    _require(ckv, "ckv", torch.bfloat16, 3)
    _require(kv_seqlens, "kv_seqlens", torch.int32, 1)
    B, H, Dk = q.shape
    _, Smax, _ = ckv.shape
    if scale is None:
        scale = Dk ** -0.5
    need = mk_attn_mla_decode_workspace_bytes(H, Dc, n_parts)
    if workspace is None:
        workspace = torch.empty(max(need, 1), device=q.device, dtype=torch.uint8)
    o = torch.empty((B, H, Dc), device=q.device, dtype=torch.bfloat16)
    lse = torch.empty((B, H), device=q.device, dtype=torch.float32)
    mk_attn_mla_decode(q, ckv, o, lse, B, H, Dc, Dk - Dc, Smax, scale, kv_seqlens, n_parts,
                       workspace, workspace.numel() * workspace.element_size(), stream)
    return o, lse


def fwd_varlen(q, k, v, cu_seqlens_q, cu_seqlens_k, max_seqlen_q: int, *, causal: bool = True,
               scale: float | None = None, with_lse: bool = True, stream=None):
    """Packed ragged forward.  q [total_q,Hq,D], k/v [total_k,Hkv,D] bf16,
    cu_seqlens int32 [B+1] (device) -> (o [total_q,Hq,D], lse [Hq,total_q] or None).
    Rows no sequence owns are left as allocated (uninitialised)."""
    import torch
    _require(q, "q", torch.bfloat16, 3)
    _require(k, "k", torch.bfloat16, 3)
    _require(v, "v", torch.bfloat16, 3)
    _require(cu_seqlens_q, "cu_seqlens_q", torch.int32, 1)
    _require(cu_seqlens_k, "cu_seqlens_k", torch.int32, 1)
    total_q, Hq, D = q.shape
    total_k, Hkv, _ = k.shape
    B = cu_seqlens_q.shape[0] - 1
    if cu_seqlens_k.shape[0] != B + 1:
        raise ValueError("cu_seqlens_q and cu_seqlens_k must have the same length")
    if scale is None:
        scale = D ** -0.5
    o = torch.empty((total_q, Hq, D), device=q.device, dtype=torch.bfloat16)
    lse = torch.empty((Hq, total_q), device=q.device, dtype=torch.float32) if with_lse else None
    mk_attn_fwd_varlen(q, k, v, o, lse, cu_seqlens_q, cu_seqlens_k, B, Hq, Hkv, max_seqlen_q,
                       total_q, total_k, D, causal, scale, stream)
    return o, lse


def fwd_ragged_paged(q, k_pages, v_pages, block_table, cu_seqlens_q, kv_seqlens,
                     max_seqlen_q: int, *, causal: bool = True, scale: float | None = None,
                     with_lse: bool = True, stream=None):
    """Ragged paged forward.  q [total_q,Hq,D] bf16 packed, page pools
    [n_pages,Hkv,page_size,D] bf16, block_table int32 [B,max_pages],
    cu_seqlens_q int32 [B+1], kv_seqlens int32 [B] (device)
    -> (o [total_q,Hq,D], lse [Hq,total_q] or None).  Rows no sequence owns
    are left as allocated (uninitialised)."""
    import torch
    _require(q, "q", torch.bfloat16, 3)
    _require(k_pages, "k_pages", torch.bfloat16, 4)
    _require(v_pages, "v_pages", torch.bfloat16, 4)
    _require(block_table, "block_table", torch.int32, 2)
    _require(cu_seqlens_q, "cu_seqlens_q", torch.int32, 1)
    _require(kv_seqlens, "kv_seqlens", torch.int32, 1)
    total_q, Hq, D = q.shape
    n_pages, Hkv, page_size, _ = k_pages.shape
    B, max_pages = block_table.shape
    if cu_seqlens_q.shape[0] != B + 1 or kv_seqlens.shape[0] != B:
        raise ValueError("cu_seqlens_q must be [B+1] and kv_seqlens [B]")
    if scale is None:
        scale = D ** -0.5
    o = torch.empty((total_q, Hq, D), device=q.device, dtype=torch.bfloat16)
    lse = torch.empty((Hq, total_q), device=q.device, dtype=torch.float32) if with_lse else None
    mk_attn_fwd_ragged_paged(q, k_pages, v_pages, block_table, o, lse, cu_seqlens_q, kv_seqlens,
                             B, Hq, Hkv, max_seqlen_q, total_q, page_size, max_pages, n_pages, D,
                             causal, scale, stream)
    return o, lse


def decode(q, k_cache, v_cache, kv_seqlens, *, scale: float | None = None, n_parts: int = 0,
           workspace=None, with_lse: bool = True, stream=None):
    """q [B,Hq,D], caches [B,Hkv,Smax,D] bf16, kv_seqlens int32 [B] -> (o, lse)."""
    import torch
    _require(q, "q", torch.bfloat16, 3)
    _require(k_cache, "k_cache", torch.bfloat16, 4)
    _require(v_cache, "v_cache", torch.bfloat16, 4)
    _require(kv_seqlens, "kv_seqlens", torch.int32, 1)
    B, Hq, D = q.shape
    _, Hkv, Smax, _ = k_cache.shape
    if scale is None:
        scale = D ** -0.5
    need = mk_attn_decode_workspace_bytes(Hq, Hkv, D, n_parts)
    if workspace is None:
        workspace = torch.empty(need, device=q.device, dtype=torch.uint8)
    o = torch.empty((B, Hq, D), device=q.device, dtype=torch.bfloat16)
    lse = torch.empty((B, Hq), device=q.device, dtype=torch.float32) if with_lse else None
    mk_attn_decode(q, k_cache, v_cache, o, lse, B, Hq, Hkv, Smax, D, scale, kv_seqlens, n_parts,
                   workspace, workspace.numel() * workspace.element_size(), stream)
    return o, lse


def decode_paged(q, k_pages, v_pages, block_table, kv_seqlens, *, scale: float | None = None,
                 n_parts: int = 0, workspace=None, with_lse: bool = True, stream=None):
    """q [B,Hq,D], page pools [n_pages,Hkv,page_size,D] bf16, block_table int32
    [B,max_pages], kv_seqlens int32 [B] -> (o, lse)."""
    import torch
    _require(q, "q", torch.bfloat16, 3)
    _require(k_pages, "k_pages", torch.bfloat16, 4)
    _require(v_pages, "v_pages", torch.bfloat16, 4)
    _require(block_table, "block_table", torch.int32, 2)
    _require(kv_seqlens, "kv_seqlens", torch.int32, 1)
    B, Hq, D = q.shape
    n_pages, Hkv, page_size, _ = k_pages.shape
    max_pages = block_table.shape[1]
    if scale is None:
        scale = D ** -0.5
    need = mk_attn_decode_workspace_bytes(Hq, Hkv, D, n_parts)
    if workspace is None:
        workspace = torch.empty(need, device=q.device, dtype=torch.uint8)
    o = torch.empty((B, Hq, D), device=q.device, dtype=torch.bfloat16)
    lse = torch.empty((B, Hq), device=q.device, dtype=torch.float32) if with_lse else None
    mk_attn_decode_paged(q, k_pages, v_pages, block_table, o, lse, B, Hq, Hkv, page_size,
                         max_pages, n_pages, D, scale, kv_seqlens, n_parts, workspace,
                         workspace.numel() * workspace.element_size(), stream)
    return o, lse


def decode_partials(workspace, Hq: int, Hkv: int, D: int, n_parts: int = 0):
    """Views of a decode workspace: (o_part [P,2,G,D], lse_part [P,2,G]) fp32.

    Slot 0 of part w holds its first piece and slot 1 its last, when that
    piece is part of a cut pair (see include/mk_attn.h); other entries are
    not written by the library."""
    import torch
    P = n_parts if n_parts else mk_attn_decode_default_parts(Hq, Hkv, D)
    G = Hq // Hkv
    n_o = P * 2 * G * D
    lse_off = -(-(n_o * 4) // 256) * 256
    flat = workspace.view(torch.uint8)
    o_part = flat[: n_o * 4].view(torch.float32).view(P, 2, G, D)
    lse_part = flat[lse_off: lse_off + P * 2 * G * 4].view(torch.float32).view(P, 2, G)
    return o_part, lse_part
