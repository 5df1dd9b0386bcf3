"""C-ABI boundary on the CPU: the library loads, exports what the header
declares, and rejects every invalid argument on the host before any HIP
call (so none of these calls touches a GPU)."""
import ctypes
import math
import os
import re

import pytest

import paper_2609_04523_amd as mk

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include",
                      "mk_attn.h")

# fake device addresses: never dereferenced, only checked for NULL/alignment
P = 0x10000
P_ODD = 0x10002
F = ctypes.c_void_p


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(mk.LIB_PATH):
        from paper_2609_04523_amd import build
        build.build()
    return mk.lib()


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[a-z_]+\s*\*?\s*(mk_[a-z0-9_]+)\s*\(",
                                 text, re.M)))


def test_header_declares_the_python_exports():
    assert sorted(mk.EXPORTS) == declared_functions()


def test_every_declared_symbol_is_exported(lib):
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_version_and_status_strings(lib):
    assert mk.mk_attn_version() == 10
    names = ["MK_OK", "MK_ERR_NULL", "MK_ERR_SHAPE", "MK_ERR_UNSUPPORTED", "MK_ERR_ALIGN",
             "MK_ERR_WORKSPACE", "MK_ERR_HIP", "MK_ERR_ARG", "MK_ERR_SCRATCH"]
    for code, name in enumerate(names):
        assert mk.mk_status_str(code).startswith(name)
        assert mk.MK_STATUS[code] == name
    assert "UNKNOWN" in mk.mk_status_str(99)
    assert "UNKNOWN" in mk.mk_status_str(-1)


def fwd_rc(lib, *, q=P, k=P, v=P, o=P, lse=None, B=1, Hq=2, Hkv=1, Sq=8, Skv=8, D=128,
           causal=1, scale=0.125, seqlens=None, o32=False):
    fn = lib.mk_attn_fwd_o32 if o32 else lib.mk_attn_fwd
    return fn(q, k, v, o, lse, B, Hq, Hkv, Sq, Skv, D, causal, scale, seqlens, None)


@pytest.mark.parametrize("o32", [False, True])
def test_fwd_validation(lib, o32):
    r = lambda **kw: fwd_rc(lib, o32=o32, **kw)
    for name in ("q", "k", "v", "o"):
        assert r(**{name: None}) == 1
    for name in ("B", "Hq", "Hkv", "Sq", "Skv"):
        assert r(**{name: 0}) == 2
        assert r(**{name: -3}) == 2
    assert r(D=0) == 2
    assert r(Hq=3, Hkv=2) == 2
    for D in (32, 96, 256, 80):
        assert r(D=D) == 3
    for name in ("q", "k", "v", "o"):
        assert r(**{name: P_ODD}) == 4
    assert r(lse=P + 2) == 4
    assert r(seqlens=P + 1) == 4
    assert r(causal=2) == 7
    assert r(causal=-1) == 7
    for s in (math.inf, -math.inf, math.nan):
        assert r(scale=s) == 7
    # too many workgroups for one launch
    assert r(B=65536, Hq=65536, Hkv=1, Sq=1) == 2


def fwd_ws_rc(lib, *, q=P, k=P, v=P, o=P, lse=None, B=1, Hq=2, Hkv=1, Sq=8, Skv=8, D=128,
              causal=1, scale=0.125, seqlens=None, ws=P, ws_bytes=1 << 30):
    return lib.mk_attn_fwd_ws(q, k, v, o, lse, B, Hq, Hkv, Sq, Skv, D, causal, scale, seqlens, ws,
                              ws_bytes, None)


def test_fwd_ws_workspace_bytes(lib):
    # B * Hkv * ceil(Skv / 64) tiles of 64 keys x D bf16, then 1 KiB of
    # work-item counters
    assert mk.mk_attn_fwd_workspace_bytes(1, 8, 32768, 128) == 8 * 512 * 64 * 128 * 2 + 1024
    assert mk.mk_attn_fwd_workspace_bytes(2, 3, 65, 64) == 2 * 3 * 2 * 64 * 64 * 2 + 1024
    assert mk.mk_attn_fwd_workspace_bytes(4, 16, 1, 128) == 4 * 16 * 64 * 128 * 2 + 1024
    for args in ((0, 1, 8, 128), (1, 0, 8, 128), (1, 1, 0, 128), (1, 1, 8, 96), (1, 1, 8, 0)):
        assert mk.mk_attn_fwd_workspace_bytes(*args) == 0


def test_fwd_ws_validation(lib):
    r = lambda **kw: fwd_ws_rc(lib, **kw)
    assert r(ws=None) == 1
    assert r(ws=P + 8) == 4
    need = mk.mk_attn_fwd_workspace_bytes(1, 1, 8, 128)
    assert r(ws_bytes=need - 1) == 7
    assert r(ws_bytes=0) == 7
    # everything mk_attn_fwd rejects, with a large enough workspace
    for name in ("q", "k", "v", "o"):
        assert r(**{name: None}) == 1
        assert r(**{name: P_ODD}) == 4
    for name in ("B", "Hq", "Hkv", "Sq", "Skv"):
        assert r(**{name: 0}) == 2
    assert r(Hq=3, Hkv=2) == 2
    assert r(D=96) == 3
    assert r(causal=2) == 7
    assert r(scale=math.nan) == 7
    assert r(lse=P + 2) == 4
    assert r(seqlens=P + 1) == 4


def varlen_rc(lib, *, q=P, k=P, v=P, o=P, lse=None, cq=P, ck=P, B=3, Hq=8, Hkv=2, max_sq=100,
              total_q=300, total_k=400, D=128, causal=1, scale=0.125):
    return lib.mk_attn_fwd_varlen(q, k, v, o, lse, cq, ck, B, Hq, Hkv, max_sq, total_q, total_k,
                                  D, causal, scale, None)


def rpa_rc(lib, *, q=P, kp=P, vp=P, bt=P, o=P, lse=None, cq=P, sl=P, B=3, Hq=8, Hkv=2,
           max_sq=100, total_q=300, ps=16, mp=64, npg=200, D=128, causal=1, scale=0.125):
    return lib.mk_attn_fwd_ragged_paged(q, kp, vp, bt, o, lse, cq, sl, B, Hq, Hkv, max_sq,
                                        total_q, ps, mp, npg, D, causal, scale, None)


def test_fwd_ragged_paged_validation(lib):
    for name in ("q", "kp", "vp", "bt", "o", "cq", "sl"):
        assert rpa_rc(lib, **{name: None}) == 1
    for name in ("B", "Hq", "Hkv", "max_sq", "total_q", "ps", "mp", "npg"):
        assert rpa_rc(lib, **{name: 0}) == 2
    assert rpa_rc(lib, Hq=6, Hkv=4) == 2
    assert rpa_rc(lib, mp=1 << 20, ps=4096) == 2           # key positions past 31 bits
    assert rpa_rc(lib, B=1 << 16, mp=1 << 16) == 2          # table entries past 31 bits
    assert rpa_rc(lib, D=96) == 3
    for ps in (8, 24, 40):
        assert rpa_rc(lib, ps=ps) == 3                      # pages of a multiple of 16 keys
    assert rpa_rc(lib, causal=2) == 7
    assert rpa_rc(lib, scale=math.inf) == 7
    for name in ("q", "kp", "vp", "o"):
        assert rpa_rc(lib, **{name: P_ODD}) == 4
    for name in ("cq", "sl", "bt"):
        assert rpa_rc(lib, **{name: P + 2}) == 4
    assert rpa_rc(lib, lse=P + 2) == 4


def test_fwd_varlen_validation(lib):
    for name in ("q", "k", "v", "o", "cq", "ck"):
        assert varlen_rc(lib, **{name: None}) == 1
    for name in ("B", "Hq", "Hkv", "max_sq", "total_q", "total_k"):
        assert varlen_rc(lib, **{name: 0}) == 2
    assert varlen_rc(lib, Hq=6, Hkv=4) == 2
    assert varlen_rc(lib, B=1 << 16, Hq=64, Hkv=64, max_sq=1 << 20) == 2  # too many workgroups
    assert varlen_rc(lib, D=96) == 3
    assert varlen_rc(lib, causal=3) == 7
    assert varlen_rc(lib, scale=math.nan) == 7
    for name in ("q", "k", "v", "o"):
        assert varlen_rc(lib, **{name: P_ODD}) == 4
    assert varlen_rc(lib, cq=P + 2) == 4
    assert varlen_rc(lib, ck=P + 1) == 4
    assert varlen_rc(lib, lse=P + 2) == 4


def dec_rc(lib, *, q=P, kc=P, vc=P, o=P, lse=None, B=2, Hq=8, Hkv=2, Smax=512, D=128,
           scale=0.1, seqlens=P, parts=0, ws=P, ws_bytes=None):
    if ws_bytes is None:
        ws_bytes = lib.mk_attn_decode_workspace_bytes(max(Hq, 1), max(Hkv, 1), D, max(parts, 0))
    return lib.mk_attn_decode(q, kc, vc, o, lse, B, Hq, Hkv, Smax, D, scale, seqlens, parts, ws,
                              ws_bytes, None)


def test_decode_validation(lib):
    for name in ("q", "kc", "vc", "o", "seqlens"):
        assert dec_rc(lib, **{name: None}) == 1
    for name in ("B", "Hq", "Hkv", "Smax"):
        assert dec_rc(lib, **{name: 0}) == 2
    assert dec_rc(lib, Hq=6, Hkv=4) == 2
    # (batch, head) rows or key stages past 32-bit indexing
    assert dec_rc(lib, B=1 << 20, Hq=4096, Hkv=4096) == 2
    assert dec_rc(lib, B=1 << 16, Hq=8, Hkv=2, Smax=1 << 20) == 2
    assert dec_rc(lib, D=96) == 3
    assert dec_rc(lib, Hq=34, Hkv=2) == 3  # group of 17 query heads
    assert dec_rc(lib, parts=-1, ws_bytes=1 << 30) == 7
    assert dec_rc(lib, parts=mk.DECODE_MAX_PARTS + 1, ws_bytes=1 << 40) == 7
    assert dec_rc(lib, scale=math.nan) == 7
    for name in ("q", "kc", "vc", "o"):
        assert dec_rc(lib, **{name: P_ODD}) == 4
    assert dec_rc(lib, seqlens=P + 2) == 4
    assert dec_rc(lib, lse=P + 1) == 4
    assert dec_rc(lib, ws=None) == 5
    need = lib.mk_attn_decode_workspace_bytes(8, 2, 128, 0)
    assert dec_rc(lib, ws_bytes=need - 1) == 5
    assert dec_rc(lib, parts=100, ws_bytes=lib.mk_attn_decode_workspace_bytes(8, 2, 128, 99)) == 5
    assert dec_rc(lib, ws=P + 16) == 4  # workspace must be 256-byte aligned


def noalloc_rc(lib, *, q=P, kc=P, vc=P, o=P, lse=None, B=2, Hq=8, Hkv=2, Smax=512, D=128,
               scale=0.1, seqlens=P, parts=0):
    return lib.mk_attn_decode_noalloc(q, kc, vc, o, lse, B, Hq, Hkv, Smax, D, scale, seqlens,
                                      parts, None)


def test_decode_noalloc_validation(lib):
    # every check runs on the host before any HIP call, so nothing here
    # reaches the device
    assert lib.mk_attn_decode_noalloc_max_bytes() == 16 << 20
    for name in ("q", "kc", "vc", "o", "seqlens"):
        assert noalloc_rc(lib, **{name: None}) == 1
    for name in ("B", "Hq", "Hkv", "Smax"):
        assert noalloc_rc(lib, **{name: 0}) == 2
    assert noalloc_rc(lib, D=96) == 3
    assert noalloc_rc(lib, Hq=34, Hkv=2) == 3
    assert noalloc_rc(lib, parts=-1) == 7
    assert noalloc_rc(lib, scale=math.nan) == 7
    for name in ("q", "kc", "vc", "o"):
        assert noalloc_rc(lib, **{name: P_ODD}) == 4
    # a part count whose workspace passes the fixed array's size
    cap = lib.mk_attn_decode_noalloc_max_bytes()
    big = 1
    while lib.mk_attn_decode_workspace_bytes(32, 2, 128, big) <= cap:
        big *= 2
    assert noalloc_rc(lib, Hq=32, Hkv=2, parts=big) == 8


def paged_rc(lib, *, q=P, kp=P, vp=P, bt=P, o=P, lse=None, B=2, Hq=8, Hkv=2, ps=16,
             max_pages=32, n_pages=64, D=128, scale=0.1, seqlens=P, parts=0, ws=P,
             ws_bytes=None):
    if ws_bytes is None:
        ws_bytes = lib.mk_attn_decode_workspace_bytes(max(Hq, 1), max(Hkv, 1), D, max(parts, 0))
    return lib.mk_attn_decode_paged(q, kp, vp, bt, o, lse, B, Hq, Hkv, ps, max_pages, n_pages, D,
                                    scale, seqlens, parts, ws, ws_bytes, None)


def test_decode_paged_validation(lib):
    for name in ("q", "kp", "vp", "bt", "o", "seqlens"):
        assert paged_rc(lib, **{name: None}) == 1
    for name in ("B", "Hq", "Hkv", "max_pages", "n_pages"):
        assert paged_rc(lib, **{name: 0}) == 2
    for ps in (0, 8, 24, -16):  # page size: a positive multiple of 16
        assert paged_rc(lib, ps=ps) == 2
    assert paged_rc(lib, Hq=6, Hkv=4) == 2
    # 32-bit limits: table entries, keys per sequence, key stages
    assert paged_rc(lib, B=1 << 16, max_pages=1 << 16) == 2
    assert paged_rc(lib, B=1, ps=1 << 16, max_pages=1 << 16) == 2
    assert paged_rc(lib, B=1 << 12, Hkv=64, Hq=64, ps=4096, max_pages=64) == 2
    assert paged_rc(lib, D=96) == 3
    assert paged_rc(lib, Hq=34, Hkv=2) == 3
    assert paged_rc(lib, parts=-1, ws_bytes=1 << 30) == 7
    assert paged_rc(lib, scale=math.inf) == 7
    for name in ("q", "kp", "vp", "o"):
        assert paged_rc(lib, **{name: P_ODD}) == 4
    assert paged_rc(lib, bt=P + 2) == 4
    assert paged_rc(lib, seqlens=P + 2) == 4
    assert paged_rc(lib, ws=None) == 5
    need = lib.mk_attn_decode_workspace_bytes(8, 2, 128, 0)
    assert paged_rc(lib, ws_bytes=need - 1) == 5
    assert paged_rc(lib, ws=P + 64) == 4


def test_decode_default_parts(lib):
    # 256 compute units x the single-wave workgroups whose LDS ring (three
    # slots of K and V for 32 keys plus the group's query rows in 1 KB
    # loads) fits in 160 KiB
    def expect(G, D):
        q_kb = -(-G // (512 // D))
        q_kb = 1 if q_kb <= 1 else (2 if q_kb <= 2 else 4)
        ring = 3 * (2 * 32 * D * 2 + q_kb * 1024)
        return 256 * max(1, (160 * 1024) // ring)
    for Hq, Hkv, D in ((32, 8, 128), (8, 1, 128), (16, 1, 128), (4, 4, 64), (16, 1, 64)):
        assert mk.mk_attn_decode_default_parts(Hq, Hkv, D) == expect(Hq // Hkv, D)
    assert mk.mk_attn_decode_default_parts(32, 8, 128) == 768
    assert mk.mk_attn_decode_default_parts(34, 2, 128) == 0
    assert mk.mk_attn_decode_default_parts(6, 4, 128) == 0
    assert mk.mk_attn_decode_default_parts(8, 2, 96) == 0


def test_decode_workspace_size(lib):
    rnd = lambda x: -(-x // 256) * 256
    for Hq, Hkv, D, P in ((32, 8, 128, 768), (16, 1, 64, 3), (4, 4, 128, 1)):
        G = Hq // Hkv
        # partial outputs, their LSEs, then one int32 [4] record per part
        want = rnd(P * 2 * G * D * 4) + rnd(P * 2 * G * 4) + rnd(P * 4 * 4)
        assert lib.mk_attn_decode_workspace_bytes(Hq, Hkv, D, P) == want
    assert lib.mk_attn_decode_workspace_bytes(32, 8, 128, 0) == \
        lib.mk_attn_decode_workspace_bytes(32, 8, 128, 768)
    assert lib.mk_attn_decode_workspace_bytes(0, 1, 64, 0) == 0
    assert lib.mk_attn_decode_workspace_bytes(8, 2, 64, -1) == 0
    assert lib.mk_attn_decode_workspace_bytes(8, 2, 80, 0) == 0
    assert lib.mk_attn_decode_workspace_bytes(8, 2, 64, mk.DECODE_MAX_PARTS + 1) == 0


def test_missing_library_fails_loudly(monkeypatch, tmp_path):
    monkeypatch.setattr(mk, "_lib", None)
    monkeypatch.setattr(mk, "LIB_PATH", str(tmp_path / "libmk_attn.so"))
    with pytest.raises(RuntimeError, match="has not been built"):
        mk.lib()


def bwd_rc(lib, *, q=P, k=P, v=P, o=P, do=P, lse=P, dq=P, dk=P, dv=P, B=2, Hq=8, Hkv=2, Sq=100,
           Skv=200, D=128, causal=1, scale=0.125, seqlens=None, ws=P, ws_bytes=None):
    if ws_bytes is None:
        ws_bytes = lib.mk_attn_bwd_workspace_bytes(max(B, 1), max(Hq, 1), max(Sq, 1))
    return lib.mk_attn_bwd(q, k, v, o, do, lse, dq, dk, dv, B, Hq, Hkv, Sq, Skv, D, causal, scale,
                           seqlens, ws, ws_bytes, None)


def test_bwd_workspace_bytes(lib):
    # two arrays of B * Hq * round_up(Sq, 128) fp32, each 256-byte aligned
    assert lib.mk_attn_bwd_workspace_bytes(2, 8, 100) == 2 * 2 * 8 * 128 * 4
    assert lib.mk_attn_bwd_workspace_bytes(1, 1, 1) == 2 * 512
    assert lib.mk_attn_bwd_workspace_bytes(1, 3, 130) == 2 * 3 * 256 * 4
    assert lib.mk_attn_bwd_workspace_bytes(0, 8, 100) == 0
    assert lib.mk_attn_bwd_workspace_bytes(2, 8, -1) == 0


def test_bwd_validation(lib):
    for name in ("q", "k", "v", "o", "do", "lse", "dq", "dk", "dv"):
        assert bwd_rc(lib, **{name: None}) == 1
    for name in ("B", "Hq", "Hkv", "Sq", "Skv"):
        assert bwd_rc(lib, **{name: 0}) == 2
    assert bwd_rc(lib, Hq=6, Hkv=4) == 2
    assert bwd_rc(lib, B=1 << 16, Hq=1 << 12, Hkv=1 << 12, Sq=1 << 10, ws_bytes=1 << 62) == 2
    assert bwd_rc(lib, D=96) == 3
    assert bwd_rc(lib, causal=2) == 7
    assert bwd_rc(lib, scale=math.inf) == 7
    for name in ("q", "k", "v", "o", "do", "dq", "dk", "dv"):
        assert bwd_rc(lib, **{name: P_ODD}) == 4
    assert bwd_rc(lib, lse=P + 2) == 4
    assert bwd_rc(lib, seqlens=P + 1) == 4
    assert bwd_rc(lib, ws=None) == 5
    assert bwd_rc(lib, ws_bytes=lib.mk_attn_bwd_workspace_bytes(2, 8, 100) - 1) == 5
    assert bwd_rc(lib, ws=P + 16) == 4


def mla_rc(lib, *, q=P, ckv=P, o=P, lse=None, B=4, H=16, Dc=512, Dr=64, Smax=1000, scale=0.07,
           seqlens=P, parts=0, ws=P, ws_bytes=None):
    if ws_bytes is None:
        ws_bytes = lib.mk_attn_mla_decode_workspace_bytes(16, 512, max(parts, 0))
    return lib.mk_attn_mla_decode(q, ckv, o, lse, B, H, Dc, Dr, Smax, scale, seqlens, parts, ws,
                                  ws_bytes, None)


def test_mla_workspace_bytes(lib):
    # default: 256 parts x 2 pieces x 16 heads x 512 fp32, then 256 x 2 x 16 fp32
    assert lib.mk_attn_mla_decode_workspace_bytes(16, 512, 0) == 256 * 2 * 16 * 512 * 4 + 32768
    assert lib.mk_attn_mla_decode_workspace_bytes(16, 512, 3) == 3 * 2 * 16 * 512 * 4 + 512
    assert lib.mk_attn_mla_decode_workspace_bytes(8, 512, 0) == 0
    assert lib.mk_attn_mla_decode_workspace_bytes(16, 256, 0) == 0


def test_mla_decode_validation(lib):
    for name in ("q", "ckv", "o", "seqlens"):
        assert mla_rc(lib, **{name: None}) == 1
    for name in ("B", "H", "Dc", "Smax"):
        assert mla_rc(lib, **{name: 0}) == 2
    assert mla_rc(lib, Dr=-1) == 2
    assert mla_rc(lib, B=1 << 20, Smax=1 << 20) == 2  # key stages past 32-bit indexing
    assert mla_rc(lib, H=32) == 3
    assert mla_rc(lib, Dc=256) == 3
    assert mla_rc(lib, Dr=0) == 3
    assert mla_rc(lib, parts=-1) == 7
    assert mla_rc(lib, scale=math.nan) == 7
    for name in ("q", "ckv", "o"):
        assert mla_rc(lib, **{name: P_ODD}) == 4
    assert mla_rc(lib, seqlens=P + 2) == 4
    assert mla_rc(lib, lse=P + 1) == 4
    assert mla_rc(lib, ws=None) == 5
    assert mla_rc(lib, ws_bytes=lib.mk_attn_mla_decode_workspace_bytes(16, 512, 0) - 1) == 5
    assert mla_rc(lib, ws=P + 16) == 4
