"""Paged-cache decode on the GPU (paper_2609_04523_amd.mk_attn_decode_paged,
through the C ABI) against the fp64 oracle's paged decode, and against the
contiguous decode kernel on the same keys."""
import numpy as np
import pytest
import torch

import paper_2609_04523_amd as mk
import workloads
from oracle import oracle as orc
from parity import assert_parity

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def run_paged(q, kp, vp, bt, lens, *, scale, n_parts=0):
    sl = torch.as_tensor(np.asarray(lens, dtype=np.int32)).to(DEV)
    o, lse = mk.decode_paged(q.to(DEV), kp.to(DEV), vp.to(DEV), bt.to(DEV), sl, scale=scale,
                             n_parts=n_parts)
    torch.cuda.synchronize()
    return o, lse


def oracle_paged(q, kp, vp, bt, lens, scale):
    return orc.decode_paged(workloads.bits(q), workloads.bits(kp), workloads.bits(vp),
                            bt.numpy(), np.asarray(lens, dtype=np.int32), scale=scale)


def test_paged_decode_workload_page16():
    # the decode workload with its cache scattered over 16-key pages in a
    # seeded random order, unused pages and rows past each length NaN
    cfg = workloads.CONFIGS["c5_decode_b64"]
    q, kc, vc, lens = workloads.config_inputs(cfg)
    kp, vp, bt = workloads.paged_layout(kc, vc, 16, seed=77, extra_pages=64, lens=lens)
    o, lse = run_paged(q, kp, vp, bt, lens, scale=cfg.scale)
    o_ref, lse_ref = oracle_paged(q, kp, vp, bt, lens, cfg.scale)
    assert_parity("paged c5 ps16", o, lse, o_ref, lse_ref)


# name, B, Hq, Hkv, Smax, D, page_size, lens
SHAPES = [
    ("ps16_edges", 6, 8, 2, 128, 128, 16, [0, 1, 15, 16, 17, 128]),
    ("ps32_d64_g8", 3, 16, 2, 256, 64, 32, [31, 32, 33]),
    ("ps48_odd_multiple", 3, 4, 1, 240, 128, 48, [47, 48, 239]),
    ("ps64_g16", 2, 16, 1, 320, 128, 64, [320, 65]),
    ("ps256_g1", 4, 4, 4, 512, 128, 256, [511, 256, 257, 3]),
    ("ps16_d64_g12", 2, 12, 1, 160, 64, 16, [160, 95]),
]


@pytest.mark.parametrize("case", SHAPES, ids=[c[0] for c in SHAPES])
def test_paged_decode_shapes(case):
    name, B, Hq, Hkv, Smax, D, ps, lens = case
    g = torch.Generator().manual_seed(len(name) * 7)
    q = torch.randn((B, Hq, D), generator=g).to(torch.bfloat16)
    kc = torch.randn((B, Hkv, Smax, D), generator=g).to(torch.bfloat16)
    vc = torch.randn((B, Hkv, Smax, D), generator=g).to(torch.bfloat16)
    kp, vp, bt = workloads.paged_layout(kc, vc, ps, seed=len(name), extra_pages=3, lens=lens)
    scale = D ** -0.5
    o, lse = run_paged(q, kp, vp, bt, lens, scale=scale)
    o_ref, lse_ref = oracle_paged(q, kp, vp, bt, lens, scale)
    assert_parity(name, o, lse, o_ref, lse_ref)


@pytest.mark.parametrize("n_parts", [1, 7, 768, 5000])
def test_paged_equals_contiguous_bitwise(n_parts):
    # same stream of stages, same arithmetic: the paged kernel must give the
    # contiguous kernel's bits on the same keys, for any part count
    B, Hq, Hkv, Smax, D = 8, 32, 8, 1024, 128
    q, kc, vc, lens = workloads.decode_inputs(B, Hq, Hkv, Smax, D, seed=41, lmin=1, lmax=Smax)
    kp, vp, bt = workloads.paged_layout(kc, vc, 16, seed=42, extra_pages=5, lens=lens)
    sl = lens.to(DEV)
    o_c, lse_c = mk.decode(q.to(DEV), kc.to(DEV), vc.to(DEV), sl, scale=D ** -0.5,
                           n_parts=n_parts)
    o_p, lse_p = run_paged(q, kp, vp, bt, lens, scale=D ** -0.5, n_parts=n_parts)
    assert torch.equal(o_c, o_p) and torch.equal(lse_c, lse_p)


def test_paged_table_entries_clamped_and_pages_shared():
    # out-of-range table entries read the nearest valid page; two sequences
    # may list the same pages (a shared prefix)
    B, Hq, Hkv, D, ps, mp = 3, 8, 2, 128, 16, 6
    n_pages = 10
    g = torch.Generator().manual_seed(51)
    q = torch.randn((B, Hq, D), generator=g).to(torch.bfloat16)
    kp = torch.randn((n_pages, Hkv, ps, D), generator=g).to(torch.bfloat16)
    vp = torch.randn((n_pages, Hkv, ps, D), generator=g).to(torch.bfloat16)
    bt = torch.tensor([[4, 7, -3, 9, 2, 0], [4, 7, 1, 55, 8, 3], [2, 2, 2, 2, 2, 2]],
                      dtype=torch.int32)
    lens = [96, 70, 40]
    scale = D ** -0.5
    o, lse = run_paged(q, kp, vp, bt, lens, scale=scale)
    o_cl, lse_cl = run_paged(q, kp, vp, bt.clamp(0, n_pages - 1), lens, scale=scale)
    assert torch.equal(o, o_cl) and torch.equal(lse, lse_cl)
    o_ref, lse_ref = oracle_paged(q, kp, vp, bt, lens, scale)
    assert_parity("clamped/shared", o, lse, o_ref, lse_ref)


def test_paged_decode_deterministic_bitwise():
    q, kc, vc, lens = workloads.decode_inputs(16, 32, 8, 1024, 128, seed=61)
    kp, vp, bt = workloads.paged_layout(kc, vc, 32, seed=62, lens=lens)
    a = run_paged(q, kp, vp, bt, lens, scale=128 ** -0.5)
    b = run_paged(q, kp, vp, bt, lens, scale=128 ** -0.5)
    assert torch.equal(a[0], b[0]) and torch.equal(a[1], b[1])
