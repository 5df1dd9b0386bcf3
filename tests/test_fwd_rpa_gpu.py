"""Ragged paged forward on the GPU (paper_2609_04523_amd.mk_attn_fwd_ragged_paged,
through the C ABI): packed query chunks and decode tokens over a paged key/value
cache, against the fp64 oracle's ragged paged forward, and bitwise against the
packed forward run on the keys and values gathered from the pages.  Page pools
hold NaN in every row past a sequence's length and in every page no table
lists, so a read of them would show in the result."""
import numpy as np
import pytest
import torch

import paper_2609_04523_amd as mk
import workloads
from oracle import oracle as orc
from parity import assert_parity

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def run_rpa(q, kp, vp, bt, cu, lens, *, causal, scale, max_sq=None):
    max_sq = max_sq or max(1, int(np.max(np.diff(cu.numpy()))))
    o, lse = mk.fwd_ragged_paged(q.to(DEV), kp.to(DEV), vp.to(DEV), bt.to(DEV), cu.to(DEV),
                                 lens.to(DEV), max_sq, causal=causal, scale=scale)
    torch.cuda.synchronize()
    return o, lse


def oracle_rpa(q, kp, vp, bt, cu, lens, *, causal, scale):
    return orc.attn_fwd_ragged_paged(workloads.bits(q), workloads.bits(kp), workloads.bits(vp),
                                     cu.numpy(), lens.numpy(), bt.numpy(), causal=causal,
                                     scale=scale)


def check(name, o, lse, o_ref, lse_ref, total_q):
    # the [1, Hq, total_q, D] / [1, Hq, total_q] shapes the checker takes
    assert_parity(name, o[:total_q].permute(1, 0, 2)[None], lse[:, :total_q][None],
                  o_ref[:total_q].transpose(1, 0, 2)[None], lse_ref[:, :total_q][None])


# name, Hq, Hkv, D, page_size, sequences [(Sq, L)]
CASES = [
    ("mixed_ps16", 8, 2, 128, 16, [(1, 700), (300, 300), (1, 65), (129, 900), (1, 1), (0, 50)]),
    ("chunks_ps32", 4, 4, 128, 32, [(64, 64), (200, 450), (3, 3), (130, 130)]),
    ("queries_past_keys_ps48", 8, 2, 128, 48, [(150, 40), (70, 200)]),
    ("empty_ps64_d64", 4, 1, 64, 64, [(0, 10), (90, 90), (20, 0), (33, 100)]),
    ("gqa16_ps128_d64", 16, 1, 64, 128, [(257, 257), (1, 513)]),
    ("long_ps256", 8, 1, 128, 256, [(600, 1500), (1, 2000), (64, 64)]),
]


@pytest.mark.parametrize("causal", [True, False])
@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_rpa_against_oracle(case, causal):
    name, Hq, Hkv, D, ps, seqs = case
    q, kp, vp, bt, cu, lens, _, _ = workloads.ragged_paged_inputs(seqs, Hq, Hkv, D, ps,
                                                                  seed=len(name), extra_pages=7)
    scale = D ** -0.5
    o, lse = run_rpa(q, kp, vp, bt, cu, lens, causal=causal, scale=scale)
    o_ref, lse_ref = oracle_rpa(q, kp, vp, bt, cu, lens, causal=causal, scale=scale)
    check(f"{name} causal={causal}", o, lse, o_ref, lse_ref, int(cu[-1]))


@pytest.mark.parametrize("causal", [True, False])
@pytest.mark.parametrize("ps", [16, 64, 256])
def test_rpa_equals_varlen_on_gathered_keys_bitwise(ps, causal):
    seqs = [(2048, 2048), (1, 3000), (700, 1800), (1, 17), (64, 64), (5, 4000)]
    Hq, Hkv, D = 32, 8, 128
    q, kp, vp, bt, cu, lens, kc, vc = workloads.ragged_paged_inputs(seqs, Hq, Hkv, D, ps,
                                                                    seed=11 + ps)
    o, lse = run_rpa(q, kp, vp, bt, cu, lens, causal=causal, scale=D ** -0.5)
    # the same keys packed token-major for the packed forward
    k = torch.cat([kc[b, :, :L].permute(1, 0, 2) for b, (_, L) in enumerate(seqs)]).contiguous()
    v = torch.cat([vc[b, :, :L].permute(1, 0, 2) for b, (_, L) in enumerate(seqs)]).contiguous()
    ck = torch.zeros(len(seqs) + 1, dtype=torch.int32)
    ck[1:] = torch.cumsum(lens, 0)
    ov, lv = mk.fwd_varlen(q.to(DEV), k.to(DEV), v.to(DEV), cu.to(DEV), ck.to(DEV),
                           int(np.max(np.diff(cu.numpy()))), causal=causal, scale=D ** -0.5)
    torch.cuda.synchronize()
    tq = int(cu[-1])
    assert torch.equal(o[:tq], ov[:tq]), "O differs from the packed forward"
    assert torch.equal(lse[:, :tq], lv[:, :tq]), "LSE differs from the packed forward"


def test_rpa_table_entries_clamped_and_unread():
    seqs = [(100, 300), (1, 130), (40, 40)]
    Hq, Hkv, D, ps = 8, 2, 128, 32
    q, kp, vp, bt, cu, lens, _, _ = workloads.ragged_paged_inputs(seqs, Hq, Hkv, D, ps, seed=5,
                                                                  extra_pages=3)
    base = run_rpa(q, kp, vp, bt, cu, lens, causal=True, scale=D ** -0.5)
    n_pages = kp.shape[0]
    # entries past each sequence's last page are never read
    bt2 = bt.clone()
    for b, (_, L) in enumerate(seqs):
        bt2[b, -(-L // ps):] = torch.tensor([-(10 ** 6), 10 ** 6, -1, n_pages])[
            torch.arange(bt.shape[1] - (-(-L // ps))) % 4]
    got = run_rpa(q, kp, vp, bt2, cu, lens, causal=True, scale=D ** -0.5)
    assert torch.equal(base[0][:141], got[0][:141]) and torch.equal(base[1][:, :141], got[1][:, :141])
    # an entry outside the pool inside a sequence reads the nearest valid page
    # (pages 0 and n_pages - 1, given finite rows here)
    g = torch.Generator().manual_seed(55)
    for pg in (0, n_pages - 1):
        kp[pg] = torch.randn(kp[pg].shape, generator=g).to(torch.bfloat16)
        vp[pg] = torch.randn(vp[pg].shape, generator=g).to(torch.bfloat16)
    bt3 = bt.clone()
    bt3[0, 2] = -5
    bt3[0, 4] = n_pages + 9
    o3, l3 = run_rpa(q, kp, vp, bt3, cu, lens, causal=True, scale=D ** -0.5)
    o_ref, lse_ref = oracle_rpa(q, kp, vp, bt3, cu, lens, causal=True, scale=D ** -0.5)
    check("clamped table entries", o3, l3, o_ref, lse_ref, int(cu[-1]))


def test_rpa_lengths_clamped():
    # lengths past the table clamp to max_pages * page_size, negative ones to 0
    seqs = [(50, 256), (20, 256), (30, 128)]
    Hq, Hkv, D, ps = 4, 2, 128, 64
    q, kp, vp, bt, cu, lens, _, _ = workloads.ragged_paged_inputs(seqs, Hq, Hkv, D, ps, seed=9)
    lens_x = torch.tensor([10 ** 7, -3, 128], dtype=torch.int32)
    o, lse = run_rpa(q, kp, vp, bt, cu, lens_x, causal=True, scale=D ** -0.5)
    o_ref, lse_ref = oracle_rpa(q, kp, vp, bt, cu, lens_x, causal=True, scale=D ** -0.5)
    check("clamped lengths", o, lse, o_ref, lse_ref, int(cu[-1]))
    assert torch.all(o[50:70] == 0) and torch.all(torch.isneginf(lse[:, 50:70]))


@pytest.mark.parametrize("ps", [16, 64])
def test_rpa_steeply_rising_scores(ps):
    # keys after each sequence's first 128 scaled up steeply (q x12, later
    # keys x4 against x0.05 for the first ones): tiles weighed against the
    # running maximum overflow and are formed again from K read through the
    # block table
    seqs = [(400, 400), (1, 300), (260, 520)]
    Hq, Hkv, D = 4, 2, 128
    q, kp, vp, bt, cu, lens, kc, vc = workloads.ragged_paged_inputs(seqs, Hq, Hkv, D, ps,
                                                                    seed=4242)
    q = (q.float() * 12.0).to(torch.bfloat16)
    kf = kc.float()
    kf[:, :, :128] *= 0.05
    kf[:, :, 128:] *= 4.0
    kp, vp, bt = workloads.paged_layout(kf.to(torch.bfloat16), vc, ps, seed=4243, lens=lens)
    o, lse = run_rpa(q, kp, vp, bt, cu, lens, causal=True, scale=D ** -0.5)
    o_ref, lse_ref = oracle_rpa(q, kp, vp, bt, cu, lens, causal=True, scale=D ** -0.5)
    check(f"rising scores ps={ps}", o, lse, o_ref, lse_ref, int(cu[-1]))


def test_rpa_deterministic_bitwise():
    seqs = [(1000, 3000), (1, 2000), (777, 777)]
    q, kp, vp, bt, cu, lens, _, _ = workloads.ragged_paged_inputs(seqs, 32, 8, 128, 16, seed=31)
    a = run_rpa(q, kp, vp, bt, cu, lens, causal=True, scale=128 ** -0.5)
    b = run_rpa(q, kp, vp, bt, cu, lens, causal=True, scale=128 ** -0.5)
    assert torch.equal(a[0], b[0]) and torch.equal(a[1], b[1])
