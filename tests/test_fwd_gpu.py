"""Attention forward on the GPU against the fp64 oracle (parity) and
against facts that hold at any size (invariants).  Calls go through the
C ABI (paper_2609_04523_amd.mk_attn_fwd / mk_attn_fwd_o32)."""
import math
import zlib

import numpy as np
import pytest
import torch

import paper_2609_04523_amd as mk
import workloads
from oracle import oracle as orc
from parity import assert_parity, to_f64

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def run_fwd(q, k, v, *, causal, scale, kv_seqlens=None, out_fp32=False):
    qd, kd, vd = q.to(DEV), k.to(DEV), v.to(DEV)
    sl = None if kv_seqlens is None else torch.tensor(kv_seqlens, dtype=torch.int32, device=DEV)
    o, lse = mk.fwd(qd, kd, vd, causal=causal, scale=scale, kv_seqlens=sl, out_fp32=out_fp32)
    torch.cuda.synchronize()
    return o, lse


def oracle_fwd(q, k, v, *, causal, scale, kv_seqlens=None, rows=None):
    return orc.attn_fwd(workloads.bits(q), workloads.bits(k), workloads.bits(v), causal=causal,
                        scale=scale, kv_seqlens=kv_seqlens, rows=rows)


# name, B, Hq, Hkv, Sq, Skv, D, causal, kv_seqlens, out_fp32, k_mult
CASES = [
    ("c1_mha_s128_d64_o32", 1, 2, 2, 128, 128, 64, True, None, True, 1.0),
    ("s1_d128", 1, 2, 1, 1, 1, 128, True, None, False, 1.0),
    ("s17_gqa2", 2, 4, 2, 17, 17, 128, True, None, False, 1.0),
    ("s129_noncausal", 1, 4, 4, 129, 129, 128, False, None, True, 1.0),
    ("s1000_gqa4_d64", 1, 8, 2, 1000, 1000, 64, True, None, False, 1.0),
    ("s300_d64_o32", 2, 2, 1, 300, 300, 64, True, None, True, 2.0),
    ("sq100_skv300_bottom_right", 2, 4, 1, 100, 300, 128, True, None, False, 1.0),
    ("ragged_lens", 3, 4, 2, 200, 300, 128, True, [300, 57, 0], False, 1.0),
    ("clamped_lens", 2, 2, 2, 64, 64, 128, True, [-5, 1000], False, 1.0),
    ("noncausal_lens_d64", 2, 4, 4, 77, 260, 64, False, [260, 100], True, 1.0),
    ("len_below_sq", 1, 2, 2, 300, 300, 128, True, [150], False, 1.0),
    ("s513_gqa8", 1, 16, 2, 513, 513, 128, True, None, False, 2.0),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_fwd_parity_shapes(case):
    name, B, Hq, Hkv, Sq, Skv, D, causal, sl, o32, kmul = case
    q, k, v = workloads.prefill_inputs(B, Hq, Hkv, Sq, Skv, D, seed=zlib.crc32(name.encode()) % 100000,
                                       k_mult=kmul)
    scale = 1.0 / math.sqrt(D)
    o, lse = run_fwd(q, k, v, causal=causal, scale=scale, kv_seqlens=sl, out_fp32=o32)
    o_ref, lse_ref = oracle_fwd(q, k, v, causal=causal, scale=scale, kv_seqlens=sl)
    assert_parity(name, o, lse, o_ref, lse_ref)


def _config_parity(cfg, rows_per_head=0):
    q, k, v = workloads.config_inputs(cfg)
    o, lse = run_fwd(q, k, v, causal=True, scale=cfg.scale, out_fp32=cfg.out_fp32)
    if rows_per_head:
        rows = workloads.sample_rows(cfg.B, cfg.Hq, cfg.S, rows_per_head, cfg.seed)
        o_ref, lse_ref = oracle_fwd(q, k, v, causal=True, scale=cfg.scale, rows=rows.numpy())
        idx = rows.long()
        o_s = torch.gather(o.cpu(), 2, idx[..., None].expand(-1, -1, -1, cfg.D))
        lse_s = torch.gather(lse.cpu(), 2, idx)
        return assert_parity(cfg.name, o_s, lse_s, o_ref, lse_ref)
    o_ref, lse_ref = oracle_fwd(q, k, v, causal=True, scale=cfg.scale)
    return assert_parity(cfg.name, o, lse, o_ref, lse_ref)


def test_fwd_mha_s128_d64_full():
    _config_parity(workloads.CONFIGS["c1_mha_s128_d64"])


def test_fwd_mha_s2k_full():
    _config_parity(workloads.CONFIGS["c2_mha_s2k"])


def test_fwd_gqa_s8k_k2_full():
    # every row of all 2 x 32 x 8192: the sharpened scores (K x 2) make
    # the largest |O|, and so the bf16 rounding of O, largest here
    _config_parity(workloads.CONFIGS["c3_gqa_s8k_k2"])


def test_fwd_gqa_s32k_sampled_rows():
    cfg = workloads.CONFIGS["c4_gqa_s32k"]
    _config_parity(cfg, rows_per_head=cfg.sample_rows)


# ---------------------------------------------------------------- invariants
def test_causal_row0_is_v0():
    # Row 0 sees key 0 alone: weight exp2(c*s - m) with m = c*s up to the
    # rounding of one fp32 product, so O = v_0 to a few fp32 ulps.
    B, Hq, Hkv, S, D = 2, 8, 2, 300, 128
    q, k, v = workloads.prefill_inputs(B, Hq, Hkv, S, S, D, seed=7)
    o, lse = run_fwd(q, k, v, causal=True, scale=0.0883883, out_fp32=True)
    G = Hq // Hkv
    for h in range(Hq):
        assert torch.allclose(o[:, h, 0].cpu(), v[:, h // G, 0].float(), rtol=1e-6, atol=0), \
            "row 0 != v_0"
    qf, kf = q.double(), k.double()
    s0 = torch.stack([(qf[:, h, 0] * kf[:, h // G, 0]).sum(-1) for h in range(Hq)], 1)
    ref = s0 * float(np.float32(0.0883883))
    assert torch.allclose(lse[:, :, 0].cpu().double(), ref, atol=1e-4, rtol=1e-5)


def test_scale_zero_prefix_mean():
    B, Hq, Hkv, S, D = 1, 4, 1, 333, 128
    q, k, v = workloads.prefill_inputs(B, Hq, Hkv, S, S, D, seed=8)
    o, lse = run_fwd(q, k, v, causal=True, scale=0.0, out_fp32=True)
    vf = v[0, 0].double()
    mean = torch.cumsum(vf, 0) / torch.arange(1, S + 1, dtype=torch.float64)[:, None]
    for h in range(Hq):
        assert torch.allclose(o[0, h].cpu().double(), mean, atol=1e-5, rtol=1e-5)
        assert torch.allclose(lse[0, h].cpu().double(),
                              torch.log(torch.arange(1, S + 1, dtype=torch.float64)),
                              atol=1e-5, rtol=0)


def test_equal_value_rows():
    B, Hq, Hkv, S, D = 1, 4, 2, 257, 128
    q, k, _ = workloads.prefill_inputs(B, Hq, Hkv, S, S, D, seed=9, k_mult=2.0)
    r = torch.randn(D, generator=torch.Generator().manual_seed(3)).to(torch.bfloat16)
    v = r.expand(B, Hkv, S, D).contiguous()
    for causal in (True, False):
        o, _ = run_fwd(q, k, v, causal=causal, scale=D ** -0.5, out_fp32=True)
        err = (o.cpu().double() - r.double()).abs()
        # numerator uses bf16 P, denominator fp32 P: relative error <= 2^-8
        assert float(err.max()) <= 2.0 ** -8 * float(r.double().abs().max()) + 1e-6


def test_gqa_equals_repeated_mha_bitwise():
    B, Hq, Hkv, S, D = 2, 8, 2, 200, 128
    q, k, v = workloads.prefill_inputs(B, Hq, Hkv, S, S, D, seed=10)
    o1, l1 = run_fwd(q, k, v, causal=True, scale=D ** -0.5)
    G = Hq // Hkv
    o2, l2 = run_fwd(q, k.repeat_interleave(G, 1).contiguous(),
                     v.repeat_interleave(G, 1).contiguous(), causal=True, scale=D ** -0.5)
    assert torch.equal(o1, o2) and torch.equal(l1, l2)


def test_deterministic_bitwise():
    cfg = workloads.CONFIGS["c2_mha_s2k"]
    q, k, v = workloads.prefill_inputs(1, 4, 4, 1024, 1024, 128, seed=11)
    a = run_fwd(q, k, v, causal=True, scale=cfg.scale)
    b = run_fwd(q, k, v, causal=True, scale=cfg.scale)
    assert torch.equal(a[0], b[0]) and torch.equal(a[1], b[1])


def test_lse_null_and_output_only():
    q, k, v = workloads.prefill_inputs(1, 2, 2, 70, 70, 128, seed=12)
    qd, kd, vd = q.to(DEV), k.to(DEV), v.to(DEV)
    o1, _ = mk.fwd(qd, kd, vd, causal=True, with_lse=False)
    o2, _ = mk.fwd(qd, kd, vd, causal=True)
    torch.cuda.synchronize()
    assert torch.equal(o1, o2)


def test_stream_argument_is_used():
    q, k, v = workloads.prefill_inputs(1, 4, 4, 256, 256, 128, seed=13)
    qd, kd, vd = q.to(DEV), k.to(DEV), v.to(DEV)
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        o, lse = mk.fwd(qd, kd, vd, causal=True, stream=s)
    s.synchronize()
    o_ref, lse_ref = oracle_fwd(q, k, v, causal=True, scale=128 ** -0.5)
    assert_parity("side_stream", o, lse, o_ref, lse_ref)


# Scores that rise steeply after the first tiles: tiles after the first are
# weighed against the running maximum without their own, so these rows make
# the kernel re-form a tile against its maximum (with q x12 and the later
# keys x4, c*s reaches ~166 > 128 above the first tile's maximum, where the
# first weighing overflows fp32).  name, Hq, Hkv, S, causal, q_mult, k_low,
# k_high, tiles of low keys
RISE_CASES = [
    ("rise_finite_causal", 4, 2, 512, True, 8.0, 0.05, 2.0, 1),
    ("rise_overflow_causal", 4, 2, 512, True, 12.0, 0.05, 4.0, 3),
    ("rise_overflow_noncausal_tail", 2, 1, 300, False, 12.0, 0.05, 4.0, 2),
]


@pytest.mark.parametrize("case", RISE_CASES, ids=[c[0] for c in RISE_CASES])
def test_fwd_steeply_rising_scores(case):
    name, Hq, Hkv, S, causal, qm, klo, khi, ntl = case
    q, k, v = workloads.prefill_inputs(1, Hq, Hkv, S, S, 128, seed=zlib.crc32(name.encode()) % 100000)
    q = (q.float() * qm).to(torch.bfloat16)
    kf = k.float()
    kf[:, :, :64 * ntl] *= klo
    kf[:, :, 64 * ntl:] *= khi
    k = kf.to(torch.bfloat16)
    scale = 128 ** -0.5
    o, lse = run_fwd(q, k, v, causal=causal, scale=scale)
    o_ref, lse_ref = oracle_fwd(q, k, v, causal=causal, scale=scale)
    assert_parity(name, o, lse, o_ref, lse_ref)
