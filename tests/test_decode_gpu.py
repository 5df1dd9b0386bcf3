"""Split-KV decode on the GPU against the fp64 oracle, through the C ABI
(paper_2609_04523_amd.mk_attn_decode)."""
import math

import numpy as np
import pytest
import torch

import paper_2609_04523_amd as mk
import workloads
from oracle import oracle as orc
from parity import assert_parity, to_f64

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
NAN_BF16 = 0x7FC0


def poison_padding(cache: torch.Tensor, lens) -> torch.Tensor:
    """NaN into every cache position at or past the sequence length."""
    c = cache.clone()
    bits = c.view(torch.int16)
    for b, L in enumerate(lens):
        L = max(0, min(int(L), c.shape[2]))
        bits[b, :, L:, :] = NAN_BF16
    return c


def run_decode(q, kc, vc, lens, *, scale, split=0, return_ws=False):
    sl = torch.as_tensor(np.asarray(lens, dtype=np.int32)).to(DEV)
    B, Hq, D = q.shape
    Smax = kc.shape[2]
    ws = torch.empty(mk.mk_attn_decode_workspace_bytes(B, Hq, Smax, D, split), device=DEV,
                     dtype=torch.uint8)
    o, lse = mk.decode(q.to(DEV), kc.to(DEV), vc.to(DEV), sl, scale=scale, split=split,
                       workspace=ws)
    torch.cuda.synchronize()
    return (o, lse, ws) if return_ws else (o, lse)


def oracle_decode(q, kc, vc, lens, scale):
    return orc.decode(workloads.bits(q), workloads.bits(kc), workloads.bits(vc),
                      np.asarray(lens, dtype=np.int32), scale=scale)


def test_decode_config5_full_with_poisoned_padding():
    cfg = workloads.CONFIGS["c5_decode_b64"]
    q, kc, vc, lens = workloads.config_inputs(cfg)
    kcp, vcp = poison_padding(kc, lens.tolist()), poison_padding(vc, lens.tolist())
    o, lse = run_decode(q, kcp, vcp, lens, scale=cfg.scale)
    o_ref, lse_ref = oracle_decode(q, kc, vc, lens, cfg.scale)
    assert_parity(cfg.name, o, lse, o_ref, lse_ref)


@pytest.mark.parametrize("split", [0, 64, 100, 512, 1000, 4096])
def test_decode_split_lengths(split):
    B, Hq, Hkv, Smax, D = 8, 32, 8, 2048, 128
    q, kc, vc, lens = workloads.decode_inputs(B, Hq, Hkv, Smax, D, seed=21, lmin=1, lmax=Smax)
    scale = D ** -0.5
    o, lse = run_decode(q, kc, vc, lens, scale=scale, split=split)
    o_ref, lse_ref = oracle_decode(q, kc, vc, lens, scale)
    assert_parity(f"split{split}", o, lse, o_ref, lse_ref)


# name, B, Hq, Hkv, Smax, D, lens
SHAPES = [
    ("mha_d64", 3, 4, 4, 300, 64, [300, 1, 65]),
    ("gqa8_d128", 2, 16, 2, 1000, 128, [999, 128]),
    ("gqa16_d64", 2, 16, 1, 700, 64, [700, 63]),
    ("gqa4_lengths_edge", 4, 8, 2, 512, 128, [0, 1, 511, 512]),
    ("clamped_lengths", 3, 8, 2, 256, 128, [-7, 100000, 129]),
    ("single_key_cache", 2, 4, 1, 1, 128, [1, 1]),
]


@pytest.mark.parametrize("case", SHAPES, ids=[c[0] for c in SHAPES])
def test_decode_shapes(case):
    name, B, Hq, Hkv, Smax, D, lens = case
    g = torch.Generator().manual_seed(len(name))
    q = torch.randn((B, Hq, D), generator=g).to(torch.bfloat16)
    kc = torch.randn((B, Hkv, Smax, D), generator=g).to(torch.bfloat16)
    vc = torch.randn((B, Hkv, Smax, D), generator=g).to(torch.bfloat16)
    scale = D ** -0.5
    o, lse = run_decode(q, poison_padding(kc, lens), poison_padding(vc, lens), lens, scale=scale)
    o_ref, lse_ref = oracle_decode(q, kc, vc, lens, scale)
    assert_parity(name, o, lse, o_ref, lse_ref)


def test_decode_partials_match_oracle_split_steps():
    B, Hq, Hkv, Smax, D = 4, 8, 2, 1500, 128
    q, kc, vc, lens = workloads.decode_inputs(B, Hq, Hkv, Smax, D, seed=22, lmin=1, lmax=Smax)
    scale = D ** -0.5
    split = 256
    o, lse, ws = run_decode(q, kc, vc, lens, scale=scale, split=split, return_ws=True)
    o_part, lse_part = mk.decode_partials(ws, B, Hq, Smax, D, split)
    _, _, op_ref, lp_ref = orc.decode_split(workloads.bits(q), workloads.bits(kc),
                                            workloads.bits(vc), lens.numpy(), scale=scale,
                                            split=split)
    for b in range(B):
        ns = -(-int(lens[b]) // split)
        assert_parity(f"partials b{b}", o_part[b, :, :ns], lse_part[b, :, :ns],
                      op_ref[b, :, :ns], lp_ref[b, :, :ns])


def test_decode_equals_last_prefill_row():
    B, Hq, Hkv, S, D = 2, 8, 2, 700, 128
    q, k, v = workloads.prefill_inputs(B, Hq, Hkv, S, S, D, seed=23)
    o_p, lse_p = mk.fwd(q.to(DEV), k.to(DEV), v.to(DEV), causal=True)
    o_d, lse_d = run_decode(q[:, :, -1].contiguous(), k, v, [S] * B, scale=D ** -0.5)
    e = (o_p[:, :, -1].double() - o_d.double()).abs().max().item()
    assert e <= 2e-2
    assert (lse_p[:, :, -1] - lse_d).abs().max().item() <= 1e-3


def test_decode_deterministic_bitwise():
    q, kc, vc, lens = workloads.decode_inputs(16, 32, 8, 1024, 128, seed=24)
    a = run_decode(q, kc, vc, lens, scale=128 ** -0.5)
    b = run_decode(q, kc, vc, lens, scale=128 ** -0.5)
    assert torch.equal(a[0], b[0]) and torch.equal(a[1], b[1])
