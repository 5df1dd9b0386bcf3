"""MLA decode on the GPU (paper_2609_04523_amd.mk_attn_mla_decode, through
the C ABI) against the fp64 oracle's MLA decode on the same bf16 inputs,
with the decode parity bar (O max 2e-2, mean 2e-3, LSE 1e-3)."""
import numpy as np
import pytest
import torch

import paper_2609_04523_amd as mk
import workloads
from oracle import oracle as orc
from parity import assert_parity

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
W = workloads.MLA
NAN_BITS = 0x7FC0


def run(q, ckv, lens, *, scale, n_parts=0):
    o, lse = mk.mla_decode(q.to(DEV), ckv.to(DEV), torch.as_tensor(lens, dtype=torch.int32).to(DEV),
                           Dc=W["Dc"], scale=scale, n_parts=n_parts)
    torch.cuda.synchronize()
    return o, lse


def oracle(q, ckv, lens, scale):
    return orc.mla_decode(workloads.bits(q), workloads.bits(ckv), np.asarray(lens, np.int32),
                          Dc=W["Dc"], scale=scale)


def poison_padding(ckv, lens):
    """NaN in every cache row at or past a sequence's length."""
    bits = ckv.view(torch.int16).clone()
    for b, L in enumerate(lens):
        L = max(0, min(int(L), ckv.shape[1]))
        bits[b, L:] = NAN_BITS
    return bits.view(torch.bfloat16)


def test_mla_workload_full():
    q, ckv, lens = workloads.mla_inputs(W["B"], W["H"], W["Dc"], W["Dr"], W["Smax"], W["seed"],
                                        W["lmin"], W["lmax"])
    ckv = poison_padding(ckv, lens.tolist())
    o, lse = run(q, ckv, lens, scale=W["scale"])
    o_ref, lse_ref = oracle(q, ckv, lens, W["scale"])
    assert_parity("mla_decode_b64", o, lse, o_ref, lse_ref)


# lengths: one key, one stage, a ragged tail, empty, past Smax (clamped), negative
SHAPES = [
    ("ragged", [1, 31, 32, 33, 700], 704),
    ("empty_and_clamped", [0, 5000, -4, 129], 1024),
    ("one_sequence", [3000], 3072),
]


@pytest.mark.parametrize("case", SHAPES, ids=[c[0] for c in SHAPES])
@pytest.mark.parametrize("n_parts", [0, 1, 7, 5000])
def test_mla_shapes_and_parts(case, n_parts):
    name, lens, smax = case
    q, ckv, _ = workloads.mla_inputs(len(lens), W["H"], W["Dc"], W["Dr"], smax, 77)
    ckv = poison_padding(ckv, lens)
    o, lse = run(q, ckv, lens, scale=W["scale"], n_parts=n_parts)
    o_ref, lse_ref = oracle(q, ckv, lens, W["scale"])
    assert_parity(f"mla {name} parts={n_parts}", o, lse, o_ref, lse_ref)


def test_mla_rope_part_enters_the_scores():
    # a query whose latent part is zero scores the keys by the rotary part alone
    lens = [200, 64]
    q, ckv, _ = workloads.mla_inputs(2, W["H"], W["Dc"], W["Dr"], 256, 91)
    q[:, :, :W["Dc"]] = 0
    o, lse = run(q, ckv, lens, scale=0.3)
    o_ref, lse_ref = oracle(q, ckv, lens, 0.3)
    assert_parity("mla rope only", o, lse, o_ref, lse_ref)


def test_mla_is_deterministic():
    q, ckv, lens = workloads.mla_inputs(8, W["H"], W["Dc"], W["Dr"], 1024, 5)
    a = run(q, ckv, lens, scale=W["scale"], n_parts=37)
    b = run(q, ckv, lens, scale=W["scale"], n_parts=37)
    assert torch.equal(a[0].view(torch.int16), b[0].view(torch.int16))
    assert torch.equal(a[1], b[1])
