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


def run_decode(q, kc, vc, lens, *, scale, n_parts=0, return_ws=False):
    sl = torch.as_tensor(np.asarray(lens, dtype=np.int32)).to(DEV)
    B, Hq, D = q.shape
    Hkv = kc.shape[1]
    ws = torch.empty(mk.mk_attn_decode_workspace_bytes(Hq, Hkv, D, n_parts), device=DEV,
                     dtype=torch.uint8)
    o, lse = mk.decode(q.to(DEV), kc.to(DEV), vc.to(DEV), sl, scale=scale, n_parts=n_parts,
                       workspace=ws)
    torch.cuda.synchronize()
    return (o, lse, ws) if return_ws else (o, lse)


def oracle_decode(q, kc, vc, lens, scale):
    return orc.decode(workloads.bits(q), workloads.bits(kc), workloads.bits(vc),
                      np.asarray(lens, dtype=np.int32), scale=scale)


def test_decode_b64_ragged_full_with_poisoned_padding():
    cfg = workloads.CONFIGS["c5_decode_b64"]
    q, kc, vc, lens = workloads.config_inputs(cfg)
    kcp, vcp = poison_padding(kc, lens.tolist()), poison_padding(vc, lens.tolist())
    o, lse = run_decode(q, kcp, vcp, lens, scale=cfg.scale)
    o_ref, lse_ref = oracle_decode(q, kc, vc, lens, cfg.scale)
    assert_parity(cfg.name, o, lse, o_ref, lse_ref)


@pytest.mark.parametrize("n_parts", [0, 1, 7, 100, 768, 5000])
def test_decode_part_counts(n_parts):
    # 5000 parts exceed the 1992 stages of this input: most parts are empty
    B, Hq, Hkv, Smax, D = 8, 32, 8, 2048, 128
    q, kc, vc, lens = workloads.decode_inputs(B, Hq, Hkv, Smax, D, seed=21, lmin=1, lmax=Smax)
    scale = D ** -0.5
    o, lse = run_decode(q, kc, vc, lens, scale=scale, n_parts=n_parts)
    o_ref, lse_ref = oracle_decode(q, kc, vc, lens, scale)
    assert_parity(f"parts{n_parts}", o, lse, o_ref, lse_ref)


# name, B, Hq, Hkv, Smax, D, lens
SHAPES = [
    ("mha_d64", 3, 4, 4, 300, 64, [300, 1, 65]),
    ("gqa8_d128", 2, 16, 2, 1000, 128, [999, 128]),
    ("gqa16_d64", 2, 16, 1, 700, 64, [700, 63]),
    ("gqa4_lengths_edge", 4, 8, 2, 512, 128, [0, 1, 511, 512]),
    ("clamped_lengths", 3, 8, 2, 256, 128, [-7, 100000, 129]),
    ("single_key_cache", 2, 4, 1, 1, 128, [1, 1]),
    ("all_empty", 2, 8, 2, 64, 128, [0, 0]),
    ("many_short", 70, 4, 2, 40, 128, [(7 * b) % 41 for b in range(70)]),
    ("gqa6_d128", 3, 12, 2, 300, 128, [300, 33, 150]),
    ("gqa12_d64", 2, 12, 1, 200, 64, [1, 200]),
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


def stream_parts(T, P):
    """Part boundaries the library documents: P equal parts, part w holding
    stages [floor(w T / P), floor((w + 1) T / P))."""
    return [(w * T // P, (w + 1) * T // P) for w in range(P)]


def stream_pieces(lens, Hkv, Smax, P):
    """Pieces of the stage stream: the 32-key stages of pairs (b, g), pair
    after pair, cut at the part boundaries.  Yields (part, slot, b, g, key0,
    key1, whole) per piece; slot 0 is a part's first piece, 1 its last."""
    nts = [-(-max(0, min(int(L), Smax)) // 32) for L in lens]
    T = Hkv * sum(nts)
    pairs, A = [], 0
    for b, nt in enumerate(nts):
        for g in range(Hkv):
            if nt:
                pairs.append((A, A + nt, b, g))
            A += nt
    for p, (s0, s1) in enumerate(stream_parts(T, P)):
        pieces = [(max(a0, s0), min(a1, s1), a0, a1, b, g) for a0, a1, b, g in pairs
                  if a0 < s1 and a1 > s0]
        for i, (p0, p1, a0, a1, b, g) in enumerate(pieces):
            L = max(0, min(int(lens[b]), Smax))
            yield (p, 0 if i == 0 else 1, b, g, 32 * (p0 - a0), min(32 * (p1 - a0), L),
                   p0 == a0 and p1 == a1)


def test_decode_pieces_match_oracle_on_their_keys():
    # every cut piece in the workspace is the attention of its query heads
    # over exactly its own keys
    B, Hq, Hkv, Smax, D = 4, 8, 2, 1500, 128
    G = Hq // Hkv
    q, kc, vc, lens = workloads.decode_inputs(B, Hq, Hkv, Smax, D, seed=22, lmin=1, lmax=Smax)
    scale = D ** -0.5
    P = 37
    o, lse, ws = run_decode(q, kc, vc, lens, scale=scale, n_parts=P, return_ws=True)
    o_part, lse_part = mk.decode_partials(ws, Hq, Hkv, D, P)
    n_cut = 0
    for p, slot, b, g, k0, k1, whole in stream_pieces(lens.tolist(), Hkv, Smax, P):
        if whole:
            continue
        n_cut += 1
        qs = q[b:b + 1, g * G:(g + 1) * G]
        o_ref, lse_ref = oracle_decode(qs, kc[b:b + 1, g:g + 1, k0:k1].contiguous(),
                                       vc[b:b + 1, g:g + 1, k0:k1].contiguous(), [k1 - k0],
                                       scale)
        assert_parity(f"piece p{p} s{slot} b{b} g{g} [{k0},{k1})", o_part[p, slot][None],
                      lse_part[p, slot][None], o_ref, lse_ref)
    assert n_cut > P // 2


@pytest.mark.parametrize("n_parts", [3, 50])
def test_decode_many_sequences_few_parts(n_parts):
    # 130 sequences: the stream is located across several 64-sequence
    # chunks and each part walks through many sequences, empty ones included
    B, Hq, Hkv, Smax, D = 130, 8, 2, 300, 64
    g = torch.Generator().manual_seed(31)
    lens = torch.randint(0, Smax + 1, (B,), generator=g).tolist()
    lens[5] = lens[64] = lens[129] = 0
    q = torch.randn((B, Hq, D), generator=g).to(torch.bfloat16)
    kc = torch.randn((B, Hkv, Smax, D), generator=g).to(torch.bfloat16)
    vc = torch.randn((B, Hkv, Smax, D), generator=g).to(torch.bfloat16)
    scale = D ** -0.5
    o, lse = run_decode(q, poison_padding(kc, lens), poison_padding(vc, lens), lens, scale=scale,
                        n_parts=n_parts)
    o_ref, lse_ref = oracle_decode(q, kc, vc, lens, scale)
    assert_parity(f"B130 parts{n_parts}", o, lse, o_ref, lse_ref)


def test_decode_workspace_reuse_and_uninitialised_partials():
    # one workspace, filled with NaN, for calls of different part counts:
    # the library needs no initialised workspace contents
    B, Hq, Hkv, Smax, D = 6, 16, 4, 900, 128
    q, kc, vc, lens = workloads.decode_inputs(B, Hq, Hkv, Smax, D, seed=25, lmin=0, lmax=Smax)
    scale = D ** -0.5
    P_max = 200
    ws = torch.empty(mk.mk_attn_decode_workspace_bytes(Hq, Hkv, D, P_max), device=DEV,
                     dtype=torch.uint8)
    ws.view(torch.float32).fill_(float("nan"))
    o_ref, lse_ref = oracle_decode(q, kc, vc, lens, scale)
    sl = lens.to(DEV)
    for P in (200, 37, 1, 150, 37):
        o, lse = mk.decode(q.to(DEV), kc.to(DEV), vc.to(DEV), sl, scale=scale, n_parts=P,
                           workspace=ws)
        torch.cuda.synchronize()
        assert_parity(f"reuse P={P}", o, lse, o_ref, lse_ref)


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
