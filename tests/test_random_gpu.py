"""Seeded random sweeps on the GPU against the fp64 oracle, through the C ABI:
dense forward (mixed head groups, head dims, causal or not, ragged and
clamped lengths, scales of either sign or zero, sharpened keys; its V^T
workspace path bitwise against it), packed
ragged forward, decode with random lengths and part counts (contiguous and
paged caches), MLA decode, and the backward (gradients against the
oracle's backward).  Every
configuration is drawn from a fixed seed, so a failure names a case that
reruns identically."""

import numpy as np
import pytest
import torch

import paper_2609_04523_amd as mk
import workloads
from oracle import oracle as orc
from parity import assert_parity

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
N_FWD, N_VARLEN, N_DEC, N_BWD, N_PAGED, N_MLA = 48, 20, 24, 10, 12, 8


def _fwd_case(i):
    r = np.random.default_rng(9000 + i)
    D = int(r.choice([64, 128]))
    G = int(r.choice([1, 2, 4, 8]))
    Hkv = int(r.integers(1, 3))
    B = int(r.integers(1, 3))
    Sq = int(r.integers(1, 520))
    Skv = Sq if r.random() < 0.5 else int(r.integers(1, 600))
    causal = bool(r.random() < 0.7)
    lens = None
    if r.random() < 0.35:
        lens = [int(x) for x in r.integers(-3, Skv + 40, size=B)]  # includes clamped values
    scale = float(r.choice([D ** -0.5, D ** -0.5, 0.37 * D ** -0.5, -0.5 * D ** -0.5, 0.0]))
    k_mult = float(r.choice([1.0, 1.0, 2.0, 4.0]))
    return dict(B=B, Hq=G * Hkv, Hkv=Hkv, Sq=Sq, Skv=Skv, D=D, causal=causal, lens=lens,
                scale=scale, k_mult=k_mult, seed=9000 + i)


@pytest.mark.parametrize("i", range(N_FWD))
def test_fwd_random(i):
    c = _fwd_case(i)
    print(f"[case] {c}", flush=True)
    q, k, v = workloads.prefill_inputs(c["B"], c["Hq"], c["Hkv"], c["Sq"], c["Skv"], c["D"],
                                       seed=c["seed"], k_mult=c["k_mult"])
    sl = None if c["lens"] is None else torch.tensor(c["lens"], dtype=torch.int32, device=DEV)
    o, lse = mk.fwd(q.to(DEV), k.to(DEV), v.to(DEV), causal=c["causal"], scale=c["scale"],
                    kv_seqlens=sl)
    torch.cuda.synchronize()
    o_ref, lse_ref = orc.attn_fwd(workloads.bits(q), workloads.bits(k), workloads.bits(v),
                                  causal=c["causal"], scale=c["scale"], kv_seqlens=c["lens"])
    assert_parity(f"fwd_random_{i}", o, lse, o_ref, lse_ref)
    # the V^T workspace path forms the same products in the same order
    ws = torch.empty(mk.mk_attn_fwd_workspace_bytes(c["B"], c["Hkv"], c["Skv"], c["D"]),
                     dtype=torch.uint8, device=DEV)
    o_ws, lse_ws = mk.fwd(q.to(DEV), k.to(DEV), v.to(DEV), causal=c["causal"], scale=c["scale"],
                          kv_seqlens=sl, workspace=ws)
    torch.cuda.synchronize()
    assert torch.equal(o_ws.view(torch.int16), o.view(torch.int16)), f"fwd_random_{i}: ws O"
    assert torch.equal(lse_ws.view(torch.int32), lse.view(torch.int32)), f"fwd_random_{i}: ws LSE"


@pytest.mark.parametrize("i", range(N_VARLEN))
def test_varlen_random(i):
    r = np.random.default_rng(9500 + i)
    B = int(r.integers(1, 7))
    D = int(r.choice([64, 128]))
    Hkv = int(r.integers(1, 3))
    Hq = Hkv * int(r.choice([1, 2, 4]))
    seqs = []
    for _ in range(B):
        kind = r.random()
        if kind < 0.25:
            sk = int(r.integers(1, 900))
            seqs.append((1, sk))                      # a decode token
        elif kind < 0.35:
            seqs.append((int(r.integers(0, 3)), int(r.integers(0, 3))))  # tiny or empty
        else:
            sk = int(r.integers(1, 700))
            seqs.append((int(r.integers(1, sk + 1)), sk))  # a prefill chunk
    causal = bool(r.random() < 0.75)
    cq = np.concatenate([[0], np.cumsum([a for a, _ in seqs])]).astype(np.int32)
    ck = np.concatenate([[0], np.cumsum([b for _, b in seqs])]).astype(np.int32)
    print(f"[case] varlen {i}: seqs={seqs} Hq={Hq} Hkv={Hkv} D={D} causal={causal}", flush=True)
    if cq[-1] == 0:
        return  # nothing to compute; the ABI rejects total_q = 0
    g = torch.Generator().manual_seed(9500 + i)
    q = torch.randn((int(cq[-1]), Hq, D), generator=g).to(torch.bfloat16)
    k = torch.randn((max(int(ck[-1]), 1), Hkv, D), generator=g).to(torch.bfloat16)
    v = torch.randn((max(int(ck[-1]), 1), Hkv, D), generator=g).to(torch.bfloat16)
    scale = D ** -0.5
    max_sq = max(int(np.max(np.diff(cq))), 1)
    o, lse = mk.fwd_varlen(q.to(DEV), k.to(DEV), v.to(DEV), torch.from_numpy(cq).to(DEV),
                           torch.from_numpy(ck).to(DEV), max_sq, causal=causal, scale=scale)
    torch.cuda.synchronize()
    o_ref, lse_ref = orc.attn_fwd_varlen(workloads.bits(q), workloads.bits(k), workloads.bits(v),
                                         cq, ck, causal=causal, scale=scale)
    assert_parity(f"varlen_random_{i}", o.permute(1, 0, 2)[None], lse[None],
                  o_ref.transpose(1, 0, 2)[None], lse_ref[None])


@pytest.mark.parametrize("i", range(N_DEC))
def test_decode_random(i):
    r = np.random.default_rng(9800 + i)
    B = int(r.integers(1, 21))
    D = int(r.choice([64, 128]))
    Hkv = int(r.integers(1, 5))
    G = int(r.choice([1, 2, 4, 8, 16]))
    Smax = int(r.choice([64, 700, 3000]))
    lens = [int(x) for x in r.integers(0, Smax + 1, size=B)]
    n_parts = int(r.choice([0, 1, 7, 100, 1000]))
    scale = float(r.choice([D ** -0.5, 2.0 * D ** -0.5]))
    print(f"[case] decode {i}: B={B} Hq={G * Hkv} Hkv={Hkv} D={D} Smax={Smax} parts={n_parts} "
          f"lens={lens}", flush=True)
    q, kc, vc, _ = workloads.decode_inputs(B, G * Hkv, Hkv, Smax, D, seed=9800 + i, lmin=0,
                                           lmax=Smax)
    sl = torch.tensor(lens, dtype=torch.int32, device=DEV)
    Hq = G * Hkv
    ws = torch.empty(mk.mk_attn_decode_workspace_bytes(Hq, Hkv, D, n_parts), device=DEV,
                     dtype=torch.uint8)
    o, lse = mk.decode(q.to(DEV), kc.to(DEV), vc.to(DEV), sl, scale=scale, n_parts=n_parts,
                       workspace=ws)
    torch.cuda.synchronize()
    o_ref, lse_ref = orc.decode(workloads.bits(q), workloads.bits(kc), workloads.bits(vc),
                                np.asarray(lens, dtype=np.int32), scale=scale)
    assert_parity(f"decode_random_{i}", o, lse, o_ref, lse_ref)


@pytest.mark.parametrize("i", range(N_BWD))
def test_bwd_random(i):
    from test_bwd_gpu import check
    r = np.random.default_rng(9900 + i)
    D = int(r.choice([64, 128]))
    Hkv = int(r.integers(1, 3))
    Hq = Hkv * int(r.choice([1, 2, 4]))
    B = int(r.integers(1, 3))
    Sq = int(r.integers(1, 300))
    Skv = Sq if r.random() < 0.5 else int(r.integers(1, 350))
    causal = bool(r.random() < 0.7)
    seqlens = [int(x) for x in r.integers(0, Skv + 1, size=B)] if r.random() < 0.3 else None
    k_mult = float(r.choice([1.0, 2.0]))
    print(f"[case] bwd {i}: B={B} Hq={Hq} Hkv={Hkv} Sq={Sq} Skv={Skv} D={D} causal={causal} "
          f"lens={seqlens} k_mult={k_mult}", flush=True)
    check(f"bwd_random_{i}", B, Hq, Hkv, Sq, Skv, D, causal, seed=9900 + i, seqlens=seqlens,
          k_mult=k_mult)


@pytest.mark.parametrize("i", range(N_PAGED))
def test_decode_paged_random(i):
    r = np.random.default_rng(9700 + i)
    B = int(r.integers(1, 13))
    D = int(r.choice([64, 128]))
    Hkv = int(r.integers(1, 4))
    G = int(r.choice([1, 4, 8]))
    ps = int(r.choice([16, 32, 48, 64, 256]))
    Smax = ps * int(r.integers(1, max(2, 2048 // ps)))
    lens = [int(x) for x in r.integers(0, Smax + 1, size=B)]
    n_parts = int(r.choice([0, 1, 50, 700]))
    scale = D ** -0.5
    print(f"[case] paged {i}: B={B} Hq={G * Hkv} Hkv={Hkv} D={D} page={ps} Smax={Smax} "
          f"parts={n_parts} lens={lens}", flush=True)
    q, kc, vc, _ = workloads.decode_inputs(B, G * Hkv, Hkv, Smax, D, seed=9700 + i, lmin=0,
                                           lmax=Smax)
    kp, vp, bt = workloads.paged_layout(kc, vc, ps, seed=9700 + i, extra_pages=int(r.integers(0, 9)),
                                        lens=torch.tensor(lens))
    sl = torch.tensor(lens, dtype=torch.int32, device=DEV)
    o, lse = mk.decode_paged(q.to(DEV), kp.to(DEV), vp.to(DEV), bt.to(DEV), sl, scale=scale,
                             n_parts=n_parts)
    torch.cuda.synchronize()
    o_ref, lse_ref = orc.decode_paged(workloads.bits(q), workloads.bits(kp), workloads.bits(vp),
                                      bt.numpy(), np.asarray(lens, dtype=np.int32), scale=scale)
    assert_parity(f"paged_random_{i}", o, lse, o_ref, lse_ref)


@pytest.mark.parametrize("i", range(N_MLA))
def test_mla_random(i):
    W = workloads.MLA
    r = np.random.default_rng(9600 + i)
    B = int(r.integers(1, 17))
    Smax = int(r.choice([32, 600, 2500]))
    lens = [int(x) for x in r.integers(0, Smax + 1, size=B)]
    n_parts = int(r.choice([0, 1, 13, 300]))
    print(f"[case] mla {i}: B={B} Smax={Smax} parts={n_parts} lens={lens}", flush=True)
    q, ckv, _ = workloads.mla_inputs(B, W["H"], W["Dc"], W["Dr"], Smax, 9600 + i, 0, Smax)
    o, lse = mk.mla_decode(q.to(DEV), ckv.to(DEV), torch.tensor(lens, dtype=torch.int32).to(DEV),
                           Dc=W["Dc"], scale=W["scale"], n_parts=n_parts)
    torch.cuda.synchronize()
    o_ref, lse_ref = orc.mla_decode(workloads.bits(q), workloads.bits(ckv),
                                    np.asarray(lens, np.int32), Dc=W["Dc"], scale=W["scale"])
    assert_parity(f"mla_random_{i}", o, lse, o_ref, lse_ref)
