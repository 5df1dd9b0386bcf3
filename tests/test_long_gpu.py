"""Long sequences on the GPU against the fp64 oracle, through the C ABI:
a few query rows over 128k keys (dense forward, causal and not), decode
over caches of up to 128k keys (thousands of stages per sequence, parts
that lie inside one sequence), and a packed ragged batch of ~200k key
tokens.  The oracle computes only the rows checked."""
import numpy as np
import pytest
import torch

import paper_2609_04523_amd as mk
import workloads
from oracle import oracle as orc
from parity import assert_parity

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


@pytest.mark.parametrize("causal", [True, False])
def test_fwd_few_queries_over_128k_keys(causal):
    B, Hq, Hkv, Sq, Skv, D = 1, 4, 2, 5, 131072, 128
    q, k, v = workloads.prefill_inputs(B, Hq, Hkv, Sq, Skv, D, seed=7100 + causal)
    lens = [Skv - 3]  # a ragged tail tile at the end of the key range
    sl = torch.tensor(lens, dtype=torch.int32, device=DEV)
    o, lse = mk.fwd(q.to(DEV), k.to(DEV), v.to(DEV), causal=causal, scale=D ** -0.5, kv_seqlens=sl)
    torch.cuda.synchronize()
    o_ref, lse_ref = orc.attn_fwd(workloads.bits(q), workloads.bits(k), workloads.bits(v),
                                  causal=causal, scale=D ** -0.5, kv_seqlens=lens)
    assert_parity(f"fwd_128k_causal{int(causal)}", o, lse, o_ref, lse_ref)


@pytest.mark.parametrize("n_parts", [0, 64])
def test_decode_128k_cache(n_parts):
    B, Hq, Hkv, Smax, D = 3, 16, 4, 131072, 128
    q, kc, vc, _ = workloads.decode_inputs(B, Hq, Hkv, Smax, D, seed=7200 + n_parts, lmin=1,
                                           lmax=Smax)
    lens = [131072, 70001, 33]
    sl = torch.tensor(lens, dtype=torch.int32, device=DEV)
    ws = torch.empty(mk.mk_attn_decode_workspace_bytes(Hq, Hkv, D, n_parts), device=DEV,
                     dtype=torch.uint8)
    o, lse = mk.decode(q.to(DEV), kc.to(DEV), vc.to(DEV), sl, scale=D ** -0.5, n_parts=n_parts,
                       workspace=ws)
    torch.cuda.synchronize()
    o_ref, lse_ref = orc.decode(workloads.bits(q), workloads.bits(kc), workloads.bits(vc),
                                np.asarray(lens, dtype=np.int32), scale=D ** -0.5)
    assert_parity(f"decode_128k_parts{n_parts}", o, lse, o_ref, lse_ref)


def test_varlen_200k_key_tokens():
    # decode tokens and short chunks over long contexts, ~200k key tokens
    seqs = [(1, 90000), (3, 60000), (1, 1), (40, 50000), (2, 123)]
    Hq, Hkv, D = 8, 2, 128
    cq = np.concatenate([[0], np.cumsum([a for a, _ in seqs])]).astype(np.int32)
    ck = np.concatenate([[0], np.cumsum([b for _, b in seqs])]).astype(np.int32)
    g = torch.Generator().manual_seed(7300)
    q = torch.randn((int(cq[-1]), Hq, D), generator=g).to(torch.bfloat16)
    k = torch.randn((int(ck[-1]), Hkv, D), generator=g).to(torch.bfloat16)
    v = torch.randn((int(ck[-1]), Hkv, D), generator=g).to(torch.bfloat16)
    o, lse = mk.fwd_varlen(q.to(DEV), k.to(DEV), v.to(DEV), torch.from_numpy(cq).to(DEV),
                           torch.from_numpy(ck).to(DEV), 40, causal=True, scale=D ** -0.5)
    torch.cuda.synchronize()
    o_ref, lse_ref = orc.attn_fwd_varlen(workloads.bits(q), workloads.bits(k), workloads.bits(v),
                                         cq, ck, causal=True, scale=D ** -0.5)
    assert_parity("varlen_200k", o.permute(1, 0, 2)[None], lse[None],
                  o_ref.transpose(1, 0, 2)[None], lse_ref[None])
