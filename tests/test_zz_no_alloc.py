"""The allocation-free decode entry point (mk_attn_decode_noalloc) against
mk_attn_decode with a caller workspace, through the C ABI: bitwise the same
output on two calls in a row, the second with a smaller batch, and both
within the decode parity bar of the fp64 oracle."""
import numpy as np
import pytest
import torch

import paper_2609_04523_amd as mk
import workloads
from oracle import oracle as orc
from parity import assert_parity

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def _both(qd, kc, vc, lens, n_parts, scale):
    B, Hq, D = qd.shape
    _, Hkv, Smax, _ = kc.shape
    q_, k_, v_, l_ = qd.to(DEV), kc.to(DEV), vc.to(DEV), lens.to(DEV)
    ws_bytes = mk.mk_attn_decode_workspace_bytes(Hq, Hkv, D, n_parts)
    ws = torch.empty(ws_bytes, device=DEV, dtype=torch.uint8)
    o_ref = torch.empty((B, Hq, D), device=DEV, dtype=torch.bfloat16)
    lse_ref = torch.empty((B, Hq), device=DEV, dtype=torch.float32)
    mk.mk_attn_decode(q_, k_, v_, o_ref, lse_ref, B, Hq, Hkv, Smax, D, scale, l_, n_parts, ws,
                      ws_bytes)
    o = torch.full((B, Hq, D), float("nan"), device=DEV, dtype=torch.bfloat16)
    lse = torch.full((B, Hq), float("nan"), device=DEV, dtype=torch.float32)
    mk.mk_attn_decode_noalloc(q_, k_, v_, o, lse, B, Hq, Hkv, Smax, D, scale, l_, n_parts)
    torch.cuda.synchronize()
    return o, lse, o_ref, lse_ref


def test_noalloc_decode_matches_workspace_decode_twice():
    # first call: the decode workload at its full size, default parts;
    # second: a smaller ragged batch with another part count, so the array
    # still holds the first call's pieces when the second runs
    cfg = workloads.CONFIGS["c5_decode_b64"]
    cases = [(workloads.config_inputs(cfg), 0, cfg.scale),
             (workloads.decode_inputs(5, 16, 4, 700, 128, seed=4242, lmin=0, lmax=700), 37,
              128 ** -0.5)]
    for n, ((qd, kc, vc, lens), parts, scale) in enumerate(cases):
        print(f"[noalloc] call {n}: B={qd.shape[0]} Hq={qd.shape[1]} Hkv={kc.shape[1]} "
              f"Smax={kc.shape[2]} parts={parts}", flush=True)
        o, lse, o_ref, lse_ref = _both(qd, kc, vc, lens, parts, scale)
        assert torch.equal(o.view(torch.int16), o_ref.view(torch.int16)), "O differs"
        assert torch.equal(lse.view(torch.int32), lse_ref.view(torch.int32)), "LSE differs"
        od, ld = orc.decode(workloads.bits(qd), workloads.bits(kc), workloads.bits(vc),
                            lens.numpy(), scale=scale)
        assert_parity(f"noalloc call {n}", o, lse, od, ld)


def test_noalloc_decode_rejects_oversized_requests():
    cap = mk.mk_attn_decode_noalloc_max_bytes()
    assert cap == 16 << 20
    # the most parts whose workspace fits, and one more part that does not
    Hq, Hkv, D = 32, 2, 128
    lo, hi = 1, mk.DECODE_MAX_PARTS
    while lo < hi:
        mid = (lo + hi + 1) // 2
        if mk.mk_attn_decode_workspace_bytes(Hq, Hkv, D, mid) <= cap:
            lo = mid
        else:
            hi = mid - 1
    qd, kc, vc, lens = workloads.decode_inputs(2, Hq, Hkv, 64, D, seed=5, lmin=1, lmax=64)
    q_, k_, v_, l_ = qd.to(DEV), kc.to(DEV), vc.to(DEV), lens.to(DEV)
    o = torch.empty((2, Hq, D), device=DEV, dtype=torch.bfloat16)
    with pytest.raises(mk.MkAttnError) as exc:
        mk.mk_attn_decode_noalloc(q_, k_, v_, o, None, 2, Hq, Hkv, 64, D, 0.1, l_, lo + 1)
    assert exc.value.status == 8 and "MK_ERR_SCRATCH" in str(exc.value)
    mk.mk_attn_decode_noalloc(q_, k_, v_, o, None, 2, Hq, Hkv, 64, D, 0.1, l_, lo)
    torch.cuda.synchronize()
