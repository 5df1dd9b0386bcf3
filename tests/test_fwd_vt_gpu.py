"""Forward through the V^T workspace (mk_attn_fwd_ws) on the GPU.

The workspace path forms the same products in the same order as
mk_attn_fwd, only its V operand comes from a re-laid-out copy, so its O and
LSE must equal mk_attn_fwd's bit for bit; mk_attn_fwd itself is held to the
oracle by test_fwd_gpu.py, and three cases here go to the oracle directly.
The copy's layout is checked against one built on the host from V."""
import math
import zlib

import numpy as np
import pytest
import torch

import paper_2609_04523_amd as mk
import workloads
from oracle import oracle as orc
from parity import assert_parity

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def ws_for(B, Hkv, Skv, D, extra=0):
    n = mk.mk_attn_fwd_workspace_bytes(B, Hkv, Skv, D)
    return torch.empty(n + extra, dtype=torch.uint8, device=DEV)


def both(q, k, v, *, causal, scale, kv_seqlens=None, ws=None):
    qd, kd, vd = q.to(DEV), k.to(DEV), v.to(DEV)
    sl = None if kv_seqlens is None else torch.tensor(kv_seqlens, dtype=torch.int32, device=DEV)
    B, Hq, Sq, D = q.shape
    Skv = k.shape[2]
    if ws is None:
        ws = ws_for(B, k.shape[1], Skv, D)
    o_ref, lse_ref = mk.fwd(qd, kd, vd, causal=causal, scale=scale, kv_seqlens=sl)
    o, lse = mk.fwd(qd, kd, vd, causal=causal, scale=scale, kv_seqlens=sl, workspace=ws)
    torch.cuda.synchronize()
    return o, lse, o_ref, lse_ref, ws


def assert_bitwise(name, o, lse, o_ref, lse_ref):
    assert torch.equal(o.view(torch.int16), o_ref.view(torch.int16)), name
    assert torch.equal(lse.view(torch.int32), lse_ref.view(torch.int32)), name


# name, B, Hq, Hkv, Sq, Skv, D, causal, kv_seqlens, scale (None: D^-1/2)
CASES = [
    ("s1_d128", 1, 2, 1, 1, 1, 128, True, None, None),
    ("s17_gqa2", 2, 4, 2, 17, 17, 128, True, None, None),
    ("s129_noncausal", 1, 4, 4, 129, 129, 128, False, None, None),
    ("s1000_gqa4_d64", 1, 8, 2, 1000, 1000, 64, True, None, None),
    ("s300_d64_noncausal", 2, 2, 1, 300, 300, 64, False, None, None),
    ("sq100_skv300_bottom_right", 2, 4, 1, 100, 300, 128, True, None, None),
    ("ragged_lens", 3, 4, 2, 200, 300, 128, True, [300, 57, 0], None),
    ("clamped_lens", 2, 2, 2, 64, 64, 128, True, [-5, 1000], None),
    ("noncausal_lens_d64", 2, 4, 4, 77, 260, 64, False, [260, 100], None),
    ("s513_gqa8", 1, 16, 2, 513, 513, 128, True, None, None),
    ("scale_negative", 1, 4, 2, 190, 190, 128, True, None, -0.05),
    ("scale_zero_d64", 1, 2, 1, 150, 150, 64, True, None, 0.0),
    # the persistent grid's queues: 8 (one per XCD) when B * Hkv is a
    # multiple of 8, else 1; one item per queue; items without keys; more
    # items than workgroups (taken from the other queues at the end)
    ("xcd8_one_item_each", 1, 8, 8, 100, 100, 128, True, None, None),
    ("xcd8_empty_sequences", 8, 8, 1, 300, 300, 128, True, [300, 0, 17, 256, 0, 1, 299, 64], None),
    ("xcd8_many_items_d64", 2, 32, 4, 2000, 2000, 64, True, None, None),
    ("one_queue_many_items", 3, 12, 3, 1100, 1100, 128, True, None, None),
    # long sequences: many items per workgroup, items taken across XCDs,
    # the other head dim and the non-causal instantiation
    ("long_d64_s16k", 1, 16, 8, 16384, 16384, 64, True, None, None),
    ("long_noncausal_s8k", 1, 16, 8, 8192, 8192, 128, False, None, None),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_fwd_ws_bitwise_equals_fwd(case):
    name, B, Hq, Hkv, Sq, Skv, D, causal, sl, scale = case
    q, k, v = workloads.prefill_inputs(B, Hq, Hkv, Sq, Skv, D,
                                       seed=zlib.crc32(name.encode()) % 100000)
    scale = 1.0 / math.sqrt(D) if scale is None else scale
    o, lse, o_ref, lse_ref, _ = both(q, k, v, causal=causal, scale=scale, kv_seqlens=sl)
    assert_bitwise(name, o, lse, o_ref, lse_ref)


@pytest.mark.parametrize("name", ["ragged_lens", "s1000_gqa4_d64", "xcd8_empty_sequences"])
def test_fwd_ws_oracle_parity(name):
    case = next(c for c in CASES if c[0] == name)
    _, B, Hq, Hkv, Sq, Skv, D, causal, sl, scale = case
    q, k, v = workloads.prefill_inputs(B, Hq, Hkv, Sq, Skv, D,
                                       seed=zlib.crc32(name.encode()) % 100000)
    scale = 1.0 / math.sqrt(D)
    o, lse, _, _, _ = both(q, k, v, causal=causal, scale=scale, kv_seqlens=sl)
    o_or, lse_or = orc.attn_fwd(workloads.bits(q), workloads.bits(k), workloads.bits(v),
                                causal=causal, scale=scale, kv_seqlens=sl)
    assert_parity(name, o, lse, o_or, lse_or)


def test_fwd_ws_ignores_values_past_the_lengths():
    # V rows past a sequence's length may hold anything (here NaN): the copy
    # writes zeros there, so the output is finite and equals mk_attn_fwd's
    B, Hq, Hkv, S, D = 2, 4, 2, 200, 128
    q, k, v = workloads.prefill_inputs(B, Hq, Hkv, S, S, D, seed=731)
    lens = [130, 65]
    v = v.clone()
    for b, L in enumerate(lens):
        v[b, :, L:] = float("nan")
    o, lse, o_ref, lse_ref, _ = both(q, k, v, causal=True, scale=D ** -0.5, kv_seqlens=lens)
    assert torch.isfinite(o.float()).all()
    assert_bitwise("nan_past_lengths", o, lse, o_ref, lse_ref)


def expected_tiles(v, lens):
    """The V^T tiles built on the host: [B, Hkv, tiles, 4, D, 16] with row
    (kc, d) holding, in half p, the keys 16 kc + (e % 4) + 4 h + 8 (e // 4),
    e = 0..7, of k-group h = p ^ ((d // 8) % 2); zero past the length."""
    B, Hkv, Skv, D = v.shape
    tiles = (Skv + 63) // 64
    vf = np.zeros((B, Hkv, tiles * 64, D), dtype=np.uint16)
    vb = workloads.bits(v)
    for b in range(B):
        L = Skv if lens is None else max(0, min(lens[b], Skv))
        vf[b, :, :L] = vb[b, :, :L]
    out = np.zeros((B, Hkv, tiles, 4, D, 16), dtype=np.uint16)
    for kc in range(4):
        for d in range(D):
            for p in range(2):
                h = p ^ ((d // 8) % 2)
                for e in range(8):
                    key = 16 * kc + (e % 4) + 4 * h + 8 * (e // 4)
                    out[:, :, :, kc, d, 8 * p + e] = vf[:, :, key::64, d][:, :, :tiles]
    return out


@pytest.mark.parametrize("D,lens", [(128, None), (64, [70, 130])])
def test_fwd_ws_tile_layout(D, lens):
    B, Hq, Hkv, S = 2, 2, 1, 130
    q, k, v = workloads.prefill_inputs(B, Hq, Hkv, S, S, D, seed=77 + D)
    ws = ws_for(B, Hkv, S, D)
    both(q, k, v, causal=True, scale=D ** -0.5, kv_seqlens=lens, ws=ws)
    tiles = (S + 63) // 64
    got = ws.cpu().numpy().view(np.uint16)[:B * Hkv * tiles * 64 * D]
    got = got.reshape(B, Hkv, tiles, 4, D, 16)
    assert np.array_equal(got, expected_tiles(v, lens))


@pytest.mark.parametrize("fill", [0x00, 0xFF, 0x7F])
def test_fwd_ws_workspace_contents_do_not_matter(fill):
    # the call sets up its own work-item counters: a workspace holding
    # anything (here all bytes `fill`) gives the same result
    B, Hq, Hkv, S, D = 2, 16, 4, 900, 128
    q, k, v = workloads.prefill_inputs(B, Hq, Hkv, S, S, D, seed=4400 + fill)
    ws = ws_for(B, Hkv, S, D)
    ws.fill_(fill)
    torch.cuda.synchronize()
    o, lse, o_ref, lse_ref, _ = both(q, k, v, causal=True, scale=D ** -0.5, ws=ws)
    assert_bitwise(f"fill_{fill}", o, lse, o_ref, lse_ref)


def test_fwd_ws_reused_workspace_smaller_second_call():
    ws = ws_for(2, 4, 700, 128)
    q, k, v = workloads.prefill_inputs(2, 8, 4, 700, 700, 128, seed=901)
    o, lse, o_ref, lse_ref, _ = both(q, k, v, causal=True, scale=128 ** -0.5, ws=ws)
    assert_bitwise("first", o, lse, o_ref, lse_ref)
    q, k, v = workloads.prefill_inputs(1, 4, 2, 333, 333, 128, seed=902)
    o, lse, o_ref, lse_ref, _ = both(q, k, v, causal=True, scale=128 ** -0.5, ws=ws)
    assert_bitwise("second", o, lse, o_ref, lse_ref)


@pytest.mark.parametrize("cfg_name", ["c3_gqa_s8k_k2", "c4_gqa_s32k"])
def test_fwd_ws_full_size_bitwise(cfg_name):
    # the sizes the bench times, in the same launch configuration
    cfg = workloads.CONFIGS[cfg_name]
    q, k, v = workloads.config_inputs(cfg)
    o, lse, o_ref, lse_ref, _ = both(q, k, v, causal=True, scale=cfg.scale)
    assert_bitwise(cfg_name, o, lse, o_ref, lse_ref)
