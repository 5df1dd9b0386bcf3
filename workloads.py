"""Seeded synthetic inputs for the attention path.

Shared by the tests (which feed both the HIP library and the CPU oracle
with the same bits) and by the benchmark.  This module holds no attention
arithmetic: it only draws random numbers and rounds them to bf16.

Recipe (one place, so both sides see identical bits):
  * ``torch.Generator().manual_seed(seed)`` on the CPU;
  * prefill: draw Q, then K, then V with ``randn`` in fp32, multiply K by
    ``k_mult`` (a power of two, so exact), round to bf16 (round to nearest
    even);
  * decode: draw the lengths first (integers uniform in [lmin, lmax],
    inclusive), then q, then the K and V caches.

The workloads stand in for the paper's flash / grouped-query attention
benchmark items (Table 2), whose shapes the paper does not give; they use
N(0,1) values, causal masking and 1/sqrt(D) scaling.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import torch


@dataclass(frozen=True)
class PrefillConfig:
    name: str
    B: int
    Hq: int
    Hkv: int
    S: int
    D: int
    seed: int
    k_mult: float = 1.0
    out_fp32: bool = False
    sample_rows: int = 0  # 0: check every row; else rows per head
    causal: bool = True

    @property
    def scale(self) -> float:
        return float(torch.tensor(1.0 / math.sqrt(self.D), dtype=torch.float32))

    @property
    def pairs_per_head(self) -> int:
        # unmasked (query, key) pairs of one causal head
        return self.S * (self.S + 1) // 2 if self.causal else self.S * self.S

    @property
    def flops(self) -> int:
        # 4*D per unmasked pair per query head (QK^T and PV, 2 FLOP per MAC)
        return 4 * self.D * self.pairs_per_head * self.B * self.Hq


@dataclass(frozen=True)
class DecodeConfig:
    name: str
    B: int
    Hq: int
    Hkv: int
    Smax: int
    D: int
    seed: int
    lmin: int = 512
    lmax: int = 4096
    split: int = 0  # 0: library default

    @property
    def scale(self) -> float:
        return float(torch.tensor(1.0 / math.sqrt(self.D), dtype=torch.float32))


# Workload table.  The first entry is the small case the oracle checks in
# full in well under a second; the next three are prefill workloads of
# growing length (MHA at 2k, grouped heads at 8k with a sharpened softmax,
# grouped heads at 32k), the last one a ragged decode batch.
CONFIGS = {
    "c1_mha_s128_d64": PrefillConfig("c1_mha_s128_d64", B=1, Hq=2, Hkv=2, S=128, D=64,
                                     seed=1001, out_fp32=True),
    "c2_mha_s2k": PrefillConfig("c2_mha_s2k", B=4, Hq=16, Hkv=16, S=2048, D=128, seed=1002),
    "c3_gqa_s8k_k2": PrefillConfig("c3_gqa_s8k_k2", B=2, Hq=32, Hkv=8, S=8192, D=128,
                                   seed=1003, k_mult=2.0),
    "c4_gqa_s32k": PrefillConfig("c4_gqa_s32k", B=1, Hq=32, Hkv=8, S=32768, D=128,
                                 seed=1004, sample_rows=256),
    "c5_decode_b64": DecodeConfig("c5_decode_b64", B=64, Hq=32, Hkv=8, Smax=4096, D=128,
                                  seed=1005),
}


def _gen(seed: int) -> torch.Generator:
    g = torch.Generator(device="cpu")
    g.manual_seed(int(seed))
    return g


def prefill_inputs(B: int, Hq: int, Hkv: int, Sq: int, Skv: int, D: int, seed: int,
                   k_mult: float = 1.0):
    """bf16 CPU tensors q [B,Hq,Sq,D], k and v [B,Hkv,Skv,D]."""
    g = _gen(seed)
    q = torch.randn((B, Hq, Sq, D), generator=g, dtype=torch.float32)
    k = torch.randn((B, Hkv, Skv, D), generator=g, dtype=torch.float32)
    v = torch.randn((B, Hkv, Skv, D), generator=g, dtype=torch.float32)
    if k_mult != 1.0:
        k = k * float(k_mult)
    return q.to(torch.bfloat16), k.to(torch.bfloat16), v.to(torch.bfloat16)


def decode_inputs(B: int, Hq: int, Hkv: int, Smax: int, D: int, seed: int,
                  lmin: int = 512, lmax: int = 4096):
    """(q [B,Hq,D] bf16, k_cache/v_cache [B,Hkv,Smax,D] bf16, lens int32 [B])."""
    g = _gen(seed)
    lens = torch.randint(lmin, lmax + 1, (B,), generator=g, dtype=torch.int64).to(torch.int32)
    q = torch.randn((B, Hq, D), generator=g, dtype=torch.float32)
    kc = torch.randn((B, Hkv, Smax, D), generator=g, dtype=torch.float32)
    vc = torch.randn((B, Hkv, Smax, D), generator=g, dtype=torch.float32)
    return q.to(torch.bfloat16), kc.to(torch.bfloat16), vc.to(torch.bfloat16), lens


# MLA decode workload: the per-GPU share (16 of 128 query heads) of a
# DeepSeek-V3-style absorbed MLA decode, latent 512 + rotary 64, with the
# decode workload's batch and length recipe; the scale is 1/sqrt(192), the
# head dim of the un-absorbed query-key product (128 + 64).
MLA = dict(name="mla_decode_b64", B=64, H=16, Dc=512, Dr=64, Smax=4096, lmin=512, lmax=4096,
           seed=1007, scale=float(torch.tensor(192 ** -0.5, dtype=torch.float32)))


def mla_inputs(B: int, H: int, Dc: int, Dr: int, Smax: int, seed: int, lmin: int = 512,
               lmax: int = 4096):
    """(q [B,H,Dc+Dr] bf16, ckv [B,Smax,Dc+Dr] bf16, lens int32 [B]): lengths
    U{lmin..lmax} first, then N(0,1) draws rounded to bf16."""
    g = _gen(seed)
    lens = torch.randint(lmin, lmax + 1, (B,), generator=g, dtype=torch.int64).to(torch.int32)
    q = torch.randn((B, H, Dc + Dr), generator=g, dtype=torch.float32)
    ckv = torch.randn((B, Smax, Dc + Dr), generator=g, dtype=torch.float32)
    return q.to(torch.bfloat16), ckv.to(torch.bfloat16), lens


def varlen_inputs(B: int, Hq: int, Hkv: int, D: int, lmin: int, lmax: int, seed: int):
    """Packed ragged prefill batch: lengths U{lmin..lmax} (queries = keys per
    sequence), then q [total,Hq,D], k/v [total,Hkv,D] bf16 N(0,1), and
    cu_seqlens int32 [B+1]."""
    g = _gen(seed)
    lens = torch.randint(lmin, lmax + 1, (B,), generator=g, dtype=torch.int64)
    cu = torch.zeros(B + 1, dtype=torch.int32)
    cu[1:] = torch.cumsum(lens, 0).to(torch.int32)
    T = int(cu[-1])
    q = torch.randn((T, Hq, D), generator=g, dtype=torch.float32).to(torch.bfloat16)
    k = torch.randn((T, Hkv, D), generator=g, dtype=torch.float32).to(torch.bfloat16)
    v = torch.randn((T, Hkv, D), generator=g, dtype=torch.float32).to(torch.bfloat16)
    return q, k, v, cu


NAN_BF16_BITS = 0x7FC0


def paged_layout(k_cache: torch.Tensor, v_cache: torch.Tensor, page_size: int, seed: int,
                 extra_pages: int = 0, lens=None):
    """Scatter contiguous caches [B,Hkv,Smax,D] into page pools
    [n_pages,Hkv,page_size,D] under a seeded random page assignment.

    Page i of sequence b (keys [i*page_size, (i+1)*page_size)) goes to
    physical page block_table[b, i], a seeded permutation of all
    B*max_pages + extra_pages pool pages.  Pool pages no table lists, and
    rows at or past a sequence's length when ``lens`` is given, hold NaN,
    so a read of them poisons the result.  Returns (k_pages, v_pages,
    block_table int32 [B, max_pages])."""
    B, Hkv, Smax, D = k_cache.shape
    if Smax % page_size:
        raise ValueError("Smax must be a multiple of page_size")
    mp = Smax // page_size
    n_pages = B * mp + extra_pages
    perm = torch.randperm(n_pages, generator=_gen(seed))
    bt = perm[: B * mp].reshape(B, mp).to(torch.int32)
    kp = torch.full((n_pages, Hkv, page_size, D), float("nan"), dtype=torch.bfloat16)
    vp = torch.full_like(kp, float("nan"))
    # [B, Hkv, mp, ps, D] -> [B, mp, Hkv, ps, D] -> rows of the pool
    src_k = k_cache.reshape(B, Hkv, mp, page_size, D).transpose(1, 2).reshape(B * mp, Hkv,
                                                                                page_size, D)
    src_v = v_cache.reshape(B, Hkv, mp, page_size, D).transpose(1, 2).reshape(B * mp, Hkv,
                                                                                page_size, D)
    if lens is not None:
        src_k, src_v = src_k.clone(), src_v.clone()
        key = torch.arange(Smax).reshape(mp, page_size)
        for b in range(B):
            L = max(0, min(int(lens[b]), Smax))
            dead = key >= L                                   # [mp, ps]
            src_k[b * mp:(b + 1) * mp].view(torch.int16).masked_fill_(
                dead[:, None, :, None].expand(mp, Hkv, page_size, D), NAN_BF16_BITS)
            src_v[b * mp:(b + 1) * mp].view(torch.int16).masked_fill_(
                dead[:, None, :, None].expand(mp, Hkv, page_size, D), NAN_BF16_BITS)
    kp[bt.reshape(-1).long()] = src_k
    vp[bt.reshape(-1).long()] = src_v
    return kp, vp, bt


def ragged_paged_inputs(seqs, Hq: int, Hkv: int, D: int, page_size: int, seed: int,
                        extra_pages: int = 0, k_mult: float = 1.0):
    """Seeded inputs of a ragged paged batch, sequences [(Sq_b, L_b), ...]:
    Sq_b packed query tokens and L_b keys each (L_b may be 0, negative or past
    the table, exercising the clamps).  q [total_q,Hq,D] randn in fp32 (then
    bf16); contiguous caches [B,Hkv,max_pages*page_size,D] randn (K times
    k_mult) scattered into NaN-poisoned page pools by paged_layout.  Returns
    (q, k_pages, v_pages, block_table, cu_q int32 [B+1], lens int32 [B],
    k_cache, v_cache)."""
    g = _gen(seed)
    cu = torch.zeros(len(seqs) + 1, dtype=torch.int32)
    cu[1:] = torch.cumsum(torch.tensor([a for a, _ in seqs], dtype=torch.int32), 0)
    lens = torch.tensor([b for _, b in seqs], dtype=torch.int32)
    mp = max(1, max(-(-max(0, b) // page_size) for _, b in seqs))
    q = torch.randn((max(int(cu[-1]), 1), Hq, D), generator=g).to(torch.bfloat16)
    kc = (torch.randn((len(seqs), Hkv, mp * page_size, D), generator=g) * k_mult).to(torch.bfloat16)
    vc = torch.randn((len(seqs), Hkv, mp * page_size, D), generator=g).to(torch.bfloat16)
    kp, vp, bt = paged_layout(kc, vc, page_size, seed + 1, extra_pages=extra_pages, lens=lens)
    return q, kp, vp, bt, cu, lens, kc, vc


# The ragged paged bench batch: prefill chunks over earlier context and decode
# tokens in one call, Hq = 32, Hkv = 8, D = 128, 64-key pages.
RPA = dict(name="rpa_mixed_b64", n_prefill=8, n_decode=56, Hq=32, Hkv=8, D=128, page_size=64,
           seed=1008)


def ragged_paged_mix(n_prefill: int, n_decode: int, seed: int):
    """Seeded (Sq, L) list of a serving step: n_prefill chunks of U{512..2048}
    queries after U{0..4096} keys of earlier context (L = context + chunk),
    then n_decode single tokens over U{512..4096} keys."""
    g = _gen(seed)
    seqs = []
    for _ in range(n_prefill):
        sq = int(torch.randint(512, 2049, (1,), generator=g))
        ctx = int(torch.randint(0, 4097, (1,), generator=g))
        seqs.append((sq, ctx + sq))
    for _ in range(n_decode):
        seqs.append((1, int(torch.randint(512, 4097, (1,), generator=g))))
    return seqs


def sample_rows(B: int, Hq: int, S: int, nrows: int, seed: int) -> torch.Tensor:
    """int32 [B,Hq,nrows] of query rows: 0 and S-1 plus nrows-2 distinct
    rows drawn from a per-(b, hq) seeded permutation."""
    out = torch.empty((B, Hq, nrows), dtype=torch.int32)
    for b in range(B):
        for h in range(Hq):
            g = _gen(seed * 1_000_003 + b * 1009 + h)
            perm = torch.randperm(S, generator=g)
            extra = [int(x) for x in perm.tolist() if 0 < int(x) < S - 1][: nrows - 2]
            rows = sorted([0, S - 1] + extra)
            out[b, h] = torch.tensor(rows, dtype=torch.int32)
    return out


def config_inputs(cfg):
    """Inputs of a table entry."""
    if isinstance(cfg, DecodeConfig):
        return decode_inputs(cfg.B, cfg.Hq, cfg.Hkv, cfg.Smax, cfg.D, cfg.seed, cfg.lmin, cfg.lmax)
    return prefill_inputs(cfg.B, cfg.Hq, cfg.Hkv, cfg.S, cfg.S, cfg.D, cfg.seed, cfg.k_mult)


def bits(t: torch.Tensor):
    """bf16 tensor -> numpy uint16 of the same bits (for the oracle)."""
    return t.contiguous().view(torch.int16).numpy().view("uint16")
