"""Pins for the CPU oracle: checks against facts fixed by the mathematics.

Each ``pin_*`` function takes an oracle ctypes handle and raises
``AssertionError`` when the oracle disagrees with the fact it checks.  The
test suite runs them against the real oracle (they must pass) and against
deliberately broken copies of the oracle built on the CPU (at least one
must fail for every planted mistake).

The facts, none of which re-types the oracle's own formula:
  * brute force: a pure-Python evaluation that materialises the masked
    score matrix and exponentiates without max-subtraction (tiny inputs);
  * hand-derived closed forms stored under tests/golden/;
  * rows of the attention weights sum to 1, and vanish where masked;
  * all value rows equal to r  =>  every output row equals r;
  * causal query 0 returns v_0 with LSE = scale * q_0 . k_0;
  * a single key returns v_0 for every query;
  * scale 0 turns softmax into a prefix mean with LSE = log(count);
  * grouped heads equal plain multi-head attention on K/V heads repeated
    G times in order (the contiguous grouping);
  * a decode step equals the last row of the causal prefill over the same
    keys;
  * the split-KV form with its log-sum-exp merge equals the unsplit result
    for any split length;
  * a paged cache is a relayout: paged decode equals contiguous decode on
    the cache gathered through the block table (numpy indexing), whatever
    the page size, with out-of-range table entries read as the nearest
    valid page and pages no sequence lists ignored;
  * a packed ragged batch equals each of its sequences run alone through
    the batched forward (bottom-right causal per sequence), rows no
    sequence owns are not written, and out-of-range offsets clamp;
  * the backward equals central finite differences of <dO, O> computed
    with the pure-Python forward in float64 (independent of the gradient
    formulas), and grouped heads' dK/dV are the sums over the group of the
    repeated-head gradients.
"""
from __future__ import annotations

import json
import math
import os

import numpy as np
import torch

import workloads
from oracle import brute
from oracle import oracle as orc

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "hand_cases.json")


def _bits_of_floats(x) -> np.ndarray:
    t = torch.tensor(x, dtype=torch.float32).to(torch.bfloat16)
    # values in the golden file are exact in bf16
    assert torch.equal(t.float(), torch.tensor(x, dtype=torch.float32)), "inexact bf16 value"
    return workloads.bits(t)


def _f(bits: np.ndarray) -> np.ndarray:
    """uint16 bf16 bits -> float64, via torch (independent of the oracle)."""
    t = torch.from_numpy(bits.astype(np.int16)).view(torch.bfloat16)
    return t.double().numpy()


def _rand(shape, seed, lo=-2.0, hi=2.0):
    g = torch.Generator().manual_seed(seed)
    x = torch.rand(shape, generator=g) * (hi - lo) + lo
    return workloads.bits(x.to(torch.bfloat16))


def _close(a, b, tol, what):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    both_inf = np.isinf(a) & np.isinf(b) & (np.sign(a) == np.sign(b))
    with np.errstate(invalid="ignore"):
        err = np.where(both_inf, 0.0, np.abs(a - b))
    scale = np.maximum(1.0, np.where(both_inf, 1.0, np.abs(b)))
    bad = ~(err <= tol * scale)
    assert not bad.any(), f"{what}: max err {np.nanmax(np.where(bad, err, 0))} (tol {tol})"


# --------------------------------------------------------------------------
def pin_golden(lib):
    with open(GOLDEN) as fh:
        cases = json.load(fh)["cases"]
    env = {"e": math.e, "exp": math.exp, "log": math.log, "sqrt": math.sqrt,
           "inf": math.inf, "__builtins__": {}}
    for c in cases:
        q = _bits_of_floats(c["q"])
        k = _bits_of_floats(c["k"])
        v = _bits_of_floats(c["v"])
        o, lse = orc.attn_fwd(q, k, v, causal=c["causal"], scale=c["scale"],
                              kv_seqlens=c["kv_seqlens"], lib=lib, threads=1)
        o_exp = np.vectorize(lambda s: float(eval(s, env)))(np.array(c["o"], dtype=object))
        lse_exp = np.vectorize(lambda s: float(eval(s, env)))(np.array(c["lse"], dtype=object))
        _close(o, o_exp.astype(np.float64), 1e-14, c["name"] + " O")
        _close(lse, lse_exp.astype(np.float64), 1e-14, c["name"] + " LSE")


BRUTE_CASES = [
    # B, Hq, Hkv, Sq, Skv, D, causal, seqlens
    (1, 1, 1, 5, 5, 4, True, None),
    (1, 2, 2, 7, 7, 1, False, None),
    (2, 4, 2, 6, 6, 4, True, None),
    (1, 4, 1, 3, 9, 8, True, None),          # Sq < Skv, bottom-right
    (2, 2, 1, 4, 8, 4, True, [5, 8]),        # ragged lengths
    (2, 2, 2, 8, 8, 4, False, [3, 0]),       # an empty sequence
    (3, 2, 1, 4, 6, 2, True, [9, -3, 2]),    # out-of-range lengths clamp
    (1, 2, 1, 16, 16, 64, True, None),
]


def pin_brute_force(lib):
    for n, (B, Hq, Hkv, Sq, Skv, D, causal, sl) in enumerate(BRUTE_CASES):
        q = _rand((B, Hq, Sq, D), 10 + n)
        k = _rand((B, Hkv, Skv, D), 20 + n)
        v = _rand((B, Hkv, Skv, D), 30 + n)
        scale = 0.7 / math.sqrt(D)
        o, lse = orc.attn_fwd(q, k, v, causal=causal, scale=scale, kv_seqlens=sl, lib=lib,
                              threads=2)
        ob, lb = brute.attention(q.tolist(), k.tolist(), v.tolist(), causal=causal,
                                 scale=scale, kv_seqlens=sl)
        _close(o, np.array(ob), 1e-12, f"brute case {n} O")
        _close(lse, np.array(lb), 1e-12, f"brute case {n} LSE")


def pin_rows_sum_to_one(lib):
    B, Hq, Hkv, Sq, Skv, D = 2, 4, 2, 9, 13, 8
    q = _rand((B, Hq, Sq, D), 41, -3, 3)
    k = _rand((B, Hkv, Skv, D), 42, -3, 3)
    for causal in (True, False):
        for sl in (None, [13, 6]):
            p = orc.attn_probs(q, k, causal=causal, scale=0.9, kv_seqlens=sl, lib=lib)
            for b in range(B):
                L = Skv if sl is None else sl[b]
                for i in range(Sq):
                    last = i + (L - Sq) if causal else L - 1
                    lim = max(0, min(L, last + 1))  # admissible keys are [0, lim)
                    row = p[b, :, i]
                    if lim == 0:
                        assert np.all(row == 0.0), "weights on an empty row"
                        continue
                    s = row.sum(axis=-1)
                    assert np.all(np.abs(s - 1.0) <= 1e-13), f"rows sum {s.min()}..{s.max()}"
                    # weights vanish exactly outside the admissible set
                    assert np.all(row[:, lim:] == 0.0), "weight on a masked key"
                    assert np.all(row[:, :lim] > 0.0), "zero weight on an admissible key"


def pin_probs_brute_force(lib):
    """The weights themselves: equal to the brute-force exp(s) / sum exp(s)
    (materialised mask, no max-subtraction) on the brute cases, which fixes
    the scale, the head mapping and the mask inside them."""
    for n, (B, Hq, Hkv, Sq, Skv, D, causal, sl) in enumerate(BRUTE_CASES):
        q = _rand((B, Hq, Sq, D), 10 + n)
        k = _rand((B, Hkv, Skv, D), 20 + n)
        scale = 0.7 / math.sqrt(D)
        p = orc.attn_probs(q, k, causal=causal, scale=scale, kv_seqlens=sl, lib=lib)
        pb = brute.probs(q.tolist(), k.tolist(), causal=causal, scale=scale, kv_seqlens=sl)
        _close(p, np.array(pb), 1e-13, f"brute case {n} P")


def pin_probs_times_values(lib):
    """P V (a numpy product, V's heads repeated G times in order) equals the
    forward's O: the weights are the ones the output is formed with."""
    B, Hq, Hkv, Sq, Skv, D = 2, 6, 2, 7, 11, 8
    q = _rand((B, Hq, Sq, D), 61, -3, 3)
    k = _rand((B, Hkv, Skv, D), 62, -3, 3)
    v = _rand((B, Hkv, Skv, D), 63)
    vr = np.repeat(_f(v), Hq // Hkv, axis=1)
    for causal in (True, False):
        for sl in (None, [11, 4]):
            p = orc.attn_probs(q, k, causal=causal, scale=0.8, kv_seqlens=sl, lib=lib)
            o, _ = orc.attn_fwd(q, k, v, causal=causal, scale=0.8, kv_seqlens=sl, lib=lib)
            _close(p @ vr, o, 1e-13, "P V against O")


def pin_equal_value_rows(lib):
    B, Hq, Hkv, S, D = 1, 4, 2, 33, 16
    q = _rand((B, Hq, S, D), 51, -4, 4)
    k = _rand((B, Hkv, S, D), 52, -4, 4)
    r = _rand((1, 1, 1, D), 53)
    v = np.broadcast_to(r, (B, Hkv, S, D)).copy()
    for causal in (True, False):
        o, _ = orc.attn_fwd(q, k, v, causal=causal, scale=0.5, lib=lib)
        _close(o, np.broadcast_to(_f(r), o.shape), 1e-13, "equal V rows")


def pin_causal_row0(lib):
    B, Hq, Hkv, S, D = 2, 4, 1, 11, 32
    q = _rand((B, Hq, S, D), 61)
    k = _rand((B, Hkv, S, D), 62)
    v = _rand((B, Hkv, S, D), 63)
    scale = 0.125
    o, lse = orc.attn_fwd(q, k, v, causal=True, scale=scale, lib=lib)
    qf, kf, vf = _f(q), _f(k), _f(v)
    for b in range(B):
        for h in range(Hq):
            assert np.array_equal(o[b, h, 0], vf[b, 0, 0]), "causal row 0 is not v_0"
            dot = math.fsum(qf[b, h, 0, d] * kf[b, 0, 0, d] for d in range(D))
            _close(lse[b, h, 0], scale * dot, 1e-15, "causal row 0 LSE")


def pin_single_key(lib):
    B, Hq, Hkv, Sq, D = 1, 2, 2, 6, 8
    q = _rand((B, Hq, Sq, D), 71)
    k = _rand((B, Hkv, 1, D), 72)
    v = _rand((B, Hkv, 1, D), 73)
    o, lse = orc.attn_fwd(q, k, v, causal=False, scale=0.3, lib=lib)
    qf, kf, vf = _f(q), _f(k), _f(v)
    for h in range(Hq):
        for i in range(Sq):
            assert np.array_equal(o[0, h, i], vf[0, h, 0]), "single key output is not v_0"
            dot = math.fsum(qf[0, h, i, d] * kf[0, h, 0, d] for d in range(D))
            _close(lse[0, h, i], 0.3 * dot, 1e-15, "single key LSE")


def pin_scale_zero(lib):
    B, Hq, Hkv, S, D = 2, 2, 1, 19, 8
    q = _rand((B, Hq, S, D), 81)
    k = _rand((B, Hkv, S, D), 82)
    v = _rand((B, Hkv, S, D), 83)
    vf = _f(v)
    sl = [19, 7]
    o, lse = orc.attn_fwd(q, k, v, causal=True, scale=0.0, kv_seqlens=sl, lib=lib)
    for b in range(B):
        L = sl[b]
        for i in range(S):
            n = max(0, min(L, i + (L - S) + 1))
            if n == 0:
                assert np.all(o[b, :, i] == 0) and np.all(np.isneginf(lse[b, :, i]))
                continue
            mean = vf[b, 0, :n].mean(axis=0)
            _close(o[b, :, i], np.broadcast_to(mean, (Hq, D)), 1e-14, "scale 0 prefix mean")
            _close(lse[b, :, i], math.log(n), 1e-15, "scale 0 LSE")
    o, lse = orc.attn_fwd(q, k, v, causal=False, scale=0.0, kv_seqlens=sl, lib=lib)
    for b in range(B):
        _close(o[b], np.broadcast_to(vf[b, 0, :sl[b]].mean(axis=0), o[b].shape), 1e-14,
               "scale 0 non-causal mean")
        _close(lse[b], math.log(sl[b]), 1e-15, "scale 0 non-causal LSE")


def pin_gqa_equals_repeated_mha(lib):
    B, Hq, Hkv, S, D = 2, 8, 2, 12, 16
    q = _rand((B, Hq, S, D), 91)
    k = _rand((B, Hkv, S, D), 92)
    v = _rand((B, Hkv, S, D), 93)
    G = Hq // Hkv
    k_rep = np.repeat(k, G, axis=1)  # head h of the repeat is KV head h // G
    v_rep = np.repeat(v, G, axis=1)
    for causal in (True, False):
        o1, l1 = orc.attn_fwd(q, k, v, causal=causal, scale=0.25, lib=lib)
        o2, l2 = orc.attn_fwd(q, k_rep, v_rep, causal=causal, scale=0.25, lib=lib)
        _close(o1, o2, 1e-15, "GQA vs repeated MHA O")
        _close(l1, l2, 1e-15, "GQA vs repeated MHA LSE")
    # and the grouping really is contiguous: perturbing KV head 1 moves query
    # heads G..2G-1 and no other
    k2 = k.copy()
    k2[:, 1] = _rand((B, 1, S, D), 94)[:, 0]
    o3, _ = orc.attn_fwd(q, k2, v, causal=True, scale=0.25, lib=lib)
    o1, _ = orc.attn_fwd(q, k, v, causal=True, scale=0.25, lib=lib)
    same = np.all(o1 == o3, axis=(0, 2, 3))
    assert list(same) == [True] * G + [False] * G, f"head grouping {same}"


def pin_decode_equals_last_prefill_row(lib):
    B, Hq, Hkv, Smax, D = 3, 4, 2, 20, 16
    q_all = _rand((B, Hq, Smax, D), 101)
    kc = _rand((B, Hkv, Smax, D), 102)
    vc = _rand((B, Hkv, Smax, D), 103)
    lens = [20, 1, 13]
    q_dec = np.stack([q_all[b, :, lens[b] - 1] for b in range(B)])
    od, ld = orc.decode(q_dec, kc, vc, lens, scale=0.2, lib=lib)
    for b in range(B):
        L = lens[b]
        o, lse = orc.attn_fwd(q_all[b:b + 1, :, :L], kc[b:b + 1, :, :L], vc[b:b + 1, :, :L],
                              causal=True, scale=0.2, lib=lib)
        _close(od[b], o[0, :, L - 1], 1e-15, "decode vs prefill row O")
        _close(ld[b], lse[0, :, L - 1], 1e-15, "decode vs prefill row LSE")
    # one-query prefill with a length mask is the same decode step
    o1, l1 = orc.attn_fwd(q_dec[:, :, None, :], kc, vc, causal=True, scale=0.2,
                          kv_seqlens=lens, lib=lib)
    _close(o1[:, :, 0], od, 1e-15, "Sq=1 bottom-right causal vs decode")
    _close(l1[:, :, 0], ld, 1e-15, "Sq=1 bottom-right causal vs decode LSE")


def pin_split_combine(lib):
    B, Hq, Hkv, Smax, D = 3, 4, 1, 37, 8
    q = _rand((B, Hq, D), 111, -3, 3)
    kc = _rand((B, Hkv, Smax, D), 112, -3, 3)
    vc = _rand((B, Hkv, Smax, D), 113)
    lens = [37, 5, 0]
    od, ld = orc.decode(q, kc, vc, lens, scale=0.6, lib=lib)
    for split in (1, 4, 7, 16, 37, 64):
        o, lse, op, lp = orc.decode_split(q, kc, vc, lens, scale=0.6, split=split, lib=lib)
        _close(o, od, 1e-13, f"split {split} O")
        _close(lse, ld, 1e-13, f"split {split} LSE")
        # splits past the sequence end are empty
        nsplit = op.shape[2]
        for b in range(B):
            for s in range(nsplit):
                if s * split >= lens[b]:
                    assert np.all(np.isneginf(lp[b, :, s])) and np.all(op[b, :, s] == 0)


def pin_row_subset(lib):
    B, Hq, Hkv, S, D = 1, 4, 2, 40, 8
    q = _rand((B, Hq, S, D), 121)
    k = _rand((B, Hkv, S, D), 122)
    v = _rand((B, Hkv, S, D), 123)
    rows = workloads.sample_rows(B, Hq, S, 6, seed=5).numpy()
    o_all, l_all = orc.attn_fwd(q, k, v, causal=True, scale=0.3, lib=lib)
    o_sub, l_sub = orc.attn_fwd(q, k, v, causal=True, scale=0.3, rows=rows, lib=lib)
    for b in range(B):
        for h in range(Hq):
            assert np.array_equal(o_sub[b, h], o_all[b, h, rows[b, h]])
            assert np.array_equal(l_sub[b, h], l_all[b, h, rows[b, h]])


def _gather_pages(pages: np.ndarray, block_table: np.ndarray) -> np.ndarray:
    """Page pool [n_pages, Hkv, ps, D] + table [B, max_pages] -> contiguous
    cache [B, Hkv, max_pages * ps, D], by numpy fancy indexing."""
    n_pages, Hkv, ps, D = pages.shape
    B, max_pages = block_table.shape
    g = pages[np.clip(block_table, 0, n_pages - 1)]          # [B, max_pages, Hkv, ps, D]
    return np.ascontiguousarray(g.transpose(0, 2, 1, 3, 4).reshape(B, Hkv, max_pages * ps, D))


PAGED_CASES = [
    # B, Hq, Hkv, page_size, max_pages, n_pages, D, lengths
    (3, 4, 2, 16, 4, 15, 8, [64, 1, 37]),
    (2, 2, 1, 3, 5, 12, 4, [15, 7]),        # odd page size
    (2, 4, 4, 1, 9, 20, 4, [9, 0]),         # one key per page, an empty sequence
    (1, 8, 2, 32, 3, 3, 16, [96]),
    (2, 2, 2, 16, 2, 6, 8, [40, -3]),       # lengths clamp to [0, 32]
]


def pin_paged_equals_gathered(lib):
    for n, (B, Hq, Hkv, ps, mp, npg, D, lens) in enumerate(PAGED_CASES):
        q = _rand((B, Hq, D), 130 + n, -3, 3)
        kp = _rand((npg, Hkv, ps, D), 140 + n, -3, 3)
        vp = _rand((npg, Hkv, ps, D), 150 + n)
        bt = np.random.default_rng(160 + n).integers(0, npg, size=(B, mp), dtype=np.int32)
        o, lse = orc.decode_paged(q, kp, vp, bt, lens, scale=0.45, lib=lib)
        og, lg = orc.decode(q, _gather_pages(kp, bt), _gather_pages(vp, bt), lens, scale=0.45,
                            lib=lib)
        _close(o, og, 1e-13, f"paged case {n} O")
        _close(lse, lg, 1e-13, f"paged case {n} LSE")


def pin_paged_table_clamp_and_unused_pages(lib):
    B, Hq, Hkv, ps, mp, npg, D = 2, 4, 2, 4, 5, 9, 8
    lens = [20, 11]
    q = _rand((B, Hq, D), 171, -3, 3)
    kp = _rand((npg, Hkv, ps, D), 172, -3, 3)
    vp = _rand((npg, Hkv, ps, D), 173)
    bt = np.array([[3, -7, 8, 14, 0], [5, 2, 2, 100, 1]], dtype=np.int32)
    o, lse = orc.decode_paged(q, kp, vp, bt, lens, scale=0.3, lib=lib)
    oc, lc = orc.decode_paged(q, kp, vp, np.clip(bt, 0, npg - 1), lens, scale=0.3, lib=lib)
    assert np.array_equal(o, oc) and np.array_equal(lse, lc), "table entries not clamped"
    og, lg = orc.decode(q, _gather_pages(kp, bt), _gather_pages(vp, bt), lens, scale=0.3, lib=lib)
    _close(o, og, 1e-13, "clamped table vs gathered O")
    _close(lse, lg, 1e-13, "clamped table vs gathered LSE")
    # pages 4, 6 and 7 are listed by no sequence (and 1 only past sequence 1's
    # length): changing them changes nothing; changing page 5 changes sequence 1
    used = set(np.clip(bt[0, :5], 0, npg - 1).tolist()) | set(np.clip(bt[1, :3], 0, npg - 1).tolist())
    kp2, vp2 = kp.copy(), vp.copy()
    for pg in range(npg):
        if pg not in used:
            kp2[pg] = _rand((Hkv, ps, D), 180 + pg)
            vp2[pg] = _rand((Hkv, ps, D), 190 + pg)
    o2, l2 = orc.decode_paged(q, kp2, vp2, bt, lens, scale=0.3, lib=lib)
    assert np.array_equal(o, o2) and np.array_equal(lse, l2), "an unused page changed the result"
    vp2[5, :, 0] = _rand((Hkv, D), 199)
    o3, _ = orc.decode_paged(q, kp2, vp2, bt, lens, scale=0.3, lib=lib)
    assert np.array_equal(o3[0], o[0]) and not np.array_equal(o3[1], o[1]), "page 5 row 0 ignored"


VARLEN_CASES = [
    # Hq, Hkv, D, [(Sq_b, Skv_b), ...]
    (4, 2, 8, [(5, 5), (1, 9), (0, 4), (7, 3), (6, 6)]),  # decode-like, empty, Sq > Skv
    (2, 1, 16, [(12, 20), (3, 3)]),                        # a chunk of a longer prompt
    (3, 3, 4, [(4, 0), (2, 2)]),                           # a sequence without keys
]


def _varlen_inputs(n, Hq, Hkv, D, seqs):
    cq = np.concatenate([[0], np.cumsum([a for a, _ in seqs])]).astype(np.int32)
    ck = np.concatenate([[0], np.cumsum([b for _, b in seqs])]).astype(np.int32)
    q = _rand((int(cq[-1]), Hq, D), 200 + n, -2.5, 2.5)
    k = _rand((max(int(ck[-1]), 1), Hkv, D), 210 + n, -2.5, 2.5)
    v = _rand((max(int(ck[-1]), 1), Hkv, D), 220 + n)
    return q, k, v, cq, ck


def pin_varlen_equals_each_sequence(lib):
    for causal in (True, False):
        for n, (Hq, Hkv, D, seqs) in enumerate(VARLEN_CASES):
            q, k, v, cq, ck = _varlen_inputs(n, Hq, Hkv, D, seqs)
            o, lse = orc.attn_fwd_varlen(q, k, v, cq, ck, causal=causal, scale=0.4, lib=lib)
            for b, (Sq, Skv) in enumerate(seqs):
                if Sq == 0:
                    continue
                ob = o[cq[b]:cq[b + 1]].transpose(1, 0, 2)
                lb = lse[:, cq[b]:cq[b + 1]]
                if Skv == 0:
                    assert np.all(ob == 0) and np.all(np.isneginf(lb)), "keyless sequence"
                    continue
                qb = np.ascontiguousarray(q[cq[b]:cq[b + 1]].transpose(1, 0, 2)[None])
                kb = np.ascontiguousarray(k[ck[b]:ck[b + 1]].transpose(1, 0, 2)[None])
                vb = np.ascontiguousarray(v[ck[b]:ck[b + 1]].transpose(1, 0, 2)[None])
                o1, l1 = orc.attn_fwd(qb, kb, vb, causal=causal, scale=0.4, lib=lib)
                _close(ob, o1[0], 1e-14, f"varlen case {n} seq {b} causal={causal} O")
                _close(lb, l1[0], 1e-14, f"varlen case {n} seq {b} causal={causal} LSE")


def pin_varlen_gaps_and_clamped_offsets(lib):
    Hq, Hkv, D = 2, 1, 8
    q = _rand((12, Hq, D), 231)
    k = _rand((10, Hkv, D), 232)
    v = _rand((10, Hkv, D), 233)
    # query rows 3..4 and 9..11 belong to no sequence; offsets past the
    # totals clamp
    cq = np.array([0, 3, 5, 9], np.int32)
    ck = np.array([0, 4, 4, 99], np.int32)
    cq_gap = np.array([0, 3, 3, 3], np.int32)  # same first sequence, nothing else
    o, lse = orc.attn_fwd_varlen(q, k, v, np.array([0, 3, 5, 9], np.int32), ck, causal=True,
                                 scale=0.5, lib=lib)
    og, lg = orc.attn_fwd_varlen(q, k, v, cq_gap, ck, causal=True, scale=0.5, lib=lib)
    assert np.array_equal(o[:3], og[:3]) and np.array_equal(lse[:, :3], lg[:, :3])
    assert np.all(np.isnan(og[3:])) and np.all(np.isnan(lg[:, 3:])), "unowned rows written"
    # sequence 2: queries 5..8, keys clamp to [4, 10)
    oc, lc = orc.attn_fwd_varlen(q, k, v, cq, np.array([0, 4, 4, 10], np.int32), causal=True,
                                 scale=0.5, lib=lib)
    assert np.array_equal(o[:9], oc[:9]) and np.array_equal(lse[:, :9], lc[:, :9]), \
        "offsets not clamped"


RAGGED_PAGED_CASES = [
    # Hq, Hkv, D, page_size, max_pages, n_pages, [(Sq_b, L_b), ...]
    (4, 2, 8, 16, 4, 20, [(5, 37), (1, 64), (0, 10), (7, 3), (16, 16), (3, 0)]),
    (2, 1, 4, 3, 6, 9, [(4, 17), (2, 2), (6, 5)]),       # odd page size, Sq > L
    (3, 3, 8, 8, 2, 7, [(2, 100), (1, -4), (4, 16)]),    # lengths clamp to [0, 16]
]


def _ragged_paged_inputs(n, Hq, Hkv, D, ps, mp, npg, seqs):
    cq = np.concatenate([[0], np.cumsum([a for a, _ in seqs])]).astype(np.int32)
    q = _rand((max(int(cq[-1]), 1), Hq, D), 240 + n, -2.5, 2.5)
    kp = _rand((npg, Hkv, ps, D), 250 + n, -2.5, 2.5)
    vp = _rand((npg, Hkv, ps, D), 260 + n)
    bt = np.random.default_rng(270 + n).integers(-2, npg + 2, size=(len(seqs), mp),
                                                  dtype=np.int32)  # some entries out of range
    lens = np.array([b for _, b in seqs], np.int32)
    return q, kp, vp, cq, lens, bt


def _gather_keys(pages, bt, lens):
    """Packed [sum L, Hkv, D] rows of every sequence's valid keys, read
    through the table by numpy indexing (entries clamped into the pool)."""
    n_pages, Hkv, ps, D = pages.shape
    rows = []
    for b, L in enumerate(lens):
        L = min(max(int(L), 0), bt.shape[1] * ps)
        j = np.arange(L)
        rows.append(pages[np.clip(bt[b, j // ps], 0, n_pages - 1), :, j % ps, :])
    out = np.concatenate(rows) if rows else np.zeros((0, Hkv, D), pages.dtype)
    return np.ascontiguousarray(out if out.shape[0] else np.zeros((1, Hkv, D), pages.dtype))


def pin_ragged_paged_equals_gathered_varlen(lib):
    for causal in (True, False):
        for n, (Hq, Hkv, D, ps, mp, npg, seqs) in enumerate(RAGGED_PAGED_CASES):
            q, kp, vp, cq, lens, bt = _ragged_paged_inputs(n, Hq, Hkv, D, ps, mp, npg, seqs)
            o, lse = orc.attn_fwd_ragged_paged(q, kp, vp, cq, lens, bt, causal=causal, scale=0.4,
                                               lib=lib)
            lc = np.clip(lens, 0, mp * ps)
            ck = np.concatenate([[0], np.cumsum(lc)]).astype(np.int32)
            og, lg = orc.attn_fwd_varlen(q, _gather_keys(kp, bt, lens), _gather_keys(vp, bt, lens),
                                         cq, ck, causal=causal, scale=0.4, lib=lib)
            tq = int(cq[-1])
            _close(o[:tq], og[:tq], 1e-13, f"ragged paged case {n} causal={causal} O")
            _close(lse[:, :tq], lg[:, :tq], 1e-13, f"ragged paged case {n} causal={causal} LSE")


def pin_ragged_paged_decode_tokens(lib):
    # one query token per sequence: the paged decode step
    Hq, Hkv, D, ps, mp, npg = 4, 2, 8, 4, 6, 11
    seqs = [(1, 21), (1, 1), (1, 24), (1, 0), (1, 9)]
    q, kp, vp, cq, lens, bt = _ragged_paged_inputs(7, Hq, Hkv, D, ps, mp, npg, seqs)
    for causal in (True, False):
        o, lse = orc.attn_fwd_ragged_paged(q, kp, vp, cq, lens, bt, causal=causal, scale=0.35,
                                           lib=lib)
        od, ld = orc.decode_paged(q, kp, vp, bt, lens, scale=0.35, lib=lib)
        _close(o, od, 1e-13, f"ragged paged decode tokens causal={causal} O")
        _close(lse.T, ld, 1e-13, f"ragged paged decode tokens causal={causal} LSE")


BWD_FD_CASES = [
    # B, Hq, Hkv, Sq, Skv, D, causal, seqlens
    (1, 2, 1, 4, 4, 3, True, None),
    (1, 2, 2, 3, 5, 2, False, [4]),
    (2, 2, 1, 3, 3, 2, True, [3, 1]),   # a short sequence: rows without keys
    (1, 1, 1, 2, 4, 2, True, None),     # bottom-right causal, Sq < Skv
]


def pin_bwd_finite_differences(lib):
    h = 1e-4
    for n, (B, Hq, Hkv, Sq, Skv, D, causal, sl) in enumerate(BWD_FD_CASES):
        q = _rand((B, Hq, Sq, D), 240 + n, -1.5, 1.5)
        k = _rand((B, Hkv, Skv, D), 250 + n, -1.5, 1.5)
        v = _rand((B, Hkv, Skv, D), 260 + n)
        do = _rand((B, Hq, Sq, D), 270 + n)
        scale = 0.8
        dq, dk, dv = orc.attn_bwd(q, k, v, do, causal=causal, scale=scale, kv_seqlens=sl, lib=lib)
        qf, kf, vf, dof = _f(q), _f(k), _f(v), _f(do)

        def loss(qx, kx, vx):
            o, _ = brute.attention_f(qx.tolist(), kx.tolist(), vx.tolist(), causal=causal,
                                     scale=scale, kv_seqlens=sl)
            return float(np.sum(np.array(o) * dof))

        for name, x, got in (("dq", qf, dq), ("dk", kf, dk), ("dv", vf, dv)):
            fd = np.zeros_like(x)
            for idx in np.ndindex(x.shape):
                xp, xm = x.copy(), x.copy()
                xp[idx] += h
                xm[idx] -= h
                args_p = [xp if t is x else t for t in (qf, kf, vf)]
                args_m = [xm if t is x else t for t in (qf, kf, vf)]
                fd[idx] = (loss(*args_p) - loss(*args_m)) / (2 * h)
            _close(got, fd, 1e-6, f"bwd case {n} {name} vs finite differences")


def pin_bwd_gqa_sums_repeated_heads(lib):
    B, Hq, Hkv, S, D = 1, 6, 2, 7, 4
    G = Hq // Hkv
    q = _rand((B, Hq, S, D), 281)
    k = _rand((B, Hkv, S, D), 282)
    v = _rand((B, Hkv, S, D), 283)
    do = _rand((B, Hq, S, D), 284)
    dq, dk, dv = orc.attn_bwd(q, k, v, do, causal=True, scale=0.5, lib=lib)
    dq2, dk2, dv2 = orc.attn_bwd(q, np.repeat(k, G, axis=1), np.repeat(v, G, axis=1), do,
                                 causal=True, scale=0.5, lib=lib)
    _close(dq, dq2, 1e-14, "GQA dq")
    _close(dk, dk2.reshape(B, Hkv, G, S, D).sum(axis=2), 1e-13, "GQA dk = group sum")
    _close(dv, dv2.reshape(B, Hkv, G, S, D).sum(axis=2), 1e-13, "GQA dv = group sum")


MLA_CASES = [
    # B, H, Dc, Dr, Smax, lengths
    (1, 1, 4, 2, 5, [5]),
    (2, 3, 8, 4, 7, [7, 3]),
    (3, 2, 6, 0, 4, [0, 4, 9]),        # no rotary part; an empty and a clamped sequence
    (2, 4, 16, 8, 6, [-2, 6]),
]


def _mla_inputs(B, H, Dc, Dr, Smax, seed):
    return _rand((B, H, Dc + Dr), seed), _rand((B, Smax, Dc + Dr), seed + 1)


def pin_mla_brute_force(lib):
    for n, (B, H, Dc, Dr, Smax, lens) in enumerate(MLA_CASES):
        q, ckv = _mla_inputs(B, H, Dc, Dr, Smax, 300 + 2 * n)
        scale = 0.6 / math.sqrt(Dc + Dr)
        o, lse = orc.mla_decode(q, ckv, lens, Dc=Dc, scale=scale, lib=lib)
        ob, lb = brute.mla_decode(q.tolist(), ckv.tolist(), lens, Dc=Dc, scale=scale)
        _close(o, np.array(ob), 1e-12, f"MLA brute case {n} O")
        _close(lse, np.array(lb), 1e-12, f"MLA brute case {n} LSE")


def pin_mla_equals_padded_decode(lib):
    """MLA decode = the plain decode with one kv head whose K rows are the
    whole cache rows and whose V rows are the same rows with the rotary
    part zeroed, output truncated to the latent part."""
    B, H, Dc, Dr, Smax = 3, 8, 32, 16, 20
    lens = [20, 7, 1]
    q, ckv = _mla_inputs(B, H, Dc, Dr, Smax, 320)
    scale = 1.0 / math.sqrt(Dc + Dr)
    o, lse = orc.mla_decode(q, ckv, lens, Dc=Dc, scale=scale, lib=lib)
    v = ckv.copy()
    v[:, :, Dc:] = 0
    od, ld = orc.decode(q, ckv[:, None], v[:, None], np.array(lens, np.int32), scale=scale,
                        lib=lib)
    _close(o, od[:, :, :Dc], 1e-13, "MLA = padded decode O")
    assert np.all(od[:, :, Dc:] == 0.0)
    _close(lse, ld, 1e-13, "MLA = padded decode LSE")


def pin_mla_single_key_and_rope(lib):
    B, H, Dc, Dr, Smax = 1, 3, 8, 4, 6
    q, ckv = _mla_inputs(B, H, Dc, Dr, Smax, 340)
    o, lse = orc.mla_decode(q, ckv, [1], Dc=Dc, scale=0.4, lib=lib)
    qf, cf = _f(q), _f(ckv)
    for h in range(H):
        assert np.array_equal(o[0, h], cf[0, 0, :Dc]), "one key: O is the latent row"
        _close(lse[0, h], 0.4 * math.fsum(qf[0, h] * cf[0, 0]), 1e-15, "one key LSE")
    # with the query's rotary part zero, the cache's rotary part cannot matter
    q0 = q.copy()
    q0[:, :, Dc:] = 0
    ckv2 = ckv.copy()
    ckv2[:, :, Dc:] = _rand((B, Smax, Dr), 341)
    a = orc.mla_decode(q0, ckv, [Smax], Dc=Dc, scale=0.4, lib=lib)
    b = orc.mla_decode(q0, ckv2, [Smax], Dc=Dc, scale=0.4, lib=lib)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])
    # and with it nonzero, the rotary part enters the scores
    c = orc.mla_decode(q, ckv2, [Smax], Dc=Dc, scale=0.4, lib=lib)
    d = orc.mla_decode(q, ckv, [Smax], Dc=Dc, scale=0.4, lib=lib)
    assert np.abs(c[1] - d[1]).max() > 1e-6


ALL_PINS = [pin_golden, pin_brute_force, pin_rows_sum_to_one, pin_probs_brute_force,
            pin_probs_times_values, pin_equal_value_rows,
            pin_causal_row0, pin_single_key, pin_scale_zero, pin_gqa_equals_repeated_mha,
            pin_decode_equals_last_prefill_row, pin_split_combine, pin_row_subset,
            pin_paged_equals_gathered, pin_paged_table_clamp_and_unused_pages,
            pin_varlen_equals_each_sequence, pin_varlen_gaps_and_clamped_offsets,
            pin_ragged_paged_equals_gathered_varlen, pin_ragged_paged_decode_tokens,
            pin_bwd_finite_differences, pin_bwd_gqa_sums_repeated_heads,
            pin_mla_brute_force, pin_mla_equals_padded_decode, pin_mla_single_key_and_rope]
