"""Brute-force attention in pure Python, for tiny inputs only.

TEST INFRASTRUCTURE ONLY.  An independent second route to the same result
as ``oracle_attn.c``, used to pin it: it materialises the whole masked
score matrix with -inf entries, exponentiates WITHOUT subtracting the row
maximum, and sums with ``math.fsum``.  Nothing here is shared with the C
oracle or with the HIP library (its own bf16 decoding, its own mask
construction from the definition of causal and length masking).

Keep the inputs small and of moderate magnitude (|s| well below 700) so
that exp() without max-subtraction cannot overflow.
"""
from __future__ import annotations

import math
import struct


def bf16_bits_to_float(bits: int) -> float:
    return struct.unpack("<f", struct.pack("<I", (int(bits) & 0xFFFF) << 16))[0]


def _mask(Sq: int, Skv: int, L: int, causal: bool):
    """allowed[i][j]: key j is inside the sequence (j < L) and, under the
    causal rule with queries sitting at the last Sq positions of the
    length-L sequence, not in the future of query i."""
    allowed = [[False] * Skv for _ in range(Sq)]
    for i in range(Sq):
        pos_i = (L - Sq) + i  # absolute position of query i
        for j in range(Skv):
            ok = j < L
            if causal:
                ok = ok and j <= pos_i
            allowed[i][j] = ok
    return allowed


def attention(q, k, v, *, causal: bool, scale: float, kv_seqlens=None):
    """q: nested lists [B][Hq][Sq][D] of bf16 bit patterns; k, v: [B][Hkv][Skv][D].

    Returns (o [B][Hq][Sq][D], lse [B][Hq][Sq]) as Python floats.
    """
    dec = lambda t: [[[[bf16_bits_to_float(x) for x in row] for row in h] for h in bb] for bb in t]
    return attention_f(dec(q), dec(k), dec(v), causal=causal, scale=scale,
                       kv_seqlens=kv_seqlens)


def attention_f(q, k, v, *, causal: bool, scale: float, kv_seqlens=None):
    """The same on nested lists of Python floats (for finite differences)."""
    B, Hq, Sq, D = len(q), len(q[0]), len(q[0][0]), len(q[0][0][0])
    Hkv, Skv = len(k[0]), len(k[0][0])
    G = Hq // Hkv
    o = [[[[0.0] * D for _ in range(Sq)] for _ in range(Hq)] for _ in range(B)]
    lse = [[[0.0] * Sq for _ in range(Hq)] for _ in range(B)]
    for b in range(B):
        L = Skv if kv_seqlens is None else max(0, min(Skv, int(kv_seqlens[b])))
        allowed = _mask(Sq, Skv, L, causal)
        for hq in range(Hq):
            kh = hq // G
            Kf = k[b][kh]
            Vf = v[b][kh]
            for i in range(Sq):
                qi = q[b][hq][i]
                scores = []
                for j in range(Skv):
                    if allowed[i][j]:
                        scores.append(scale * math.fsum(qi[d] * Kf[j][d] for d in range(D)))
                    else:
                        scores.append(-math.inf)
                e = [math.exp(s) for s in scores]  # exp(-inf) = 0
                z = math.fsum(e)
                if z == 0.0:
                    o[b][hq][i] = [0.0] * D
                    lse[b][hq][i] = -math.inf
                    continue
                o[b][hq][i] = [math.fsum(e[j] * Vf[j][d] for j in range(Skv)) / z
                               for d in range(D)]
                lse[b][hq][i] = math.log(z)
    return o, lse


def mla_decode(q, ckv, kv_seqlens, *, Dc: int, scale: float):
    """MLA decode by brute force.  q: nested lists [B][H][Dc+Dr] of bf16 bit
    patterns; ckv: [B][Smax][Dc+Dr].  Scores use every column of the cache
    row, outputs the first Dc columns.  Returns (o [B][H][Dc], lse [B][H])."""
    B, H = len(q), len(q[0])
    Smax = len(ckv[0])
    o = [[[0.0] * Dc for _ in range(H)] for _ in range(B)]
    lse = [[0.0] * H for _ in range(B)]
    for b in range(B):
        L = max(0, min(Smax, int(kv_seqlens[b])))
        rows = [[bf16_bits_to_float(x) for x in ckv[b][j]] for j in range(L)]
        for h in range(H):
            qv = [bf16_bits_to_float(x) for x in q[b][h]]
            if L == 0:
                lse[b][h] = -math.inf
                continue
            w = [math.exp(scale * math.fsum(a * c for a, c in zip(qv, row))) for row in rows]
            z = math.fsum(w)
            lse[b][h] = math.log(z)
            for e in range(Dc):
                o[b][h][e] = math.fsum(w[j] * rows[j][e] for j in range(L)) / z
    return o, lse


def probs(q, k, *, causal: bool, scale: float, kv_seqlens=None):
    """The normalised attention weights by brute force: the whole masked
    score matrix (-inf where a key is not admissible), exp without
    max-subtraction, each row divided by its fsum.  q: nested lists
    [B][Hq][Sq][D] of bf16 bit patterns; k: [B][Hkv][Skv][D].  Returns
    p [B][Hq][Sq][Skv] (rows without an admissible key are all zero)."""
    dec = lambda t: [[[[bf16_bits_to_float(x) for x in row] for row in h] for h in bb] for bb in t]
    qf, kf = dec(q), dec(k)
    B, Hq, Sq, D = len(qf), len(qf[0]), len(qf[0][0]), len(qf[0][0][0])
    Hkv, Skv = len(kf[0]), len(kf[0][0])
    G = Hq // Hkv
    out = [[[[0.0] * Skv for _ in range(Sq)] for _ in range(Hq)] for _ in range(B)]
    for b in range(B):
        L = Skv if kv_seqlens is None else max(0, min(Skv, int(kv_seqlens[b])))
        allowed = _mask(Sq, Skv, L, causal)
        for hq in range(Hq):
            Kh = kf[b][hq // G]
            for i in range(Sq):
                qi = qf[b][hq][i]
                e = [math.exp(scale * math.fsum(qi[d] * Kh[j][d] for d in range(D)))
                     if allowed[i][j] else 0.0 for j in range(Skv)]
                z = math.fsum(e)
                if z > 0.0:
                    out[b][hq][i] = [x / z for x in e]
    return out
