"""Brute-force attention in pure Python -- TEST INFRASTRUCTURE ONLY.

The literal formula of exact softmax attention (paper Sec. 3.5: each GPU
attends over every token of the window for its heads), one query row
at a time, with math.exp and correctly rounded sums (math.fsum).  For tiny
inputs only; it pins the C oracle, it is not used to check the GPU.
"""
from __future__ import annotations

import math
import struct


def bf16_to_float(bits: int) -> float:
    return struct.unpack("<f", struct.pack("<I", (int(bits) & 0xFFFF) << 16))[0]


def attn_row(qrow, keys, values, scale: float):
    """qrow: list of D floats; keys/values: lists of Skv rows of D floats.
    Returns (o: list of D floats, lse: float)."""
    s = [scale * math.fsum(a * b for a, b in zip(qrow, krow)) for krow in keys]
    m = max(s)
    w = [math.exp(x - m) for x in s]
    l = math.fsum(w)
    D = len(values[0])
    o = [math.fsum(w[j] * values[j][t] for j in range(len(values))) / l for t in range(D)]
    return o, m + math.log(l)


def attn(q, k, v, scale: float):
    """q [B,Sq,H,D], k/v [B,Skv,H,D] as nested sequences (or numpy arrays) of bf16 bits.
    Returns (O as nested lists [B][Sq][H][D], LSE [B][H][Sq])."""
    B, Sq, H, D = len(q), len(q[0]), len(q[0][0]), len(q[0][0][0])
    Skv = len(k[0])
    O = [[[None] * H for _ in range(Sq)] for _ in range(B)]
    L = [[[0.0] * Sq for _ in range(H)] for _ in range(B)]
    for b in range(B):
        for h in range(H):
            keys = [[bf16_to_float(k[b][j][h][t]) for t in range(D)] for j in range(Skv)]
            vals = [[bf16_to_float(v[b][j][h][t]) for t in range(D)] for j in range(Skv)]
            for i in range(Sq):
                qrow = [bf16_to_float(q[b][i][h][t]) for t in range(D)]
                o, lse = attn_row(qrow, keys, vals, scale)
                O[b][i][h] = o
                L[b][h][i] = lse
    return O, L
