"""Micro-oracle for tiny inputs (test infrastructure only; see the package docstring).

Independent of ``oracle.predictor``: router logits (Eq. 4) are computed as exact rationals from the
stored bit patterns and rounded once, to nearest-even float32; selections are made with Python's
``sorted`` over (score descending, index ascending) tuples with explicit loops.  Used to pin the
float64-GEMM oracle on small shapes.
"""
from __future__ import annotations

import math
import struct
from fractions import Fraction
from typing import List, Optional, Sequence

import numpy as np


def bf16_bits_to_fraction(bits: int) -> Fraction:
    """Exact value of one bfloat16 bit pattern (finite values only)."""
    bits = int(bits) & 0xFFFF
    sign = -1 if bits >> 15 else 1
    exp = (bits >> 7) & 0xFF
    man = bits & 0x7F
    if exp == 0xFF:
        raise ValueError("non-finite bfloat16")
    if exp == 0:
        return sign * Fraction(man, 1 << (126 + 7))
    return sign * Fraction(man | 0x80, 1) * (Fraction(2) ** (exp - 127 - 7))


def f32_to_fraction(v: float) -> Fraction:
    v = float(np.float32(v))
    if not math.isfinite(v):
        raise ValueError("non-finite float32")
    return Fraction(*v.as_integer_ratio())


def fraction_to_f32(q: Fraction) -> np.float32:
    """Round an exact rational to the nearest binary32 value, ties to even (overflow -> inf)."""
    if q == 0:
        return np.float32(0.0)
    sign = -1.0 if q < 0 else 1.0
    q = abs(q)
    n, d = q.numerator, q.denominator
    e = n.bit_length() - d.bit_length()
    while Fraction(2) ** e > q:
        e -= 1
    while q >= Fraction(2) ** (e + 1):
        e += 1                                   # now 2^e <= q < 2^(e+1)
    e = max(e, -126)                             # subnormals share the minimum exponent
    scaled = q / (Fraction(2) ** (e - 23))       # 24-bit significand field (for normals)
    m = scaled.numerator // scaled.denominator
    rem = scaled - m
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and m % 2 == 1):
        m += 1
    if m >= (1 << 24):
        m >>= 1
        e += 1
    if e > 127:
        return np.float32(sign * math.inf)
    return np.float32(sign * math.ldexp(m, e - 23))


def exact_logits(x: np.ndarray, w: np.ndarray, dtype: str,
                 logit_bias: Optional[np.ndarray] = None) -> np.ndarray:
    """z[t, e] = round_f32( sum_h x[t,h] * w[e,h] + b[e] ), every operation exact before the one
    rounding.  ``x`` T x H and ``w`` E x H hold bf16 bits (uint16) or float32 values."""
    conv = bf16_bits_to_fraction if dtype == "bf16" else f32_to_fraction
    X = [[conv(v) for v in row] for row in np.asarray(x)]
    W = [[conv(v) for v in row] for row in np.asarray(w)]
    B = None if logit_bias is None else [f32_to_fraction(v) for v in logit_bias]
    T, E = len(X), len(W)
    out = np.empty((T, E), dtype=np.float32)
    for t in range(T):
        for e in range(E):
            acc = sum((a * b for a, b in zip(X[t], W[e])), Fraction(0))
            if B is not None:
                acc += B[e]
            out[t, e] = fraction_to_f32(acc)
    return out


def f32_round(v: float) -> float:
    """Round a Python float to float32 via the IEEE pack/unpack of the struct module."""
    return struct.unpack("<f", struct.pack("<f", v))[0]


def brute_scores(z_row: Sequence[float], kind: str, bias: Optional[Sequence[float]]) -> List[float]:
    if kind == "softmax":
        return [float(v) for v in z_row]
    out = []
    for e, v in enumerate(z_row):
        s = f32_round(1.0 / (1.0 + math.exp(-float(v))))
        if bias is not None:
            s = f32_round(s + float(np.float32(bias[e])))
        out.append(s)
    return out


def brute_select(z_row: Sequence[float], k: int, kind: str = "softmax",
                 bias: Optional[Sequence[float]] = None, n_group: int = 1, topk_group: int = 1,
                 group_topn: int = 1) -> List[int]:
    """Top-k (with optional group limit) of one token by explicit sorting."""
    if kind == "softmax" and n_group > 1 and group_topn > 1:
        raise ValueError("softmax routing takes group_topn 1 only")
    s = brute_scores(z_row, kind, bias)
    E = len(s)
    allowed = list(range(E))
    if n_group > 1:
        gsz = E // n_group
        gscore = []
        for g in range(n_group):
            vals = sorted((s[e] for e in range(g * gsz, (g + 1) * gsz)), reverse=True)
            acc = vals[0]
            for v in vals[1:group_topn]:
                acc = f32_round(acc + v)
            gscore.append(acc)
        kept = sorted(range(n_group), key=lambda g: (-gscore[g], g))[:topk_group]
        allowed = [e for e in range(E) if e // gsz in kept]
    return sorted(allowed, key=lambda e: (-s[e], e))[:k]
