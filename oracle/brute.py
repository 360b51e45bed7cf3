"""Exact-rational brute force of the binary-delta matmul -- TEST INFRASTRUCTURE.

Pure-Python loops over ``fractions.Fraction`` for tiny inputs only.  bf16 and
fp32 values are dyadic rationals, so the real-number result of

    y[m][n] = sum_k x[m][k] W[n][k] + alpha[t] * sum_k x[m][k] (2 b[t][n][k] - 1)

(the BitDelta GEMM of Section 4.4, with the ``2b-1`` decode of Appendix A.2)
is computed with no rounding at all.  Shares nothing with ``oracle.c``: its own
bf16 decode, its own bit extraction, its own loops.
"""
from __future__ import annotations

import struct
from fractions import Fraction


def bf16_bits_to_fraction(h: int) -> Fraction:
    """Exact value of a bf16 bit pattern (finite values only)."""
    h &= 0xFFFF
    sign = -1 if (h >> 15) & 1 else 1
    exp = (h >> 7) & 0xFF
    man = h & 0x7F
    if exp == 0xFF:
        raise ValueError("non-finite bf16")
    if exp == 0:
        val = Fraction(man, 1 << 7) * Fraction(1, 1 << 126)
    else:
        val = (1 + Fraction(man, 1 << 7)) * (Fraction(2) ** (exp - 127))
    return sign * val


def f16_bits_to_fraction(h: int) -> Fraction:
    """Exact value of an IEEE binary16 bit pattern (finite values only)."""
    h &= 0xFFFF
    sign = -1 if (h >> 15) & 1 else 1
    exp = (h >> 10) & 0x1F
    man = h & 0x3FF
    if exp == 0x1F:
        raise ValueError("non-finite fp16")
    if exp == 0:
        val = Fraction(man, 1 << 10) * Fraction(1, 1 << 14)
    else:
        val = (1 + Fraction(man, 1 << 10)) * (Fraction(2) ** (exp - 15))
    return sign * val


def f32_to_fraction(v: float) -> Fraction:
    """Exact value of a float32 (the float is first rounded to fp32)."""
    (bits,) = struct.unpack("<I", struct.pack("<f", v))
    return Fraction(struct.unpack("<f", struct.pack("<I", bits))[0])


def sign_from_words(words, k: int) -> int:
    """+1 when bit (k % 32) of word (k // 32) is set, else -1."""
    return 1 if (int(words[k // 32]) >> (k % 32)) & 1 else -1


def matmul_exact(x_bits, w_bits, packed, alpha, tenant_ids=None, dtype="bf16"):
    """Exact y as a nested list of Fractions (None for out-of-range tenants).

    x_bits [M][K] and w_bits [N][K] are bf16 (or, with dtype="f16", IEEE
    binary16) bit patterns, packed is [T][N][K/32] of uint32 words, alpha a
    length-T sequence of fp32 values.
    """
    dec = f16_bits_to_fraction if dtype == "f16" else bf16_bits_to_fraction
    M = len(x_bits)
    K = len(x_bits[0]) if M else 0
    N = len(w_bits)
    T = len(packed)
    y = []
    for m in range(M):
        t = 0 if tenant_ids is None else int(tenant_ids[m])
        row = []
        for n in range(N):
            if not (0 <= t < T):
                row.append(None)
                continue
            a = f32_to_fraction(float(alpha[t]))
            acc = Fraction(0)
            for k in range(K):
                xv = dec(int(x_bits[m][k]))
                wv = dec(int(w_bits[n][k]))
                s = sign_from_words(packed[t][n], k)
                acc += xv * wv + a * xv * s
            row.append(acc)
        y.append(row)
    return y
