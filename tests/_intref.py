"""Independent scalar references used to pin the oracle (test helper, not the oracle).

Everything here works on exact integers: a finite float32 value v is decomposed as
|v| = M * 2**p with M a non-negative integer, and every comparison the formats need is a
comparison of two such numbers, done with Python's arbitrary-precision integers.  The
rounding rules are written as threshold counts (one comparison per midpoint, strict or not
according to which neighbour is the even code), a different method from the oracle's
nearest-grid search, so that a mistake in either shows up as a disagreement.
"""
from __future__ import annotations

import struct

import numpy as np


def decompose_f32(u: int):
    """float32 bit pattern -> (sign, M, p) with |v| = M * 2**p (finite values only)."""
    sign = (u >> 31) & 1
    ef = (u >> 23) & 0xFF
    frac = u & 0x7FFFFF
    if ef == 0xFF:
        raise ValueError("NaN/Inf are outside the contract")
    if ef == 0:
        return sign, frac, -149
    return sign, frac | 0x800000, ef - 150


def f32_bits(x: float) -> int:
    return struct.unpack("<I", struct.pack("<f", x))[0]


def cmp(m1: int, p1: int, m2: int, p2: int) -> int:
    """Sign of m1*2**p1 - m2*2**p2 (exact)."""
    q = min(p1, p2)
    a = m1 << (p1 - q)
    b = m2 << (p2 - q)
    return (a > b) - (a < b)


def floor_log2(m: int, p: int) -> int:
    return p + m.bit_length() - 1


# ----------------------------------------------------------------------------------------
# MXFP4 (OCP MX conversion rule)
# ----------------------------------------------------------------------------------------
# E2M1 midpoints times 4: 0.25 0.75 1.25 1.75 2.5 3.5 5 ; tie goes up when the upper code is
# even (codes 2, 4, 6 sit above the midpoints 0.75, 1.75, 3.5)
_MX_MID4 = [(1, False), (3, True), (5, False), (7, True), (10, False), (14, True), (20, False)]


def mx_block_ref(bits):
    """MXFP4 codes and E8M0 byte of one block given as float32 bit patterns."""
    dec = [decompose_f32(int(u)) for u in bits]
    amax = (0, 0)
    for _, m, p in dec:
        if m and (amax[0] == 0 or cmp(m, p, *amax) > 0):
            amax = (m, p)
    if amax[0] == 0:
        e = -127
    else:
        e = max(-127, min(127, floor_log2(*amax) - 2))
    codes = []
    for s, m, p in dec:
        k = 0
        if m == 0:
            codes.append(s << 3)
            continue
        for t4, inclusive in _MX_MID4:
            c = cmp(4 * m, p - e, t4, 0)  # compare 4*|v|/2**e with t4
            k += (c >= 0) if inclusive else (c > 0)
        codes.append((s << 3) | k)
    return codes, e + 127


# ----------------------------------------------------------------------------------------
# HiF4 (readings H1-H6)
# ----------------------------------------------------------------------------------------
def _s1_175(c: int):
    """1.75 * E6M2(c) as (M, p): 7 * (4 + m) * 2**(e - 31 - 4)."""
    return 7 * (4 + (c & 3)), (c >> 2) - 31 - 4


def hif4_block_ref(bits):
    """HiF4 codes and metadata word of one 64-element block of float32 bit patterns."""
    assert len(bits) == 64
    dec = [decompose_f32(int(u)) for u in bits]

    def amax(idx):
        best = (0, 0)
        for i in idx:
            _, m, p = dec[i]
            if m and (best[0] == 0 or cmp(m, p, *best) > 0):
                best = (m, p)
        return best

    a = amax(range(64))
    # level 1: binary search for the smallest code with 1.75*s1 >= A (all codes if A == 0)
    lo, hi = 0, 255
    if a[0] != 0 and cmp(*_s1_175(255), *a) < 0:
        c1 = 255
    else:
        while lo < hi:
            mid = (lo + hi) // 2
            if a[0] == 0 or cmp(*_s1_175(mid), *a) >= 0:
                hi = mid
            else:
                lo = mid + 1
        c1 = lo
    ms, ps = _s1_175(c1)  # 1.75 * s1
    meta = c1
    codes = [0] * 64
    for g in range(8):
        ag = amax(range(8 * g, 8 * g + 8))
        b2 = 1 if (ag[0] == 0 or cmp(*ag, ms, ps - 1) <= 0) else 0
        meta |= b2 << (8 + g)
        for half in range(2):
            h = 2 * g + half
            ah = amax(range(4 * h, 4 * h + 4))
            b3 = 1 if (ah[0] == 0 or cmp(*ah, ms, ps - 1 - b2) <= 0) else 0
            meta |= b3 << (16 + h)
            b = b2 + b3
            # s = (4+m) * 2**(e-31-2-b); midpoint (2k'+1)*s/8 = (2k'+1)(4+m) 2**(e-31-5-b)
            mm = 4 + (c1 & 3)
            pe = (c1 >> 2) - 31 - 5 - b
            for i in range(4 * h, 4 * h + 4):
                s, m, p = dec[i]
                k = 0
                for kp in range(7 if m else 0):
                    c = cmp(m, p, (2 * kp + 1) * mm, pe)
                    k += (c > 0) if kp % 2 == 0 else (c >= 0)
                codes[i] = (s << 3) | k
    return codes, meta


def finite_bf16_as_f32_bits() -> np.ndarray:
    """All finite bfloat16 values, as float32 bit patterns (65024 of them)."""
    b = np.arange(1 << 16, dtype=np.uint32)
    b = b[((b >> 7) & 0xFF) != 0xFF]
    return b << 16
