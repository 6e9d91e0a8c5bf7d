"""Exact brute force for tiny cases (pure Python, ``fractions.Fraction``).

TEST INFRASTRUCTURE ONLY (see ``grinqh_oracle``).  This file is a second,
independent route to the same numbers, used to pin the numpy oracle:

* the b-bit nested code is found by taking the first b characters of the
  b_max-character binary string of the code (Sec. 3.3: the b most
  significant bits), not by shifting;
* the reconstruction point is found from the *bin* of b_max-bit codes that
  share that prefix: its lowest member (what truncation, a floor, lands on)
  plus half the bin's width (Sec. 3.3: phi moves the value from the lower
  bound of the bin to its centre; at full depth the bin has one member and is
  used as is, reading R1), and the offset is the middle code 2^(b_max-1);
* ranks for the top-p assignment are counted pairwise, O(K^2);
* RTN is done with exact rational arithmetic and explicit half-even rounding,
  with the fp16/fp32 roundings of the scale done by Python's float machinery.
"""
from __future__ import annotations

import struct
from fractions import Fraction


def code_bits(q: int, b_max: int = 8) -> str:
    return format(int(q), f"0{b_max}b")


def bin_of_prefix(prefix: str, b_max: int = 8):
    """All b_max-bit codes whose binary string starts with ``prefix``."""
    return [c for c in range(2 ** b_max) if code_bits(c, b_max).startswith(prefix)]


def reconstruction_point(q: int, b: int, b_max: int = 8) -> Fraction:
    """Code-space value (before scale/offset) that a b-bit read reconstructs."""
    if b == 0:
        raise ValueError("level 0 is skipped")
    members = bin_of_prefix(code_bits(q, b_max)[:b], b_max)
    lo = min(members)
    if len(members) == 1:
        return Fraction(lo)
    return Fraction(lo) + Fraction(len(members), 2)


def w_hat(q: int, s: Fraction, b: int, b_max: int = 8) -> Fraction:
    """Weight value reconstructed from a b-bit read (0 when skipped)."""
    if b == 0:
        return Fraction(0)
    return s * (reconstruction_point(q, b, b_max) - 2 ** (b_max - 1))


def vmm_exact(codes, scales, x, levels, level_bits, group):
    """y[n] = sum_k x_k * w_hat[n, k] exactly, codes [N][K] ints,
    scales [K//group][N] Fractions, x [K] Fractions, levels [K] ints; the
    top level's width is b_max."""
    b_max = level_bits[-1]
    N = len(codes)
    K = len(codes[0])
    y = []
    for n in range(N):
        acc = Fraction(0)
        for k in range(K):
            b = level_bits[levels[k]]
            if b == 0:
                continue
            acc += x[k] * w_hat(codes[n][k], scales[k // group][n], b, b_max)
        y.append(acc)
    return y


def topk_levels_pairwise(keys, counts):
    """Level per channel from explicit ranks: rank_i = #{j: key_j > key_i}
    + #{j < i: key_j == key_i}; the top counts[n] ranks get level n, etc."""
    K = len(keys)
    n = len(counts) - 1
    cum_top = []                      # number of channels at level >= j
    for j in range(n + 1):
        cum_top.append(sum(counts[j:]))
    out = []
    for i in range(K):
        rank = sum(1 for j in range(K) if keys[j] > keys[i])
        rank += sum(1 for j in range(i) if keys[j] == keys[i])
        lvl = 0
        for j in range(n + 1):
            if rank < cum_top[j]:
                lvl = j
        out.append(lvl)
    return out


def _round_f32(v: float) -> float:
    return struct.unpack("<f", struct.pack("<f", v))[0]


def _round_f16(v: float) -> float:
    return struct.unpack("<e", struct.pack("<e", v))[0]


def round_half_even(r: Fraction) -> int:
    fl = r.numerator // r.denominator
    rem = r - fl
    if rem > Fraction(1, 2):
        return fl + 1
    if rem < Fraction(1, 2):
        return fl
    return fl if fl % 2 == 0 else fl + 1


def rtn_group_exact(ws, b_max: int = 8):
    """RTN of one group of fp16 weights (Python floats holding fp16 values).

    Returns (codes list, scale as float).  The scale follows reading R4:
    fp32 division by 2^(b_max-1) - 1 (127 at 8 bits), then rounding to fp16;
    the code is the half-even rounding of the fp32 quotient w/s, clamped to
    [-2^(b_max-1), 2^(b_max-1) - 1], plus 2^(b_max-1).
    """
    half = 2 ** (b_max - 1)
    amax = max(abs(w) for w in ws)
    s = _round_f16(_round_f32(amax / float(half - 1))) if amax != 0.0 else 0.0
    # amax / 127 in fp32: Python divides in double; the double quotient of two
    # fp32 values rounded to fp32 equals the fp32 IEEE quotient (the double has
    # more than 2*24+2 bits), so this is the correctly rounded fp32 result.
    codes = []
    for w in ws:
        if s == 0.0:
            codes.append(half)
            continue
        quot = _round_f32(w / s)      # same double-rounding argument as above
        r = round_half_even(Fraction(quot))
        r = max(-half, min(half - 1, r))
        codes.append(r + half)
    return codes, s
