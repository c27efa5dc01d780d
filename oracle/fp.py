"""IEEE rounding emulation (oracle; test infrastructure only).

The paper computes in fp32 and simulates fp16 and bf16 by casting results of
single-precision operations to the lower precision (Section 3.2).  This module
supplies the roundings that the oracle's same-algorithm emulation applies:

* ``fraction_to_f32``: an exact rational rounded once to the nearest fp32,
  ties to even (used for the transform matrices);
* ``to_dtype``: fp32 values rounded to fp32 / fp16 / bf16, round to nearest
  even (fp16 through numpy's IEEE half conversion, bf16 by the bit-level
  rule on the fp32 encoding, NaN kept quiet with its sign).
"""
from fractions import Fraction

import numpy as np

DTYPES = ("f32", "f16", "bf16")

# unit roundoff (half an ulp at 1) of each storage type
UNIT_ROUNDOFF = {"f32": 2.0 ** -24, "f16": 2.0 ** -11, "bf16": 2.0 ** -8}


def fraction_to_f32(q):
    """Nearest fp32 to the rational q, ties to even; returned as a Python float."""
    q = Fraction(q)
    if q == 0:
        return 0.0
    sign = -1.0 if q < 0 else 1.0
    a = abs(q)
    num, den = a.numerator, a.denominator
    # e = floor(log2(a))
    e = num.bit_length() - den.bit_length()
    if Fraction(num, den) < Fraction(2) ** e:
        e -= 1
    if e > 127:
        return sign * float("inf")
    # quantum of the result: 2^(e-23) for normals, 2^-149 for subnormals
    qexp = max(e, -126) - 23
    # scaled = a / 2^qexp, split into integer part and remainder
    if qexp >= 0:
        sn, sd = num, den << qexp
    else:
        sn, sd = num << (-qexp), den
    mant, r = divmod(sn, sd)
    twice = 2 * r
    if twice > sd or (twice == sd and (mant & 1)):
        mant += 1
    val = Fraction(mant) * (Fraction(2) ** qexp)
    if val >= Fraction(2) ** 128:
        return sign * float("inf")
    return sign * float(val)


def f32(x):
    return np.asarray(x, dtype=np.float32)


def round_bf16(x):
    """fp32 -> bf16 -> fp32, round to nearest even, NaN preserved (quieted)."""
    a = np.ascontiguousarray(np.asarray(x, dtype=np.float32))
    u = a.view(np.uint32).astype(np.uint64)
    nan = np.isnan(a)
    lsb = (u >> 16) & 1
    r = ((u + 0x7FFF + lsb) >> 16) << 16
    r = np.where(nan, (u | 0x00400000) & 0xFFFF0000, r)
    return r.astype(np.uint32).view(np.float32).reshape(a.shape)


def round_f16(x):
    """fp32 -> fp16 -> fp32 (IEEE round to nearest even)."""
    return np.asarray(x, dtype=np.float32).astype(np.float16).astype(np.float32)


def to_dtype(x, dtype):
    """Round fp32 values to the storage dtype and return them as fp32."""
    x = np.asarray(x, dtype=np.float32)
    if dtype == "f32":
        return x.copy()
    if dtype == "f16":
        return round_f16(x)
    if dtype == "bf16":
        return round_bf16(x)
    raise ValueError(f"unknown dtype {dtype!r}")


def fma_f32(a, b, c):
    """a * b + c rounded once to fp32 (round to nearest even), elementwise.

    The transforms of the library accumulate each term with one fused
    multiply-add, so the emulation rounds a product and its sum together.
    The product of two fp32 values is exact in float64 (48 significant bits);
    the float64 sum s = p + c is then exact up to the error e that TwoSum
    recovers.  Rounding s to fp32 gives the correctly rounded p + c unless s
    lies exactly half-way between two fp32 numbers while e is not zero (a
    double rounding); then the exact sum p + c lies on e's side of that
    midpoint and rounds to the neighbour there.
    """
    a = np.asarray(a, dtype=np.float32)
    b = np.asarray(b, dtype=np.float32)
    c = np.asarray(c, dtype=np.float32)
    p = a.astype(np.float64) * b.astype(np.float64)
    c64 = c.astype(np.float64)
    s = p + c64
    bv = s - p
    e = (p - (s - bv)) + (c64 - bv)                  # TwoSum: p + c == s + e exactly
    with np.errstate(over="ignore", invalid="ignore"):
        r = s.astype(np.float32)
        r64 = r.astype(np.float64)
        other = np.nextafter(r, np.where(s > r64, np.float32(np.inf), np.float32(-np.inf)).astype(np.float32))
        mid = (r64 + other.astype(np.float64)) * 0.5
        tie = (s != r64) & (s == mid) & (e != 0)
        up = np.maximum(r, other)
        down = np.minimum(r, other)
        out = np.where(tie, np.where(e > 0, up, down), r)
    return out.astype(np.float32)
