"""FP8 encode / decode, written from the format definitions.

The paper trains in FP8 without naming the encodings (§2.1 "Temporal Latency
and Hidden State in Delayed Scaling", which cites Micikevicius et al., "FP8
Formats for Deep Learning").  That cited work defines the two formats used
here, as later standardised by OCP:

* E4M3: 1 sign, 4 exponent (bias 7), 3 mantissa bits.  No infinities; the
  single pattern S.1111.111 is NaN, so the largest finite value is
  1.75 * 2^8 = 448.  Subnormals are 2^-6 * f/8.
* E5M2: 1 sign, 5 exponent (bias 15), 2 mantissa bits, IEEE-like: exponent 31
  with f = 0 is infinity, f != 0 is NaN.  Largest finite value
  1.75 * 2^15 = 57344.  Subnormals are 2^-14 * f/4.

Encoding rule (the paper is silent; this is the saturating
round-to-nearest-even reading):
  NaN            -> 0x7F with the input's sign bit
  |v| >= fmax    -> +-fmax (this includes +-inf)
  otherwise      -> nearest representable magnitude, ties to even mantissa,
                    then the input's sign bit (so a negative value that rounds
                    to zero gives 0x80).

Everything is evaluated in float64, where every step below is exact for
float32 / bfloat16 inputs.
"""
from __future__ import annotations

import dataclasses

import numpy as np


@dataclasses.dataclass(frozen=True)
class FP8Format:
    name: str
    mbits: int        # mantissa bits
    bias: int
    emin: int         # exponent of the smallest normal
    emax: int         # exponent of the largest finite value
    fmax: float       # largest finite magnitude
    fmax_code: int    # its code (positive)
    has_inf: bool


E4M3 = FP8Format("E4M3", mbits=3, bias=7, emin=-6, emax=8, fmax=448.0, fmax_code=0x7E, has_inf=False)
E5M2 = FP8Format("E5M2", mbits=2, bias=15, emin=-14, emax=15, fmax=57344.0, fmax_code=0x7B, has_inf=True)
FORMATS = {"E4M3": E4M3, "E5M2": E5M2}


def fmt_of(f) -> FP8Format:
    return f if isinstance(f, FP8Format) else FORMATS[f]


def decode(codes, fmt) -> np.ndarray:
    """FP8 code -> float64 value (NaN codes give NaN, E5M2 inf codes give +-inf)."""
    fmt = fmt_of(fmt)
    c = np.asarray(codes).astype(np.int64)
    sign = (c >> 7) & 1
    ebits = 7 - fmt.mbits
    e = (c >> fmt.mbits) & ((1 << ebits) - 1)
    f = c & ((1 << fmt.mbits) - 1)
    sub = np.ldexp(f.astype(np.float64), fmt.emin - fmt.mbits)
    nrm = np.ldexp((f + (1 << fmt.mbits)).astype(np.float64), e - fmt.bias - fmt.mbits)
    val = np.where(e == 0, sub, nrm)
    top = (1 << ebits) - 1
    if fmt.has_inf:
        val = np.where((e == top) & (f == 0), np.inf, val)
        val = np.where((e == top) & (f != 0), np.nan, val)
    else:
        val = np.where((e == top) & (f == (1 << fmt.mbits) - 1), np.nan, val)
    return np.where(sign == 1, -val, val)


def encode(values, fmt) -> np.ndarray:
    """float -> FP8 code (uint8), saturating round-to-nearest-even."""
    fmt = fmt_of(fmt)
    v = np.asarray(values, dtype=np.float64)
    sign = np.signbit(v).astype(np.int64)
    nan = np.isnan(v)
    a = np.where(nan, 0.0, np.abs(v))
    sat = a >= fmt.fmax
    a = np.where(sat, 0.0, a)
    # a = m * 2^E with m in [1, 2); zero belongs to the subnormal range.
    _, e2 = np.frexp(a)
    E = np.where(a == 0.0, fmt.emin, e2.astype(np.int64) - 1)
    Eq = np.maximum(E, fmt.emin)
    # quantum of the binade (or of the subnormal range), then an integer count
    n = np.rint(np.ldexp(a, (fmt.mbits - Eq).astype(np.int64))).astype(np.int64)
    # ((Eq - emin) << mbits) + n covers subnormals (Eq = emin, n < 2^mbits),
    # normals (n in [2^mbits, 2^(mbits+1))) and the carry into the next binade.
    mag = ((Eq - fmt.emin) << fmt.mbits) + n
    code = np.where(nan, 0x7F, np.where(sat, fmt.fmax_code, mag))
    return (code | (sign << 7)).astype(np.uint8)
