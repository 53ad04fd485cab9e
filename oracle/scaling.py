"""Per-tensor amax recording and the delayed scale update.

§2.1 of the paper: delayed scaling derives its scaling factors from moving
amax histories instead of inspecting each operand as it is quantized; an
invocation reads the persistent state, quantizes and multiplies, and records
statistics that later microbatches use.  §3.2 fixes *when* the state moves:
F turns S0 into S1, dI turns S1 into S2 (quantizing dY once), dW never touches
it.  The paper prints neither the history algorithm nor the scale formula;
the readings taken here are:

* amax is max |x| over the whole unscaled tensor; NaN propagates.
* Recording keeps the running maximum in history slot 0.
* An update takes a = max over the whole history (slot 0 included).  If a is
  finite and positive, the new exponent is e = floor(log2(fmax / a)) - margin,
  clamped to [-126, 126] so that both 2^e and 2^-e are normal float32;
  scale = 2^e and scale_inv = 2^-e.  Otherwise the scale is kept.
* Then the history rotates one place towards slot 0 (slot 0's value moves to
  the last slot) and slot 0 is cleared, so the update after the k-th record
  sees the last H recorded amaxes.
* Initial state: history all zero, scale = scale_inv = 1.

Current (dynamic) scaling, which §2.1 names beside delayed scaling as a
target and which §4.2 allows at the last stage's output boundary, inspects
the operand itself: its scale comes from the amax of the tensor about to be
cast.
The paper prints no formula for it either; the reading taken here keeps the
delayed rule's exponent and its degenerate case, applied to that one amax:
e = floor(log2(fmax / max|x|)) - margin (clamped as above), and a tensor whose
amax is 0, inf or NaN keeps the role's previous scale.  No history is kept.
"""
from __future__ import annotations

import math

import numpy as np

from .fp8 import fmt_of

EXP_LO, EXP_HI = -126, 126


def amax(x) -> float:
    """max |x| over the tensor as float64 (exact for float32 / bf16 data); 0 for an empty tensor."""
    x = np.asarray(x, dtype=np.float64)
    if x.size == 0:
        return 0.0
    return float(np.max(np.abs(x)))


def scale_exponent(a: float, fmt, margin: int):
    """floor(log2(fmax / a)) - margin, clamped; None when a is 0, inf or NaN.

    Evaluated exactly: with a = m * 2^E (m in [1, 2)) and fmax = 1.75 * 2^Emax,
    a * 2^e <= fmax holds for e = Emax - E when m <= 1.75 and for one less when
    m > 1.75, so that is the floor."""
    fmt = fmt_of(fmt)
    if not (math.isfinite(a) and a > 0.0):
        return None
    m, e2 = math.frexp(a)          # a = m * 2^e2, m in [0.5, 1)
    m, E = 2.0 * m, e2 - 1          # a = m * 2^E,  m in [1, 2)
    e0 = fmt.emax - E - (1 if m > 1.75 else 0)
    return max(EXP_LO, min(EXP_HI, e0 - margin))


class DelayedScaler:
    """Amax history + scale of one tensor role of one layer."""

    def __init__(self, fmt, history_len: int, margin: int):
        if history_len < 1:
            raise ValueError("history_len must be >= 1")
        self.fmt = fmt_of(fmt)
        self.margin = int(margin)
        self.hist = np.zeros(history_len, dtype=np.float64)
        self.scale = 1.0
        self.scale_inv = 1.0

    def record(self, a: float) -> None:
        h0 = self.hist[0]
        self.hist[0] = a if (math.isnan(a) or a > h0) else h0

    def update(self) -> None:
        a = float(np.max(self.hist))          # NaN propagates
        e = scale_exponent(a, self.fmt, self.margin)
        if e is not None:
            self.scale = math.ldexp(1.0, e)
            self.scale_inv = math.ldexp(1.0, -e)
        self.hist = np.roll(self.hist, -1)
        self.hist[0] = 0.0

    def copy(self) -> "DelayedScaler":
        s = DelayedScaler(self.fmt, len(self.hist), self.margin)
        s.hist = self.hist.copy()
        s.scale, s.scale_inv = self.scale, self.scale_inv
        return s


class CurrentScaler:
    """Scale of one tensor role under current (dynamic) scaling: no history;
    the scale is set from the amax of the tensor it is about to cast."""

    def __init__(self, fmt, margin: int):
        self.fmt = fmt_of(fmt)
        self.margin = int(margin)
        self.scale = 1.0
        self.scale_inv = 1.0

    def set_from(self, x) -> None:
        e = scale_exponent(amax(x), self.fmt, self.margin)
        if e is not None:
            self.scale = math.ldexp(1.0, e)
            self.scale_inv = math.ldexp(1.0, -e)
