"""Pins for amax recording and the delayed scale update: exact rationals,
hand-computed rollover sequences, and a window computed by slicing."""
import math
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle import fp8, scaling

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _parse(v):
    return float(v) if v in ("nan", "inf", "-inf") else float.fromhex(v)


def exponent_by_definition(a: float, fmt, margin: int) -> int:
    """Largest integer e with a * 2^e <= fmax, found by stepping over exact rationals."""
    fa, fm = Fraction(a), Fraction(fmt.fmax)
    e = 0
    while fa * Fraction(2) ** e > fm:
        e -= 1
    while fa * Fraction(2) ** (e + 1) <= fm:
        e += 1
    return max(-126, min(126, e - margin))


def edge_values():
    out = []
    for E in range(-40, 40):
        base = 1.75 * 2.0 ** E
        f = np.float32(base)
        out += [float(f), float(np.nextafter(f, np.float32(np.inf))), float(np.nextafter(f, np.float32(0))),
                2.0 ** E, float(np.nextafter(np.float32(2.0 ** E), np.float32(0)))]
    return out


@pytest.mark.parametrize("fmt", [fp8.E4M3, fp8.E5M2], ids=lambda f: f.name)
@pytest.mark.parametrize("margin", [0, 1, 3])
def test_scale_exponent_exact(fmt, margin):
    rng = np.random.default_rng(11)
    rand = (rng.random(400) * np.exp2(rng.integers(-60, 60, 400))).astype(np.float32)
    for a in edge_values() + [float(x) for x in rand if x > 0]:
        assert scaling.scale_exponent(a, fmt, margin) == exponent_by_definition(a, fmt, margin), (a, margin)


def test_scale_exponent_degenerate():
    for a in (0.0, math.inf, math.nan, -0.0):
        assert scaling.scale_exponent(a, fp8.E4M3, 0) is None


def test_rollover_golden():
    n = 0
    with open(os.path.join(GOLDEN, "scale_rollover.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            head, amaxes, scales = [p.strip() for p in line.split("|")]
            name, H, margin = head.split()
            s = scaling.DelayedScaler(name, int(H), int(margin))
            for a, want in zip(amaxes.split(","), scales.split(",")):
                s.record(_parse(a))
                s.update()
                assert s.scale == _parse(want), (line, a, s.scale)
                assert s.scale * s.scale_inv == 1.0
            n += 1
    assert n >= 5


@pytest.mark.parametrize("H", [1, 2, 4, 16])
def test_update_uses_last_H_amaxes(H):
    """The scale after the k-th record is the scale of the max over the last H
    records, or the previous scale when that max is 0 (window by slicing)."""
    rng = np.random.default_rng(H)
    seq = [float(np.float32(x)) for x in rng.random(50) * np.exp2(rng.integers(-8, 8, 50))]
    seq[10:14] = [0.0] * 4
    s = scaling.DelayedScaler("E4M3", H, 0)
    expect = 1.0
    for k, a in enumerate(seq):
        s.record(a)
        s.update()
        w = max(seq[max(0, k - H + 1):k + 1])
        if w > 0:
            expect = 2.0 ** exponent_by_definition(w, fp8.E4M3, 0)
        assert s.scale == expect


def test_record_keeps_running_max_and_propagates_nan():
    s = scaling.DelayedScaler("E4M3", 4, 0)
    s.record(2.0)
    s.record(1.0)
    assert s.hist[0] == 2.0
    s.record(float("nan"))
    s.record(5.0)
    assert math.isnan(s.hist[0])


def test_amax():
    assert scaling.amax(np.array([[-3.0, 2.0], [1.0, 0.5]], dtype=np.float32)) == 3.0
    assert scaling.amax(np.zeros((0, 4), dtype=np.float32)) == 0.0
    assert math.isnan(scaling.amax(np.array([1.0, np.nan, 7.0], dtype=np.float32)))
    assert scaling.amax(np.array([-np.inf, 1.0], dtype=np.float32)) == math.inf
