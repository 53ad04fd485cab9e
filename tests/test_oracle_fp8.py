"""Pins for the oracle's FP8 codec: brute force over all codes, a library cast,
and hand-derived values.  None of these re-types the encoder's formula."""
import math
import os
from fractions import Fraction

import numpy as np
import pytest
import torch

from oracle import fp8

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
FMTS = [fp8.E4M3, fp8.E5M2]
TORCH_DT = {"E4M3": torch.float8_e4m3fn, "E5M2": torch.float8_e5m2}


def _parse(v):
    return float(v) if v in ("nan", "inf", "-inf") else float.fromhex(v)


def brute_force_encode(v: float, fmt) -> int:
    """Nearest code by exhaustive search: among the finite codes with the sign of v,
    the one whose value is nearest |v|, ties to the even code, clamped to fmax."""
    if math.isnan(v):
        return 0x7F | (0x80 if math.copysign(1.0, v) < 0 else 0)
    sign = 0x80 if math.copysign(1.0, v) < 0 else 0
    a = Fraction(min(abs(v), fmt.fmax))      # saturate, then search exactly
    vals = fp8.decode(np.arange(128), fmt)   # non-negative codes
    best, best_d = None, None
    for c in range(128):
        x = float(vals[c])
        if not math.isfinite(x):
            continue
        d = abs(a - Fraction(x))
        if best is None or d < best_d or (d == best_d and (c & 1) == 0 and (best & 1) == 1):
            best, best_d = c, d
    return best | sign


def probe_values(fmt):
    """Every code value, every midpoint between neighbours, +-1 float32 ulp around
    each midpoint, edges around fmax, tiny values, zeros, infinities and NaN."""
    vals = fp8.decode(np.arange(128), fmt)
    fin = np.sort(vals[np.isfinite(vals)])
    mids = (fin[1:] + fin[:-1]) / 2
    mids32 = mids.astype(np.float32)
    up = np.nextafter(mids32, np.float32(np.inf))
    dn = np.nextafter(mids32, np.float32(0))
    extra = np.array([fmt.fmax, fmt.fmax * (1 + 2.0 ** -(fmt.mbits + 1)), fmt.fmax * 1.01, fmt.fmax * 2, 1e30,
                      np.inf, 0.0, 2.0 ** (fmt.emin - fmt.mbits - 1), 2.0 ** (fmt.emin - fmt.mbits - 2),
                      1e-30, 1e-45], dtype=np.float64)
    pos = np.concatenate([fin, mids, mids32, up, dn, extra]).astype(np.float32).astype(np.float64)
    return np.concatenate([pos, -pos, [np.nan, -np.nan, -0.0]])


@pytest.mark.parametrize("fmt", FMTS, ids=lambda f: f.name)
def test_decode_all_codes_match_torch(fmt):
    codes = torch.arange(256, dtype=torch.int32).to(torch.uint8)
    ref = codes.view(TORCH_DT[fmt.name]).to(torch.float64).numpy()
    got = fp8.decode(np.arange(256), fmt)
    np.testing.assert_array_equal(np.isnan(got), np.isnan(ref))
    ok = ~np.isnan(ref)
    np.testing.assert_array_equal(got[ok], ref[ok])
    np.testing.assert_array_equal(np.signbit(got[ok]), np.signbit(ref[ok]))


def test_decode_hand_values():
    assert fp8.decode(0x7E, fp8.E4M3) == 448.0
    assert math.isnan(fp8.decode(0x7F, fp8.E4M3)) and math.isnan(fp8.decode(0xFF, fp8.E4M3))
    assert fp8.decode(0x01, fp8.E4M3) == 2.0 ** -9
    assert fp8.decode(0x08, fp8.E4M3) == 2.0 ** -6
    assert fp8.decode(0x7B, fp8.E5M2) == 57344.0
    assert fp8.decode(0x7C, fp8.E5M2) == math.inf and fp8.decode(0xFC, fp8.E5M2) == -math.inf
    assert math.isnan(fp8.decode(0x7D, fp8.E5M2))
    assert fp8.decode(0x01, fp8.E5M2) == 2.0 ** -16


@pytest.mark.parametrize("fmt", FMTS, ids=lambda f: f.name)
def test_encode_equals_brute_force(fmt):
    vals = probe_values(fmt)
    got = fp8.encode(vals, fmt)
    for v, g in zip(vals, got):
        assert int(g) == brute_force_encode(float(v), fmt), (fmt.name, float(v).hex(), hex(int(g)))


@pytest.mark.parametrize("fmt", FMTS, ids=lambda f: f.name)
def test_encode_random_equals_brute_force(fmt):
    rng = np.random.default_rng(7)
    e = rng.integers(fmt.emin - fmt.mbits - 3, fmt.emax + 2, size=600)
    vals = (rng.random(600) + 1.0) * np.exp2(e.astype(np.float64)) * np.where(rng.random(600) < 0.5, -1, 1)
    vals = vals.astype(np.float32).astype(np.float64)
    got = fp8.encode(vals, fmt)
    for v, g in zip(vals, got):
        assert int(g) == brute_force_encode(float(v), fmt)


@pytest.mark.parametrize("fmt", FMTS, ids=lambda f: f.name)
def test_encode_matches_torch_cast_after_clamp(fmt):
    """torch's float8 casts round to nearest even but do not saturate, so clamp first."""
    rng = np.random.default_rng(3)
    x = (rng.standard_normal(20000) * np.exp2(rng.integers(-20, 18, 20000))).astype(np.float32)
    x = np.concatenate([x, probe_values(fmt).astype(np.float32)])
    x = x[np.isfinite(x)]
    clamped = np.clip(x, -fmt.fmax, fmt.fmax)
    ref = torch.from_numpy(clamped).to(TORCH_DT[fmt.name]).view(torch.uint8).numpy()
    got = fp8.encode(x.astype(np.float64), fmt)
    np.testing.assert_array_equal(got, ref)


def test_encode_hand_fixture():
    n = 0
    with open(os.path.join(GOLDEN, "fp8_encode_hand.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            name, val, code = line.split()[:3]
            got = int(fp8.encode(np.array([_parse(val)]), name)[0])
            assert got == int(code, 16), (name, val, hex(got), code)
            n += 1
    assert n >= 25


@pytest.mark.parametrize("fmt", FMTS, ids=lambda f: f.name)
def test_roundtrip_every_finite_code(fmt):
    vals = fp8.decode(np.arange(256), fmt)
    ok = np.isfinite(vals)
    back = fp8.encode(vals[ok], fmt)
    np.testing.assert_array_equal(back, np.arange(256)[ok].astype(np.uint8))
