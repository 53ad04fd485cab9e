"""Pins for quantize, the TN GEMM and affine placement: exact integer products,
exact rational sums, plain loops, and explicit index arithmetic."""
from fractions import Fraction

import numpy as np
import pytest

from oracle import fp8, gemm


def test_integer_codes_equal_exact_int64_matmul():
    """Integers |n| <= 16 are exact in E4M3 and |n| <= 8 in E5M2, so the product of
    their codes must equal an int64 matmul exactly, in every operand format pair."""
    rng = np.random.default_rng(0)
    for fa, fb, lim_a, lim_b in [("E4M3", "E4M3", 16, 16), ("E5M2", "E4M3", 8, 16), ("E5M2", "E5M2", 8, 8)]:
        a = rng.integers(-lim_a, lim_a + 1, size=(37, 129))
        b = rng.integers(-lim_b, lim_b + 1, size=(23, 129))
        ca = fp8.encode(a.astype(np.float64), fa)
        cb = fp8.encode(b.astype(np.float64), fb)
        got = gemm.gemm_tn(ca, fa, cb, fb, 1.0, 1.0)
        np.testing.assert_array_equal(got, (a @ b.T).astype(np.float64))
        got_s = gemm.gemm_tn(ca, fa, cb, fb, 2.0 ** -3, 2.0 ** 5)
        np.testing.assert_array_equal(got_s, (a @ b.T).astype(np.float64) * 4.0)


def test_gemm_equals_exact_rational_sum():
    rng = np.random.default_rng(1)
    ca = rng.integers(0, 256, size=(5, 33)).astype(np.uint8)
    cb = rng.integers(0, 256, size=(4, 33)).astype(np.uint8)
    ca[(ca & 0x7F) == 0x7F] = 0x10      # no NaN codes
    cb[((cb & 0x7C) == 0x7C)] = 0x11    # no E5M2 inf / NaN codes
    got = gemm.gemm_tn(ca, "E4M3", cb, "E5M2", 0.5, 0.25)
    va, vb = fp8.decode(ca, "E4M3"), fp8.decode(cb, "E5M2")
    for i in range(5):
        for j in range(4):
            exact = sum(Fraction(float(va[i, r])) * Fraction(float(vb[j, r])) for r in range(33)) / 8
            # float64 accumulation of <= 33 exact products: relative error <= 33 * 2^-53
            assert abs(Fraction(float(got[i, j])) - exact) <= Fraction(33, 2 ** 53) * sum(
                abs(Fraction(float(va[i, r])) * Fraction(float(vb[j, r]))) for r in range(33)) / 8


def test_gemm_equals_loops():
    rng = np.random.default_rng(2)
    x = (rng.standard_normal((6, 40)) * 3).astype(np.float32)
    w = (rng.standard_normal((5, 40)) * 0.02).astype(np.float32)
    cx, cw = gemm.quantize(x, 16.0, "E4M3"), gemm.quantize(w, 1024.0, "E4M3")
    np.testing.assert_allclose(gemm.gemm_tn(cx, "E4M3", cw, "E4M3", 1 / 16, 1 / 1024),
                               gemm.gemm_tn_loops(cx, "E4M3", cw, "E4M3", 1 / 16, 1 / 1024), rtol=1e-13, atol=0)


@pytest.mark.parametrize("fmt", ["E4M3", "E5M2"])
@pytest.mark.parametrize("e", [-7, 0, 5])
def test_quantize_inverts_decode(fmt, e):
    """Every finite code c satisfies quantize(decode(c) / 2^e, scale=2^e) == c."""
    codes = np.arange(256)
    vals = fp8.decode(codes, fmt)
    ok = np.isfinite(vals)
    x = (vals[ok] * 2.0 ** -e).astype(np.float32)
    np.testing.assert_array_equal(gemm.quantize(x, 2.0 ** e, fmt), codes[ok].astype(np.uint8))


def test_quantize_transpose_and_amax():
    rng = np.random.default_rng(4)
    x = rng.standard_normal((7, 19)).astype(np.float32)
    q, qt, a = gemm.quantize_with_amax(x, 8.0, "E4M3")
    np.testing.assert_array_equal(qt, q.T)
    assert a == float(np.max(np.abs(x)))


def test_place_init_accum_and_untouched():
    n, k, ld, off = 3, 4, 6, 5
    buf = np.full(off + (n - 1) * ld + k + 3, -7.0, dtype=np.float32)
    d = np.arange(n * k, dtype=np.float64).reshape(n, k) + 0.5
    gemm.place(buf, d, off, ld, accumulate=False)
    for i in range(buf.size):
        r, c = divmod(i - off, ld)
        inside = i >= off and r < n and c < k
        assert buf[i] == (d[r, c] if inside else -7.0), i
    gemm.place(buf, d, off, ld, accumulate=True)
    for r in range(n):
        for c in range(k):
            assert buf[off + r * ld + c] == np.float32(2 * d[r, c])
    assert buf[off + k] == -7.0 and buf[-1] == -7.0
