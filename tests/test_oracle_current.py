"""Pins for the oracle's current (dynamic) scaling: the scale is fixed by the
amax of the tensor being cast.  Checked against exact rationals (the scaled
amax lands in the top binade below fmax), closed forms, the equivalence with a
one-entry delayed history recorded before its update (two separately written
code paths), the degenerate cases, and an error bound on a whole forward."""
import math
from fractions import Fraction

import numpy as np
import pytest

from oracle import contract as OC
from oracle import fp8, gemm, scaling
from oracle.layer import Stage


def _tensors(rng):
    out = []
    for lo in (-60, -20, -3, 0, 5, 30):
        x = rng.standard_normal((17, 23)) * 2.0 ** (lo + rng.integers(0, 6))
        out.append(x.astype(np.float32))
    out.append(np.full((3, 3), np.float32(448.0 * 2 ** -7)))
    out.append(np.array([[np.nextafter(np.float32(1.75), np.float32(2))]], dtype=np.float32))
    return out


@pytest.mark.parametrize("fmt", [fp8.E4M3, fp8.E5M2], ids=lambda f: f.name)
def test_scaled_amax_in_top_binade(fmt):
    """margin 0: amax * scale <= fmax < 2 * amax * scale, in exact rationals."""
    rng = np.random.default_rng(5)
    for x in _tensors(rng):
        s = scaling.CurrentScaler(fmt, 0)
        s.set_from(x)
        a = Fraction(float(np.max(np.abs(x.astype(np.float64)))))
        sc = Fraction(s.scale)
        assert a * sc <= Fraction(fmt.fmax) < 2 * a * sc, (float(a), s.scale)
        assert s.scale * s.scale_inv == 1.0


@pytest.mark.parametrize("margin", [0, 2])
def test_margin_divides_scale(margin):
    x = np.array([[3.0, -5.0]], dtype=np.float32)
    s0, sm = scaling.CurrentScaler(fp8.E4M3, 0), scaling.CurrentScaler(fp8.E4M3, margin)
    s0.set_from(x)
    sm.set_from(x)
    assert sm.scale == s0.scale / 2 ** margin


def test_closed_forms():
    cases = [(fp8.E4M3, 448.0 * 2 ** 5, 2.0 ** -5), (fp8.E4M3, 449.0, 0.5), (fp8.E4M3, 1.0, 256.0),
             (fp8.E5M2, 57344.0 * 2 ** -9, 2.0 ** 9), (fp8.E5M2, 1.0, 32768.0), (fp8.E4M3, 2.0 ** -140, 2.0 ** 126),
             (fp8.E4M3, 3.0e38, 2.0 ** -120)]
    for fmt, a, want in cases:
        s = scaling.CurrentScaler(fmt, 0)
        s.set_from(np.array([[a, -a / 3]], dtype=np.float64))
        assert s.scale == want, (fmt.name, a, s.scale)


def test_amax_element_is_never_saturated():
    """With margin 0 the largest element maps to a finite code at most fmax and
    above fmax / 2 (no saturation; delayed scaling can saturate, current cannot)."""
    rng = np.random.default_rng(9)
    for fmt in (fp8.E4M3, fp8.E5M2):
        for x in _tensors(rng):
            s = scaling.CurrentScaler(fmt, 0)
            s.set_from(x)
            a = float(np.max(np.abs(x.astype(np.float64))))
            if not 2.0 ** -100 < a < 2.0 ** 100:     # clamp not binding
                continue
            v = abs(fp8.decode(fp8.encode(np.array([a * s.scale]), fmt), fmt)[0])
            assert fmt.fmax / 2 <= v <= fmt.fmax


def test_equals_one_entry_history_recorded_first():
    rng = np.random.default_rng(3)
    for fmt in (fp8.E4M3, fp8.E5M2):
        for margin in (0, 1):
            cur = scaling.CurrentScaler(fmt, margin)
            dly = scaling.DelayedScaler(fmt, 1, margin)
            seq = _tensors(rng) + [np.zeros((2, 2), np.float32), np.array([[np.nan, 1.0]], np.float32),
                                   np.array([[np.inf]], np.float32)] + _tensors(rng)
            for x in seq:
                cur.set_from(x)
                dly.record(scaling.amax(x))
                dly.update()
                assert (cur.scale, cur.scale_inv) == (dly.scale, dly.scale_inv)
                assert dly.hist[0] == 0.0


def test_degenerate_tensor_keeps_previous_scale():
    s = scaling.CurrentScaler(fp8.E4M3, 0)
    s.set_from(np.zeros((4, 4), np.float32))
    assert s.scale == 1.0
    s.set_from(np.array([[3584.0]], np.float32))       # 448 * 8
    assert s.scale == 0.125
    for bad in (np.zeros((1, 1)), np.array([[np.nan]]), np.array([[-np.inf, 1.0]]), np.zeros((0, 3))):
        s.set_from(bad)
        assert (s.scale, s.scale_inv) == (0.125, 8.0)


def _stage(M, scaling_kind, w):
    st = Stage(M)
    st.add_layer(0, 0, w, 16, 1, 0, scaling=scaling_kind)
    st.add_buffer(64, w.size)
    for m in range(M):
        st.bind(0, m, 64, 0, w.shape[1])
    return st


def test_each_microbatch_uses_its_own_scale():
    """Two microbatches of very different magnitude: each slot keeps the
    scale_inv of its own X, and the cache keeps the one of W."""
    rng = np.random.default_rng(1)
    w = (rng.standard_normal((8, 32)) * 0.02).astype(np.float32)
    st = _stage(2, "current", w)
    xs = [(rng.standard_normal((16, 32)) * s).astype(np.float32) for s in (1.0, 1000.0)]
    for m, x in enumerate(xs):
        assert st.fwd(0, (0, 0, m, 0, 0), x)[0] == OC.OK
        e = scaling.scale_exponent(scaling.amax(x), fp8.E4M3, 0)
        assert st.layers[0].payload[m].x_scale_inv == 2.0 ** -e
    assert st.layers[0].w_scale_inv == 2.0 ** -scaling.scale_exponent(scaling.amax(w), fp8.E4M3, 0)


def test_forward_error_bound_where_delayed_saturates():
    """X ~ N(0, 1000): the first delayed cast (scale 1) saturates at 448, the
    current cast does not, so |Y - X W^T| stays within the FP8 rounding bound:
    per product at most (2^-4 + 2^-4 + 2^-8) |x||w| for E4M3 normals, plus the
    subnormal spacing of either operand."""
    rng = np.random.default_rng(2)
    w = (rng.standard_normal((24, 64)) * 0.02).astype(np.float32)
    x = (rng.standard_normal((16, 64)) * 1000.0).astype(np.float32)
    exact = x.astype(np.float64) @ w.astype(np.float64).T
    bound_rel = 2.0 ** -4 + 2.0 ** -4 + 2.0 ** -8
    st = _stage(1, "current", w)
    _, y, _ = st.fwd(0, (0, 0, 0, 0, 0), x)
    L = st.layers[0]
    sub_x = 2.0 ** -9 * L.payload[0].x_scale_inv      # E4M3 subnormal spacing, unscaled
    sub_w = 2.0 ** -9 * L.w_scale_inv
    ax, aw = np.abs(x.astype(np.float64)), np.abs(w.astype(np.float64))
    bound = bound_rel * (ax @ aw.T) + sub_x * aw.sum(1)[None, :] + sub_w * ax.sum(1)[:, None] \
        + 64 * sub_x * sub_w
    assert np.all(np.abs(y - exact) <= bound)
    dl = _stage(1, "delayed", w)
    _, yd, _ = dl.fwd(0, (0, 0, 0, 0, 0), x)
    assert np.max(np.abs(yd - exact)) > 10 * np.max(np.abs(y - exact))


def test_split_dw_equals_full_backward_under_current_scaling():
    rng = np.random.default_rng(4)
    w = (rng.standard_normal((8, 32)) * 0.02).astype(np.float32)
    xs = [(rng.standard_normal((16, 32)) * s).astype(np.float32) for s in (1.0, 50.0)]
    dys = [(rng.standard_normal((16, 8)) * s).astype(np.float32) for s in (0.01, 3.0)]
    grads = []
    for split in (True, False):
        st = _stage(2, "current", w)
        refs = [st.fwd(0, (0, 0, m, 0, 0), xs[m])[2] for m in range(2)]
        for m in (1, 0):
            key = (0, 0, m, 0, 0)
            mode = OC.INIT if m == 1 else OC.ACCUM
            if split:
                assert st.dgrad(0, key, refs[m], dys[m])[0] == OC.OK
                assert st.wgrad_place(0, key, refs[m], 64, 0, 32, mode) == OC.OK
            else:
                assert st.bwd_full(0, key, refs[m], dys[m], 64, 0, 32, mode)[0] == OC.OK
        grads.append(st.arena[64].copy())
    assert np.array_equal(grads[0], grads[1])
    # and the placed sum is the two dW products with each microbatch's own scales
    want = np.zeros(8 * 32)
    for m in range(2):
        sx = scaling.CurrentScaler(fp8.E4M3, 0)
        sd = scaling.CurrentScaler(fp8.E5M2, 0)
        sx.set_from(xs[m])
        sd.set_from(dys[m])
        xq, xq_t, _ = gemm.quantize_with_amax(xs[m], sx.scale, fp8.E4M3)
        dq, dq_t, _ = gemm.quantize_with_amax(dys[m], sd.scale, fp8.E5M2)
        d = fp8.decode(dq_t, fp8.E5M2) @ fp8.decode(xq_t, fp8.E4M3).T * (sd.scale_inv * sx.scale_inv)
        want = (want.astype(np.float32) + d.astype(np.float32).ravel()).astype(np.float32) if m else \
            d.astype(np.float32).ravel()
    assert math.isclose(float(np.max(np.abs(grads[0] - want))), 0.0, abs_tol=1e-6 * float(np.max(np.abs(want))))
