"""Quantize, the three GEMMs of the split linear, and affine gradient placement.

§3.2 of the paper gives the action signatures
    (Y_m, S1, T_m)          = F(X_m, W, S0)
    (dX_m, B_m, S2, Q_m)    = dI(dY_m, T_m, S1)
    dW_m                    = dW(Q_m)
for a linear Y = X W^T this means Y = X W^T in F, dX = dY W in dI and
dW = dY^T X in the deferred dW, each on FP8-quantized operands.  All three are
written here as one "TN" product C[i, j] = sum_r A[i, r] B[j, r]:
    F : A = X_q  [M, K],  B = W_q    [N, K]   -> Y  [M, N]
    dI: A = dY_q [M, N],  B = W_q^T  [K, N]   -> dX [M, K]
    dW: A = dY_q^T [N, M], B = X_q^T [K, M]   -> dW [N, K]
The product of two FP8 values is exact in float64 and so is the sum at these
sizes up to rounding of the float64 accumulation; the result is multiplied by
the two power-of-two scale inverses (exact).

§3.4 / §4.3: the deferred dW is written into a stable view of a flat FP32
main-gradient arena at an affine offset: element (n, k) lives at
off + n * ld + k.  The first write of a view initialises it, later ones
accumulate in FP32.
"""
from __future__ import annotations

import numpy as np

from . import fp8
from .scaling import amax


def quantize(x_f32: np.ndarray, scale: float, fmt) -> np.ndarray:
    """FP8 codes of x * scale, same shape as x (§2.1: cast with the delayed scale)."""
    return fp8.encode(np.asarray(x_f32, dtype=np.float64) * scale, fmt)


def quantize_with_amax(x_f32: np.ndarray, scale: float, fmt):
    """Codes (row-wise), codes of the transpose (column-wise) and the amax of x."""
    q = quantize(x_f32, scale, fmt)
    return q, np.ascontiguousarray(q.T), amax(x_f32)


def gemm_tn(a_codes, fmt_a, b_codes, fmt_b, a_scale_inv: float, b_scale_inv: float) -> np.ndarray:
    """C = (a_scale_inv * b_scale_inv) * A B^T on decoded FP8 operands, float64."""
    a = fp8.decode(a_codes, fmt_a)
    b = fp8.decode(b_codes, fmt_b)
    c = a @ b.T
    return c * (a_scale_inv * b_scale_inv)


def gemm_tn_loops(a_codes, fmt_a, b_codes, fmt_b, a_scale_inv: float, b_scale_inv: float) -> np.ndarray:
    """The same product as three plain loops (small sizes only)."""
    a = fp8.decode(a_codes, fmt_a)
    b = fp8.decode(b_codes, fmt_b)
    m, k = a.shape
    n = b.shape[0]
    c = np.zeros((m, n), dtype=np.float64)
    for i in range(m):
        for j in range(n):
            s = 0.0
            for r in range(k):
                s += float(a[i, r]) * float(b[j, r])
            c[i, j] = s
    return c * (a_scale_inv * b_scale_inv)


def view_index(offset: int, ld: int, n_rows: int, k_cols: int) -> np.ndarray:
    """Flat indices of an [n_rows, k_cols] view at `offset` with row stride `ld`."""
    return offset + np.arange(n_rows)[:, None] * ld + np.arange(k_cols)[None, :]


def place(main_grad: np.ndarray, d: np.ndarray, offset: int, ld: int, accumulate: bool) -> None:
    """Write (or add) d [N, K] into the flat float32 buffer in place.

    INIT stores fl32(d); ACCUM stores fl32(G + d).  Elements outside the view,
    including the gap k >= K between rows when ld > K, are untouched."""
    n, k = d.shape
    idx = view_index(offset, ld, n, k)
    if accumulate:
        main_grad[idx] = (main_grad[idx].astype(np.float64) + d).astype(np.float32)
    else:
        main_grad[idx] = d.astype(np.float32)

