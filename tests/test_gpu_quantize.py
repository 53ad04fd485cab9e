"""Quantizer parity on the GPU: codes, transposed codes, amax and snapshot,
bit-exact against the oracle."""
import math

import numpy as np
import pytest

import workloads as W
from oracle import fp8, gemm, scaling
from tests.gpu_util import dev, meta_buffer, meta_of, torch, u8, upload
from tests.libqe import need_lib

pytestmark = pytest.mark.gpu


def boundary_values(fmt):
    vals = fp8.decode(np.arange(128), fmt)
    fin = np.sort(vals[np.isfinite(vals)])
    mids = ((fin[1:] + fin[:-1]) / 2).astype(np.float32)
    up = np.nextafter(mids, np.float32(np.inf))
    dn = np.nextafter(mids, np.float32(0))
    extra = np.array([fmt.fmax, fmt.fmax * 1.0001, fmt.fmax * 2, 1e30, np.inf, 0.0, 1e-30, 1e-45, 1e-39,
                      2.0 ** (fmt.emin - fmt.mbits - 1)], dtype=np.float32)
    pos = np.concatenate([fin.astype(np.float32), mids, up, dn, extra])
    return np.concatenate([pos, -pos, np.array([np.nan, -np.nan, -0.0], dtype=np.float32)]).astype(np.float32)


def run_quant(qe, d, x_t, fmt, scale=1.0, H=4, ld_row=None, ld_col=None):
    rows, cols = x_t.shape
    ld_row = cols if ld_row is None else ld_row
    ld_col = rows if ld_col is None else ld_col
    xb = upload(x_t, d)
    mb = meta_buffer(H, d, scale)
    q_row = u8(rows * ld_row, d)
    q_col = u8(cols * ld_col, d)
    snap = torch.zeros(1, dtype=torch.float32, device=d)
    st = qe.qe_quantize_fp8(xb, qe.BF16 if x_t.dtype == "bf16" else qe.F32, rows, cols, meta_of(qe, mb, fmt),
                            q_row, ld_row, q_col, ld_col, snap)
    assert st == "OK"
    torch.cuda.synchronize()
    qr = q_row.cpu().numpy()[: rows * ld_row].reshape(rows, ld_row)[:, :cols] if rows else np.zeros((0, cols))
    qc = q_col.cpu().numpy()[: cols * ld_col].reshape(cols, ld_col)[:, :rows] if cols else np.zeros((0, rows))
    return qr, qc, mb.cpu().numpy(), float(snap.cpu().numpy()[0])


def check(x_f32, fmt_name, qr, qc, mb, snap, scale, H=4):
    want = gemm.quantize(x_f32, scale, fmt_name)
    np.testing.assert_array_equal(qr, want)
    np.testing.assert_array_equal(qc, want.T)
    a = scaling.amax(x_f32)
    if math.isnan(a):
        assert math.isnan(mb[0])
    else:
        assert mb[0] == np.float32(a)
    assert snap == np.float32(1.0 / scale)


@pytest.mark.parametrize("fmt", ["E4M3", "E5M2"])
@pytest.mark.parametrize("scale", [1.0, 2.0 ** 5, 2.0 ** -3])
def test_boundary_values_all_codes(fmt, scale):
    qe = need_lib()
    d = dev()
    f = fp8.fmt_of(fmt)
    v = boundary_values(f) / np.float32(scale)
    cols = 53
    rows = (v.size + cols - 1) // cols
    x = np.zeros(rows * cols, dtype=np.float32)
    x[: v.size] = v
    x = x.reshape(rows, cols)
    fid = qe.E4M3 if fmt == "E4M3" else qe.E5M2
    qr, qc, mb, snap = run_quant(qe, d, W.Tensor(x, "f32"), fid, scale)
    check(x, fmt, qr, qc, mb, snap, scale)


@pytest.mark.parametrize("fmt", ["E4M3", "E5M2"])
def test_boundary_values_full_tiles(fmt):
    """The same vectors laid out so that every tile takes the vectorised path."""
    qe = need_lib()
    d = dev()
    f = fp8.fmt_of(fmt)
    v = boundary_values(f)
    x = np.resize(v, 256 * 384).reshape(256, 384).astype(np.float32)
    fid = qe.E4M3 if fmt == "E4M3" else qe.E5M2
    qr, qc, mb, snap = run_quant(qe, d, W.Tensor(x, "f32"), fid, 1.0)
    check(x, fmt, qr, qc, mb, snap, 1.0)


@pytest.mark.parametrize("shape", [(0, 5), (5, 0), (1, 1), (37, 53), (128, 128), (300, 200), (129, 1000),
                                   (256, 4096)])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("fmt", ["E4M3", "E5M2"])
def test_random_shapes(shape, dtype, fmt):
    qe = need_lib()
    d = dev()
    rng = W.rng_for(1, 0, 0, 0)
    x = W.normal(rng, shape, 3.0, dtype)
    scale = 2.0 ** 4 if fmt == "E4M3" else 2.0 ** 12
    fid = qe.E4M3 if fmt == "E4M3" else qe.E5M2
    qr, qc, mb, snap = run_quant(qe, d, x, fid, scale)
    check(x.as_f32(), fmt, qr, qc, mb, snap, scale)


def test_padded_leading_dimensions_untouched():
    qe = need_lib()
    d = dev()
    x = W.normal(W.rng_for(2, 0, 0, 0), (40, 70), 1.0, "bf16")
    rows, cols, ldr, ldc = 40, 70, 80, 48
    xb = upload(x, d)
    mb = meta_buffer(4, d, 8.0)
    q_row = torch.full((rows * ldr,), 0xA5, dtype=torch.uint8, device=d)
    q_col = torch.full((cols * ldc,), 0x5A, dtype=torch.uint8, device=d)
    assert qe.qe_quantize_fp8(xb, qe.BF16, rows, cols, meta_of(qe, mb, qe.E4M3), q_row, ldr, q_col, ldc) == "OK"
    torch.cuda.synchronize()
    want = gemm.quantize(x.as_f32(), 8.0, "E4M3")
    qr = q_row.cpu().numpy().reshape(rows, ldr)
    qc = q_col.cpu().numpy().reshape(cols, ldc)
    np.testing.assert_array_equal(qr[:, :cols], want)
    np.testing.assert_array_equal(qc[:, :rows], want.T)
    assert (qr[:, cols:] == 0xA5).all() and (qc[:, rows:] == 0x5A).all()


def test_amax_accumulates_and_nan_propagates():
    qe = need_lib()
    d = dev()
    mb = meta_buffer(4, d)
    m = meta_of(qe, mb, qe.E4M3)
    a = torch.tensor([[1.0, -7.5], [2.0, 3.0]], device=d)
    b = torch.tensor([[5.0, 0.5]], device=d)
    assert qe.qe_quantize_fp8(a, qe.F32, 2, 2, m) == "OK"
    assert qe.qe_quantize_fp8(b, qe.F32, 1, 2, m) == "OK"
    torch.cuda.synchronize()
    assert mb[0].item() == 7.5
    c = torch.tensor([[float("nan"), 1.0]], device=d)
    assert qe.qe_quantize_fp8(c, qe.F32, 1, 2, m) == "OK"
    torch.cuda.synchronize()
    assert math.isnan(mb[0].item())


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("fmt", ["E4M3", "E5M2"])
@pytest.mark.parametrize("shape", [(256, 384), (37, 53)], ids=["full_tiles", "ragged"])
def test_subnormal_inputs_scaled_to_normal(dtype, fmt, shape):
    """An all-subnormal tensor (FP32 / BF16 subnormals, both signs, with zeros):
    the scale update clamps its exponent to 126, and the cast multiplies every
    subnormal input by 2^126, which lands in the normal range; codes and the
    recorded amax must match the oracle bit for bit (a flush of subnormal
    inputs to zero would make every code zero)."""
    qe = need_lib()
    d = dev()
    rng = np.random.default_rng(5)
    mant = rng.integers(0, 1 << 23, size=shape, dtype=np.int64).astype(np.uint32)
    if dtype == "bf16":
        mant &= np.uint32(0x007F0000)            # bf16 subnormals: the top 7 mantissa bits
    sign = rng.integers(0, 2, size=shape, dtype=np.int64).astype(np.uint32) << 31
    bits = (sign | mant).astype(np.uint32)
    x = bits.view(np.float32)
    assert not np.any(np.isfinite(x) & (np.abs(x) >= np.float32(2.0 ** -126)))
    t = W.Tensor((bits >> 16).astype(np.uint16), "bf16") if dtype == "bf16" else W.Tensor(x, "f32")
    x_f32 = t.as_f32()
    f = qe.E4M3 if fmt == "E4M3" else qe.E5M2
    # the exponent the scale update derives from this amax, clamped to 126
    a = scaling.amax(x_f32)
    assert 0.0 < a < 2.0 ** -126
    assert scaling.scale_exponent(a, fmt, 0) == 126
    H = 4
    mb = meta_buffer(H, d, 1.0)
    meta = meta_of(qe, mb, f)
    # first cast at scale 1 records the amax; the update sets scale = 2^126
    qr, qc, mb1, snap = run_quant(qe, d, t, f, 1.0, H=H)
    mb.copy_(torch.from_numpy(mb1).to(d))
    assert qe.qe_amax_scale_update([meta]) == "OK"
    torch.cuda.synchronize()
    m = mb.cpu().numpy()
    assert m[H] == np.float32(2.0 ** 126) and m[H + 1] == np.float32(2.0 ** -126)
    qr, qc, _, snap = run_quant(qe, d, t, f, 2.0 ** 126, H=H)
    check(x_f32, fmt, qr, qc, mb1, snap, 2.0 ** 126)
    assert np.count_nonzero(qr) > qr.size // 2


def _bf16_rows_f32(bits_i16):
    """bf16 bit patterns (int16) -> float32 values."""
    return (bits_i16.view(np.uint16).astype(np.uint32) << 16).view(np.float32)


def test_tensor_past_2_31_elements():
    """A bf16 tensor of 65,613 x 32,808 elements (2^31 plus 5.9 M, 4.3 GB;
    ragged tiles in both dimensions) through the delayed cast, then through
    the current-scaling cast (whose amax pass takes the streamed path): the
    amax of every element against the oracle's (a max over row blocks), sampled
    rows of the row-wise codes and sampled columns of the transposed codes
    (first, last and tile-edge indices, random ones) against the oracle's
    cast, and every transposed code equal to its row-wise one."""
    qe = need_lib()
    d = dev()
    rows, cols = 65_613, 32_808
    assert rows * cols > 1 << 31
    g = torch.Generator(device=d)
    g.manual_seed(31)
    x = torch.randn((rows, cols), dtype=torch.bfloat16, device=d, generator=g) * 3.0
    x[rows - 1, cols - 1] = -776.0                     # the largest magnitude, in the last (ragged) tile
    xh = x.view(torch.int16).cpu().numpy()
    amax = max(scaling.amax(_bf16_rows_f32(xh[r:r + 4096])) for r in range(0, rows, 4096))
    assert amax == 776.0
    rng = np.random.default_rng(31)
    rpick = np.unique(np.concatenate([[0, 1, 127, 128, 65535, 65536, rows - 1], rng.integers(0, rows, 5)]))
    cpick = np.unique(np.concatenate([[0, 127, 128, 32767, 32768, cols - 1], rng.integers(0, cols, 5)]))
    xr = _bf16_rows_f32(xh[rpick])                     # [rpick, cols]
    xc = _bf16_rows_f32(np.ascontiguousarray(xh[:, cpick].T))  # [cpick, rows]
    del xh
    q_row = u8(rows * cols, d)
    q_col = u8(rows * cols, d)

    def check_codes(scale):
        np.testing.assert_array_equal(q_row.view(rows, cols)[torch.from_numpy(rpick).to(d)].cpu().numpy(),
                                      gemm.quantize(xr, scale, "E5M2"))
        np.testing.assert_array_equal(q_col.view(cols, rows)[torch.from_numpy(cpick).to(d)].cpu().numpy(),
                                      gemm.quantize(xc, scale, "E5M2"))
        assert torch.equal(q_row.view(rows, cols).t(), q_col.view(cols, rows))

    # delayed: the meta's scale, the amax recorded into history[0]
    mb = meta_buffer(4, d, 2.0 ** 4)
    snap = torch.zeros(1, dtype=torch.float32, device=d)
    assert qe.qe_quantize_fp8(x, qe.BF16, rows, cols, meta_of(qe, mb, qe.E5M2), q_row, cols, q_col, rows,
                              snap) == "OK"
    torch.cuda.synchronize()
    assert mb[0].item() == amax and snap.item() == 2.0 ** -4
    check_codes(2.0 ** 4)
    # current scaling: the scale is set from this tensor's amax first
    mc = meta_buffer(1, d)
    token = torch.zeros(1, dtype=torch.int64, device=d)
    assert qe.qe_quantize_fp8_current(x, qe.BF16, rows, cols, meta_of(qe, mc, qe.E5M2), q_row, cols, q_col, rows,
                                      snap, token) == "OK"
    torch.cuda.synchronize()
    e = scaling.scale_exponent(amax, "E5M2", 0)
    m = mc.cpu().numpy()
    assert (m[0], m[1], m[2]) == (0.0, np.float32(2.0 ** e), np.float32(2.0 ** -e))
    assert snap.item() == 2.0 ** -e and token.item() == 1
    check_codes(2.0 ** e)
