"""Current (dynamic) scaling on the GPU: the amax pass, the one-call current
cast, and whole layers whose casts take the scale of the tensor being cast;
codes, amax and scales bit-exact against the oracle, GEMM outputs within 1e-3,
split = full and graph = eager bitwise."""
import math

import numpy as np
import pytest

import workloads as W
from oracle import gemm, scaling
from tests import schedules as S
from tests.gpu_util import accum_buffer, accum_value, dev, meta_buffer, meta_of, torch, u8
from tests.libqe import need_lib
from tests.stage_driver import Spec
from tests.test_gpu_layer import _assert_bitwise, _run_variant, run_pair

pytestmark = pytest.mark.gpu


def _device_tensor(x_f32, dtype, offset, d):
    """x (float32 numpy) on the device `offset` elements into a larger buffer,
    as float32 or bf16 bits; returns (buffer, address, the values as float32)."""
    n = x_f32.size
    if dtype == "bf16":
        bits = W.f32_to_bf16_bits(x_f32.ravel())
        host = np.zeros(n + offset, dtype=np.uint16)
        host[offset:] = bits
        buf = torch.from_numpy(host.view(np.int16)).to(d)
        return buf, buf.data_ptr() + 2 * offset, W.bf16_bits_to_f32(bits).reshape(x_f32.shape)
    host = np.zeros(n + offset, dtype=np.float32)
    host[offset:] = x_f32.ravel()
    buf = torch.from_numpy(host).to(d)
    return buf, buf.data_ptr() + 4 * offset, x_f32


def _amax_via(qe, d, addr, dtype, numel, use_accum, init=0.0):
    """Run qe_amax into a fresh one-entry role (history[0] = init) with or
    without an accumulator; return the folded value."""
    mb = meta_buffer(1, d)
    mb[0] = init
    acc = accum_buffer(d) if use_accum else None
    st = qe.qe_amax(addr, qe.BF16 if dtype == "bf16" else qe.F32, numel, meta_of(qe, mb, qe.E4M3, accum=acc))
    assert st == "OK"
    torch.cuda.synchronize()
    if use_accum:
        assert mb[0].item() == init        # the history is untouched until an update folds the accumulator
        return accum_value(acc)
    return mb[0].item()


@pytest.mark.parametrize("use_accum", [False, True])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("numel", [0, 1, 5, 8, 9, 63, 1000, 4096 * 33 + 5, (1 << 22) + 3])
@pytest.mark.parametrize("offset", [0, 1, 7])
def test_amax_matches_oracle(dtype, numel, offset, use_accum):
    qe = need_lib()
    d = dev()
    rng = np.random.default_rng(numel * 8 + offset)
    x = (rng.standard_normal(numel) * 3.0).astype(np.float32)
    places = sorted({0, numel // 2, numel - 1}) if numel else []
    for p in places + [None]:
        y = x.copy()
        if p is not None:
            y[p] = -1234.5 * (1 + p % 3)       # the max sits in the head, the body or the tail
        buf, addr, vals = _device_tensor(y, dtype, offset, d)
        got = _amax_via(qe, d, addr, dtype, numel, use_accum)
        assert got == np.float32(scaling.amax(vals)), (p, got)
    if numel and not use_accum:                # max semantics with a larger value already in the slot
        buf, addr, vals = _device_tensor(x, dtype, offset, d)
        assert _amax_via(qe, d, addr, dtype, numel, False, init=1e30) == np.float32(1e30)
    for special, want_nan in ((np.inf, False), (-np.inf, False), (np.nan, True)):
        if not numel:
            break
        y = x.copy()
        y[places[-1]] = special
        buf, addr, vals = _device_tensor(y, dtype, offset, d)
        got = _amax_via(qe, d, addr, dtype, numel, use_accum)
        assert math.isnan(got) if want_nan else got == math.inf


@pytest.mark.parametrize("dtype,numel,offset", [("f32", (80 << 20) + 3, 1), ("bf16", (150 << 20) + 5, 7)])
def test_amax_streamed_tensor_matches_oracle(dtype, numel, offset):
    """Tensors larger than the 256 MB memory-side cache take the amax pass's
    non-temporal path: same exact max, NaN still propagates."""
    qe = need_lib()
    d = dev()
    rng = np.random.default_rng(numel)
    x = rng.standard_normal(numel, dtype=np.float32)
    x[numel // 3] = -777.25                    # the max in the body
    buf, addr, vals = _device_tensor(x, dtype, offset, d)
    assert _amax_via(qe, d, addr, dtype, numel, True) == np.float32(scaling.amax(vals))
    assert _amax_via(qe, d, addr, dtype, numel, False) == np.float32(scaling.amax(vals))
    del buf
    x[numel - 2] = np.nan
    buf, addr, vals = _device_tensor(x, dtype, offset, d)
    assert math.isnan(_amax_via(qe, d, addr, dtype, numel, True))
    del buf
    torch.cuda.empty_cache()


def test_amax_rejects_bad_arguments():
    qe = need_lib()
    d = dev()
    buf = torch.zeros(16, dtype=torch.float32, device=d)
    m = meta_of(qe, meta_buffer(1, d), qe.E4M3)
    assert qe.qe_amax(buf.data_ptr() + 2, qe.F32, 4, m) == "INVALID_ARG"
    assert qe.qe_amax(buf, qe.F32, -1, m) == "INVALID_ARG"
    assert qe.qe_amax(buf, 7, 4, m) == "INVALID_ARG"
    assert qe.qe_amax(buf, qe.F32, 4, qe.FP8Meta()) == "INVALID_ARG"


@pytest.mark.parametrize("fmt", ["E4M3", "E5M2"])
def test_accumulator_folds_into_history_at_update(fmt):
    """Two delayed casts fold into the accumulator, not the history; the next
    update folds the accumulator into history[0], clears it, and gives the
    oracle's history and scale (the same as recording straight into history[0])."""
    qe = need_lib()
    d = dev()
    rng = np.random.default_rng(23)
    H = 4
    mb, acc = meta_buffer(H, d), accum_buffer(d)
    meta = meta_of(qe, mb, qe.E4M3 if fmt == "E4M3" else qe.E5M2, accum=acc)
    ref = scaling.DelayedScaler(fmt, H, 0)
    for step in range(6):
        for j in range(2):
            x = (rng.standard_normal((200, 136)) * 10.0 ** (step - 2 + j)).astype(np.float32)
            if step == 4 and j == 1:
                x[7, 9] = np.nan
            xb = torch.from_numpy(x).to(d)
            q = u8(x.size, d)
            assert qe.qe_quantize_fp8(xb, qe.F32, 200, 136, meta, q, 136, None, 0) == "OK"
            ref.record(scaling.amax(x))
        torch.cuda.synchronize()
        assert mb[0].item() == 0.0
        got = accum_value(acc)
        assert math.isnan(got) if math.isnan(ref.hist[0]) else got == np.float32(ref.hist[0])
        assert qe.qe_amax_scale_update([meta]) == "OK"
        ref.update()
        torch.cuda.synchronize()
        m = mb.cpu().numpy()
        np.testing.assert_array_equal(m[:H], ref.hist.astype(np.float32))
        assert (m[H], m[H + 1]) == (np.float32(ref.scale), np.float32(ref.scale_inv))
        assert not acc.cpu().numpy().any()


def _current_cast(qe, d, x_f32, dtype, fmt, mb, token, margin=0):
    rows, cols = x_f32.shape
    buf, addr, vals = _device_tensor(x_f32, dtype, 0, d)
    q_row, q_col = u8(rows * cols, d), u8(rows * cols, d)
    snap = torch.zeros(1, dtype=torch.float32, device=d)
    st = qe.qe_quantize_fp8_current(addr, qe.BF16 if dtype == "bf16" else qe.F32, rows, cols,
                                    meta_of(qe, mb, qe.E4M3 if fmt == "E4M3" else qe.E5M2, margin), q_row, cols,
                                    q_col, rows, snap, token)
    assert st == "OK"
    torch.cuda.synchronize()
    qr = q_row.cpu().numpy()[: rows * cols].reshape(rows, cols)
    qc = q_col.cpu().numpy()[: rows * cols].reshape(cols, rows)
    return vals, qr, qc, float(snap.item())


@pytest.mark.parametrize("fmt", ["E4M3", "E5M2"])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("margin", [0, 1])
def test_current_cast_sequence_matches_oracle(fmt, dtype, margin):
    """Successive casts on one role: each takes the scale of its own tensor
    (a larger, then a much smaller tensor), a zero tensor keeps the last scale,
    history[0] is clear after every call, and the token counts the calls."""
    qe = need_lib()
    d = dev()
    rng = np.random.default_rng(17)
    mb = meta_buffer(1, d)
    token = torch.zeros(1, dtype=torch.int64, device=d)
    ref = scaling.CurrentScaler(fmt, margin)
    shapes = [(128, 128), (300, 200), (1, 1), (257, 129), (64, 48), (33, 700)]
    mags = [1.0, 2000.0, 1e-3, 0.0, 37.0, 1e-30]
    for i, ((rows, cols), mag) in enumerate(zip(shapes, mags)):
        x = (rng.standard_normal((rows, cols)) * mag).astype(np.float32)
        vals, qr, qc, snap = _current_cast(qe, d, x, dtype, fmt, mb, token, margin)
        ref.set_from(vals)
        want = gemm.quantize(vals, ref.scale, fmt)
        np.testing.assert_array_equal(qr, want, err_msg=f"call {i}")
        np.testing.assert_array_equal(qc, want.T, err_msg=f"call {i}")
        m = mb.cpu().numpy()
        assert m[0] == 0.0
        assert (m[1], m[2]) == (np.float32(ref.scale), np.float32(ref.scale_inv)), (i, m, ref.scale)
        assert snap == np.float32(ref.scale_inv)
        assert token.item() == i + 1


def test_current_cast_rejects_history():
    qe = need_lib()
    d = dev()
    mb = meta_buffer(4, d)
    x = torch.zeros(16, dtype=torch.float32, device=d)
    q = u8(16, d)
    assert qe.qe_quantize_fp8_current(x, qe.F32, 4, 4, meta_of(qe, mb, qe.E4M3), q, 4, q, 4) == "INVALID_ARG"


def test_current_layer_single_schedule():
    spec = Spec([(256, 256)], tokens=128, M=2, history=1, margin=0, in_dtype="f32", shared_view=True, cfg=0,
                scaling="current")
    run_pair(spec, [S.SINGLE] * 3, check_codes_after=4)


def test_current_layer_ragged_bf16_outliers():
    """Outlier activations and log-normal gradients: current scaling never
    saturates the largest element, and codes still match bit for bit."""
    spec = Spec([(200, 136), (72, 300)], tokens=100, M=2, history=1, margin=1, in_dtype="bf16",
                shared_view=False, cfg=91, outliers=True, scaling="current")
    run_pair(spec, [S.SINGLE, S.SINGLE], check_codes_after=4)


@pytest.mark.parametrize("use_graphs", [False, True])
def test_current_layer_zero_bubble_schedule(use_graphs):
    spec = Spec([(96, 160), (160, 64)], tokens=48, M=8, history=1, margin=0, in_dtype="bf16", shared_view=False,
                cfg=2, scaling="current")
    run_pair(spec, [S.ZB_STEP0, S.ZB_STEP1], use_graphs=use_graphs, check_codes_after=13)


def test_current_layer_empty_microbatch():
    spec = Spec([(64, 96)], tokens=0, M=1, history=1, margin=0, in_dtype="f32", shared_view=False, cfg=93,
                scaling="current")
    g, o = run_pair(spec, [[("F", 0), ("dI", 0), ("dW", 0)]] * 2)
    assert np.all(g.grad.cpu().numpy() == 0)


def test_current_split_equals_full_and_graph_equals_eager():
    spec = Spec([(96, 160), (72, 200)], tokens=48, M=8, history=1, margin=0, in_dtype="bf16", shared_view=False,
                cfg=2, scaling="current")
    steps = [S.ZB_STEP0, S.ZB_STEP1]
    split = _run_variant(spec, steps, False, False)
    _assert_bitwise(split, _run_variant(spec, steps, False, True))
    _assert_bitwise(split, _run_variant(spec, steps, True, False))
