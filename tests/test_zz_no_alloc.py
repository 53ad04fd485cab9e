"""The allocation-free current-scaling cast (qe_quantize_fp8_current_noalloc):
called through the C ABI, its codes, transposed codes, scale, scale_inv,
snapshot, cleared history and effect token equal those of
qe_quantize_fp8_current with a caller-allocated amax accumulator, bit for bit,
on two calls in a row (the second with a smaller tensor, after the first left
the library's scratch behind), also for an unaligned input and one that holds
a NaN (whose scale is kept)."""
import numpy as np
import pytest

import workloads as W
from tests.gpu_util import accum_buffer, dev, meta_buffer, meta_of, torch, u8, upload
from tests.libqe import need_lib

pytestmark = pytest.mark.gpu


def _cast(qe, d, fn, t, meta_buf, fmt, accum, token, offset=0):
    rows, cols = t.shape
    ldr, ldc = cols + 3, rows + 5
    src = upload(t, d)
    if offset:
        buf = torch.empty(src.numel() + offset, dtype=src.dtype, device=d)
        buf[offset:].copy_(src.reshape(-1))
        addr = buf.data_ptr() + offset * src.element_size()
    else:
        buf, addr = src, src.data_ptr()
    q_row = torch.full((rows * ldr,), 0xA5, dtype=torch.uint8, device=d)
    q_col = torch.full((cols * ldc,), 0x5A, dtype=torch.uint8, device=d)
    snap = torch.zeros(1, dtype=torch.float32, device=d)
    st = fn(addr, qe.BF16 if t.dtype == "bf16" else qe.F32, rows, cols, meta_of(qe, meta_buf, fmt, accum=accum),
            q_row, ldr, q_col, ldc, snap, token)
    assert st == "OK", st
    torch.cuda.synchronize()
    del buf
    return q_row.cpu().numpy(), q_col.cpu().numpy(), snap.item()


@pytest.mark.parametrize("fmt_name", ["E4M3", "E5M2"])
def test_noalloc_equals_current_cast_two_calls(fmt_name):
    qe = need_lib()
    d = dev()
    fmt = qe.E4M3 if fmt_name == "E4M3" else qe.E5M2
    big = W.normal(W.rng_for(4, 0, 0, 0), (700, 1300), 3.0, "bf16")
    small = W.normal(W.rng_for(4, 0, 0, 1), (129, 37), 0.25, "f32")
    nan = W.normal(W.rng_for(4, 0, 0, 2), (64, 200), 1.0, "f32")
    nan.data[17, 33] = np.nan
    ref_meta, new_meta = meta_buffer(1, d), meta_buffer(1, d)
    ref_tok = torch.zeros(1, dtype=torch.int64, device=d)
    new_tok = torch.zeros(1, dtype=torch.int64, device=d)
    acc = accum_buffer(d)
    for t, offset in ((big, 0), (small, 0), (small, 3), (nan, 1)):
        ref = _cast(qe, d, qe.qe_quantize_fp8_current, t, ref_meta, fmt, acc, ref_tok, offset)
        got = _cast(qe, d, qe.qe_quantize_fp8_current_noalloc, t, new_meta, fmt, None, new_tok, offset)
        np.testing.assert_array_equal(got[0], ref[0])
        np.testing.assert_array_equal(got[1], ref[1])
        assert got[2] == ref[2]
        np.testing.assert_array_equal(new_meta.cpu().numpy().view(np.uint32), ref_meta.cpu().numpy().view(np.uint32))
        assert new_meta[0].item() == 0.0            # the one-entry history is left clear, as the update leaves it
        assert new_tok.item() == ref_tok.item()
    assert np.count_nonzero(got[0]) > 0
    assert not bool(torch.any(acc != 0))            # the caller's accumulator was cleared by its update


def test_noalloc_rejects_a_caller_accumulator():
    qe = need_lib()
    d = dev()
    mb = meta_buffer(1, d)
    x = torch.ones((4, 4), device=d)
    assert qe.qe_quantize_fp8_current_noalloc(x, qe.F32, 4, 4, meta_of(qe, mb, qe.E4M3, accum=accum_buffer(d)),
                                              u8(16, d), 4, u8(16, d), 4) == "INVALID_ARG"
    assert qe.qe_quantize_fp8_current_noalloc(x, qe.F32, 4, 4, meta_of(qe, meta_buffer(4, d), qe.E4M3),
                                              u8(16, d), 4, u8(16, d), 4) == "INVALID_ARG"
