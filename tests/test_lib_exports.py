"""The C ABI library loads without a GPU and exports every declared entry point."""
import ctypes

from tests.libqe import header_symbols, need_lib


def test_exports_every_declared_symbol():
    qe = need_lib()
    L = qe.lib()
    names = header_symbols()
    assert len(names) >= 25
    missing = [n for n in names if not hasattr(L, n)]
    assert not missing, missing
    # the binding forwards exactly the declared calls
    assert sorted(qe.exported_symbols()) == names


def test_status_strings_match_binding():
    qe = need_lib()
    for code, name in enumerate(qe.STATUS):
        assert qe.qe_status_str(code) == name


def test_struct_sizes():
    qe = need_lib()
    assert ctypes.sizeof(qe.TapeKey) == 20
    assert ctypes.sizeof(qe.TapeRef) == 8
    assert ctypes.sizeof(qe.FP8Meta) == 40
    assert ctypes.sizeof(qe.LayerDesc) == 72


def test_invalid_args_rejected_without_device():
    qe = need_lib()
    meta = qe.FP8Meta(0, 0, 0, 4, 0, 0, 0)
    assert qe.qe_quantize_fp8(0, qe.F32, 4, 4, meta, stream=0) == "INVALID_ARG"
    assert qe.qe_fp8_gemm_tn(16, qe.E4M3, 8, 16, qe.E4M3, 16, 4, 4, 16, 16, 16, 16, qe.F32, 4, stream=0) \
        == "INVALID_ARG"
    assert qe.qe_fp8_gemm_tn(16, 7, 16, 16, qe.E4M3, 16, 4, 4, 16, 16, 16, 16, qe.F32, 4, stream=0) == "INVALID_ARG"
    assert qe.qe_amax_scale_update([meta], stream=0) == "INVALID_ARG"
