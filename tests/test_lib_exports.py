"""The C ABI library loads without a GPU and exports every declared entry point."""
import ctypes

import pytest

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
    """The binding's ctypes structs have the sizes the C compiler gives the header's structs."""
    import os
    import shutil
    import subprocess
    import tempfile
    qe = need_lib()
    pairs = {"qe_tape_key": qe.TapeKey, "qe_tape_ref": qe.TapeRef, "qe_fp8_meta": qe.FP8Meta,
             "qe_config": qe.Config, "qe_layer_desc": qe.LayerDesc, "qe_ctx_state": qe.CtxState,
             "qe_layer_state": qe.LayerState, "qe_slot_state": qe.SlotState,
             "qe_prebuild_desc": qe.PrebuildDesc}
    if shutil.which("gcc") is None:
        pytest.skip("no C compiler")
    inc = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include")
    src = '#include <stdio.h>\n#include "qe.h"\nint main(void) {\n' + "".join(
        f'  printf("{n} %zu\\n", sizeof({n}));\n' for n in pairs) + "  return 0;\n}\n"
    with tempfile.TemporaryDirectory() as td:
        c, exe = os.path.join(td, "sizes.c"), os.path.join(td, "sizes")
        open(c, "w").write(src)
        subprocess.run(["gcc", "-std=c99", "-I", inc, c, "-o", exe], check=True)
        out = subprocess.run([exe], check=True, capture_output=True, text=True).stdout
    sizes = dict((n, int(v)) for n, v in (line.split() for line in out.splitlines()))
    for n, cls in pairs.items():
        assert ctypes.sizeof(cls) == sizes[n], (n, ctypes.sizeof(cls), sizes[n])


def test_invalid_args_rejected_without_device():
    qe = need_lib()
    meta = qe.FP8Meta(0, 0, 0, 4, 0, 0, 0)
    assert qe.qe_quantize_fp8(0, qe.F32, 4, 4, meta, stream=0) == "INVALID_ARG"
    assert qe.qe_fp8_gemm_tn(16, qe.E4M3, 8, 16, qe.E4M3, 16, 4, 4, 16, 16, 16, 16, qe.F32, 4, stream=0) \
        == "INVALID_ARG"
    assert qe.qe_fp8_gemm_tn(16, 7, 16, 16, qe.E4M3, 16, 4, 4, 16, 16, 16, 16, qe.F32, 4, stream=0) == "INVALID_ARG"
    # a reduction length of 2^31 or more is refused before any device call
    k = 1 << 31
    assert qe.qe_fp8_gemm_tn(16, qe.E4M3, k, 16, qe.E4M3, k, 4, 4, k, 16, 16, 16, qe.F32, 4, stream=0) \
        == "INVALID_ARG"
    assert qe.qe_amax_scale_update([meta], stream=0) == "INVALID_ARG"
    assert qe.qe_set_gemm_tile(6) == "INVALID_ARG"
    assert qe.qe_set_gemm_tile(-1) == "INVALID_ARG"
    assert qe.qe_set_gemm_tile(qe.TILE_AUTO) == "OK"
