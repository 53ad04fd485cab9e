"""Thin ctypes binding of libqe.so (the C ABI in include/qe.h).

Argument marshalling only: every function here has the name of the C entry
point it forwards to, turns tensors into device pointers and streams into
hipStream_t handles, and returns the C status as a string ("OK", "STALE_REF",
...).  All device work happens inside the library.  If libqe.so has not been
built, importing works but the first call raises: there is no fallback path.
"""
from __future__ import annotations

import ctypes as C
import os
from typing import Optional

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libqe.so")

E4M3, E5M2 = 0, 1
F32, BF16 = 0, 1
INIT, ACCUM = 0, 1
ROLE_X, ROLE_W, ROLE_DY = 0, 1, 2
SCALING_DELAYED, SCALING_CURRENT = 0, 1
AMAX_LINES, AMAX_STRIDE = 64, 64   # amax accumulator: lines x floats between lines
KC_QUANT, KC_UPDATE, KC_GEMM, KC_COPY, KC_AMAX = 0, 1, 2, 3, 4
GRAPH_INPUTS_REBIND, GRAPH_INPUTS_RECAPTURE, GRAPH_INPUTS_COPY = 0, 1, 2

STATUS = ["OK", "INVALID_ARG", "STALE_REF", "KEY_MISMATCH", "KEY_LIVE", "POOL_FULL", "DUPLICATE_CONSUMER", "ORDER",
          "EPOCH", "STALE_CACHE", "DEST_MISMATCH", "DEST_ALIAS", "DUP_WRITE", "ARENA_INVALID", "INCOMPLETE",
          "NOT_QUIESCENT", "HIP", "UNSUPPORTED"]


class TapeKey(C.Structure):
    _fields_ = [("epoch", C.c_uint32), ("stage", C.c_uint32), ("microbatch", C.c_uint32), ("unit", C.c_uint32),
                ("invocation", C.c_uint32)]

    def astuple(self):
        return (self.epoch, self.stage, self.microbatch, self.unit, self.invocation)


class TapeRef(C.Structure):
    _fields_ = [("slot", C.c_uint32), ("generation", C.c_uint32)]

    def astuple(self):
        return (self.slot, self.generation)


class FP8Meta(C.Structure):
    _fields_ = [("amax_history", C.c_void_p), ("scale", C.c_void_p), ("scale_inv", C.c_void_p),
                ("history_len", C.c_int32), ("margin", C.c_int32), ("fmt", C.c_int32), ("reserved", C.c_int32),
                ("amax_accum", C.c_void_p)]


class Config(C.Structure):
    _fields_ = [("device", C.c_int32), ("microbatches", C.c_int32), ("use_graphs", C.c_int32),
                ("null_executor", C.c_int32), ("one_way_handoff", C.c_int32), ("copy_gradients", C.c_int32),
                ("replay_on_caller", C.c_int32), ("graph_inputs", C.c_int32)]


class LayerDesc(C.Structure):
    _fields_ = [("stage", C.c_uint32), ("unit", C.c_uint32), ("n_out", C.c_int64), ("k_in", C.c_int64),
                ("max_tokens", C.c_int64), ("w", C.c_void_p), ("w_dtype", C.c_int32), ("history_len", C.c_int32),
                ("margin", C.c_int32), ("fmt_x", C.c_int32), ("fmt_w", C.c_int32), ("fmt_dy", C.c_int32),
                ("scaling", C.c_int32)]


class CtxState(C.Structure):
    _fields_ = [("e_w", C.c_int64), ("token", C.c_int64), ("device_token", C.c_int64), ("arena_valid", C.c_int32),
                ("finalized", C.c_int32), ("graphs", C.c_int64), ("captures", C.c_int64), ("replays", C.c_int64),
                ("handoffs", C.c_int64), ("capture_ns", C.c_int64), ("arena_bytes", C.c_int64),
                ("device_bytes", C.c_int64), ("rebinds", C.c_int64), ("rebound_nodes", C.c_int64),
                ("prebuild_ns", C.c_int64)]


class PrebuildDesc(C.Structure):
    _fields_ = [("tokens", C.c_int64), ("x_dtype", C.c_int32), ("y_dtype", C.c_int32), ("dy_dtype", C.c_int32),
                ("dx_dtype", C.c_int32)]


class LayerState(C.Structure):
    _fields_ = [("e_c", C.c_int64), ("refreshes", C.c_int64), ("n_slots", C.c_int32), ("reserved", C.c_int32)]


class SlotState(C.Structure):
    _fields_ = [("live", C.c_int32), ("generation", C.c_uint32), ("bits", C.c_uint32), ("reserved", C.c_uint32),
                ("key", TapeKey), ("tokens", C.c_int64), ("bound", C.c_int32), ("written", C.c_int32),
                ("view_offset", C.c_int64), ("view_ld", C.c_int64), ("view_buf", C.c_void_p)]


_P, _I32, _U32, _I64 = C.c_void_p, C.c_int32, C.c_uint32, C.c_int64
_SIGS = {
    "qe_amax_scale_update": [C.POINTER(FP8Meta), _I32, _P, _P],
    "qe_quantize_fp8": [_P, _I32, _I64, _I64, C.POINTER(FP8Meta), _P, _I64, _P, _I64, _P, _P],
    "qe_amax": [_P, _I32, _I64, C.POINTER(FP8Meta), _P],
    "qe_quantize_fp8_current": [_P, _I32, _I64, _I64, C.POINTER(FP8Meta), _P, _I64, _P, _I64, _P, _P, _P],
    "qe_quantize_fp8_current_noalloc": [_P, _I32, _I64, _I64, C.POINTER(FP8Meta), _P, _I64, _P, _I64, _P, _P, _P],
    "qe_fp8_gemm_tn": [_P, _I32, _I64, _P, _I32, _I64, _I64, _I64, _I64, _P, _P, _P, _I32, _I64, _I32, _P],
    "qe_set_gemm_tile": [_I32],
    "qe_ctx_create": [C.POINTER(Config), C.POINTER(_P)],
    "qe_layer_register": [_P, C.POINTER(LayerDesc), C.POINTER(_I32)],
    "qe_layer_meta": [_P, _I32, _I32, C.POINTER(FP8Meta)],
    "qe_layer_cache": [_P, _I32, C.POINTER(_P), C.POINTER(_I64), C.POINTER(_P), C.POINTER(_I64), C.POINTER(_P)],
    "qe_layer_slot_payload": [_P, _I32, _I32, C.POINTER(_P), C.POINTER(_I64), C.POINTER(_P), C.POINTER(_I64),
                              C.POINTER(_P), C.POINTER(_P)],
    "qe_fp8_linear_fwd": [_P, _I32, TapeKey, _P, _I32, _I64, _P, _I32, C.POINTER(TapeRef), _P],
    "qe_fp8_linear_dgrad": [_P, _I32, TapeKey, TapeRef, _P, _I32, _P, _I32, _P],
    "qe_fp8_linear_wgrad_place": [_P, _I32, TapeKey, TapeRef, _P, _I64, _I64, _I32, _P],
    "qe_fp8_linear_bwd_full": [_P, _I32, TapeKey, TapeRef, _P, _I32, _P, _I32, _P, _I64, _I64, _I32, _P],
    "qe_arena_bind": [_P, _I32, _U32, _P, _I64, _I64, _I64],
    "qe_prebuild_graphs": [_P, C.POINTER(PrebuildDesc)],
    "qe_arena_finalize": [_P],
    "qe_optimizer_commit": [_P],
    "qe_abort_epoch": [_P],
    "qe_arena_rebuild": [_P],
    "qe_checkpoint_export": [_P, _P, _I64, C.POINTER(_I64)],
    "qe_checkpoint_import": [_P, _P, _I64],
    "qe_sync": [_P],
    "qe_get_state": [_P, C.POINTER(CtxState)],
    "qe_get_layer_state": [_P, _I32, C.POINTER(LayerState)],
    "qe_get_slot_state": [_P, _I32, _I32, C.POINTER(SlotState)],
    "qe_inject_fault": [_P, _I32],
    "qe_set_kernel_timing": [_P, _I32],
    "qe_get_kernel_timing": [_P, _I32, C.POINTER(C.c_double), C.POINTER(_I64)],
}

_lib = None


def lib():
    """Load libqe.so; raises if it has not been built (no fallback)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2609_23536_amd.build`")
        # torch ships its own HIP runtime under the same soname; load it first so
        # that the library and torch's allocator and streams share one runtime.
        try:
            import torch  # noqa: F401
        except ImportError:
            pass
        L = C.CDLL(LIB_PATH)
        for name, args in _SIGS.items():
            fn = getattr(L, name)
            fn.argtypes = args
            fn.restype = C.c_int
        L.qe_ctx_destroy.argtypes = [_P]
        L.qe_ctx_destroy.restype = None
        L.qe_status_str.argtypes = [C.c_int]
        L.qe_status_str.restype = C.c_char_p
        _lib = L
    return _lib


def ptr(x) -> int:
    """Device (or host) address of a tensor, an int, or None (0)."""
    if x is None:
        return 0
    if isinstance(x, int):
        return x
    return int(x.data_ptr())


def stream_handle(s) -> int:
    if s is None:
        import torch
        return int(torch.cuda.current_stream().cuda_stream)
    if isinstance(s, int):
        return s
    return int(s.cuda_stream)


def _st(code: int) -> str:
    return STATUS[code] if 0 <= code < len(STATUS) else f"UNKNOWN({code})"


def key(epoch: int, stage: int, microbatch: int, unit: int, invocation: int = 0) -> TapeKey:
    return TapeKey(epoch, stage, microbatch, unit, invocation)


# --------------------------------------------------------------------------- stateless hot-path calls
def qe_amax_scale_update(metas, device_token=None, stream=None) -> str:
    arr = (FP8Meta * len(metas))(*metas)
    return _st(lib().qe_amax_scale_update(arr, len(metas), ptr(device_token), stream_handle(stream)))


def qe_quantize_fp8(inp, in_dtype: int, rows: int, cols: int, meta: FP8Meta, q_row=None, ld_row: int = 0,
                    q_col=None, ld_col: int = 0, scale_inv_snapshot=None, stream=None) -> str:
    return _st(lib().qe_quantize_fp8(ptr(inp), in_dtype, rows, cols, C.byref(meta), ptr(q_row), ld_row, ptr(q_col),
                                     ld_col, ptr(scale_inv_snapshot), stream_handle(stream)))


def qe_amax(inp, in_dtype: int, numel: int, meta: FP8Meta, stream=None) -> str:
    return _st(lib().qe_amax(ptr(inp), in_dtype, numel, C.byref(meta), stream_handle(stream)))


def qe_quantize_fp8_current(inp, in_dtype: int, rows: int, cols: int, meta: FP8Meta, q_row=None, ld_row: int = 0,
                            q_col=None, ld_col: int = 0, scale_inv_snapshot=None, device_token=None,
                            stream=None) -> str:
    return _st(lib().qe_quantize_fp8_current(ptr(inp), in_dtype, rows, cols, C.byref(meta), ptr(q_row), ld_row,
                                             ptr(q_col), ld_col, ptr(scale_inv_snapshot), ptr(device_token),
                                             stream_handle(stream)))


def qe_quantize_fp8_current_noalloc(inp, in_dtype: int, rows: int, cols: int, meta: FP8Meta, q_row=None,
                                    ld_row: int = 0, q_col=None, ld_col: int = 0, scale_inv_snapshot=None,
                                    device_token=None, stream=None) -> str:
    return _st(lib().qe_quantize_fp8_current_noalloc(ptr(inp), in_dtype, rows, cols, C.byref(meta), ptr(q_row),
                                                     ld_row, ptr(q_col), ld_col, ptr(scale_inv_snapshot),
                                                     ptr(device_token), stream_handle(stream)))


def qe_fp8_gemm_tn(a, fmt_a: int, lda: int, b, fmt_b: int, ldb: int, m: int, n: int, k: int, a_scale_inv,
                   b_scale_inv, c, c_dtype: int, ldc: int, mode: int = INIT, stream=None) -> str:
    return _st(lib().qe_fp8_gemm_tn(ptr(a), fmt_a, lda, ptr(b), fmt_b, ldb, m, n, k, ptr(a_scale_inv),
                                    ptr(b_scale_inv), ptr(c), c_dtype, ldc, mode, stream_handle(stream)))


TILE_AUTO, TILE_256x256, TILE_256x192, TILE_192x256, TILE_256x128, TILE_256x224 = 0, 1, 2, 3, 4, 5


def qe_set_gemm_tile(tile: int) -> str:
    return _st(lib().qe_set_gemm_tile(tile))


def make_meta(hist, scale, scale_inv, fmt: int, margin: int = 0, amax_accum=None) -> FP8Meta:
    return FP8Meta(ptr(hist), ptr(scale), ptr(scale_inv), int(hist.numel()), margin, fmt, 0, ptr(amax_accum))


# --------------------------------------------------------------------------- context
class Context:
    """Owns one qe_ctx.  Methods forward to the C calls of the same name."""

    def __init__(self, microbatches: int, use_graphs: bool = False, null_executor: bool = False, device: int = 0,
                 one_way_handoff: bool = False, copy_gradients: bool = False, replay_on_caller: bool = False,
                 graph_inputs: int = GRAPH_INPUTS_REBIND):
        cfg = Config(device, microbatches, int(use_graphs), int(null_executor), int(one_way_handoff),
                     int(copy_gradients), int(replay_on_caller), int(graph_inputs))
        h = C.c_void_p()
        st = _st(lib().qe_ctx_create(C.byref(cfg), C.byref(h)))
        if st != "OK":
            raise RuntimeError(f"qe_ctx_create failed: {st}")
        self.h = h
        self.null = null_executor

    def close(self):
        if self.h:
            lib().qe_ctx_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def qe_layer_register(self, stage: int, unit: int, n_out: int, k_in: int, max_tokens: int, w, w_dtype: int,
                          history_len: int, margin: int, fmt_x: int = E4M3, fmt_w: int = E4M3,
                          fmt_dy: int = E5M2, scaling: int = SCALING_DELAYED):
        d = LayerDesc(stage, unit, n_out, k_in, max_tokens, ptr(w), w_dtype, history_len, margin, fmt_x, fmt_w,
                      fmt_dy, scaling)
        out = C.c_int32()
        return _st(lib().qe_layer_register(self.h, C.byref(d), C.byref(out))), out.value

    def qe_layer_meta(self, layer: int, role: int) -> FP8Meta:
        m = FP8Meta()
        st = _st(lib().qe_layer_meta(self.h, layer, role, C.byref(m)))
        if st != "OK":
            raise RuntimeError(st)
        return m

    def qe_layer_cache(self, layer: int):
        w, wt, s = C.c_void_p(), C.c_void_p(), C.c_void_p()
        lw, lwt = C.c_int64(), C.c_int64()
        _st(lib().qe_layer_cache(self.h, layer, C.byref(w), C.byref(lw), C.byref(wt), C.byref(lwt), C.byref(s)))
        return {"w_q": w.value, "ld_w_q": lw.value, "w_q_t": wt.value, "ld_w_q_t": lwt.value, "w_scale_inv": s.value}

    def qe_layer_slot_payload(self, layer: int, slot: int):
        x, dy, sx, sdy = C.c_void_p(), C.c_void_p(), C.c_void_p(), C.c_void_p()
        lx, ldy = C.c_int64(), C.c_int64()
        _st(lib().qe_layer_slot_payload(self.h, layer, slot, C.byref(x), C.byref(lx), C.byref(dy), C.byref(ldy),
                                        C.byref(sx), C.byref(sdy)))
        return {"x_q_t": x.value, "ld_x_q_t": lx.value, "dy_q_t": dy.value, "ld_dy_q_t": ldy.value,
                "x_scale_inv": sx.value, "dy_scale_inv": sdy.value}

    def qe_fp8_linear_fwd(self, layer: int, k: TapeKey, x, x_dtype: int, tokens: int, y, y_dtype: int,
                          caller=None):
        ref = TapeRef()
        st = _st(lib().qe_fp8_linear_fwd(self.h, layer, k, ptr(x), x_dtype, tokens, ptr(y), y_dtype, C.byref(ref),
                                         self._caller(caller)))
        return st, (ref.astuple() if st == "OK" else None)

    def qe_fp8_linear_dgrad(self, layer: int, k: TapeKey, ref, dy, dy_dtype: int, dx, dx_dtype: int,
                            caller=None) -> str:
        return _st(lib().qe_fp8_linear_dgrad(self.h, layer, k, TapeRef(*ref), ptr(dy), dy_dtype, ptr(dx), dx_dtype,
                                             self._caller(caller)))

    def qe_fp8_linear_wgrad_place(self, layer: int, k: TapeKey, ref, main_grad, offset: int, ld: int, mode: int,
                                  caller=None) -> str:
        return _st(lib().qe_fp8_linear_wgrad_place(self.h, layer, k, TapeRef(*ref), ptr(main_grad), offset, ld,
                                                   mode, self._caller(caller)))

    def qe_fp8_linear_bwd_full(self, layer: int, k: TapeKey, ref, dy, dy_dtype: int, dx, dx_dtype: int, main_grad,
                               offset: int, ld: int, mode: int, caller=None) -> str:
        return _st(lib().qe_fp8_linear_bwd_full(self.h, layer, k, TapeRef(*ref), ptr(dy), dy_dtype, ptr(dx),
                                                dx_dtype, ptr(main_grad), offset, ld, mode, self._caller(caller)))

    def qe_arena_bind(self, layer: int, microbatch: int, buf, buf_elems: int, offset: int, ld: int) -> str:
        return _st(lib().qe_arena_bind(self.h, layer, microbatch, ptr(buf), buf_elems, offset, ld))

    def qe_prebuild_graphs(self, tokens: int, x_dtype: int, y_dtype: int, dy_dtype: int, dx_dtype: int) -> str:
        d = PrebuildDesc(tokens, x_dtype, y_dtype, dy_dtype, dx_dtype)
        return _st(lib().qe_prebuild_graphs(self.h, C.byref(d)))

    def qe_arena_finalize(self) -> str:
        return _st(lib().qe_arena_finalize(self.h))

    def qe_optimizer_commit(self) -> str:
        return _st(lib().qe_optimizer_commit(self.h))

    def qe_abort_epoch(self) -> str:
        return _st(lib().qe_abort_epoch(self.h))

    def qe_arena_rebuild(self) -> str:
        return _st(lib().qe_arena_rebuild(self.h))

    def qe_checkpoint_export(self):
        """(status, payload bytes or None)."""
        size = C.c_int64()
        st = _st(lib().qe_checkpoint_export(self.h, None, 0, C.byref(size)))
        if st != "OK":
            return st, None
        buf = C.create_string_buffer(size.value)
        st = _st(lib().qe_checkpoint_export(self.h, buf, size.value, C.byref(size)))
        return (st, buf.raw[: size.value]) if st == "OK" else (st, None)

    def qe_checkpoint_import(self, payload: bytes) -> str:
        buf = C.create_string_buffer(payload, len(payload))
        return _st(lib().qe_checkpoint_import(self.h, buf, len(payload)))

    def qe_sync(self) -> str:
        return _st(lib().qe_sync(self.h))

    def qe_inject_fault(self, n: int) -> str:
        return _st(lib().qe_inject_fault(self.h, n))

    def qe_set_kernel_timing(self, enable: bool) -> str:
        return _st(lib().qe_set_kernel_timing(self.h, int(enable)))

    def qe_get_kernel_timing(self, kernel_class: int):
        """(total milliseconds, launches) of one kernel class; raises on a non-OK status."""
        ms, n = C.c_double(), C.c_int64()
        st = _st(lib().qe_get_kernel_timing(self.h, kernel_class, C.byref(ms), C.byref(n)))
        if st != "OK":
            raise RuntimeError(f"qe_get_kernel_timing: {st}")
        return ms.value, n.value

    def qe_get_state(self) -> dict:
        s = CtxState()
        lib().qe_get_state(self.h, C.byref(s))
        return {f: getattr(s, f) for f, _ in CtxState._fields_}

    def qe_get_layer_state(self, layer: int) -> dict:
        s = LayerState()
        lib().qe_get_layer_state(self.h, layer, C.byref(s))
        return {"e_c": s.e_c, "refreshes": s.refreshes, "n_slots": s.n_slots}

    def qe_get_slot_state(self, layer: int, slot: int) -> dict:
        s = SlotState()
        lib().qe_get_slot_state(self.h, layer, slot, C.byref(s))
        return {"live": bool(s.live), "generation": s.generation, "bits": s.bits, "key": s.key.astuple(),
                "tokens": s.tokens, "bound": bool(s.bound), "written": bool(s.written),
                "view_offset": s.view_offset, "view_ld": s.view_ld, "view_buf": s.view_buf or 0}

    def _caller(self, caller) -> int:
        if self.null:
            return 0
        return stream_handle(caller)


def qe_status_str(code: int) -> str:
    return lib().qe_status_str(code).decode()


def exported_symbols():
    """Names of the C entry points this binding forwards to."""
    return sorted(list(_SIGS) + ["qe_ctx_destroy", "qe_status_str"])
