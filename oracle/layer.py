"""A stage of FP8 linears driven through F / dI / dW actions in schedule order.

Each action follows Algorithm 1 (§4.1): check through the contract, run the
physical work, commit.  The physical work is §3.2's transition:

F(m):  [first forward of an epoch only] quantize W with the W scale, keep
       W_q, W_q^T and the W scale_inv as the cache, record amax(W);
       quantize X_m with the X scale, keep X_q^T and the X scale_inv in slot m,
       record amax(X_m); Y_m = X_q W_q^T; then one scale update of the X and W
       roles (S0 -> S1).
dI(m): quantize dY_m with the dY scale, keep dY_q^T and the dY scale_inv in
       slot m, record amax(dY_m); dX_m = dY_q (W_q^T)^T; then one scale
       update of the dY role (S1 -> S2).  dY is quantized once, here.
dW(m): dW_m = dY_q^T X_q using the two scale_inv values kept in slot m, never
       the live scales; placed into the bound arena view; no state update.

The W role is updated with every forward but records an amax only when the
cache is refreshed (§2.1: the quantized weight is cached across microbatches
and refreshed only in the first forward after an optimizer step).

A layer with current (dynamic) scaling runs the same actions, but each tensor
is cast with a scale set from its own amax just before the cast (X in F, W on
a cache refresh, dY in dI); there is no history and nothing is recorded.

A checkpoint (§3.5) is the persistent part of the stage: e_W, each layer's
static configuration and precision recipe, and the FP8 state of its three
roles.  The weight cache, tapes and token are rebuilt by the process that
restores it; the restore marks the caches stale so the first forward
re-quantizes W with the restored W scale, exactly as the first forward after
any optimizer commit does.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional

import numpy as np

from . import contract as C
from .gemm import gemm_tn, place, quantize_with_amax
from .scaling import CurrentScaler, DelayedScaler


@dataclasses.dataclass
class Payload:
    xq_t: Optional[np.ndarray] = None     # [K, tokens] codes
    x_scale_inv: float = 1.0
    dyq_t: Optional[np.ndarray] = None    # [N, tokens] codes
    dy_scale_inv: float = 1.0


class OracleLayer:
    def __init__(self, w_f32: np.ndarray, history: int, margin: int, fmt_x: str, fmt_w: str, fmt_dy: str,
                 microbatches: int, scaling: str = "delayed"):
        self.w = np.asarray(w_f32, dtype=np.float32)
        self.fmt_x, self.fmt_w, self.fmt_dy = fmt_x, fmt_w, fmt_dy
        if scaling not in ("delayed", "current"):
            raise ValueError(scaling)
        self.current = scaling == "current"
        self.scaling, self.history, self.margin = scaling, int(history), int(margin)
        if self.current:
            self.sx = CurrentScaler(fmt_x, margin)
            self.sw = CurrentScaler(fmt_w, margin)
            self.sdy = CurrentScaler(fmt_dy, margin)
        else:
            self.sx = DelayedScaler(fmt_x, history, margin)
            self.sw = DelayedScaler(fmt_w, history, margin)
            self.sdy = DelayedScaler(fmt_dy, history, margin)
        self.wq = self.wq_t = None
        self.w_scale_inv = 1.0
        self.payload: List[Payload] = [Payload() for _ in range(microbatches)]


class Stage:
    """One pipeline stage: its linears, its contract and their FP8 state."""

    def __init__(self, microbatches: int):
        self.contract = C.Contract(microbatches)
        self.layers: List[OracleLayer] = []
        self.arena: Dict[int, np.ndarray] = {}   # buffer address -> float32 flat buffer

    def add_layer(self, stage: int, unit: int, w_f32: np.ndarray, max_tokens: int, history: int, margin: int,
                  fmt_x: str = "E4M3", fmt_w: str = "E4M3", fmt_dy: str = "E5M2", scaling: str = "delayed") -> int:
        n, k = w_f32.shape
        idx = self.contract.add_layer(stage, unit, n, k, max_tokens)
        self.layers.append(OracleLayer(w_f32, history, margin, fmt_x, fmt_w, fmt_dy, self.contract.M, scaling))
        return idx

    def set_weight(self, layer: int, w_f32: np.ndarray) -> None:
        """In-place master-weight update between finalize and commit."""
        self.layers[layer].w = np.asarray(w_f32, dtype=np.float32)

    def add_buffer(self, address: int, elems: int, init: Optional[np.ndarray] = None) -> np.ndarray:
        buf = np.zeros(elems, dtype=np.float32) if init is None else np.array(init, dtype=np.float32)
        self.arena[address] = buf
        return buf

    # ---------------------------------------------------------------- F
    def fwd(self, layer: int, key, x_f32: np.ndarray):
        x_f32 = np.asarray(x_f32, dtype=np.float32)
        tokens = x_f32.shape[0]
        st, refresh = self.contract.check_fwd(layer, key, tokens)
        if st != C.OK:
            return st, None, None
        if self.contract._physical_fails():
            self.contract.abort()
            return C.EXEC_FAILED, None, None
        L = self.layers[layer]
        if L.current:
            if refresh:
                L.sw.set_from(L.w)
                L.wq, L.wq_t, _ = quantize_with_amax(L.w, L.sw.scale, L.fmt_w)
                L.w_scale_inv = L.sw.scale_inv
            L.sx.set_from(x_f32)
            xq, xq_t, _ = quantize_with_amax(x_f32, L.sx.scale, L.fmt_x)
            P = L.payload[key[2]]
            P.xq_t, P.x_scale_inv = xq_t, L.sx.scale_inv
            y = gemm_tn(xq, L.fmt_x, L.wq, L.fmt_w, P.x_scale_inv, L.w_scale_inv)
            ref = self.contract.commit_fwd(layer, key, tokens, refresh)
            return C.OK, y, ref
        if refresh:
            L.wq, L.wq_t, a_w = quantize_with_amax(L.w, L.sw.scale, L.fmt_w)
            L.w_scale_inv = L.sw.scale_inv
            L.sw.record(a_w)
        xq, xq_t, a_x = quantize_with_amax(x_f32, L.sx.scale, L.fmt_x)
        P = L.payload[key[2]]
        P.xq_t, P.x_scale_inv = xq_t, L.sx.scale_inv
        L.sx.record(a_x)
        y = gemm_tn(xq, L.fmt_x, L.wq, L.fmt_w, P.x_scale_inv, L.w_scale_inv)
        L.sx.update()
        L.sw.update()
        ref = self.contract.commit_fwd(layer, key, tokens, refresh)
        return C.OK, y, ref

    # ---------------------------------------------------------------- dI
    def _dgrad_physical(self, layer: int, ref, dy_f32: np.ndarray):
        L = self.layers[layer]
        P = L.payload[ref[0]]
        if L.current:
            L.sdy.set_from(dy_f32)
        dyq, dyq_t, a_dy = quantize_with_amax(dy_f32, L.sdy.scale, L.fmt_dy)
        P.dyq_t, P.dy_scale_inv = dyq_t, L.sdy.scale_inv
        dx = gemm_tn(dyq, L.fmt_dy, L.wq_t, L.fmt_w, P.dy_scale_inv, L.w_scale_inv)
        if not L.current:
            L.sdy.record(a_dy)
            L.sdy.update()
        return dx

    def dgrad(self, layer: int, key, ref, dy_f32: np.ndarray):
        st = self.contract.check_dgrad(layer, key, ref)
        if st != C.OK:
            return st, None
        dy_f32 = np.asarray(dy_f32, dtype=np.float32)
        assert dy_f32.shape == (self.contract.layers[layer].slots[ref[0]].tokens, self.contract.layers[layer].n)
        if self.contract._physical_fails():
            self.contract.abort()
            return C.EXEC_FAILED, None
        dx = self._dgrad_physical(layer, ref, dy_f32)
        self.contract.commit_dgrad(layer, ref)
        return C.OK, dx

    # ---------------------------------------------------------------- dW
    def _wgrad_physical(self, layer: int, ref, buf: int, offset: int, ld: int, mode: int):
        L = self.layers[layer]
        P = L.payload[ref[0]]
        d = gemm_tn(P.dyq_t, L.fmt_dy, P.xq_t, L.fmt_x, P.dy_scale_inv, P.x_scale_inv)
        place(self.arena[buf], d, offset, ld, accumulate=(mode == C.ACCUM))
        return d

    def wgrad_place(self, layer: int, key, ref, buf: int, offset: int, ld: int, mode: int):
        st = self.contract.check_wgrad(layer, key, ref, buf, offset, ld, mode)
        if st != C.OK:
            return st
        if self.contract._physical_fails():
            self.contract.abort()
            return C.EXEC_FAILED
        self._wgrad_physical(layer, ref, buf, offset, ld, mode)
        self.layers[layer].payload[ref[0]] = Payload()
        self.contract.commit_wgrad(layer, ref)
        return C.OK

    # ---------------------------------------------------------------- dI immediately followed by dW
    def bwd_full(self, layer: int, key, ref, dy_f32: np.ndarray, buf: int, offset: int, ld: int, mode: int):
        st = self.contract.check_bwd_full(layer, key, ref, buf, offset, ld, mode)
        if st != C.OK:
            return st, None
        dy_f32 = np.asarray(dy_f32, dtype=np.float32)
        assert dy_f32.shape == (self.contract.layers[layer].slots[ref[0]].tokens, self.contract.layers[layer].n)
        if self.contract._physical_fails():
            self.contract.abort()
            return C.EXEC_FAILED, None
        dx = self._dgrad_physical(layer, ref, dy_f32)
        self._wgrad_physical(layer, ref, buf, offset, ld, mode)
        self.layers[layer].payload[ref[0]] = Payload()
        self.contract.commit_bwd_full(layer, ref)
        return C.OK, dx

    # ---------------------------------------------------------------- arena / epoch
    def bind(self, layer: int, m: int, buf: int, offset: int, ld: int) -> str:
        return self.contract.bind(layer, m, buf, self.arena[buf].size, offset, ld)

    def finalize(self) -> str:
        return self.contract.finalize()

    def optimizer_commit(self) -> str:
        return self.contract.optimizer_commit()

    def abort(self) -> None:
        self.contract.abort()

    def rebuild(self) -> str:
        return self.contract.rebuild()

    # ---------------------------------------------------------------- checkpoint
    def checkpoint_export(self):
        """(status, payload): the persistent state, only at a quiescent point."""
        st = self.contract.checkpoint_check()
        if st != C.OK:
            return st, None
        layers = []
        for info, L in zip(self.contract.layers, self.layers):
            roles = {}
            for r, s in (("x", L.sx), ("w", L.sw), ("dy", L.sdy)):
                hist = np.zeros(1) if L.current else s.hist.copy()
                roles[r] = (hist, s.scale, s.scale_inv)
            layers.append({"stage": info.stage, "unit": info.unit, "n": info.n, "k": info.k,
                           "max_tokens": info.max_tokens, "history": L.history, "margin": L.margin,
                           "fmts": (L.fmt_x, L.fmt_w, L.fmt_dy), "scaling": L.scaling, "roles": roles})
        return C.OK, {"e_w": self.contract.e_w, "microbatches": self.contract.M, "layers": layers}

    def checkpoint_import(self, payload) -> str:
        """Restore a payload into this process's stage, whose layers were
        registered with the same configuration; nothing changes on a mismatch
        or when the stage is not quiescent."""
        if payload["microbatches"] != self.contract.M or len(payload["layers"]) != len(self.layers):
            return C.INVALID_ARG
        for p, info, L in zip(payload["layers"], self.contract.layers, self.layers):
            mine = (info.stage, info.unit, info.n, info.k, info.max_tokens, L.history, L.margin,
                    (L.fmt_x, L.fmt_w, L.fmt_dy), L.scaling)
            theirs = (p["stage"], p["unit"], p["n"], p["k"], p["max_tokens"], p["history"], p["margin"],
                      tuple(p["fmts"]), p["scaling"])
            if mine != theirs:
                return C.INVALID_ARG
        st = self.contract.checkpoint_check()
        if st != C.OK:
            return st
        for p, L in zip(payload["layers"], self.layers):
            for r, s in (("x", L.sx), ("w", L.sw), ("dy", L.sdy)):
                hist, scale, scale_inv = p["roles"][r]
                if not L.current:
                    s.hist = np.array(hist, dtype=np.float64)
                s.scale, s.scale_inv = float(scale), float(scale_inv)
            L.wq = L.wq_t = None
        return self.contract.restore(payload["e_w"])

    def fp8_state(self, layer: int) -> dict:
        L = self.layers[layer]
        if L.current:   # no history: a one-entry history that is always clear
            return {r: (np.zeros(1), s.scale, s.scale_inv) for r, s in (("x", L.sx), ("w", L.sw), ("dy", L.sdy))}
        return {r: (s.hist.copy(), s.scale, s.scale_inv) for r, s in (("x", L.sx), ("w", L.sw), ("dy", L.sdy))}
