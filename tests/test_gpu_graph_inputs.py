"""Static binding and dynamic inputs of the graph executor (§4.3 eq. G_r,
§4.4): qe_prebuild_graphs captures the G = 3 M L graphs of a stage up front,
and a caller that hands every action new X / dY / Y / dX buffers (rotated
each step, as activations and gradients are in a training loop) gets no
further capture: the call's buffers are bound into the existing graph, by
rewriting its kernel-node arguments (the default) or, in the paper's scheme,
by copies into and out of static library buffers.  Every replay must give the
bits the same actions give launched directly."""
import numpy as np
import pytest

import workloads as W
from tests.gpu_util import dev, torch, upload
from tests.libqe import need_lib
from tests.stage_driver import Spec

pytestmark = pytest.mark.gpu

M = 4
SPEC = Spec([(192, 160), (96, 272)], tokens=200, M=M, history=8, margin=0, in_dtype="bf16", shared_view=False,
            cfg=7)
SCHED = [("F", m) for m in range(M)] + [("dI", m) for m in range(M)] + [("dW", m) for m in reversed(range(M))]
STEPS = 3
ROT = 3  # buffer sets rotated over the steps


def _run(qe, use_graphs, graph_inputs=0, replay_on_caller=False, rotate=True, prebuild=True, current=False,
         full=False, copy_gradients=False, prebuild_tokens=0):
    """`full`: dI and dW of each microbatch as one full-backward action (in the dW slots of the
    schedule, dI slots skipped); `prebuild_tokens`: the token count the graphs are prebuilt for
    (0: the layers' max_tokens, which is what the calls use)."""
    d = dev()
    ctx = qe.Context(M, use_graphs=use_graphs, replay_on_caller=replay_on_caller, graph_inputs=graph_inputs,
                     copy_gradients=copy_gradients)
    L = len(SPEC.shapes)
    ws = [upload(SPEC.weight(u), d) for u in range(L)]
    for u, (n, k) in enumerate(SPEC.shapes):
        st, idx = ctx.qe_layer_register(0, u, n, k, SPEC.tokens, ws[u], qe.BF16, 1 if current else SPEC.history,
                                        SPEC.margin, scaling=qe.SCALING_CURRENT if current else qe.SCALING_DELAYED)
        assert st == "OK" and idx == u
    grad = torch.zeros(SPEC.grad_elems(), dtype=torch.float32, device=d)
    for u, (n, k) in enumerate(SPEC.shapes):
        for m in range(M):
            assert ctx.qe_arena_bind(u, m, grad, grad.numel(), SPEC.offset(u, m), k) == "OK"
    G = 3 * M * L
    if prebuild and use_graphs:
        assert ctx.qe_prebuild_graphs(prebuild_tokens, qe.BF16, qe.F32, qe.BF16, qe.F32) == "OK"
        st = ctx.qe_get_state()
        assert st["captures"] == G and st["graphs"] == G and st["prebuild_ns"] > 0, st
    t = SPEC.tokens
    # ROT distinct buffers per (layer, microbatch, tensor)
    bufs = {}
    for u, (n, k) in enumerate(SPEC.shapes):
        for m in range(M):
            bufs[("x", u, m)] = [torch.empty((t, k), dtype=torch.int16, device=d) for _ in range(ROT)]
            bufs[("dy", u, m)] = [torch.empty((t, n), dtype=torch.int16, device=d) for _ in range(ROT)]
            bufs[("y", u, m)] = [torch.empty((t, n), dtype=torch.float32, device=d) for _ in range(ROT)]
            bufs[("dx", u, m)] = [torch.empty((t, k), dtype=torch.float32, device=d) for _ in range(ROT)]
    outs, grads, rebinds = {}, [], []
    for step in range(STEPS):
        refs = {}
        for a, m in SCHED:
            for u, (n, k) in enumerate(SPEC.shapes):
                r = (step + m) % ROT if rotate else 0
                key = qe.key(step, 0, m, u)
                x, dy = SPEC.inputs(u, m, step)
                if a == "F":
                    xb, yb = bufs[("x", u, m)][r], bufs[("y", u, m)][r]
                    xb.copy_(upload(x, d))
                    yb.fill_(float("nan"))
                    st, refs[(u, m)] = ctx.qe_fp8_linear_fwd(u, key, xb, qe.BF16, t, yb, qe.F32)
                    assert st == "OK", (a, m, u, st)
                    outs[("y", step, u, m)] = yb.clone()
                elif a == "dI" and full:
                    continue
                elif a == "dW" and full:
                    dyb, dxb = bufs[("dy", u, m)][r], bufs[("dx", u, m)][r]
                    dyb.copy_(upload(dy, d))
                    dxb.fill_(float("nan"))
                    st = ctx.qe_fp8_linear_bwd_full(u, key, refs[(u, m)], dyb, qe.BF16, dxb, qe.F32, grad,
                                                    SPEC.offset(u, m), k, qe.INIT)
                    assert st == "OK", (a, m, u, st)
                    outs[("dx", step, u, m)] = dxb.clone()
                elif a == "dI":
                    dyb, dxb = bufs[("dy", u, m)][r], bufs[("dx", u, m)][r]
                    dyb.copy_(upload(dy, d))
                    dxb.fill_(float("nan"))
                    st = ctx.qe_fp8_linear_dgrad(u, key, refs[(u, m)], dyb, qe.BF16, dxb, qe.F32)
                    assert st == "OK", (a, m, u, st)
                    outs[("dx", step, u, m)] = dxb.clone()
                else:
                    st = ctx.qe_fp8_linear_wgrad_place(u, key, refs[(u, m)], grad, SPEC.offset(u, m), k, qe.INIT)
                    assert st == "OK", (a, m, u, st)
        assert ctx.qe_arena_finalize() == "OK"
        torch.cuda.synchronize()
        grads.append(grad.cpu().numpy().copy())
        for u in range(L):  # a new weight version, in place
            ws[u].copy_(upload(W.normal(W.rng_for(1, 7, u, W.ROLE_W, 0, step), SPEC.shapes[u], 0.02, "bf16"), d))
        torch.cuda.synchronize()
        assert ctx.qe_optimizer_commit() == "OK"
        rebinds.append(ctx.qe_get_state()["rebinds"])
    assert ctx.qe_sync() == "OK"
    st = ctx.qe_get_state()
    assert st["device_token"] == st["token"]
    host = {k: v.cpu().numpy() for k, v in outs.items()}
    ctx.close()
    return host, grads, st, rebinds


def _same(ref, got):
    assert ref[0].keys() == got[0].keys()
    for k in ref[0]:
        np.testing.assert_array_equal(ref[0][k].view(np.uint32), got[0][k].view(np.uint32), err_msg=str(k))
    for a, b in zip(ref[1], got[1]):
        np.testing.assert_array_equal(a.view(np.uint32), b.view(np.uint32))


@pytest.mark.parametrize("replay_on_caller", [False, True], ids=["graph_stream", "caller_stream"])
def test_rotating_buffers_rebind_without_capture(replay_on_caller):
    qe = need_lib()
    ref = _run(qe, use_graphs=False, replay_on_caller=replay_on_caller)
    got = _run(qe, use_graphs=True, graph_inputs=qe.GRAPH_INPUTS_REBIND, replay_on_caller=replay_on_caller)
    _same(ref, got)
    st = got[2]
    G = 3 * M * len(SPEC.shapes)
    assert st["captures"] == G and st["graphs"] == G, st
    assert st["replays"] == STEPS * G
    # every F and dI graph is rebound in every step (its buffers rotate); dW graphs never (their view is fixed)
    assert got[3] == [2 * M * len(SPEC.shapes) * (s + 1) for s in range(STEPS)], got[3]


def test_fixed_buffers_bind_once():
    qe = need_lib()
    got = _run(qe, use_graphs=True, graph_inputs=qe.GRAPH_INPUTS_REBIND, rotate=False)
    G = 3 * M * len(SPEC.shapes)
    assert got[2]["captures"] == G
    # the first call of each F / dI binds its buffers into the prebuilt graph; later calls change nothing
    assert got[3] == [2 * M * len(SPEC.shapes)] * STEPS, got[3]
    _same(_run(qe, use_graphs=False, rotate=False), got)


def test_paper_static_buffers_with_copies():
    qe = need_lib()
    ref = _run(qe, use_graphs=False)
    got = _run(qe, use_graphs=True, graph_inputs=qe.GRAPH_INPUTS_COPY)
    _same(ref, got)
    G = 3 * M * len(SPEC.shapes)
    assert got[2]["captures"] == G and got[2]["rebinds"] == 0


def test_recapture_mode_and_no_prebuild():
    qe = need_lib()
    ref = _run(qe, use_graphs=False)
    got = _run(qe, use_graphs=True, graph_inputs=qe.GRAPH_INPUTS_RECAPTURE)
    _same(ref, got)
    G = 3 * M * len(SPEC.shapes)
    assert got[2]["captures"] > G and got[2]["rebinds"] == 0
    lazy = _run(qe, use_graphs=True, prebuild=False)
    _same(ref, lazy)
    assert lazy[2]["captures"] == G  # captured on first use, then rebound


@pytest.mark.parametrize("variant", ["current_scaling", "full_backward", "copied_gradients"])
def test_rotating_buffers_other_plans(variant):
    """The same rotation on the other kernel sequences an action can have: current
    scaling (amax pass, update, cast, GEMM), the full backward (dI and dW in one
    action, with the graphs of its own key captured on first use) and the
    copied-gradient path (GEMM into the private buffer, then the copy kernel)."""
    qe = need_lib()
    kw = {"current": variant == "current_scaling", "full": variant == "full_backward",
          "copy_gradients": variant == "copied_gradients"}
    ref = _run(qe, use_graphs=False, **kw)
    got = _run(qe, use_graphs=True, graph_inputs=qe.GRAPH_INPUTS_REBIND, **kw)
    _same(ref, got)
    G = 3 * M * len(SPEC.shapes)
    if variant == "full_backward":
        # F graphs prebuilt and rebound; dI / dW graphs prebuilt but unused; one full-backward graph per
        # (layer, slot) captured on first use and rebound afterwards
        assert got[2]["captures"] == G + M * len(SPEC.shapes), got[2]
    else:
        assert got[2]["captures"] == G, got[2]
    assert got[2]["rebinds"] > 0


def test_prebuilt_for_other_token_count_recaptures_once():
    """Graphs prebuilt for fewer tokens than the calls use have another launch
    shape: each is captured again on its first use (bits unchanged), then only
    rebound."""
    qe = need_lib()
    ref = _run(qe, use_graphs=False)
    got = _run(qe, use_graphs=True, prebuild_tokens=SPEC.tokens - 72)
    _same(ref, got)
    G = 3 * M * len(SPEC.shapes)
    assert G < got[2]["captures"] <= 2 * G, got[2]
