"""Quiescent checkpoint on the GPU (§3.5, Invariant 4): a stage saved at an
optimizer boundary and restored into a fresh context reproduces the
uninterrupted run bit for bit (outputs, placed gradients, FP8 state) across
an amax-history rollover, in eager and graph mode, for delayed and current
scaling; both runs match the oracle at every step, the oracle going through
its own checkpoint."""
import numpy as np
import pytest

from tests import schedules as S
from tests.gpu_util import dev, rel_err, torch
from tests.libqe import need_lib
from tests.stage_driver import GpuStage, OracleStage, Spec
from tests.test_gpu_layer import compare_state

pytestmark = pytest.mark.gpu


def _steps(kind, n):
    if kind == "single":
        return [S.SINGLE] * n
    return [S.ZB_STEP0 if i % 2 == 0 else S.ZB_STEP1 for i in range(n)]


def _spec(kind, scaling):
    H = 1 if scaling == "current" else 4
    if kind == "single":
        return Spec([(256, 256)], tokens=128, M=2, history=H, margin=0, in_dtype="f32", shared_view=True, cfg=0,
                    scaling=scaling)
    return Spec([(96, 160), (72, 200)], tokens=48, M=8, history=H, margin=0, in_dtype="bf16", shared_view=False,
                cfg=2, scaling=scaling)


def _run(spec, kind, total, use_graphs, save_after=None):
    qe = need_lib()
    d = dev()
    g, o = GpuStage(qe, spec, use_graphs=use_graphs, device=d), OracleStage(spec)
    outs, grads, states, w = {}, [], [], None
    for step, sched in enumerate(_steps(kind, total)):
        if step == save_after:
            torch.cuda.synchronize()
            st, payload = g.ctx.qe_checkpoint_export()
            assert st == "OK" and payload is not None
            ost, opayload = o.st.checkpoint_export()
            g.ctx.close()
            g = GpuStage(qe, spec, use_graphs=use_graphs, device=d, weights=w)
            assert g.ctx.qe_checkpoint_import(payload) == "OK"
            cs = g.ctx.qe_get_state()
            assert cs["e_w"] == step and cs["token"] == 0
            o = OracleStage(spec, weights=w)
            assert o.st.checkpoint_import(opayload) == "OK"
            compare_state_no_cache(g, o, spec)
        g.run(sched, step, step)
        o.run(sched, step, step)
        torch.cuda.synchronize()
        compare_state(g, o, spec)
        grads.append(g.grad.cpu().numpy().copy())
        assert rel_err(grads[-1], o.st.arena[o.buf]) <= 1e-3
        for k, v in g.outs.items():
            outs[k] = v.cpu().numpy().copy()
        for k, ref in o.outs.items():
            got = outs[k]
            assert rel_err(got, ref) <= 1e-3, k
        states.append([g.fp8_state(u) for u in range(len(spec.shapes))])
        w = o.sgd_weights()
        g.end_step(w)
        o.end_step(w)
        g.outs, o.outs = {}, {}
    assert g.ctx.qe_sync() == "OK"
    cs = g.ctx.qe_get_state()
    assert cs["device_token"] == cs["token"]
    if save_after is not None:
        assert g.ctx.qe_get_layer_state(0)["refreshes"] == total - save_after
    return outs, grads, states


def compare_state_no_cache(g, o, spec):
    """FP8 state right after a restore (the weight cache is stale, not compared)."""
    for u in range(len(spec.shapes)):
        gs, os_ = g.fp8_state(u), o.st.fp8_state(u)
        for r in ("x", "w", "dy"):
            np.testing.assert_array_equal(gs[r][0], os_[r][0].astype(np.float32))
            assert gs[r][1] == os_[r][1] and gs[r][2] == os_[r][2]
        assert g.ctx.qe_get_layer_state(u)["e_c"] == -1


@pytest.mark.parametrize("use_graphs", [False, True])
@pytest.mark.parametrize("scaling", ["delayed", "current"])
@pytest.mark.parametrize("kind", ["single", "zb"])
def test_resume_bitwise_equals_uninterrupted(kind, scaling, use_graphs):
    spec = _spec(kind, scaling)
    total, save = 6, 3
    full = _run(spec, kind, total, use_graphs)
    resumed = _run(spec, kind, total, use_graphs, save_after=save)
    for k in full[0]:
        if k[3] >= save:
            np.testing.assert_array_equal(full[0][k], resumed[0][k], err_msg=str(k))
    for a, b in zip(full[1][save:], resumed[1][save:]):
        np.testing.assert_array_equal(a.view(np.uint32), b.view(np.uint32))
    for sa, sb in zip(full[2][save:], resumed[2][save:]):
        for x, y in zip(sa, sb):
            for r in x:
                np.testing.assert_array_equal(x[r][0], y[r][0])
                assert x[r][1:] == y[r][1:]


def test_checkpoint_withheld_with_live_tape_on_gpu():
    qe = need_lib()
    spec = _spec("single", "delayed")
    g = GpuStage(qe, spec, device=dev())
    g.run([("F", 0)], 0, 0)
    snap = g.ctx.qe_get_state()
    assert g.ctx.qe_checkpoint_export() == ("NOT_QUIESCENT", None)
    assert g.ctx.qe_get_state() == snap
    g.run([("dI", 0), ("dW", 0), ("F", 1), ("dI", 1), ("dW", 1)], 0, 0)
    assert g.ctx.qe_checkpoint_export()[0] == "NOT_QUIESCENT"
    g.end_step()
    assert g.ctx.qe_checkpoint_export()[0] == "OK"
