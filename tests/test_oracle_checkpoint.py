"""Pins for the oracle's quiescent checkpoint (§3.5, Invariant 4, Table
"faults"): a run saved at an optimizer boundary and resumed in a fresh stage
reproduces the uninterrupted run bit for bit across an amax-history rollover;
dropping any persistent part breaks that; live work withholds the checkpoint;
process-local state (token, generations, cache) is rebuilt."""
import copy

import numpy as np
import pytest

import workloads as W
from oracle import contract as OC
from tests import schedules as S
from tests.stage_driver import OracleStage, Spec


class ShrinkingSpec(Spec):
    """Activations 16x smaller every step (exact: a power of two), so the
    delayed scale depends on which past amaxes the history still holds."""

    def inputs(self, u, m, step):
        x, dy = super().inputs(u, m, step)
        return W.Tensor(x.data * np.float32(16.0 ** -step), x.dtype), dy


def _spec(kind, scaling):
    if kind == "single":
        return Spec([(24, 40)], tokens=16, M=2, history=1 if scaling == "current" else 4, margin=0,
                    in_dtype="f32", shared_view=True, cfg=0, scaling=scaling)
    return Spec([(24, 40), (16, 24)], tokens=8, M=8, history=1 if scaling == "current" else 4, margin=0,
                in_dtype="bf16", shared_view=False, cfg=2, scaling=scaling)


def _steps(kind, n):
    if kind == "single":
        return [S.SINGLE] * n
    return [S.ZB_STEP0 if i % 2 == 0 else S.ZB_STEP1 for i in range(n)]


def _run(o, spec, steps, first_step):
    for i, sched in enumerate(steps):
        step = first_step + i
        o.run(sched, step, step)
        new_w = o.sgd_weights()
        o.end_step(new_w)
        yield step, new_w


def _state(o):
    return ({k: v.copy() for k, v in o.outs.items()}, o.st.arena[o.buf].copy(),
            [o.st.fp8_state(u) for u in range(len(o.spec.shapes))])


def _assert_same(a, b, from_step):
    outs_a, grad_a, fp8_a = a
    outs_b, grad_b, fp8_b = b
    keys = [k for k in outs_a if k[3] >= from_step]
    assert keys and all(k in outs_b for k in keys)
    for k in keys:
        np.testing.assert_array_equal(outs_a[k], outs_b[k], err_msg=str(k))
    np.testing.assert_array_equal(grad_a, grad_b)
    for x, y in zip(fp8_a, fp8_b):
        for r in x:
            np.testing.assert_array_equal(x[r][0], y[r][0])
            assert x[r][1:] == y[r][1:]


def _resume(spec, kind, save_after, total, drop=None):
    o = OracleStage(spec)
    w = None
    for _, w in _run(o, spec, _steps(kind, save_after), 0):
        pass
    st, payload = o.st.checkpoint_export()
    assert st == OC.OK
    if drop is not None:
        payload = drop(copy.deepcopy(payload))
    r = OracleStage(spec, weights=w)
    assert r.st.checkpoint_import(payload) == OC.OK
    for _ in _run(r, spec, _steps(kind, total)[save_after:], save_after):
        pass
    return r


@pytest.mark.parametrize("kind", ["single", "zb", "shrinking"])
@pytest.mark.parametrize("scaling", ["delayed", "current"])
def test_resume_reproduces_uninterrupted_run(kind, scaling):
    """Save at step 3 and continue through step 6 (the history of 4 rolls over)."""
    spec = _spec(kind, scaling)
    if kind == "shrinking":
        spec = ShrinkingSpec([(24, 40)], tokens=16, M=2, history=1 if scaling == "current" else 4, margin=0,
                             in_dtype="f32", shared_view=True, cfg=0, scaling=scaling)
        kind = "single"
    full = OracleStage(spec)
    for _ in _run(full, spec, _steps(kind, 6), 0):
        pass
    r = _resume(spec, kind, 3, 6)
    _assert_same(_state(full), _state(r), 3)
    assert r.st.contract.e_w == full.st.contract.e_w == 6


def _drop_history(p):
    for L in p["layers"]:
        for r in L["roles"]:
            h, s, si = L["roles"][r]
            L["roles"][r] = (np.zeros_like(h), s, si)
    return p


def _drop_scales(p):
    for L in p["layers"]:
        for r in L["roles"]:
            h, s, si = L["roles"][r]
            L["roles"][r] = (h, 1.0, 1.0)
    return p


def _drop_epoch(p):
    p["e_w"] = 0
    return p


@pytest.mark.parametrize("drop", [_drop_history, _drop_scales, _drop_epoch])
def test_each_persistent_part_is_needed(drop):
    """Losing the history, the scales or e_W makes the resumed run differ (or be rejected)."""
    spec = ShrinkingSpec([(24, 40)], tokens=16, M=2, history=4, margin=0, in_dtype="f32", shared_view=True, cfg=0)
    full = OracleStage(spec)
    for _ in _run(full, spec, _steps("single", 6), 0):
        pass
    if drop is _drop_epoch:
        with pytest.raises(AssertionError):      # keys of epoch 3 are rejected with EPOCH
            _resume(spec, "single", 3, 6, drop)
        return
    r = _resume(spec, "single", 3, 6, drop)
    with pytest.raises(AssertionError):
        _assert_same(_state(full), _state(r), 3)


def test_live_work_withholds_checkpoint():
    """Table "faults": a live tape, an arena write in flight or a finalized,
    uncommitted epoch withholds the checkpoint and changes nothing."""
    spec = _spec("single", "delayed")
    o = OracleStage(spec)
    x, dy = spec.inputs(0, 0, 0)
    st, _, ref = o.st.fwd(0, (0, 0, 0, 0, 0), x.as_f32())
    snap = o.st.contract.snapshot()
    assert o.st.checkpoint_export() == (OC.NOT_QUIESCENT, None)
    assert o.st.contract.snapshot() == snap
    assert o.st.dgrad(0, (0, 0, 0, 0, 0), ref, dy.as_f32())[0] == OC.OK
    assert o.st.checkpoint_export()[0] == OC.NOT_QUIESCENT
    assert o.st.wgrad_place(0, (0, 0, 0, 0, 0), ref, o.buf, 0, 40, OC.INIT) == OC.OK
    assert o.st.checkpoint_export()[0] == OC.NOT_QUIESCENT       # view written, epoch open
    o.run([("F", 1), ("dI", 1), ("dW", 1)], 0, 0)
    assert o.st.finalize() == OC.OK
    assert o.st.checkpoint_export()[0] == OC.NOT_QUIESCENT       # finalized, not committed
    assert o.st.optimizer_commit() == OC.OK
    assert o.st.checkpoint_export()[0] == OC.OK
    # an aborted epoch leaves the arena invalid until rebuilt
    o.st.fwd(0, (1, 0, 0, 0, 0), x.as_f32())
    o.st.abort()
    assert o.st.checkpoint_export()[0] == OC.ARENA_INVALID
    assert o.st.rebuild() == OC.OK
    assert o.st.checkpoint_export()[0] == OC.OK


def test_restore_rebuilds_process_local_state():
    """After a restore: e_W is the saved one, the token and generations are the
    new process's, the cache is stale (a non-first forward is refused and the
    first forward refreshes), and import into a busy stage is refused."""
    spec = _spec("single", "delayed")
    o = OracleStage(spec)
    w = None
    for _, w in _run(o, spec, _steps("single", 2), 0):
        pass
    _, payload = o.st.checkpoint_export()
    r = OracleStage(spec, weights=w)
    assert r.st.checkpoint_import(payload) == OC.OK
    c = r.st.contract
    assert (c.e_w, c.token, c.layers[0].e_c) == (2, 0, -1)
    x, _ = spec.inputs(0, 1, 2)
    assert r.st.fwd(0, (2, 0, 1, 0, 0), x.as_f32())[0] == OC.STALE_CACHE
    x, _ = spec.inputs(0, 0, 2)
    st, _, ref = r.st.fwd(0, (2, 0, 0, 0, 0), x.as_f32())
    assert st == OC.OK and ref == (0, 1) and c.layers[0].refreshes == 1 and c.layers[0].e_c == 2
    assert r.st.checkpoint_import(payload) == OC.NOT_QUIESCENT


def test_import_rejects_other_configuration():
    spec = _spec("single", "delayed")
    o = OracleStage(spec)
    _, payload = o.st.checkpoint_export()
    for field, value in (("n", 25), ("history", 8), ("margin", 1), ("scaling", "current"),
                         ("fmts", ("E4M3", "E4M3", "E4M3")), ("max_tokens", 17), ("unit", 3)):
        p = copy.deepcopy(payload)
        p["layers"][0][field] = value
        r = OracleStage(spec)
        snap = r.st.contract.snapshot()
        assert r.st.checkpoint_import(p) == OC.INVALID_ARG, field
        assert r.st.contract.snapshot() == snap
    p = copy.deepcopy(payload)
    p["microbatches"] = 3
    assert OracleStage(spec).st.checkpoint_import(p) == OC.INVALID_ARG
