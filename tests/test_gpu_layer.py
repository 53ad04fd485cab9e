"""End-to-end layer actions on the GPU against the oracle: every FP8 code,
amax history and scale bit-exact; Y, dX and the placed dW within 1e-3; the
contract state equal.  Also the split = full-backward identity and eager =
graph replay, both bitwise on the GPU."""
import numpy as np
import pytest

from tests import schedules as S
from tests.gpu_util import dev, rel_err, torch
from tests.libqe import need_lib
from tests.stage_driver import GpuStage, OracleStage, Spec

pytestmark = pytest.mark.gpu


def as_f32(t):
    a = t.cpu().numpy()
    if a.dtype == np.int16:
        return (a.view(np.uint16).astype(np.uint32) << 16).view(np.float32)
    return a


def compare_state(g, o, spec):
    for u in range(len(spec.shapes)):
        gs, os_ = g.fp8_state(u), o.st.fp8_state(u)
        for r in ("x", "w", "dy"):
            np.testing.assert_array_equal(gs[r][0], os_[r][0].astype(np.float32), err_msg=f"hist {r} layer {u}")
            assert gs[r][1] == os_[r][1] and gs[r][2] == os_[r][2], (r, u, gs[r][1:], os_[r][1:])
        wq, wqt = g.cache_codes(u)
        np.testing.assert_array_equal(wq, o.st.layers[u].wq)
        np.testing.assert_array_equal(wqt, o.st.layers[u].wq_t)
    cs = g.ctx.qe_get_state()
    snap = o.st.contract.snapshot()
    assert cs["e_w"] == snap["e_w"] and cs["token"] == snap["token"]


def compare_outputs(g, o, tol=1e-3):
    for key, ref in o.outs.items():
        got = as_f32(g.outs[key])
        assert rel_err(got, ref) <= tol, key


def run_pair(spec, steps, use_graphs=False, check_codes_after=None, **stage_kw):
    qe = need_lib()
    d = dev()
    g = GpuStage(qe, spec, use_graphs=use_graphs, device=d, **stage_kw)
    o = OracleStage(spec)
    for step, sched in enumerate(steps):
        S.check_legal(sched, spec.M)
        if check_codes_after is not None:
            cut = check_codes_after
            g.run(sched[:cut], step, step)
            o.run(sched[:cut], step, step)
            torch.cuda.synchronize()
            # slot payloads of every live tape, bit-exact
            for u in range(len(spec.shapes)):
                for m in range(spec.M):
                    if o.st.contract.layers[u].slots[m].live and o.st.layers[u].payload[m].dyq_t is not None:
                        xt, dyt = g.slot_codes(u, m)
                        np.testing.assert_array_equal(xt, o.st.layers[u].payload[m].xq_t)
                        np.testing.assert_array_equal(dyt, o.st.layers[u].payload[m].dyq_t)
            compare_state(g, o, spec)
            g.run(sched[cut:], step, step)
            o.run(sched[cut:], step, step)
        else:
            g.run(sched, step, step)
            o.run(sched, step, step)
        torch.cuda.synchronize()
        compare_state(g, o, spec)
        assert rel_err(g.grad.cpu().numpy(), o.st.arena[o.buf]) <= 1e-3
        new_w = o.sgd_weights()
        g.end_step(new_w)
        o.end_step(new_w)
    compare_outputs(g, o)
    assert g.ctx.qe_sync() == "OK"
    cs = g.ctx.qe_get_state()
    assert cs["device_token"] == cs["token"]
    return g, o


def test_single_linear_schedule():
    """One FP8 linear, 2 microbatches of 128 tokens, K = N = 256, fp32, H = 4."""
    spec = Spec([(256, 256)], tokens=128, M=2, history=4, margin=0, in_dtype="f32", shared_view=True, cfg=0)
    run_pair(spec, [S.SINGLE] * 3, check_codes_after=4)


def test_ragged_layers_bf16_schedule():
    spec = Spec([(200, 136), (72, 300)], tokens=100, M=2, history=4, margin=1, in_dtype="bf16",
                shared_view=False, cfg=91)
    run_pair(spec, [S.SINGLE, S.SINGLE], check_codes_after=4)


@pytest.mark.parametrize("w_dtype,fmt_w", [("f32", "E4M3"), ("bf16", "E5M2")])
def test_weight_dtype_or_format_unlike_input(w_dtype, fmt_w):
    """W's cast and X's cast share a launch only when they share the input dtype and FP8
    format; here they do not (fp32 master weights under bf16 activations, or an E5M2 weight
    code), so the refresh runs them as two launches, with the same codes and scales."""
    spec = Spec([(200, 136), (256, 384)], tokens=100, M=2, history=4, margin=0, in_dtype="bf16",
                shared_view=True, cfg=93, w_dtype=w_dtype, fmt_w=fmt_w)
    run_pair(spec, [S.SINGLE] * 2, check_codes_after=4)


@pytest.mark.parametrize("use_graphs", [False, True])
def test_refresh_cast_pair_with_misaligned_input(use_graphs):
    """The refreshing forward casts W and X in one launch; with X handed over one element past
    a 16-byte boundary its tiles take the unaligned path and W's the aligned one, in the same
    grid: codes, histories and scales still equal the oracle's bit for bit."""
    spec = Spec([(256, 384), (200, 136)], tokens=192, M=2, history=4, margin=0, in_dtype="bf16",
                shared_view=True, cfg=94)
    run_pair(spec, [S.SINGLE] * 2, use_graphs=use_graphs, check_codes_after=4, x_misaligned=True)


def test_bf16_outputs():
    spec = Spec([(256, 384)], tokens=192, M=2, history=4, margin=0, in_dtype="bf16", shared_view=True,
                out_dtype="bf16", cfg=92)
    qe = need_lib()
    g = GpuStage(qe, spec, device=dev())
    o = OracleStage(spec)
    g.run(S.SINGLE, 0, 0)
    o.run(S.SINGLE, 0, 0)
    torch.cuda.synchronize()
    for key, ref in o.outs.items():
        assert rel_err(as_f32(g.outs[key]), ref) <= 2.0 ** -8 + 1e-3, key


def test_zero_bubble_schedule():
    """8 microbatches, forwards ahead of dI, deferred dW reversed then
    interleaved, history 16 (rollover mid-step), a version bump in between."""
    spec = Spec([(96, 160), (160, 64)], tokens=48, M=8, history=16, margin=0, in_dtype="bf16", shared_view=False,
                cfg=2)
    run_pair(spec, [S.ZB_STEP0, S.ZB_STEP1], check_codes_after=13)


def test_outlier_saturation_schedule():
    """Outlier activations (x300 channels) and log-normal(2) gradients saturate
    E4M3 / E5M2 under the delayed scale, then the scale backs off."""
    spec = Spec([(128, 512)], tokens=256, M=1, history=4, margin=1, in_dtype="f32", shared_view=False, cfg=3,
                outliers=True)
    run_pair(spec, [[("F", 0), ("dI", 0), ("dW", 0)]] * 3)


def test_empty_microbatch():
    spec = Spec([(64, 96)], tokens=0, M=1, history=4, margin=0, in_dtype="f32", shared_view=False, cfg=93)
    g, o = run_pair(spec, [[("F", 0), ("dI", 0), ("dW", 0)]] * 2)
    assert np.all(g.grad.cpu().numpy() == 0)


def _run_variant(spec, steps, use_graphs, full, copy_gradients=False):
    qe = need_lib()
    g = GpuStage(qe, spec, use_graphs=use_graphs, device=dev(), copy_gradients=copy_gradients)
    o = OracleStage(spec)
    grads = []
    for step, sched in enumerate(steps):
        sched = S.to_full(sched) if full else sched
        g.run(sched, step, step)
        o.run(sched, step, step)
        torch.cuda.synchronize()
        grads.append(g.grad.cpu().numpy().copy())
        new_w = o.sgd_weights()
        g.end_step(new_w)
        o.end_step(new_w)
    outs = {k: v.cpu().numpy().copy() for k, v in g.outs.items()}
    states = [g.fp8_state(u) for u in range(len(spec.shapes))]
    return g, grads, outs, states


def _assert_bitwise(a, b):
    ga, oa, sa = a[1], a[2], a[3]
    gb, ob, sb = b[1], b[2], b[3]
    for x, y in zip(ga, gb):
        np.testing.assert_array_equal(x.view(np.uint32), y.view(np.uint32))
    assert oa.keys() == ob.keys()
    for k in oa:
        np.testing.assert_array_equal(oa[k], ob[k])
    for x, y in zip(sa, sb):
        for r in x:
            np.testing.assert_array_equal(x[r][0], y[r][0])
            assert x[r][1:] == y[r][1:]


@pytest.mark.parametrize("case", ["single", "zb"])
def test_split_dw_bitwise_equals_full_backward(case):
    if case == "single":
        spec = Spec([(256, 256)], tokens=128, M=2, history=4, margin=0, in_dtype="f32", shared_view=True, cfg=0)
        steps = [S.SINGLE, S.SINGLE]
    else:
        spec = Spec([(96, 160)], tokens=48, M=8, history=16, margin=0, in_dtype="bf16", shared_view=False, cfg=2)
        steps = [S.ZB_STEP0, S.ZB_STEP1]
    _assert_bitwise(_run_variant(spec, steps, False, False), _run_variant(spec, steps, False, True))


def test_graph_replay_bitwise_equals_eager():
    spec = Spec([(96, 160), (160, 64)], tokens=48, M=8, history=16, margin=0, in_dtype="bf16", shared_view=False,
                cfg=2)
    steps = [S.ZB_STEP0, S.ZB_STEP1, S.ZB_STEP0]
    eager = _run_variant(spec, steps, False, False)
    graph = _run_variant(spec, steps, True, False)
    _assert_bitwise(eager, graph)
    st = graph[0].ctx.qe_get_state()
    # inputs are uploaded to fresh buffers per action: the buffers are bound into
    # each action's graph (kernel-node arguments rewritten), with no new capture
    assert st["replays"] == sum(len(s) for s in steps) * 2
    assert st["graphs"] > 0 and st["handoffs"] == 2 * st["replays"]
    assert st["captures"] == st["graphs"] and st["rebinds"] > 0


@pytest.mark.parametrize("case", ["single", "zb"])
@pytest.mark.parametrize("use_graphs", [False, True])
def test_copied_gradients_bitwise_equal_direct_placement(case, use_graphs):
    """The copied-gradient path (dW into a private buffer, then a copy / add into
    the view) gives the same bits as direct placement, shared views included."""
    if case == "single":
        spec = Spec([(256, 256)], tokens=128, M=2, history=4, margin=0, in_dtype="f32", shared_view=True, cfg=0)
        steps = [S.SINGLE, S.SINGLE]
    else:
        spec = Spec([(96, 160), (72, 200)], tokens=48, M=8, history=16, margin=0, in_dtype="bf16",
                    shared_view=False, cfg=2)
        steps = [S.ZB_STEP0, S.ZB_STEP1]
    direct = _run_variant(spec, steps, use_graphs, False)
    copied = _run_variant(spec, steps, use_graphs, False, copy_gradients=True)
    _assert_bitwise(direct, copied)


@pytest.mark.parametrize("case", ["single", "zb"])
@pytest.mark.parametrize("copy_gradients", [False, True], ids=["direct", "copied"])
@pytest.mark.parametrize("use_graphs", [False, True], ids=["eager", "graphs"])
def test_placement_against_oracle_padded_views(case, copy_gradients, use_graphs):
    """dW placed into views whose row stride exceeds K, by direct placement and by
    the copied-gradient path (§3.4's conservative clone path: dW into a private
    buffer, then a copy / add into the view), each against the oracle at 1e-3:
    INIT and ACCUM into a shared view (single), INIT into per-microbatch views
    (zero-bubble); the elements between rows stay untouched (zero)."""
    if case == "single":   # odd padding: the copy kernel's element-wise path
        spec = Spec([(256, 256)], tokens=128, M=2, history=4, margin=0, in_dtype="f32", shared_view=True, cfg=0,
                    ld_pad=5)
        steps = [S.SINGLE, S.SINGLE]
    else:                  # padding by 4: its 16-byte path
        spec = Spec([(96, 160), (72, 200)], tokens=48, M=8, history=16, margin=0, in_dtype="bf16",
                    shared_view=False, cfg=2, ld_pad=4)
        steps = [S.ZB_STEP0, S.ZB_STEP1]
    g, o = run_pair(spec, steps, use_graphs=use_graphs, copy_gradients=copy_gradients)
    got = g.grad.cpu().numpy()
    for u, (n, k) in enumerate(spec.shapes):
        for m in range(1 if spec.shared_view else spec.M):
            view = got[spec.offset(u, m):spec.offset(u, m) + n * spec.ld(u)].reshape(n, spec.ld(u))
            assert np.all(view[:, k:] == 0), (u, m)
            assert np.any(view[:, :k] != 0), (u, m)
