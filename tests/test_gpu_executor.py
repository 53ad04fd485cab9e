"""The caller-stream executor (qe_config.replay_on_caller): each action's graph
or kernels run on the caller's stream, so stream order replaces the two-way
handoff of §2.3 / §4.4, and a change of caller stream between actions is
chained through one event so all actions keep one total order (the ordering
the paper gets from a single graph stream).  Results must be bitwise those of
the graph-stream executor, also with every action on a different stream, and a
consumer enqueued on the caller stream right after an action must never see
stale output."""
import numpy as np
import pytest

from tests import schedules as S
from tests.gpu_util import dev, torch
from tests.libqe import need_lib
from tests.stage_driver import GpuStage, OracleStage, Spec

pytestmark = pytest.mark.gpu

SPEC = Spec([(96, 160), (160, 64)], tokens=48, M=8, history=16, margin=0, in_dtype="bf16", shared_view=False, cfg=2)
STEPS = [S.ZB_STEP0, S.ZB_STEP1, S.ZB_STEP0]


def _run(use_graphs, replay_on_caller, n_streams=0):
    qe = need_lib()
    d = dev()
    streams = [torch.cuda.Stream() for _ in range(n_streams)] if n_streams else None
    g = GpuStage(qe, SPEC, use_graphs=use_graphs, device=d, replay_on_caller=replay_on_caller, streams=streams)
    o = OracleStage(SPEC)
    grads = []
    for step, sched in enumerate(STEPS):
        g.run(sched, step, step)
        o.run(sched, step, step)
        torch.cuda.synchronize()
        grads.append(g.grad.cpu().numpy().copy())
        new_w = o.sgd_weights()
        g.end_step(new_w)
        o.end_step(new_w)
    torch.cuda.synchronize()
    outs = {k: v.cpu().numpy().copy() for k, v in g.outs.items()}
    states = [g.fp8_state(u) for u in range(len(SPEC.shapes))]
    assert g.ctx.qe_sync() == "OK"
    st = g.ctx.qe_get_state()
    assert st["device_token"] == st["token"]
    return g, grads, outs, states, st


def _same(a, b):
    for x, y in zip(a[1], b[1]):
        np.testing.assert_array_equal(x.view(np.uint32), y.view(np.uint32))
    assert a[2].keys() == b[2].keys()
    for k in a[2]:
        np.testing.assert_array_equal(a[2][k], b[2][k], err_msg=str(k))
    for x, y in zip(a[3], b[3]):
        for r in x:
            np.testing.assert_array_equal(x[r][0], y[r][0])
            assert x[r][1:] == y[r][1:]


@pytest.mark.parametrize("use_graphs", [False, True], ids=["eager", "graphs"])
def test_caller_stream_bitwise_equals_graph_stream(use_graphs):
    ref = _run(use_graphs, False)
    got = _run(use_graphs, True)
    _same(ref, got)
    assert got[4]["handoffs"] == 0 and ref[4]["handoffs"] > 0
    if use_graphs:
        assert got[4]["replays"] == ref[4]["replays"] > 0


@pytest.mark.parametrize("use_graphs", [False, True], ids=["eager", "graphs"])
def test_caller_stream_chains_actions_across_streams(use_graphs):
    """Every action on the next of three streams (F, dI and the deferred dW of
    one microbatch on different streams; scale updates in fixed order across
    them): the chaining event keeps one total order, bitwise as on one stream."""
    ref = _run(use_graphs, False)
    got = _run(use_graphs, True, n_streams=3)
    _same(ref, got)


def test_caller_stream_consumer_never_stale():
    qe = need_lib()
    d = dev()
    n, k, t = 28672, 4096, 4096
    ctx = qe.Context(1, use_graphs=True, replay_on_caller=True)
    g = torch.Generator(device=d)
    g.manual_seed(1)
    w = (torch.randn(n, k, device=d, generator=g) * 0.02).to(torch.bfloat16)
    x = torch.randn(t, k, device=d, generator=g).to(torch.bfloat16)
    st, L = ctx.qe_layer_register(0, 0, n, k, t, w, qe.BF16, 4, 0)
    assert st == "OK"
    y = torch.empty((t, n), dtype=torch.bfloat16, device=d)
    caller = torch.cuda.Stream()
    stale = 0
    for trial in range(30):
        with torch.cuda.stream(caller):
            y.fill_(float("nan"))
            st, ref = ctx.qe_fp8_linear_fwd(L, qe.key(0, 0, 0, 0), x, qe.BF16, t, y, qe.BF16, caller=caller)
            assert st == "OK"
            seen = y.clone()
        torch.cuda.synchronize()
        assert ctx.qe_sync() == "OK"
        if not torch.equal(seen.view(torch.int16), y.view(torch.int16)):
            stale += 1
        assert ctx.qe_abort_epoch() == "OK" and ctx.qe_arena_rebuild() == "OK"
    assert not torch.isnan(y.float()).any()
    assert stale == 0
    ctx.close()


def test_caller_stream_destroyed_between_actions():
    """The caller-stream executor keeps no caller stream handle between actions:
    F on a raw HIP stream that is destroyed right after the call (without a
    synchronisation), then dI and dW on a second raw stream, give the same bits
    as the same actions on torch's current stream."""
    import ctypes as C
    qe = need_lib()
    d = dev()
    hip = C.CDLL("libamdhip64.so")
    n, k, t = 256, 256, 128
    g = torch.Generator(device=d)
    g.manual_seed(7)
    w = torch.randn(n, k, device=d, generator=g) * 0.02
    x = torch.randn(t, k, device=d, generator=g)
    dy = torch.randn(t, n, device=d, generator=g) * 0.01

    def run(raw):
        ctx = qe.Context(1, use_graphs=True, replay_on_caller=True)
        st, L = ctx.qe_layer_register(0, 0, n, k, t, w, qe.F32, 4, 0)
        assert st == "OK"
        grad = torch.zeros(n * k, device=d)
        assert ctx.qe_arena_bind(L, 0, grad, n * k, 0, k) == "OK"
        y = torch.zeros(t, n, device=d)
        dx = torch.zeros(t, k, device=d)
        torch.cuda.synchronize()
        for step in range(2):
            key = qe.key(step, 0, 0, 0)
            s1, s2 = C.c_void_p(), C.c_void_p()
            if raw:
                assert hip.hipStreamCreate(C.byref(s1)) == 0 and hip.hipStreamCreate(C.byref(s2)) == 0
            st, ref = ctx.qe_fp8_linear_fwd(L, key, x, qe.F32, t, y, qe.F32, caller=s1.value if raw else None)
            assert st == "OK"
            if raw:
                assert hip.hipStreamDestroy(s1) == 0       # no synchronisation first
            c2 = s2.value if raw else None
            assert ctx.qe_fp8_linear_dgrad(L, key, ref, dy, qe.F32, dx, qe.F32, caller=c2) == "OK"
            assert ctx.qe_fp8_linear_wgrad_place(L, key, ref, grad, 0, k, qe.INIT, caller=c2) == "OK"
            assert ctx.qe_sync() == "OK"
            if raw:
                assert hip.hipStreamDestroy(s2) == 0
            assert ctx.qe_arena_finalize() == "OK" and ctx.qe_optimizer_commit() == "OK"
        torch.cuda.synchronize()
        out = (y.cpu().numpy().copy(), dx.cpu().numpy().copy(), grad.cpu().numpy().copy())
        st = ctx.qe_get_state()
        assert st["device_token"] == st["token"]
        ctx.close()
        return out

    ref = run(False)
    got = run(True)
    for a, b in zip(ref, got):
        np.testing.assert_array_equal(a.view(np.uint32), b.view(np.uint32))


@pytest.mark.parametrize("mode", ["delayed", "delayed_copied", "current"])
def test_kernel_timing_counts_each_class(mode):
    """Eager kernel timing counts every launch of the actions' kernel
    sequences (§3.2) under its class.  Per optimizer step, delayed scaling: F
    (with the weight refresh) is one paired cast and one GEMM whose extra
    workgroups run the scale update, dI one cast and one GEMM, the deferred dW
    one GEMM, plus one gradient copy on the copied-gradient path; current
    scaling adds an amax pass per cast tensor (W, X, dY) and a stand-alone
    update before each action's casts.  Totals run on across reads; with timing
    off they stop; an unknown class is refused."""
    qe = need_lib()
    d = dev()
    n, k, t = 256, 320, 160
    g = torch.Generator(device=d)
    g.manual_seed(8)
    w = torch.randn(n, k, device=d, generator=g) * 0.02
    x = torch.randn(t, k, device=d, generator=g)
    dy = torch.randn(t, n, device=d, generator=g) * 0.01
    current = mode == "current"
    ctx = qe.Context(1, copy_gradients=mode == "delayed_copied")
    st, L = ctx.qe_layer_register(0, 0, n, k, t, w, qe.F32, 1 if current else 4, 0,
                                  scaling=qe.SCALING_CURRENT if current else qe.SCALING_DELAYED)
    assert st == "OK"
    grad = torch.zeros(n * k, device=d)
    assert ctx.qe_arena_bind(L, 0, grad, n * k, 0, k) == "OK"
    y = torch.zeros(t, n, device=d)
    dx = torch.zeros(t, k, device=d)
    classes = (qe.KC_QUANT, qe.KC_UPDATE, qe.KC_GEMM, qe.KC_COPY, qe.KC_AMAX)

    def step(i):
        key = qe.key(i, 0, 0, 0)
        st, ref = ctx.qe_fp8_linear_fwd(L, key, x, qe.F32, t, y, qe.F32)
        assert st == "OK"
        assert ctx.qe_fp8_linear_dgrad(L, key, ref, dy, qe.F32, dx, qe.F32) == "OK"
        assert ctx.qe_fp8_linear_wgrad_place(L, key, ref, grad, 0, k, qe.INIT) == "OK"
        assert ctx.qe_sync() == "OK"
        assert ctx.qe_arena_finalize() == "OK" and ctx.qe_optimizer_commit() == "OK"

    def counts():
        return {c: ctx.qe_get_kernel_timing(c) for c in classes}

    per_step = {qe.KC_QUANT: 2, qe.KC_UPDATE: 2 if current else 0, qe.KC_GEMM: 3,
                qe.KC_COPY: 1 if mode == "delayed_copied" else 0, qe.KC_AMAX: 3 if current else 0}
    assert all(v == (0.0, 0) for v in counts().values())
    assert ctx.qe_set_kernel_timing(True) == "OK"
    step(0)
    first = counts()
    step(1)
    second = counts()
    for c in classes:
        assert first[c][1] == per_step[c] and second[c][1] == 2 * per_step[c], (mode, c, first, second)
        assert (second[c][0] > first[c][0] > 0.0) if per_step[c] else second[c][0] == 0.0
    assert ctx.qe_set_kernel_timing(False) == "OK"
    step(2)
    assert counts() == second
    for bad in (-1, len(classes)):
        with pytest.raises(RuntimeError):
            ctx.qe_get_kernel_timing(bad)
    ctx.close()


def test_two_contexts_interleaved_match_solo_runs():
    """Two contexts on one device, their actions interleaved call by call on
    two caller streams (graph replay, each with its own graph stream, layers
    and arena): every output equals, bit for bit, the same context's run on
    its own, so the contexts share no state."""
    qe = need_lib()
    d = dev()
    shapes = [(256, 320, 160), (384, 256, 96)]
    g = torch.Generator(device=d)
    g.manual_seed(21)
    data = []
    for n, k, t in shapes:
        w = torch.randn(n, k, device=d, generator=g) * 0.02
        x = torch.randn(t, k, device=d, generator=g)
        dy = torch.randn(t, n, device=d, generator=g) * 0.01
        data.append((n, k, t, w, x, dy))

    def make(i):
        n, k, t, w, x, dy = data[i]
        ctx = qe.Context(1, use_graphs=True)
        st, L = ctx.qe_layer_register(0, 0, n, k, t, w, qe.F32, 4, 0)
        assert st == "OK"
        grad = torch.zeros(n * k, device=d)
        assert ctx.qe_arena_bind(L, 0, grad, n * k, 0, k) == "OK"
        return {"ctx": ctx, "L": L, "grad": grad, "y": torch.zeros(t, n, device=d), "dx": torch.zeros(t, k, device=d)}

    def actions(i, s, step):
        n, k, t, w, x, dy = data[i]
        key = qe.key(step, 0, 0, 0)
        c = s["ctx"]

        def fwd():
            st, s["ref"] = c.qe_fp8_linear_fwd(s["L"], key, x, qe.F32, t, s["y"], qe.F32)
            return st
        yield fwd
        yield lambda: c.qe_fp8_linear_dgrad(s["L"], key, s["ref"], dy, qe.F32, s["dx"], qe.F32)
        yield lambda: c.qe_fp8_linear_wgrad_place(s["L"], key, s["ref"], s["grad"], 0, k, qe.INIT)

    def finish(s):
        c = s["ctx"]
        assert c.qe_sync() == "OK"
        assert c.qe_arena_finalize() == "OK" and c.qe_optimizer_commit() == "OK"

    def outputs(s):
        torch.cuda.synchronize()
        return [s[n].cpu().numpy().copy() for n in ("y", "dx", "grad")]

    solo = []
    for i in range(2):
        s = make(i)
        for step in range(2):
            for a in actions(i, s, step):
                assert a() == "OK"
            finish(s)
        solo.append(outputs(s))
        s["ctx"].close()

    both = [make(0), make(1)]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    torch.cuda.synchronize()                           # inputs and buffers ready before the side streams run
    for step in range(2):
        seqs = [list(actions(i, both[i], step)) for i in range(2)]
        for a0, a1 in zip(*seqs):
            with torch.cuda.stream(streams[0]):
                assert a0() == "OK"
            with torch.cuda.stream(streams[1]):
                assert a1() == "OK"
        for s in both:
            finish(s)
    for i in range(2):
        got = outputs(both[i])
        for a, b in zip(solo[i], got):
            np.testing.assert_array_equal(a.view(np.uint32), b.view(np.uint32))
        both[i]["ctx"].close()
