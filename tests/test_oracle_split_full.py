"""The paper's split = full-backward invariant (§5.2, Table "correctness",
stepwise state parity across amax-history rollover), checked on the oracle
itself: a deferred, reordered dW must equal dW computed right after its dI."""
import numpy as np
import pytest

import workloads as W
from oracle import contract as C
from oracle.layer import Stage
from tests import schedules as S

BUF = 1 << 16


def build(M, shapes, history, margin, seed, dtype="f32"):
    st = Stage(M)
    for u, (n, k) in enumerate(shapes):
        w = W.normal(W.rng_for(seed, 99, u, W.ROLE_W), (n, k), 0.02, dtype).as_f32()
        st.add_layer(0, u, w, max_tokens=64, history=history, margin=margin)
    return st


def run(st, schedule, shapes, tokens, epoch, seed, shared_view, step=0):
    M = st.contract.M
    total = sum(n * k for n, k in shapes)
    buf = st.arena.get(BUF)
    if buf is None:
        st.add_buffer(BUF, total * (1 if shared_view else M))
        offs = np.cumsum([0] + [n * k for n, k in shapes])
        for u, (n, k) in enumerate(shapes):
            for m in range(M):
                off = offs[u] if shared_view else m * total + offs[u]
                assert st.bind(u, m, BUF, int(off), k) == C.OK
    refs, outs = {}, {}
    for a, m in schedule:
        for u, (n, k) in enumerate(shapes):
            key = (epoch, 0, m, u, 0)
            x = W.normal(W.rng_for(seed, 7, u, W.ROLE_X, m, step), (tokens, k), 1.0, "f32").as_f32()
            dy = W.normal(W.rng_for(seed, 7, u, W.ROLE_DY, m, step), (tokens, n), 0.01, "f32").as_f32()
            b = st.contract.bindings[(u, m)]
            mode = C.INIT if not any(o.written and o.start() == b.start() for o in st.contract.bindings.values()) \
                else C.ACCUM
            if a == "F":
                s, y, refs[(u, m)] = st.fwd(u, key, x)
                outs[("y", u, m)] = y
            elif a == "dI":
                s, outs[("dx", u, m)] = st.dgrad(u, key, refs[(u, m)], dy)
            elif a == "dW":
                s = st.wgrad_place(u, key, refs[(u, m)], BUF, b.offset, b.ld, mode)
            else:
                s, outs[("dx", u, m)] = st.bwd_full(u, key, refs[(u, m)], dy, BUF, b.offset, b.ld, mode)
            assert s == C.OK, (a, m, u, s)
    return outs


@pytest.mark.parametrize("case", ["single", "zb"])
def test_split_equals_full(case):
    if case == "single":
        M, shapes, hist, steps, shared = 2, [(24, 40)], 4, [S.SINGLE, S.SINGLE], True
    else:
        M, shapes, hist, steps, shared = 8, [(24, 40), (16, 24)], 16, [S.ZB_STEP0, S.ZB_STEP1], False
    results = []
    for variant in ("split", "full"):
        st = build(M, shapes, hist, 0, seed=5)
        outs_all = []
        for step, sched in enumerate(steps):
            S.check_legal(sched, M)
            sched = sched if variant == "split" else S.to_full(sched)
            outs_all.append(run(st, sched, shapes, 32, step, 5, shared, step))
            assert st.finalize() == C.OK
            grad = st.arena[BUF].copy()
            results.append((variant, step, grad, outs_all[-1],
                            [st.fp8_state(u) for u in range(len(shapes))], st.contract.snapshot()))
            # a plain SGD step on the weights, then the version bump
            total = sum(n * k for n, k in shapes)
            offs = np.cumsum([0] + [n * k for n, k in shapes])
            for u, (n, k) in enumerate(shapes):
                g = sum(grad[(0 if shared else m * total) + offs[u]:][:n * k].reshape(n, k)
                        for m in range(1 if shared else M))
                st.set_weight(u, (st.layers[u].w - 1e-3 * g).astype(np.float32))
            assert st.optimizer_commit() == C.OK
    half = len(results) // 2
    for (v1, s1, g1, o1, f1, c1), (v2, s2, g2, o2, f2, c2) in zip(results[:half], results[half:]):
        assert s1 == s2
        np.testing.assert_array_equal(g1, g2)
        for kk in o1:
            np.testing.assert_array_equal(o1[kk], o2[kk])
        for a, b in zip(f1, f2):
            for r in a:
                np.testing.assert_array_equal(a[r][0], b[r][0])
                assert a[r][1:] == b[r][1:]
        assert c1["e_w"] == c2["e_w"]


def test_dw_with_live_scales_would_differ():
    """Sanity of the invariant test above: between dI0 and dW0 the dY scale moves
    (delayed-scaling rollover), so a dW that used the live scale instead of the
    snapshot kept in the slot would not match."""
    st = build(2, [(24, 40)], 4, 0, seed=5)
    run(st, S.SINGLE[:4], [(24, 40)], 32, 0, 5, True)
    L = st.layers[0]
    assert L.payload[0].dy_scale_inv != L.sdy.scale_inv
