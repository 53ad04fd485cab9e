"""The library's contract (null executor: no HIP call, no device) against the
oracle's state machine, call by call and state by state."""
import random

import pytest

from oracle import contract as OC
from tests.libqe import need_lib

BUF = 1 << 20          # fake buffer base address (never dereferenced in null mode)
BUF_ELEMS = 1 << 22


class Pair:
    """Runs every call on both the oracle contract and the library, compares status and state."""

    def __init__(self, M, layers):
        qe = need_lib()
        self.qe = qe
        self.o = OC.Contract(M)
        self.c = qe.Context(M, null_executor=True)
        self.M = M
        self.refs_o, self.refs_c = {}, {}
        for u, (n, k, t) in enumerate(layers):
            self.o.add_layer(0, u, n, k, t)
            st, idx = self.c.qe_layer_register(0, u, n, k, t, 0, qe.F32, 4, 0)
            assert st == "OK" and idx == u

    def state(self):
        ctx = self.c.qe_get_state()
        snap = {"e_w": ctx["e_w"], "token": ctx["token"], "arena_valid": bool(ctx["arena_valid"]),
                "finalized": bool(ctx["finalized"]), "layers": [], "written": {}}
        for l in range(len(self.o.layers)):
            ls = self.c.qe_get_layer_state(l)
            slots = []
            for m in range(self.M):
                s = self.c.qe_get_slot_state(l, m)
                slots.append((s["live"], s["key"] if s["live"] else None, s["generation"], s["bits"],
                              s["tokens"] if s["live"] else 0))
                if s["bound"]:
                    snap["written"][(l, m)] = s["written"]
            snap["layers"].append({"e_c": ls["e_c"], "refreshes": ls["refreshes"], "slots": slots})
        return snap

    def check(self):
        assert self.state() == self.o.snapshot()

    def fwd(self, l, k, tokens=8):
        st, refresh = self.o.check_fwd(l, k, tokens)
        if st == OC.OK:
            if self.o._physical_fails():
                self.o.abort()
                st = OC.EXEC_FAILED
            else:
                self.o.commit_fwd(l, k, tokens, refresh)
        st_c, ref = self.c.qe_fp8_linear_fwd(l, self.qe.key(*k), 0, self.qe.F32, tokens, 0, self.qe.F32)
        assert st_c == st, ("fwd", l, k, st_c, st)
        return st, ref

    def dgrad(self, l, k, ref):
        st = self.o.check_dgrad(l, k, ref)
        if st == OC.OK:
            if self.o._physical_fails():
                self.o.abort()
                st = OC.EXEC_FAILED
            else:
                self.o.commit_dgrad(l, ref)
        st_c = self.c.qe_fp8_linear_dgrad(l, self.qe.key(*k), ref, 0, self.qe.F32, 0, self.qe.F32)
        assert st_c == st, ("dI", l, k, ref, st_c, st)
        return st

    def wgrad(self, l, k, ref, off, ld, mode, buf=BUF):
        st = self.o.check_wgrad(l, k, ref, buf, off, ld, mode)
        if st == OC.OK:
            if self.o._physical_fails():
                self.o.abort()
                st = OC.EXEC_FAILED
            else:
                self.o.commit_wgrad(l, ref)
        st_c = self.c.qe_fp8_linear_wgrad_place(l, self.qe.key(*k), ref, buf, off, ld, mode)
        assert st_c == st, ("dW", l, k, ref, st_c, st)
        return st

    def full(self, l, k, ref, off, ld, mode, buf=BUF):
        st = self.o.check_bwd_full(l, k, ref, buf, off, ld, mode)
        if st == OC.OK:
            if self.o._physical_fails():
                self.o.abort()
                st = OC.EXEC_FAILED
            else:
                self.o.commit_bwd_full(l, ref)
        st_c = self.c.qe_fp8_linear_bwd_full(l, self.qe.key(*k), ref, 0, self.qe.F32, 0, self.qe.F32, buf, off,
                                             ld, mode)
        assert st_c == st, ("full", l, k, ref, st_c, st)
        return st

    def bind(self, l, m, off, ld, buf=BUF, elems=BUF_ELEMS):
        st = self.o.bind(l, m, buf, elems, off, ld)
        assert self.c.qe_arena_bind(l, m, buf, elems, off, ld) == st
        return st

    def finalize(self):
        st = self.o.finalize()
        assert self.c.qe_arena_finalize() == st
        return st

    def commit(self):
        st = self.o.optimizer_commit()
        assert self.c.qe_optimizer_commit() == st
        return st

    def abort(self):
        self.o.abort()
        assert self.c.qe_abort_epoch() == "OK"

    def rebuild(self):
        assert self.c.qe_arena_rebuild() == self.o.rebuild()

    def inject(self, n):
        self.o.inject_fault(n)
        assert self.c.qe_inject_fault(n) == "OK"

    def checkpoint(self):
        st = self.o.checkpoint_check()
        st_c, payload = self.c.qe_checkpoint_export()
        assert st_c == st, ("checkpoint", st_c, st)
        return st, payload

    def restore(self, payload, e_w):
        st = self.o.restore(e_w)
        assert self.c.qe_checkpoint_import(payload) == st, ("restore", st)
        return st


def K(e, m, u=0, inv=0):
    return (e, 0, m, u, inv)


def test_fault_table_rows():
    p = Pair(2, [(4, 8, 16)])
    p.bind(0, 0, 0, 8)
    p.bind(0, 1, 64, 8)
    # old reference after slot reuse
    _, r0 = p.fwd(0, K(0, 0))
    p.dgrad(0, K(0, 0), r0)
    p.wgrad(0, K(0, 0), r0, 0, 8, OC.INIT)
    _, r0b = p.fwd(0, K(0, 0, inv=1))
    assert p.dgrad(0, K(0, 0), r0) == OC.STALE_REF
    p.check()
    # repeated dI
    assert p.dgrad(0, K(0, 0, inv=1), r0b) == OC.OK
    assert p.dgrad(0, K(0, 0, inv=1), r0b) == OC.DUPLICATE_CONSUMER
    assert p.wgrad(0, K(0, 0, inv=1), r0b, 0, 8, OC.INIT) == OC.DUP_WRITE   # view 0 already written
    p.check()
    # finalize with a missing dW
    _, r1 = p.fwd(0, K(0, 1))
    p.dgrad(0, K(0, 1), r1)
    assert p.finalize() == OC.INCOMPLETE
    assert p.commit() == OC.NOT_QUIESCENT
    p.check()
    # write after an aborted write
    p.inject(1)
    assert p.wgrad(0, K(0, 1), r1, 64, 8, OC.INIT) == OC.EXEC_FAILED
    assert p.wgrad(0, K(0, 1), r1, 64, 8, OC.INIT) == OC.ARENA_INVALID
    assert p.finalize() == OC.ARENA_INVALID
    p.check()
    p.rebuild()
    p.check()
    # stale cache: after a commit, a microbatch-1 forward before microbatch 0
    _, r0 = p.fwd(0, K(0, 0, inv=2))
    p.full(0, K(0, 0, inv=2), r0, 0, 8, OC.INIT)
    _, r1 = p.fwd(0, K(0, 1, inv=2))
    p.full(0, K(0, 1, inv=2), r1, 64, 8, OC.INIT)
    assert p.finalize() == OC.OK and p.commit() == OC.OK
    assert p.fwd(0, K(1, 1))[0] == OC.STALE_CACHE
    assert p.fwd(0, K(1, 0))[0] == OC.OK
    p.check()


def test_bind_rules():
    p = Pair(2, [(4, 8, 16), (3, 5, 16)])
    assert p.bind(0, 0, 0, 8) == OC.OK
    assert p.bind(0, 1, 0, 8) == OC.OK
    assert p.bind(1, 0, 20, 5) == OC.DEST_ALIAS
    assert p.bind(1, 0, 32, 5) == OC.OK
    assert p.bind(1, 1, 33, 5) == OC.DEST_ALIAS
    assert p.bind(1, 1, 0, 4) == OC.INVALID_ARG
    assert p.bind(1, 1, BUF_ELEMS - 5, 5) == OC.INVALID_ARG
    assert p.bind(1, 1, 100, 5, buf=0) == OC.INVALID_ARG
    assert p.bind(2, 0, 100, 5) == OC.INVALID_ARG
    p.check()


@pytest.mark.parametrize("seed", range(16))
def test_random_schedules_match_oracle(seed):
    rng = random.Random(seed)
    M, nl = rng.choice([1, 2, 3, 4]), rng.choice([1, 2])
    p = Pair(M, [(4, 8, 16)] * nl)
    for u in range(nl):
        for m in range(M):
            shared = rng.random() < 0.3
            p.bind(u, m, (u * M + (0 if shared else m)) * 64, 8)
    refs = {}
    for _ in range(300):
        u, m = rng.randrange(nl), rng.randrange(M)
        e = p.o.e_w + (0 if rng.random() < 0.9 else rng.choice([-1, 1]))
        k = K(max(e, 0), m, u, rng.choice([0, 0, 0, 1]))
        ref = refs.get((u, m), (m, 0))
        if rng.random() < 0.1:
            ref = (ref[0], ref[1] + rng.choice([-1, 1, 2]))
        if rng.random() < 0.03:
            p.inject(rng.randint(1, 3))
        b = p.o.bindings.get((u, m))
        off = b.offset if b else 0
        mode = OC.ACCUM if (b and any(o.written and o.start() == b.start() for o in p.o.bindings.values())) \
            else OC.INIT
        if rng.random() < 0.05:
            mode = 1 - mode
        what = rng.choice(["f", "f", "di", "dw", "full", "fin", "commit", "abort", "rebuild", "ckpt", "restore"])
        if what == "f":
            st, r = p.fwd(u, k, tokens=rng.randint(0, 16))
            if st == OC.OK:
                refs[(u, m)] = r
                # keep the key of this tape for its consumers
                refs[("key", u, m)] = k
        elif what in ("di", "dw", "full"):
            kk = refs.get(("key", u, m), k)
            if rng.random() < 0.1:
                kk = k
            if what == "di":
                p.dgrad(u, kk, ref)
            elif what == "dw":
                p.wgrad(u, kk, ref, off, 8, mode)
            else:
                p.full(u, kk, ref, off, 8, mode)
        elif what == "fin":
            p.finalize()
        elif what == "commit":
            p.commit()
        elif what == "abort" and rng.random() < 0.2:
            p.abort()
        elif what == "rebuild":
            p.rebuild()
        elif what == "ckpt":
            e_w = p.o.e_w
            st, payload = p.checkpoint()
            if st == OC.OK:
                refs["ckpt"] = (payload, e_w)
        elif what == "restore" and "ckpt" in refs:
            p.restore(*refs["ckpt"])
        p.check()


def test_register_scaling_recipe_validation():
    """Current scaling keeps no history: it needs history_len == 1; unknown recipes are rejected."""
    qe = need_lib()
    c = qe.Context(1, null_executor=True)
    assert c.qe_layer_register(0, 0, 8, 8, 8, 0, qe.F32, 4, 0, scaling=qe.SCALING_CURRENT)[0] == "INVALID_ARG"
    assert c.qe_layer_register(0, 0, 8, 8, 8, 0, qe.F32, 1, 0, scaling=2)[0] == "INVALID_ARG"
    assert c.qe_layer_register(0, 0, 8, 8, 8, 0, qe.F32, 1, 0, scaling=qe.SCALING_CURRENT) == ("OK", 0)
    assert c.qe_layer_register(0, 1, 8, 8, 8, 0, qe.F32, 4, 0, scaling=qe.SCALING_DELAYED) == ("OK", 1)
    c.close()


def test_register_rejects_reduction_lengths_past_2_31():
    """n_out, k_in and max_tokens are each the reduction length of one GEMM
    (dI, F and dW): 2^31 - 1 is accepted, 2^31 is refused."""
    qe = need_lib()
    c = qe.Context(1, null_executor=True)
    big = 1 << 31
    for u, (n, k, t) in enumerate([(big, 8, 8), (8, big, 8), (8, 8, big)]):
        assert c.qe_layer_register(0, u, n, k, t, 0, qe.F32, 4, 0)[0] == "INVALID_ARG"
    assert c.qe_layer_register(0, 0, 8, 8, big - 1, 0, qe.F32, 4, 0) == ("OK", 0)
    c.close()


def test_executor_config_validation():
    """replay_on_caller is 0 or 1, and the one-way (testing) handoff exists only
    for the graph-stream executor."""
    qe = need_lib()
    import ctypes as C
    for replay, one_way, want in ((0, 0, "OK"), (1, 0, "OK"), (2, 0, "INVALID_ARG"), (-1, 0, "INVALID_ARG"),
                                  (1, 1, "INVALID_ARG"), (0, 1, "OK")):
        cfg = qe.Config(0, 1, 0, 1, one_way, 0, replay)
        h = C.c_void_p()
        st = qe.qe_status_str(qe.lib().qe_ctx_create(C.byref(cfg), C.byref(h)))
        assert st == want, (replay, one_way, st)
        if h:
            qe.lib().qe_ctx_destroy(h)


def _payload_fields(b):
    import struct
    magic, version, n_layers, M, _, e_w = struct.unpack_from("<8sIIiiq", b, 0)
    return magic, version, n_layers, M, e_w


def test_checkpoint_payload_and_validation():
    """Payload layout and size, withheld checkpoints, and every rejected import
    (bad hash, truncation, magic, version, other configuration, busy stage)
    leaving the state unchanged."""
    import struct
    qe = need_lib()
    p = Pair(2, [(4, 8, 16), (3, 5, 16)])
    p.bind(0, 0, 0, 8)
    p.bind(0, 1, 64, 8)
    p.bind(1, 0, 128, 5)
    p.bind(1, 1, 192, 5)
    assert p.checkpoint()[0] == OC.OK
    _, r = p.fwd(0, K(0, 0))
    assert p.checkpoint() == (OC.NOT_QUIESCENT, None)                     # live tape
    p.full(0, K(0, 0), r, 0, 8, OC.INIT)
    assert p.checkpoint()[0] == OC.NOT_QUIESCENT                          # arena write in flight
    for u in range(2):
        for m in range(2):
            if (u, m) != (0, 0):
                _, r = p.fwd(u, K(0, m, u))
                p.full(u, K(0, m, u), r, [0, 64, 128, 192][2 * u + m], [8, 5][u], OC.INIT)
    assert p.finalize() == OC.OK
    assert p.checkpoint()[0] == OC.NOT_QUIESCENT                          # finalized, not committed
    assert p.commit() == OC.OK
    st, payload = p.checkpoint()
    assert st == OC.OK
    assert len(payload) == 32 + 2 * (64 + 3 * (4 + 2) * 4) + 8
    assert _payload_fields(payload) == (b"QECKPT01", 1, 2, 2, 1)
    rec = struct.unpack_from("<IIqqqiiiiiiii", payload, 32)
    assert rec == (0, 0, 4, 8, 16, qe.F32, 4, 0, qe.E4M3, qe.E4M3, qe.E5M2, qe.SCALING_DELAYED, 0)

    def fresh():
        q = Pair(2, [(4, 8, 16), (3, 5, 16)])
        return q

    bad = []
    flipped = bytearray(payload)
    flipped[40] ^= 1
    bad.append(bytes(flipped))                                            # hash mismatch
    bad.append(payload[:-1])                                              # truncated
    for off, fmt, val in ((0, "<8s", b"QECKPT02"), (8, "<I", 2), (16, "<i", 3), (40, "<q", 9), (76, "<i", 5)):
        b = bytearray(payload[:-8])
        struct.pack_into(fmt, b, off, val)
        bad.append(bytes(b) + _fnv1a(bytes(b)).to_bytes(8, "little"))    # well-formed hash, wrong field
    for b in bad:
        q = fresh()
        snap = q.c.qe_get_state()
        assert q.c.qe_checkpoint_import(b) == "INVALID_ARG"
        assert q.c.qe_get_state() == snap
    # a busy stage refuses the import
    q = fresh()
    _, r = q.fwd(0, K(0, 0))
    assert q.c.qe_checkpoint_import(payload) == "NOT_QUIESCENT"
    # the good payload restores e_W and marks the caches stale; token stays local
    q = fresh()
    assert q.restore(payload, 1) == OC.OK
    q.check()
    assert q.c.qe_get_state()["e_w"] == 1 and q.c.qe_get_state()["token"] == 0
    assert q.c.qe_get_layer_state(0)["e_c"] == -1


def _fnv1a(b):
    h = 1469598103934665603
    for x in b:
        h = ((h ^ x) * 1099511628211) % (1 << 64)
    return h


def test_prebuild_graphs_argument_checks():
    """qe_prebuild_graphs validates before doing anything (host-only context)."""
    from tests.libqe import need_lib
    qe = need_lib()
    nog = qe.Context(2, use_graphs=False, null_executor=True)
    assert nog.qe_prebuild_graphs(0, qe.BF16, qe.F32, qe.BF16, qe.F32) == "INVALID_ARG"
    nog.close()
    c = qe.Context(2, use_graphs=True, null_executor=True)
    st, idx = c.qe_layer_register(0, 0, 64, 32, 100, None, qe.F32, 4, 0)
    assert st == "OK"
    assert c.qe_prebuild_graphs(101, qe.BF16, qe.F32, qe.BF16, qe.F32) == "INVALID_ARG"
    assert c.qe_prebuild_graphs(-1, qe.BF16, qe.F32, qe.BF16, qe.F32) == "INVALID_ARG"
    assert c.qe_prebuild_graphs(0, 7, qe.F32, qe.BF16, qe.F32) == "INVALID_ARG"
    assert c.qe_prebuild_graphs(100, qe.BF16, qe.F32, qe.BF16, qe.F32) == "OK"
    assert c.qe_get_state()["captures"] == 0  # no device: nothing captured
    c.close()


def test_graph_inputs_mode_checked():
    from tests.libqe import need_lib
    qe = need_lib()
    for bad in (-1, 3):
        with pytest.raises(RuntimeError):
            qe.Context(1, use_graphs=True, null_executor=True, graph_inputs=bad)
