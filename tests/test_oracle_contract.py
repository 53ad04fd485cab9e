"""Pins for the oracle's contract state machine: the paper's fault table, the
four invariants as properties of random schedules, and 'rejected calls change
nothing'."""
import copy
import random

import pytest

from oracle import contract as C


def key(e, m, stage=0, unit=0, inv=0):
    return (e, stage, m, unit, inv)


def make(M=2, n=4, k=8, tokens=16):
    c = C.Contract(M)
    c.add_layer(0, 0, n, k, tokens)
    return c


def run_f(c, layer, k, tokens=16):
    st, refresh = c.check_fwd(layer, k, tokens)
    if st != C.OK:
        return st, None
    return st, c.commit_fwd(layer, k, tokens, refresh)


def run_di(c, layer, k, ref):
    st = c.check_dgrad(layer, k, ref)
    if st == C.OK:
        c.commit_dgrad(layer, ref)
    return st


def run_dw(c, layer, k, ref, buf, off, ld, mode):
    st = c.check_wgrad(layer, k, ref, buf, off, ld, mode)
    if st == C.OK:
        c.commit_wgrad(layer, ref)
    return st


# ------------------------------------------------------------------ Table "faults"
def test_fault_stale_ref_after_slot_reuse_preserves_current_record():
    c = make(M=1)
    assert c.bind(0, 0, 4096, 10 ** 6, 0, 8) == C.OK
    st, r1 = run_f(c, 0, key(0, 0))
    assert run_di(c, 0, key(0, 0), r1) == C.OK
    assert run_dw(c, 0, key(0, 0), r1, 4096, 0, 8, C.INIT) == C.OK
    # slot released; reuse it in the next epoch
    assert c.finalize() == C.OK and c.optimizer_commit() == C.OK
    st, r2 = run_f(c, 0, key(1, 0))
    assert r2 == (0, 2)
    before = copy.deepcopy(c.snapshot())
    assert run_di(c, 0, key(0, 0), r1) == C.STALE_REF
    assert run_di(c, 0, key(1, 0), r1) == C.STALE_REF
    assert c.snapshot() == before


def test_fault_repeated_di_rejected():
    c = make()
    _, r = run_f(c, 0, key(0, 0))
    assert run_di(c, 0, key(0, 0), r) == C.OK
    before = copy.deepcopy(c.snapshot())
    assert run_di(c, 0, key(0, 0), r) == C.DUPLICATE_CONSUMER
    assert c.snapshot() == before


def test_fault_finalize_with_missing_dw():
    c = make(M=2)
    c.bind(0, 0, 4096, 10 ** 6, 0, 8)
    c.bind(0, 1, 4096, 10 ** 6, 100, 8)
    refs = [run_f(c, 0, key(0, m))[1] for m in range(2)]
    for m in range(2):
        assert run_di(c, 0, key(0, m), refs[m]) == C.OK
    assert run_dw(c, 0, key(0, 0), refs[0], 4096, 0, 8, C.INIT) == C.OK
    assert c.finalize() == C.INCOMPLETE
    assert c.optimizer_commit() == C.NOT_QUIESCENT
    assert c.e_w == 0


def test_fault_write_after_aborted_write():
    c = make(M=2)
    c.bind(0, 0, 4096, 10 ** 6, 0, 8)
    c.bind(0, 1, 4096, 10 ** 6, 100, 8)
    refs = [run_f(c, 0, key(0, m))[1] for m in range(2)]
    for m in range(2):
        run_di(c, 0, key(0, m), refs[m])
    c.abort()                                       # the write of mb 0 failed
    assert run_dw(c, 0, key(0, 1), refs[1], 4096, 100, 8, C.INIT) == C.ARENA_INVALID
    assert c.finalize() == C.ARENA_INVALID
    assert c.rebuild() == C.OK and c.arena_valid


def test_fault_stale_cache():
    c = make(M=2)
    c.bind(0, 0, 4096, 10 ** 6, 0, 8)
    c.bind(0, 1, 4096, 10 ** 6, 0, 8)
    refs = [run_f(c, 0, key(0, m))[1] for m in range(2)]
    for m in range(2):
        run_di(c, 0, key(0, m), refs[m])
    run_dw(c, 0, key(0, 0), refs[0], 4096, 0, 8, C.INIT)
    run_dw(c, 0, key(0, 1), refs[1], 4096, 0, 8, C.ACCUM)
    assert c.finalize() == C.OK and c.optimizer_commit() == C.OK
    # microbatch 1 runs first after the version bump: its cache is stale
    assert run_f(c, 0, key(1, 1))[0] == C.STALE_CACHE
    st, r = run_f(c, 0, key(1, 0))
    assert st == C.OK and c.layers[0].e_c == 1


def test_commit_with_live_tape_withheld():
    c = make()
    run_f(c, 0, key(0, 0))
    assert c.optimizer_commit() == C.NOT_QUIESCENT and c.e_w == 0


def test_dest_checks():
    c = make(M=2)
    c.add_layer(0, 1, 4, 8, 16)
    assert c.bind(0, 0, 4096, 10 ** 6, 0, 8) == C.OK
    assert c.bind(0, 1, 4096, 10 ** 6, 0, 8) == C.OK              # shared view, same layer
    assert c.bind(1, 0, 4096, 10 ** 6, 8, 8) == C.DEST_ALIAS      # overlaps layer 0
    assert c.bind(1, 0, 4096, 10 ** 6, 32, 8) == C.OK
    assert c.bind(1, 1, 4096, 10 ** 6, 7, 8) == C.DEST_ALIAS
    assert c.bind(1, 1, 4096, 40, 32, 8) == C.INVALID_ARG         # does not fit
    assert c.bind(1, 1, 4096, 10 ** 6, 64, 7) == C.INVALID_ARG    # ld < K
    _, r = run_f(c, 0, key(0, 0))
    run_di(c, 0, key(0, 0), r)
    assert run_dw(c, 0, key(0, 0), r, 4096, 0, 9, C.INIT) == C.DEST_MISMATCH
    assert run_dw(c, 0, key(0, 0), r, 4096, 0, 8, C.ACCUM) == C.ORDER   # not initialised yet
    assert run_dw(c, 0, key(0, 0), r, 4096, 0, 8, C.INIT) == C.OK
    _, r1 = run_f(c, 0, key(0, 1))
    assert run_dw(c, 0, key(0, 1), r1, 4096, 0, 8, C.ACCUM) == C.ORDER  # dI has not run
    run_di(c, 0, key(0, 1), r1)
    assert run_dw(c, 0, key(0, 1), r1, 4096, 0, 8, C.INIT) == C.ORDER   # shared view already initialised
    assert run_dw(c, 0, key(0, 1), r1, 4096, 0, 8, C.ACCUM) == C.OK


def test_keys_and_pool():
    c = make(M=2)
    st, r = run_f(c, 0, key(0, 0))
    assert run_f(c, 0, key(0, 0))[0] == C.KEY_LIVE
    assert run_f(c, 0, key(0, 0, inv=1))[0] == C.POOL_FULL
    assert run_f(c, 0, key(0, 2))[0] == C.INVALID_ARG
    assert run_f(c, 0, key(1, 1))[0] == C.EPOCH
    assert run_f(c, 0, key(0, 1, unit=3))[0] == C.KEY_MISMATCH
    assert run_di(c, 0, key(0, 0, inv=1), r) == C.KEY_MISMATCH
    assert run_di(c, 0, key(0, 0), (0, 7)) == C.STALE_REF


# ------------------------------------------------------------------ invariants on random schedules
def random_schedule(seed, M=3, layers=2, steps=3, ops=150):
    """Drive the contract with random legal and illegal calls and check the invariants."""
    rng = random.Random(seed)
    c = C.Contract(M)
    for u in range(layers):
        c.add_layer(0, u, 4, 8, 16)
        for m in range(M):
            assert c.bind(u, m, 1 << 20, 1 << 20, (u * M + m) * 64, 8) == C.OK
    refs = {}
    for _ in range(ops):
        before = copy.deepcopy(c.snapshot())
        tok = c.token
        u, m = rng.randrange(layers), rng.randrange(M)
        e = c.e_w if rng.random() < 0.9 else c.e_w + rng.choice([-1, 1])
        k = key(e, m, unit=u)
        ref = refs.get((u, m), (m, rng.randrange(0, 4)))
        if rng.random() < 0.1:
            ref = (m, ref[1] + rng.choice([-1, 1]))
        what = rng.choice(["f", "f", "di", "dw", "fin", "commit"])
        if what == "f":
            st, r = run_f(c, u, k)
            if st == C.OK:
                refs[(u, m)] = r
                assert c.token == tok + 1                                  # Invariant 1
                assert c.layers[u].e_c == c.e_w                            # Invariant 3
                assert r[1] == before["layers"][u]["slots"][m][2] + 1      # Invariant 2 (monotonic)
        elif what == "di":
            st = run_di(c, u, k, ref)
            if st == C.OK:
                assert c.token == tok + 1
                assert ref[1] == c.layers[u].slots[m].generation           # Invariant 2
        elif what == "dw":
            st = run_dw(c, u, k, ref, 1 << 20, (u * M + m) * 64, 8, C.INIT)
            if st == C.OK:
                assert c.token == tok                                      # dW never moves the token
        elif what == "fin":
            st = c.finalize()
        else:
            st = c.optimizer_commit()
            if st == C.OK:
                assert not any(s.live for L in before_layers(before) for s in L)   # Invariant 4
                assert c.e_w == before["e_w"] + 1
        if st != C.OK:
            assert c.snapshot() == before, (what, st)
    return c


def before_layers(snap):
    class S:
        def __init__(self, t):
            self.live = t[0]
    return [[S(t) for t in L["slots"]] for L in snap["layers"]]


@pytest.mark.parametrize("seed", range(12))
def test_invariants_on_random_schedules(seed):
    random_schedule(seed)
