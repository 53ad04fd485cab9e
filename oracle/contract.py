"""The bookkeeping contract of a pipeline stage, as a plain state machine.

Written from §3 (the contract), Algorithm 1 (§4.1), §4.3 and §4.5 of the
paper, and Table "faults".  Every action is *checked* first; a rejected call
changes nothing (§4.1: checks come before the physical work, and the state
moves only once that work has succeeded; Table "faults": rejecting a stale
reference leaves the live record intact).  Only a failure of the
physical action itself aborts the epoch (§4.5).

State:
* TapeKey K = (e, s, m, u, i): epoch, stage, microbatch, sub-layer unit,
  invocation (§3.1).  A layer is identified by (s, u).
* Slot pool: one slot per configured microbatch per layer (slot p = m; §4.2: a
  dW's explicit microbatch index and its TapeRef must point at one slot).  Allocating
  increments the slot's generation g_p, starting from 0, so the first
  reference is (p, 1); release keeps g_p (§3.1, Invariant 2).
* Consumer bits {dI, dW}; the slot is released once both have run (§3.1).
* Effect token: advanced once by every state-mutating action, i.e. F and dI;
  a deferred dW never advances it (§3.2, Invariant 1).
* Versions: e_W per stage, e_C per layer; the first forward (m = 0) of an
  epoch refreshes the cache and sets e_C <- e_W; any other forward requires
  e_C = e_W (§3.3, Invariant 3).  A never-filled cache has e_C = -1.
* Arena: per (layer, microbatch) bound views (buffer address, offset, row
  stride) of a flat FP32 buffer; exactly-once writes per epoch; shared views
  are initialised by their first write and accumulated by later ones;
  overlapping views of different layers, or different views, are aliases
  (§3.4, §4.3).  A valid flag, cleared by an abort until rebuilt (§4.5).
* Checkpoints (§3.5, Invariant 4): taken only at a quiescent point (no live
  tape, no arena write since the last commit, a valid arena; Table "faults":
  a checkpoint with live work is withheld).  e_W is persistent; tapes, slot
  generations, the effect token and cache contents are process-local, so a
  restore keeps this process's token and generations and marks every weight
  cache stale, which makes the first forward refresh it.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional, Tuple

# Status names.  The C library reports the same outcomes under QE_<NAME>.
OK = "OK"
INVALID_ARG = "INVALID_ARG"
STALE_REF = "STALE_REF"
KEY_MISMATCH = "KEY_MISMATCH"
KEY_LIVE = "KEY_LIVE"
POOL_FULL = "POOL_FULL"
DUPLICATE_CONSUMER = "DUPLICATE_CONSUMER"
ORDER = "ORDER"
EPOCH = "EPOCH"
STALE_CACHE = "STALE_CACHE"
DEST_MISMATCH = "DEST_MISMATCH"
DEST_ALIAS = "DEST_ALIAS"
DUP_WRITE = "DUP_WRITE"
ARENA_INVALID = "ARENA_INVALID"
INCOMPLETE = "INCOMPLETE"
NOT_QUIESCENT = "NOT_QUIESCENT"
EXEC_FAILED = "HIP"

DI_BIT, DW_BIT = 1, 2
INIT, ACCUM = 0, 1

Key = Tuple[int, int, int, int, int]     # (epoch, stage, microbatch, unit, invocation)
Ref = Tuple[int, int]                    # (slot, generation)


@dataclasses.dataclass
class Slot:
    live: bool = False
    key: Optional[Key] = None
    generation: int = 0
    bits: int = 0
    tokens: int = 0


@dataclasses.dataclass
class Binding:
    buf: int           # buffer base address (bytes)
    buf_elems: int
    offset: int        # elements
    ld: int            # elements
    written: bool = False

    def start(self) -> int:
        return self.buf + 4 * self.offset


@dataclasses.dataclass
class LayerInfo:
    stage: int
    unit: int
    n: int
    k: int
    max_tokens: int
    e_c: int = -1
    refreshes: int = 0
    slots: List[Slot] = dataclasses.field(default_factory=list)

    def span(self, ld: int) -> int:
        return (self.n - 1) * ld + self.k


class Contract:
    def __init__(self, microbatches: int):
        if microbatches < 1:
            raise ValueError("microbatches must be >= 1")
        self.M = microbatches
        self.layers: List[LayerInfo] = []
        self.e_w = 0
        self.token = 0
        self.arena_valid = True
        self.finalized = False
        self.bindings: Dict[Tuple[int, int], Binding] = {}
        self.fail_countdown = 0     # n > 0: the n-th next physical action fails

    # ---------------------------------------------------------------- setup
    def add_layer(self, stage: int, unit: int, n: int, k: int, max_tokens: int) -> int:
        self.layers.append(LayerInfo(stage, unit, n, k, max_tokens, slots=[Slot() for _ in range(self.M)]))
        return len(self.layers) - 1

    def inject_fault(self, n: int) -> None:
        self.fail_countdown = n

    def _physical_fails(self) -> bool:
        if self.fail_countdown > 0:
            self.fail_countdown -= 1
            if self.fail_countdown == 0:
                return True
        return False

    # ---------------------------------------------------------------- forward
    def check_fwd(self, layer: int, key: Key, tokens: int):
        """Returns (status, refresh)."""
        if not (0 <= layer < len(self.layers)):
            return INVALID_ARG, False
        L = self.layers[layer]
        e, s, m, u, _ = key
        if s != L.stage or u != L.unit:
            return KEY_MISMATCH, False
        if not (0 <= m < self.M) or not (0 <= tokens <= L.max_tokens):
            return INVALID_ARG, False
        if e != self.e_w:
            return EPOCH, False
        slot = L.slots[m]
        if slot.live:
            return (KEY_LIVE if slot.key == tuple(key) else POOL_FULL), False
        refresh = L.e_c != self.e_w
        if refresh and m != 0:
            return STALE_CACHE, False
        return OK, refresh

    def commit_fwd(self, layer: int, key: Key, tokens: int, refresh: bool) -> Ref:
        L = self.layers[layer]
        m = key[2]
        slot = L.slots[m]
        slot.generation += 1
        slot.live, slot.key, slot.bits, slot.tokens = True, tuple(key), 0, tokens
        self.token += 1
        if refresh:
            L.e_c = self.e_w
            L.refreshes += 1
        return (m, slot.generation)

    # ---------------------------------------------------------------- shared ref checks
    def _resolve(self, layer: int, key: Key, ref: Ref):
        L = self.layers[layer]
        p, g = ref
        if not (0 <= p < self.M):
            return INVALID_ARG
        slot = L.slots[p]
        if not slot.live or slot.generation != g:
            return STALE_REF
        if slot.key != tuple(key):
            return KEY_MISMATCH
        if key[0] != self.e_w:
            return EPOCH
        return OK

    def _check_dest(self, layer: int, m: int, buf: int, offset: int, ld: int, mode: int):
        b = self.bindings.get((layer, m))
        if b is None or b.buf != buf or b.offset != offset or b.ld != ld:
            return DEST_MISMATCH
        if b.written:
            return DUP_WRITE
        initialised = any(o.written and o.start() == b.start() and o.ld == b.ld
                          for o in self.bindings.values())
        if (mode == INIT) == initialised:
            return ORDER
        return OK

    # ---------------------------------------------------------------- dI
    def check_dgrad(self, layer: int, key: Key, ref: Ref):
        if not (0 <= layer < len(self.layers)):
            return INVALID_ARG
        st = self._resolve(layer, key, ref)
        if st != OK:
            return st
        if self.layers[layer].slots[ref[0]].bits & DI_BIT:
            return DUPLICATE_CONSUMER
        return OK

    def commit_dgrad(self, layer: int, ref: Ref) -> None:
        self.layers[layer].slots[ref[0]].bits |= DI_BIT
        self.token += 1

    # ---------------------------------------------------------------- dW
    def check_wgrad(self, layer: int, key: Key, ref: Ref, buf: int, offset: int, ld: int, mode: int):
        if not (0 <= layer < len(self.layers)) or mode not in (INIT, ACCUM):
            return INVALID_ARG
        if not self.arena_valid:
            return ARENA_INVALID
        st = self._resolve(layer, key, ref)
        if st != OK:
            return st
        bits = self.layers[layer].slots[ref[0]].bits
        if not bits & DI_BIT:
            return ORDER
        if bits & DW_BIT:
            return DUPLICATE_CONSUMER
        return self._check_dest(layer, ref[0], buf, offset, ld, mode)

    def _release_if_done(self, slot: Slot) -> None:
        if slot.bits == (DI_BIT | DW_BIT):
            slot.live, slot.key, slot.tokens = False, None, 0

    def commit_wgrad(self, layer: int, ref: Ref) -> None:
        slot = self.layers[layer].slots[ref[0]]
        slot.bits |= DW_BIT
        self.bindings[(layer, ref[0])].written = True
        self._release_if_done(slot)

    # ---------------------------------------------------------------- fused full backward
    def check_bwd_full(self, layer: int, key: Key, ref: Ref, buf: int, offset: int, ld: int, mode: int):
        if not (0 <= layer < len(self.layers)) or mode not in (INIT, ACCUM):
            return INVALID_ARG
        if not self.arena_valid:
            return ARENA_INVALID
        st = self._resolve(layer, key, ref)
        if st != OK:
            return st
        if self.layers[layer].slots[ref[0]].bits & (DI_BIT | DW_BIT):
            return DUPLICATE_CONSUMER
        return self._check_dest(layer, ref[0], buf, offset, ld, mode)

    def commit_bwd_full(self, layer: int, ref: Ref) -> None:
        slot = self.layers[layer].slots[ref[0]]
        slot.bits |= DI_BIT | DW_BIT
        self.token += 1
        self.bindings[(layer, ref[0])].written = True
        self._release_if_done(slot)

    # ---------------------------------------------------------------- arena
    def bind(self, layer: int, m: int, buf: int, buf_elems: int, offset: int, ld: int) -> str:
        if not (0 <= layer < len(self.layers)) or not (0 <= m < self.M):
            return INVALID_ARG
        L = self.layers[layer]
        if buf == 0 or offset < 0 or ld < L.k or buf_elems < offset + L.span(ld):
            return INVALID_ARG
        old = self.bindings.get((layer, m))
        if old is not None and old.written:
            return DUP_WRITE
        new = Binding(buf, buf_elems, offset, ld)
        lo, hi = new.start(), new.start() + 4 * L.span(ld)
        for (l2, m2), o in self.bindings.items():
            if (l2, m2) == (layer, m):
                continue
            olo = o.start()
            ohi = olo + 4 * self.layers[l2].span(o.ld)
            if lo < ohi and olo < hi:
                shared = (l2 == layer and olo == lo and o.ld == ld)
                if not shared:
                    return DEST_ALIAS
        self.bindings[(layer, m)] = new
        return OK

    def finalize(self) -> str:
        if not self.arena_valid:
            return ARENA_INVALID
        if any(not b.written for b in self.bindings.values()):
            return INCOMPLETE
        self.finalized = True
        return OK

    def optimizer_commit(self) -> str:
        if any(s.live for L in self.layers for s in L.slots):
            return NOT_QUIESCENT
        if not self.arena_valid:
            return ARENA_INVALID
        if self.bindings and not self.finalized:
            return INCOMPLETE
        self.e_w += 1
        for b in self.bindings.values():
            b.written = False
        self.finalized = False
        return OK

    def abort(self) -> None:
        for L in self.layers:
            for s in L.slots:
                if s.live and s.key[0] == self.e_w:
                    s.live, s.key, s.tokens = False, None, 0
        self.arena_valid = False
        self.finalized = False

    def rebuild(self) -> str:
        self.arena_valid = True
        for b in self.bindings.values():
            b.written = False
        self.finalized = False
        return OK

    # ---------------------------------------------------------------- checkpoint
    def checkpoint_check(self) -> str:
        if any(s.live for L in self.layers for s in L.slots):
            return NOT_QUIESCENT
        if self.finalized or any(b.written for b in self.bindings.values()):
            return NOT_QUIESCENT
        if not self.arena_valid:
            return ARENA_INVALID
        return OK

    def restore(self, e_w: int) -> str:
        st = self.checkpoint_check()
        if st != OK:
            return st
        self.e_w = int(e_w)
        for L in self.layers:
            L.e_c = -1
        return OK

    # ---------------------------------------------------------------- snapshot
    def snapshot(self) -> dict:
        """Everything a test compares against the library's reported state."""
        return {
            "e_w": self.e_w, "token": self.token, "arena_valid": self.arena_valid,
            "finalized": self.finalized,
            "layers": [{"e_c": L.e_c, "refreshes": L.refreshes,
                        "slots": [(s.live, s.key if s.live else None, s.generation, s.bits,
                                   s.tokens if s.live else 0) for s in L.slots]}
                       for L in self.layers],
            "written": {k: b.written for k, b in sorted(self.bindings.items())},
        }
