"""Action orders used by the tests (F / dI / dW per microbatch), written out.

* single-linear order: F0 F1 dI0 dI1 dW0 dW1 into one shared gradient view
  (dW0 initialises it, dW1 accumulates).
* zero-bubble-style order over 8 microbatches: forwards run ahead, each dI
  follows in order, and the deferred dWs run out of order: reversed at the end
  of step 0, interleaved (some mid-schedule) in step 1.  Every microbatch has
  its own gradient view.
"""

SINGLE = [("F", 0), ("F", 1), ("dI", 0), ("dI", 1), ("dW", 0), ("dW", 1)]

_ZB_FDI = [("F", 0), ("F", 1), ("F", 2), ("F", 3), ("dI", 0), ("F", 4), ("dI", 1), ("F", 5), ("dI", 2),
           ("F", 6), ("dI", 3), ("F", 7), ("dI", 4), ("dI", 5), ("dI", 6), ("dI", 7)]

ZB_STEP0 = _ZB_FDI + [("dW", m) for m in reversed(range(8))]
ZB_STEP1 = [("F", 0), ("F", 1), ("F", 2), ("F", 3), ("dI", 0), ("F", 4), ("dI", 1), ("dW", 1), ("F", 5),
            ("dI", 2), ("dW", 0), ("F", 6), ("dI", 3), ("dW", 3), ("F", 7), ("dI", 4), ("dW", 2), ("dI", 5),
            ("dW", 5), ("dW", 4), ("dI", 6), ("dI", 7), ("dW", 7), ("dW", 6)]


def to_full(schedule):
    """The same F / dI order with each dW fused into its dI (a full backward)."""
    return [("B", m) if a == "dI" else (a, m) for a, m in schedule if a != "dW"]


def check_legal(schedule, M):
    seen = {}
    for a, m in schedule:
        assert 0 <= m < M
        prev = seen.get(m, [])
        want = {"F": [], "dI": ["F"], "dW": ["F", "dI"], "B": ["F"]}[a]
        assert prev == want, (a, m, prev)
        seen[m] = prev + [a] if a in ("F", "dI") else []
    assert not seen or all(v == [] for v in seen.values())
