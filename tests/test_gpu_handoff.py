"""Caller / graph stream handoff (§2.3 and Table "correctness", stream-ordering
row): with the two-way handoff a consumer enqueued on the caller stream right
after a replayed action always sees the action's final output; with only the
one-way edge (testing mode) it can observe stale data.  Checked with an
explicit caller stream and with the default stream, graph replay and direct
launches: a completion event recorded by a node inside the graph was found
not to order a waiting stream on this runtime, so the executor records it
after the launch, and these trials are what shows that it orders."""
import pytest

from tests.gpu_util import dev, torch
from tests.libqe import need_lib

pytestmark = pytest.mark.gpu


def stale_count(one_way: bool, trials: int, default_stream: bool = False, use_graphs: bool = True) -> int:
    qe = need_lib()
    d = dev()
    n, k, t = 28672, 4096, 4096
    ctx = qe.Context(1, use_graphs=use_graphs, one_way_handoff=one_way)
    g = torch.Generator(device=d)
    g.manual_seed(1)
    w = (torch.randn(n, k, device=d, generator=g) * 0.02).to(torch.bfloat16)
    x = torch.randn(t, k, device=d, generator=g).to(torch.bfloat16)
    st, L = ctx.qe_layer_register(0, 0, n, k, t, w, qe.BF16, 4, 0)
    assert st == "OK"
    y = torch.empty((t, n), dtype=torch.bfloat16, device=d)
    # The runtime maps streams onto a few hardware queues in turn; a caller
    # stream that shares the graph stream's queue is serialised with it and
    # can never see stale data, so the trials cycle over four caller streams
    # (consecutive ones sit on different queues).
    callers = [torch.cuda.default_stream(d)] if default_stream else [torch.cuda.Stream() for _ in range(4)]
    stale = 0
    for trial in range(trials):
        caller = callers[trial % len(callers)]
        with torch.cuda.stream(caller):
            y.fill_(float("nan"))                      # producer's output not written yet
            st, ref = ctx.qe_fp8_linear_fwd(L, qe.key(0, 0, 0, 0), x, qe.BF16, t, y, qe.BF16, caller=caller)
            assert st == "OK"
            seen = y.clone()                           # consumer on the caller stream
        torch.cuda.synchronize()
        assert ctx.qe_sync() == "OK"
        if not torch.equal(seen.view(torch.int16), y.view(torch.int16)):
            stale += 1
        assert ctx.qe_abort_epoch() == "OK" and ctx.qe_arena_rebuild() == "OK"   # free the slot
    assert not torch.isnan(y.float()).any()
    ctx.close()
    return stale


@pytest.mark.parametrize("default_stream", [False, True], ids=["explicit_stream", "default_stream"])
@pytest.mark.parametrize("use_graphs", [True, False], ids=["graphs", "eager"])
def test_two_way_handoff_never_stale(default_stream, use_graphs):
    assert stale_count(one_way=False, trials=30, default_stream=default_stream, use_graphs=use_graphs) == 0


def test_one_way_handoff_is_observably_stale():
    assert stale_count(one_way=True, trials=30) > 0
