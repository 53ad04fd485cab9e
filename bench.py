"""Benchmark: one pass of the FP8 split-linear hot path over a Llama-shaped stage.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME] [--eager]

A step runs, for every linear of the stage (QKV, O, gate+up, down of the
Llama-3-70B shape by default, one microbatch of 8192 tokens, bf16 inputs and
master weights, amax history 1024):  F (with the weight-cache refresh, since
every step follows a version bump), then dI and the deferred dW with direct
placement into one flat FP32 main-gradient buffer, then arena finalize and
optimizer commit.  The stage's graphs are captured before the first step
(qe_prebuild_graphs) and every action is one HIP-graph replay, by default on
the caller's stream (stream order gives both directions of the handoff;
--executor two-way runs the paper's two-way handoff through the library's
graph stream instead, and the line reports the other executor's step time
beside the headline).  Inputs are synthetic, seeded, and resident in HBM
before timing starts.

Prints one JSON line.  `value` is GEMM FLOPs (fwd + dI + dW, 2*M*N*K each)
per second over the whole step, quantization and scale updates included.
`roofline` is the GEMM kernel alone, timed with HIP events that its launches
carry on the stream the library launches it on, in an instrumented eager pass
over the same steps.
`cpu_baseline` times the CPU oracle stage by stage on a bounded sample of the
same workload.  Beside the headline the line carries the same steps under the
other executor, with the actions' kernels launched the other way (direct
launches against graph replay), with copied gradients, with current scaling,
after a checkpoint restart, and with the caller's buffers rotated every step
under the three ways a replayed graph meets new buffers; per-action latencies
of a single small linear; and the deferred dW GEMM alone at the zero-bubble
microbatch, INIT- and ACCUM-placed.  A progress line after every setup phase
and every pass goes to stderr.
"""
from __future__ import annotations

import os

# Thread counts of the CPU oracle's BLAS, fixed before NumPy loads (a value
# already in the environment wins).
_THREADS = os.environ.get("OMP_NUM_THREADS") or str(min(16, len(os.sched_getaffinity(0))))
os.environ.setdefault("OMP_NUM_THREADS", _THREADS)
os.environ.setdefault("OPENBLAS_NUM_THREADS", _THREADS)

import argparse  # noqa: E402
import json  # noqa: E402
import sys  # noqa: E402
import time  # noqa: E402

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

FP8_PEAK_TFLOPS = 5000.0      # MI355X dense FP8 MFMA
HBM_PEAK_GBS = 8000.0         # MI355X HBM3E
METRIC = "FP8 fwd+dI+dW TFLOP/s (% FP8 MFMA peak); quantize/wgrad-place GB/s (% HBM)"


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100, help="timed steps (the stage replayed 100 times by default)")
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="llama3_70b_stage_8192tok")
    ap.add_argument("--eager", action="store_true", help="launch kernels directly instead of graph replay")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-ablation", action="store_true",
                    help="skip the copied-gradient passes (direct placement only)")
    ap.add_argument("--no-current", action="store_true", help="skip the current-scaling passes")
    ap.add_argument("--no-checkpoint", action="store_true", help="skip the checkpoint / restart measurement")
    ap.add_argument("--executor", choices=("caller", "two-way"), default="caller",
                    help="caller: every action replayed on the caller's stream (stream order is the handoff); "
                         "two-way: on the library's graph stream behind the paper's two-way handoff")
    ap.add_argument("--no-executor", action="store_true", help="skip the pass with the other executor")
    ap.add_argument("--no-launch-mode", action="store_true",
                    help="skip the pass that launches the same actions the other way (direct launches under graph "
                         "replay, graph replay under --eager)")
    ap.add_argument("--no-wgrad", action="store_true",
                    help="skip the dW-placement measurement at the zero-bubble workload's 2048-token microbatch")
    ap.add_argument("--no-latency", action="store_true",
                    help="skip the per-action latency of the small single-linear schedule")
    ap.add_argument("--wgrad-only", action="store_true",
                    help="run only the dW-placement leg (zero-bubble microbatch) and print its JSON")
    ap.add_argument("--no-rotate", action="store_true",
                    help="skip the passes with the caller's buffers rotated every step")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="BYTES",
                    help="only run a plain device copy of BYTES bytes (counter calibration)")
    return ap.parse_args()


GEMM_SOURCE = os.path.join(ROOT, "paper_2609_23536_amd", "csrc", "gemm_fp8.hip")


def gemm_traffic_per_launch(workload):
    """HBM bytes per GEMM launch from the committed counter runs on this
    workload, or None when there are none or they were taken on a different
    GEMM kernel source than the current one."""
    import hashlib
    path = os.path.join(ROOT, "profiles", f"gemm_{workload}_traffic.txt")
    if not os.path.exists(path):
        return None
    kv = {}
    for line in open(path):
        if ":" in line and not line.startswith("#"):
            k, v = line.split(":", 1)
            kv[k.strip()] = v.strip()
    sha = hashlib.sha256(open(GEMM_SOURCE, "rb").read()).hexdigest()
    if kv.get("kernel_source_sha256") != sha or kv.get("workload") != workload:
        return None
    return float(kv["gemm_hbm_bytes_per_launch"])


def copy_calibration(nbytes):
    import torch
    src = torch.empty(nbytes, dtype=torch.uint8, device="cuda:0")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes": nbytes, "copies": 3}))


_RESIDENT = {}  # workload -> (weights, inputs, output gradients) on the device


def resident_inputs(torch, wl, device):
    """The seeded weights, inputs and output gradients of `wl`, generated on the
    host once per workload and kept on the device (every pass only reads them)."""
    import numpy as np
    import workloads as W
    key = (wl.key, str(device))
    if key in _RESIDENT:
        return _RESIDENT[key]
    _RESIDENT.clear()
    bf = wl.in_dtype == "bf16"

    def up(t):
        a = t.data.view(np.int16) if bf else t.data
        return torch.from_numpy(a).to(device)

    ws, xs, dys = [], [], []
    for u, lin in enumerate(wl.linears):
        t0 = time.perf_counter()
        ws.append(up(W.layer_weight(wl, u)))
        inp = W.layer_inputs(wl, u)
        xs.append(up(inp["x"]))
        dys.append(up(inp["dy"]))
        del inp
        progress(f"inputs of {lin.name} ({lin.k_in}->{lin.n_out}, {wl.tokens} tokens) generated and uploaded "
                 f"in {time.perf_counter() - t0:.1f} s")
    _RESIDENT[key] = (ws, xs, dys)
    return _RESIDENT[key]


class StageBench:
    """One stage context over the workload's linears.  `rotate` > 1 hands every
    action one of `rotate` sets of X / dY / Y / dX buffers in turn (as a
    training loop hands the layer new activation and gradient tensors);
    `prebuild` captures the stage's graphs before the first step."""

    def __init__(self, qe, torch, wl, use_graphs, device, copy_gradients=False, current=False,
                 replay_on_caller=False, graph_inputs=0, rotate=1, prebuild=True):
        self.qe, self.torch, self.wl, self.d = qe, torch, wl, device
        self.ctx = qe.Context(1, use_graphs=use_graphs, copy_gradients=copy_gradients,
                              replay_on_caller=replay_on_caller, graph_inputs=graph_inputs)
        self.n_lin = len(wl.linears)
        bf = wl.in_dtype == "bf16"
        self.dt = qe.BF16 if bf else qe.F32
        tdt = torch.int16 if bf else torch.float32
        ws, xs, dys = resident_inputs(torch, wl, device)
        self.w = list(ws)
        self.rotate = rotate
        self.x = [[x] + [x.clone() for _ in range(rotate - 1)] for x in xs]
        self.dy = [[dy] + [dy.clone() for _ in range(rotate - 1)] for dy in dys]
        self.y = [[torch.empty((wl.tokens, lin.n_out), dtype=tdt, device=device) for _ in range(rotate)]
                  for lin in wl.linears]
        self.dx = [[torch.empty((wl.tokens, lin.k_in), dtype=tdt, device=device) for _ in range(rotate)]
                   for lin in wl.linears]
        for u, lin in enumerate(wl.linears):
            st, idx = self.ctx.qe_layer_register(0, u, lin.n_out, lin.k_in, wl.tokens, self.w[u], self.dt,
                                                 1 if current else wl.history, wl.margin,
                                                 scaling=qe.SCALING_CURRENT if current else qe.SCALING_DELAYED)
            assert st == "OK" and idx == u, st
        self.grad = torch.zeros(wl.flat_grad_elems(), dtype=torch.float32, device=device)
        self.offs = wl.grad_offsets()
        for u, lin in enumerate(wl.linears):
            st = self.ctx.qe_arena_bind(u, 0, self.grad, self.grad.numel(), self.offs[u], lin.k_in)
            assert st == "OK", st
        self.prebuild_ms = None
        if use_graphs and prebuild:
            st = self.ctx.qe_prebuild_graphs(wl.tokens, self.dt, self.dt, self.dt, self.dt)
            assert st == "OK", st
            self.prebuild_ms = self.ctx.qe_get_state()["prebuild_ns"] / 1e6
        self.epoch = 0
        self.nstep = 0

    def step(self):
        qe, wl, ctx = self.qe, self.wl, self.ctx
        r = self.nstep % self.rotate
        refs = []
        for u in range(self.n_lin):
            st, ref = ctx.qe_fp8_linear_fwd(u, qe.key(self.epoch, 0, 0, u), self.x[u][r], self.dt, wl.tokens,
                                            self.y[u][r], self.dt)
            assert st == "OK", st
            refs.append(ref)
        for u in reversed(range(self.n_lin)):
            k = qe.key(self.epoch, 0, 0, u)
            st = ctx.qe_fp8_linear_dgrad(u, k, refs[u], self.dy[u][r], self.dt, self.dx[u][r], self.dt)
            assert st == "OK", st
            st = ctx.qe_fp8_linear_wgrad_place(u, k, refs[u], self.grad, self.offs[u], wl.linears[u].k_in, qe.INIT)
            assert st == "OK", st
        assert ctx.qe_arena_finalize() == "OK"
        assert ctx.qe_optimizer_commit() == "OK"
        self.epoch += 1
        self.nstep += 1


def per_action_latency(qe, torch, device, steps=200, warmup=10):
    """Latency-bound case: one FP8 linear (K = N = 256), two microbatches of 128
    tokens, fp32 inputs, history 4, schedule F0 F1 dI0 dI1 dW0 dW1 (both dW into
    one shared view: INIT, then ACCUM), then finalize and commit.  Mean wall time
    per action: graph replay and direct launches, each behind the two-way
    handoff (the graph stream) and on the caller's stream; and, on the caller's
    stream, with the caller's X / dY / Y / dX buffers rotated over three sets
    every step under the three ways a replayed graph can meet new buffers
    (kernel-node arguments rewritten in place, the paper's static buffers with
    copies, a new capture)."""
    import numpy as np
    import workloads as W
    wl = W.WORKLOADS["single_linear_128x256x256"]
    lin = wl.linears[0]
    R = 3

    def up(t):
        return torch.from_numpy(np.ascontiguousarray(t.data)).to(device)

    modes = {"graph": (True, False, qe.GRAPH_INPUTS_REBIND, 1), "eager": (False, False, 0, 1),
             "graph_on_caller": (True, True, qe.GRAPH_INPUTS_REBIND, 1), "eager_on_caller": (False, True, 0, 1),
             "rotate_rebind": (True, True, qe.GRAPH_INPUTS_REBIND, R),
             "rotate_copy": (True, True, qe.GRAPH_INPUTS_COPY, R),
             "rotate_recapture": (True, True, qe.GRAPH_INPUTS_RECAPTURE, R),
             "rotate_eager": (False, True, 0, R)}
    res, counters = {}, {}
    for mode, (graphs, on_caller, gi, rot) in modes.items():
        ctx = qe.Context(wl.microbatches, use_graphs=graphs, replay_on_caller=on_caller, graph_inputs=gi)
        w = up(W.layer_weight(wl, 0))
        st, idx = ctx.qe_layer_register(0, 0, lin.n_out, lin.k_in, wl.tokens, w, qe.F32, wl.history, wl.margin)
        assert st == "OK" and idx == 0, st
        grad = torch.zeros(lin.n_out * lin.k_in, dtype=torch.float32, device=device)
        for m in range(wl.microbatches):
            assert ctx.qe_arena_bind(0, m, grad, grad.numel(), 0, lin.k_in) == "OK"
        if graphs:
            assert ctx.qe_prebuild_graphs(wl.tokens, qe.F32, qe.F32, qe.F32, qe.F32) == "OK"
        xs = [[up(W.layer_inputs(wl, 0, mb=m)["x"]) for _ in range(rot)] for m in range(wl.microbatches)]
        dys = [[up(W.layer_inputs(wl, 0, mb=m)["dy"]) for _ in range(rot)] for m in range(wl.microbatches)]
        ys = [[torch.empty((wl.tokens, lin.n_out), dtype=torch.float32, device=device) for _ in range(rot)]
              for _ in range(wl.microbatches)]
        dxs = [[torch.empty((wl.tokens, lin.k_in), dtype=torch.float32, device=device) for _ in range(rot)]
               for _ in range(wl.microbatches)]
        epoch = [0]

        def step():
            r = epoch[0] % rot
            refs = []
            for m in range(wl.microbatches):
                st, ref = ctx.qe_fp8_linear_fwd(0, qe.key(epoch[0], 0, m, 0), xs[m][r], qe.F32, wl.tokens, ys[m][r],
                                                qe.F32)
                assert st == "OK", st
                refs.append(ref)
            for m in range(wl.microbatches):
                st = ctx.qe_fp8_linear_dgrad(0, qe.key(epoch[0], 0, m, 0), refs[m], dys[m][r], qe.F32, dxs[m][r],
                                             qe.F32)
                assert st == "OK", st
            for m in range(wl.microbatches):
                st = ctx.qe_fp8_linear_wgrad_place(0, qe.key(epoch[0], 0, m, 0), refs[m], grad, 0, lin.k_in,
                                                   qe.INIT if m == 0 else qe.ACCUM)
                assert st == "OK", st
            assert ctx.qe_arena_finalize() == "OK"
            assert ctx.qe_optimizer_commit() == "OK"
            epoch[0] += 1

        for _ in range(warmup):
            step()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(steps):
            step()
        torch.cuda.synchronize()
        el = time.perf_counter() - t0
        assert ctx.qe_sync() == "OK"
        stt = ctx.qe_get_state()
        assert stt["device_token"] == stt["token"]
        res[mode] = el / (steps * 3 * wl.microbatches) * 1e6
        counters[mode] = {"captures": stt["captures"], "rebinds": stt["rebinds"]}
        ctx.close()
    out = {"workload": wl.key, "actions_per_step": 3 * wl.microbatches,
           "graph_us_per_action": round(res["graph"], 2), "eager_us_per_action": round(res["eager"], 2),
           "eager_over_graph": round(res["eager"] / res["graph"], 3),
           "graph_on_caller_us_per_action": round(res["graph_on_caller"], 2),
           "eager_on_caller_us_per_action": round(res["eager_on_caller"], 2)}
    out["rotating_buffers"] = {
        "buffer_sets": R, "executor": "replay_on_caller",
        **{m[len("rotate_"):] + "_us_per_action": round(res[m], 2) for m in res if m.startswith("rotate_")},
        "graphs_prebuilt": 3 * wl.microbatches,
        "captures": {m[len("rotate_"):]: counters[m]["captures"] for m in counters if m.startswith("rotate_")},
        "rebinds": counters["rotate_rebind"]["rebinds"]}
    return out


def wgrad_place(qe, torch, device, tokens=2048, reps=20):
    """The deferred dW GEMM with direct placement at the zero-bubble workload's
    microbatch (2048 tokens) and the Llama-3-8B stage's four linears: dW =
    dY^T X from the transposed E5M2 / E4M3 codes, placed into [N, K] views of
    one flat FP32 buffer (each view at its own offset, as per microbatch):
    INIT (the headline figures) and ACCUM (read-add-write, as when microbatches
    share one view).  Algorithmic bytes per launch: (N + K) * tokens code bytes
    read + 4 N K written (INIT) or 8 N K read and written (ACCUM); roofline time
    max(FLOPs / MFMA peak, bytes / HBM peak)."""
    import workloads as W
    wl = W.WORKLOADS["llama3_8b_zb_8x2048"]
    assert wl.tokens == tokens
    one = torch.ones(1, device=device)
    offs = wl.grad_offsets()
    grad = torch.zeros(wl.flat_grad_elems(), dtype=torch.float32, device=device)
    res = {}
    for mode, out_bytes in ((qe.INIT, 4), (qe.ACCUM, 8)):
        tot_t = tot_b = tot_f = tot_roof = 0.0
        per = []
        for u, lin in enumerate(wl.linears):
            n, k = lin.n_out, lin.k_in
            g = torch.Generator(device=device)
            g.manual_seed(u)
            a = (torch.randn(n, tokens, device=device, generator=g) * 0.5).to(torch.float8_e5m2).view(torch.uint8)
            b = (torch.randn(k, tokens, device=device, generator=g) * 0.5).to(torch.float8_e4m3fn).view(torch.uint8)
            view = grad[offs[u]:]

            def run():
                st = qe.qe_fp8_gemm_tn(a, qe.E5M2, tokens, b, qe.E4M3, tokens, n, k, tokens, one, one, view, qe.F32,
                                       k, mode)
                assert st == "OK", st

            for _ in range(3):
                run()
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(reps):
                run()
            e1.record()
            e1.synchronize()
            t = e0.elapsed_time(e1) / reps * 1e-3
            byts = (n + k) * tokens + out_bytes * n * k
            flop = 2.0 * n * k * tokens
            roof = max(flop / (FP8_PEAK_TFLOPS * 1e12), byts / (HBM_PEAK_GBS * 1e9))
            per.append({"linear": lin.name, "n": n, "k": k, "us": round(t * 1e6, 2), "gbs": round(byts / t / 1e9, 1),
                        "tflops": round(flop / t / 1e12, 1), "roofline_frac": round(roof / t, 4),
                        "bound": "hbm" if byts / (HBM_PEAK_GBS * 1e9) > flop / (FP8_PEAK_TFLOPS * 1e12) else "mfma"})
            tot_t += t
            tot_b += byts
            tot_f += flop
            tot_roof += roof
        res[mode] = {"achieved_gbs": round(tot_b / tot_t / 1e9, 1), "unit": "GB/s", "peak_gbs": HBM_PEAK_GBS,
                     "frac_hbm": round(tot_b / tot_t / 1e9 / HBM_PEAK_GBS, 4), "tflops": round(tot_f / tot_t / 1e12, 1),
                     "roofline_frac": round(tot_roof / tot_t, 4), "per_linear": per}
    out = {"workload": wl.key, "tokens": tokens, "placement": "INIT into per-view offsets of one flat FP32 buffer"}
    out.update(res[qe.INIT])
    acc = res[qe.ACCUM]
    out["accumulate"] = {"placement": "ACCUM (read-add-write) into the same views", **acc}
    return out


def timed_ms(b, torch, warmup, steps):
    """Mean wall time of `steps` steps after `warmup` untimed ones, device-synchronised."""
    for _ in range(warmup):
        b.step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        b.step()
    torch.cuda.synchronize()
    return (time.perf_counter() - t0) / steps * 1e3


def amax_bytes(wl):
    """Per step under current scaling: the amax pass reads X, dY and (refresh) W once each."""
    b_in = 2 if wl.in_dtype == "bf16" else 4
    return sum((wl.tokens * (lin.k_in + lin.n_out) + lin.n_out * lin.k_in) * b_in for lin in wl.linears)


def qbytes_per_step(wl):
    """Per step: quantize bytes (in + row codes + column codes) of X, dY and the W refresh."""
    b_in = 2 if wl.in_dtype == "bf16" else 4
    q = 0
    for lin in wl.linears:
        q += wl.tokens * lin.k_in * (b_in + 2)       # X
        q += wl.tokens * lin.n_out * (b_in + 2)      # dY
        q += lin.n_out * lin.k_in * (b_in + 2)       # W refresh
    return q


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(wl, rows=8192, tokens=4096):
    """The CPU oracle as it stands, stage by stage, on a bounded sample of the
    workload: its O projection (K = hidden) restricted to the first `rows`
    output features of the weight (the first rows of the same seeded draw) at
    `tokens` tokens, through F (with the weight-cache refresh), dI and dW with
    INIT placement, each stage timed with perf_counter on the host's cores.
    `value` is the sample's GEMM FLOPs over the time of all its stages (the
    headline's definition); the stages report GFLOP/s or GB/s of algorithmic
    work."""
    import numpy as np
    import workloads as W
    from oracle.gemm import gemm_tn, place, quantize_with_amax
    from oracle.scaling import DelayedScaler
    try:
        from threadpoolctl import threadpool_info
        cores = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:
        cores = int(os.environ.get("OMP_NUM_THREADS", len(os.sched_getaffinity(0))))
    u = 1
    lin = wl.linears[u]
    k, n, t = lin.k_in, min(rows, lin.n_out), min(tokens, wl.tokens)
    b_in = 2 if wl.in_dtype == "bf16" else 4
    w = W.normal(W.rng_for(0, wl.cfg, u, W.ROLE_W), (n, k), 0.02, wl.in_dtype).as_f32()
    inp = W.layer_inputs(wl, u, tokens=t)
    x = inp["x"].as_f32()
    dy = np.ascontiguousarray(inp["dy"].as_f32()[:, :n])
    sx, sw, sdy = (DelayedScaler(f, wl.history, wl.margin) for f in ("E4M3", "E4M3", "E5M2"))
    stages, tot = [], [0.0]

    def timed(name, fn, work, unit):
        t0 = time.perf_counter()
        r = fn()
        el = time.perf_counter() - t0
        tot[0] += el
        rate = work / el / 1e9 if el > 0 else None
        stages.append({"stage": name, "seconds": round(el, 4), "value": None if rate is None else round(rate, 3),
                       "unit": unit})
        return r

    wq, wq_t, a_w = timed("quantize W (cast + transpose + amax)",
                          lambda: quantize_with_amax(w, sw.scale, "E4M3"), n * k * (b_in + 2), "GB/s")
    xq, xq_t, a_x = timed("quantize X (cast + transpose + amax)",
                          lambda: quantize_with_amax(x, sx.scale, "E4M3"), t * k * (b_in + 2), "GB/s")
    timed("GEMM fwd Y = X W^T", lambda: gemm_tn(xq, "E4M3", wq, "E4M3", sx.scale_inv, sw.scale_inv),
          2.0 * t * n * k, "GFLOP/s")

    def upd(*ss_amax):
        for sc, a in ss_amax:
            if a is not None:
                sc.record(a)
            sc.update()
    t0 = time.perf_counter()
    upd((sx, a_x), (sw, a_w))
    el_u = time.perf_counter() - t0
    dyq, dyq_t, a_dy = timed("quantize dY (cast + transpose + amax)",
                             lambda: quantize_with_amax(dy, sdy.scale, "E5M2"), t * n * (b_in + 2), "GB/s")
    timed("GEMM dI dX = dY W", lambda: gemm_tn(dyq, "E5M2", wq_t, "E4M3", sdy.scale_inv, sw.scale_inv),
          2.0 * t * n * k, "GFLOP/s")
    t0 = time.perf_counter()
    upd((sdy, a_dy))
    el_u += time.perf_counter() - t0
    tot[0] += el_u
    stages.append({"stage": "scale updates (X, W, dY)", "seconds": round(el_u, 6),
                   "us_per_update": round(el_u / 3 * 1e6, 2)})
    d = timed("GEMM dW = dY^T X", lambda: gemm_tn(dyq_t, "E5M2", xq_t, "E4M3", sdy.scale_inv, sx.scale_inv),
              2.0 * t * n * k, "GFLOP/s")
    buf = np.zeros(n * k, dtype=np.float32)
    timed("placement INIT into the flat FP32 buffer", lambda: place(buf, d, 0, k, accumulate=False), 4.0 * n * k,
          "GB/s")
    flops = 3 * 2.0 * t * n * k
    return {"value": round(flops / tot[0] / 1e12, 6), "unit": "TFLOP/s", "cores": int(cores), "kind": "oracle",
            "cpu": cpu_model(), "omp_num_threads": os.environ.get("OMP_NUM_THREADS"),
            "sample": f"{lin.name} {k}->{n} (first {n} of {lin.n_out} output features) at {t} tokens of {wl.key}: "
                      f"F (with W refresh) + dI + dW through the float64 oracle, {tot[0]:.2f} s",
            "stages": stages}


def progress(msg):
    """One line per finished pass on stderr (stdout carries only the JSON result line)."""
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def main():
    args = parse()
    if args.copy_calibration:
        copy_calibration(args.copy_calibration)
        return
    if args.gpus != 1:
        print(json.dumps({"error": "the benchmark runs on one GPU; --gpus must be 1 (no multi-GPU path is built)"}))
        sys.exit(2)
    import torch
    import workloads as W
    from paper_2609_23536_amd import qe

    if not torch.cuda.is_available():
        print(json.dumps({"error": "no GPU visible"}))
        sys.exit(2)
    qe.lib()
    dev = torch.device("cuda:0")
    torch.zeros(1, device=dev)
    progress("torch and the library loaded, device initialised")
    if args.wgrad_only:
        print(json.dumps({"wgrad_place": wgrad_place(qe, torch, dev)}), flush=True)
        return
    wl = W.WORKLOADS[args.workload]
    use_graphs = not args.eager

    on_caller = args.executor == "caller"
    b = StageBench(qe, torch, wl, use_graphs, dev, replay_on_caller=on_caller)
    progress(f"stage registered ({len(wl.linears)} linears); graphs prebuilt in "
             f"{b.prebuild_ms if b.prebuild_ms is not None else 0:.1f} ms")
    for _ in range(args.warmup):
        b.step()
    torch.cuda.synchronize()
    progress(f"{args.warmup} warm-up steps done")
    t0 = time.perf_counter()
    for _ in range(args.steps):
        b.step()
    torch.cuda.synchronize()
    el = time.perf_counter() - t0
    assert b.ctx.qe_sync() == "OK"
    st = b.ctx.qe_get_state()
    assert st["device_token"] == st["token"]

    flops = wl.gemm_flops_per_pass()
    ms = el / args.steps * 1e3
    value = flops / (el / args.steps) / 1e12
    progress(f"timed pass: {ms:.4f} ms per step ({wl.key})")

    # quiescent checkpoint at this optimizer boundary, restart into a fresh context
    ckpt = None
    if not args.no_checkpoint:
        t0 = time.perf_counter()
        cst, payload = b.ctx.qe_checkpoint_export()
        export_ms = (time.perf_counter() - t0) * 1e3
        assert cst == "OK", cst
        epoch = b.epoch
    b.ctx.close()
    del b
    torch.cuda.empty_cache()
    if not args.no_checkpoint:
        r = StageBench(qe, torch, wl, use_graphs, dev, replay_on_caller=on_caller)
        r.epoch = epoch
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        assert r.ctx.qe_checkpoint_import(payload) == "OK"
        import_ms = (time.perf_counter() - t0) * 1e3
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        r.step()                                  # graphs prebuilt again, caches refreshed
        torch.cuda.synchronize()
        first_ms = (time.perf_counter() - t0) * 1e3
        after_ms = timed_ms(r, torch, 0, 3)
        progress("checkpoint / restart pass")
        assert r.ctx.qe_sync() == "OK"
        rst = r.ctx.qe_get_state()
        assert rst["device_token"] == rst["token"] and rst["e_w"] == epoch + 4
        ckpt = {"payload_bytes": len(payload), "export_ms": round(export_ms, 3), "import_ms": round(import_ms, 3),
                "first_step_after_restart_ms": round(first_ms, 3), "steady_step_after_restart_ms": round(after_ms, 4),
                "graphs_prebuilt_after_restart_ms": r.prebuild_ms, "graph_captures_after_restart": rst["captures"]}
        r.ctx.close()
        del r
        torch.cuda.empty_cache()

    # ablation: the copied-gradient path (dW to a private buffer, then a copy
    # into the view) against direct placement, same steps, same replay mode
    copied_ms = None
    if not args.no_ablation:
        c = StageBench(qe, torch, wl, use_graphs, dev, copy_gradients=True, replay_on_caller=on_caller)
        copied_ms = timed_ms(c, torch, args.warmup, args.steps)
        progress("copied-gradient pass")
        c.ctx.close()
        del c
        torch.cuda.empty_cache()

    # current (dynamic) scaling: the same step with every cast scaled by its own tensor's amax
    current_ms = None
    if not args.no_current:
        c = StageBench(qe, torch, wl, use_graphs, dev, current=True, replay_on_caller=on_caller)
        current_ms = timed_ms(c, torch, args.warmup, args.steps)
        progress("current-scaling pass")
        assert c.ctx.qe_sync() == "OK"
        cst = c.ctx.qe_get_state()
        assert cst["device_token"] == cst["token"]
        c.ctx.close()
        del c
        torch.cuda.empty_cache()

    # the other executor on the same steps: the paper's two-way handoff through
    # the graph stream, or (with --executor two-way) replay on the caller's stream
    other_ms = None
    if not args.no_executor:
        c = StageBench(qe, torch, wl, use_graphs, dev, replay_on_caller=not on_caller)
        other_ms = timed_ms(c, torch, args.warmup, args.steps)
        progress("other-executor pass")
        assert c.ctx.qe_sync() == "OK"
        cst = c.ctx.qe_get_state()
        assert cst["device_token"] == cst["token"] and (cst["handoffs"] == 0) == (not on_caller)
        c.ctx.close()
        del c
        torch.cuda.empty_cache()

    # the same steps with the actions' kernels launched the other way (direct
    # launches when the headline replays graphs), on the same executor
    mode_ms = None
    if not args.no_launch_mode:
        c = StageBench(qe, torch, wl, not use_graphs, dev, replay_on_caller=on_caller)
        mode_ms = timed_ms(c, torch, args.warmup, args.steps)
        assert c.ctx.qe_sync() == "OK"
        c.ctx.close()
        del c
        torch.cuda.empty_cache()
        progress("other launch-mode pass")

    # the caller's X / dY / Y / dX buffers rotated over three sets every step
    # (as a training loop hands the layer new tensors): kernel-node arguments
    # rewritten in place, the paper's static buffers with copies, re-capture
    rotation = None
    if use_graphs and not args.no_rotate:
        rotation = {"buffer_sets": 3}
        for name, gi in (("rebind", qe.GRAPH_INPUTS_REBIND), ("copy", qe.GRAPH_INPUTS_COPY),
                         ("recapture", qe.GRAPH_INPUTS_RECAPTURE)):
            c = StageBench(qe, torch, wl, True, dev, replay_on_caller=on_caller, graph_inputs=gi, rotate=3)
            r_ms = timed_ms(c, torch, args.warmup, args.steps)
            assert c.ctx.qe_sync() == "OK"
            cst = c.ctx.qe_get_state()
            assert cst["device_token"] == cst["token"]
            rotation[name] = {"ms_per_step": round(r_ms, 4), "step_time_vs_headline": round(r_ms / ms, 4),
                              "captures": cst["captures"], "rebinds": cst["rebinds"],
                              "capture_ms": round(cst["capture_ns"] / 1e6, 2)}
            c.ctx.close()
            del c
            torch.cuda.empty_cache()
            progress(f"rotating-buffer pass ({name})")

    latency = None if args.no_latency else per_action_latency(qe, torch, dev)
    progress("per-action latency leg")
    wgrad = None if args.no_wgrad else wgrad_place(qe, torch, dev)
    progress("dW-placement leg")
    torch.cuda.empty_cache()

    # instrumented eager passes: per-kernel-class times from the HIP events the launches carry
    def instrumented(copy_gradients=False, current=False):
        e = StageBench(qe, torch, wl, False, dev, copy_gradients=copy_gradients, current=current)
        e.step()
        torch.cuda.synchronize()
        e.ctx.qe_set_kernel_timing(True)
        for _ in range(args.steps):
            e.step()
        t = {k: e.ctx.qe_get_kernel_timing(k)
             for k in (qe.KC_GEMM, qe.KC_QUANT, qe.KC_UPDATE, qe.KC_COPY, qe.KC_AMAX)}
        e.ctx.close()
        del e
        torch.cuda.empty_cache()
        return t

    kt = instrumented(False)
    progress("instrumented pass")
    gemm_ms, gemm_n = kt[qe.KC_GEMM]
    q_ms, q_n = kt[qe.KC_QUANT]
    u_ms, u_n = kt[qe.KC_UPDATE]
    assert kt[qe.KC_COPY][1] == 0, "direct placement launched a gradient copy"
    if copied_ms is not None:
        c_ms, c_n = instrumented(copy_gradients=True)[qe.KC_COPY]
        progress("instrumented copied-gradient pass")
        # INIT placement (one microbatch): the copy reads the private FP32 dW and writes the view
        copy_bytes = sum(8 * lin.n_out * lin.k_in for lin in wl.linears)
        copy_gbs = copy_bytes * args.steps / (c_ms * 1e-3) / 1e9
    if current_ms is not None:
        kc = instrumented(current=True)
        progress("instrumented current-scaling pass")
        a_ms, a_n = kc[qe.KC_AMAX]
        cq_ms, cq_n = kc[qe.KC_QUANT]
        a_gbs = amax_bytes(wl) * args.steps / (a_ms * 1e-3) / 1e9
        cq_gbs = qbytes_per_step(wl) * args.steps / (cq_ms * 1e-3) / 1e9
    gemm_tflops = flops * args.steps / (gemm_ms * 1e-3) / 1e12
    qbytes = qbytes_per_step(wl)
    q_gbs = qbytes * args.steps / (q_ms * 1e-3) / 1e9

    out = {
        "metric": METRIC, "value": round(value, 2), "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "fp8(e4m3 x,w / e5m2 dy), f32 accumulate", "data": "synthetic",
        "config": {"workload": wl.key, "tokens": wl.tokens, "microbatches": wl.microbatches,
                   "linears": [[l.name, l.k_in, l.n_out] for l in wl.linears], "in_dtype": wl.in_dtype,
                   "amax_history": wl.history, "graphs": use_graphs,
                   "executor": "replay_on_caller" if on_caller else "graph_stream_two_way_handoff"},
        "frac_of_fp8_peak": round(value / FP8_PEAK_TFLOPS, 4),
        "roofline": {"bound": "mfma", "achieved": round(gemm_tflops, 2), "peak": FP8_PEAK_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(gemm_tflops / FP8_PEAK_TFLOPS, 4),
                     "traffic": gemm_traffic_per_launch(wl.key),
                     "kernel": "gemm_tn_w4_kernel / gemm_tn_kernel (fwd + dI + dW launches)",
                     "avg_launch_us": round(gemm_ms / gemm_n * 1e3, 2), "launches": gemm_n},
        "quantize": {"achieved": round(q_gbs, 1), "unit": "GB/s", "peak": HBM_PEAK_GBS,
                     "frac": round(q_gbs / HBM_PEAK_GBS, 4), "avg_launch_us": round(q_ms / q_n * 1e3, 2),
                     "launches": q_n},
        "scale_update": ({"avg_launch_us": round(u_ms / u_n * 1e3, 2), "launches": u_n} if u_n else
                         {"launches": 0, "fused": "runs in extra workgroups of the action's GEMM launch"}),
        "graph": {"graphs_prebuilt": 3 * wl.microbatches * len(wl.linears), "captures": st["captures"],
                  "replays": st["replays"], "rebinds": st["rebinds"], "handoffs": st["handoffs"],
                  "prebuild_ms": round(st["prebuild_ns"] / 1e6, 2), "capture_ms": round(st["capture_ns"] / 1e6, 2)},
        "targets": {"gemm_frac_of_fp8_peak": 0.60, "quantize_amax_wgrad_place_frac_of_hbm": 0.70},
    }
    if copied_ms is not None:
        out["direct_placement_ablation"] = {
            "copied_ms_per_step": round(copied_ms, 4), "direct_speedup_over_copied": round(copied_ms / ms, 4),
            "copies_per_step_direct": 0, "copies_per_step_copied": c_n // args.steps,
            "copy_bytes_per_step": copy_bytes, "copy_avg_launch_us": round(c_ms / c_n * 1e3, 2),
            "copy_achieved_gbs": round(copy_gbs, 1), "copy_frac_hbm": round(copy_gbs / HBM_PEAK_GBS, 4)}
    if ckpt is not None:
        out["checkpoint"] = ckpt
    if current_ms is not None:
        out["current_scaling"] = {
            "ms_per_step": round(current_ms, 4), "value": round(flops / (current_ms * 1e-3) / 1e12, 2),
            "unit": "TFLOP/s", "step_time_vs_delayed": round(current_ms / ms, 4),
            "amax": {"achieved": round(a_gbs, 1), "unit": "GB/s", "peak": HBM_PEAK_GBS,
                     "frac": round(a_gbs / HBM_PEAK_GBS, 4), "avg_launch_us": round(a_ms / a_n * 1e3, 2),
                     "launches": a_n, "bytes_per_step": amax_bytes(wl)},
            "quantize": {"achieved": round(cq_gbs, 1), "unit": "GB/s", "frac": round(cq_gbs / HBM_PEAK_GBS, 4),
                         "avg_launch_us": round(cq_ms / cq_n * 1e3, 2), "launches": cq_n}}
    if other_ms is not None:
        out["executor_" + ("two_way_handoff" if on_caller else "replay_on_caller")] = {
            "ms_per_step": round(other_ms, 4), "value": round(flops / (other_ms * 1e-3) / 1e12, 2),
            "unit": "TFLOP/s", "step_time_vs_headline": round(other_ms / ms, 4),
            "handoffs_per_step": 2 * 3 * wl.microbatches * len(wl.linears) if on_caller else 0}
    if mode_ms is not None:
        out["launch_mode_" + ("direct" if use_graphs else "graph_replay")] = {
            "ms_per_step": round(mode_ms, 4), "value": round(flops / (mode_ms * 1e-3) / 1e12, 2),
            "unit": "TFLOP/s", "step_time_vs_headline": round(mode_ms / ms, 4)}
    if rotation is not None:
        out["rotating_buffers"] = rotation
    if latency is not None:
        out["per_action_latency"] = latency
    if wgrad is not None:
        out["wgrad_place"] = wgrad
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(wl)
        progress("cpu baseline")
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
