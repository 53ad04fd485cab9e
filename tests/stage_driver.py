"""Runs an action schedule on the library (GPU) and on the oracle with the same
seeded inputs, so tests can compare them action by action."""
import numpy as np

import workloads as W
from oracle import contract as OC
from oracle.layer import Stage
from tests.gpu_util import dev_bytes, dev_f32, torch, upload


class Spec:
    def __init__(self, shapes, tokens, M, history, margin, in_dtype, shared_view, out_dtype="f32", seed=0,
                 cfg=90, outliers=False, scaling="delayed", w_dtype=None, fmt_w="E4M3", ld_pad=0):
        """`w_dtype`: the master weights' dtype (default `in_dtype`); `fmt_w`: W's FP8 format;
        `ld_pad`: each gradient view's row stride is K + ld_pad (elements between rows untouched)."""
        self.ld_pad = ld_pad
        self.shapes, self.tokens, self.M = shapes, tokens, M
        self.w_dtype, self.fmt_w = w_dtype or in_dtype, fmt_w
        self.history, self.margin, self.in_dtype = history, margin, in_dtype
        self.shared_view, self.out_dtype, self.seed, self.cfg = shared_view, out_dtype, seed, cfg
        self.outliers, self.scaling = outliers, scaling

    def ld(self, u):
        return self.shapes[u][1] + self.ld_pad

    def total(self):
        return sum(n * self.ld(u) for u, (n, k) in enumerate(self.shapes))

    def offset(self, u, m):
        offs = np.cumsum([0] + [n * self.ld(v) for v, (n, k) in enumerate(self.shapes)])
        return int(offs[u] if self.shared_view else m * self.total() + offs[u])

    def grad_elems(self):
        return self.total() * (1 if self.shared_view else self.M)

    def weight(self, u):
        n, k = self.shapes[u]
        return W.normal(W.rng_for(self.seed, self.cfg, u, W.ROLE_W), (n, k), 0.02, self.w_dtype)

    def inputs(self, u, m, step):
        n, k = self.shapes[u]
        rx = W.rng_for(self.seed, self.cfg, u, W.ROLE_X, m, step)
        rd = W.rng_for(self.seed, self.cfg, u, W.ROLE_DY, m, step)
        if self.outliers:
            x = W.outlier_activations(rx, self.tokens, k, 0.001 if k >= 1000 else 0.02, 300.0, self.in_dtype)
            dy = W.lognormal_signed(rd, (self.tokens, n), 2.0, self.in_dtype)
        else:
            x = W.normal(rx, (self.tokens, k), 1.0, self.in_dtype)
            dy = W.normal(rd, (self.tokens, n), 0.01, self.in_dtype)
        return x, dy


class GpuStage:
    def __init__(self, qe, spec, use_graphs=False, device=None, copy_gradients=False, weights=None,
                 replay_on_caller=False, streams=None, x_misaligned=False):
        """`weights`: the current master weights (workloads.Tensor per layer), default the initial ones.
        `streams`: caller streams used in turn, one per action (inputs are uploaded and outputs
        allocated on the action's stream); default torch's current stream.
        `x_misaligned`: hand F its input one element past a 16-byte boundary (so the cast of X
        takes the unaligned path while W's stays aligned)."""
        self.x_misaligned = x_misaligned
        self.qe, self.spec = qe, spec
        self.d = device
        self.ctx = qe.Context(spec.M, use_graphs=use_graphs, copy_gradients=copy_gradients,
                              replay_on_caller=replay_on_caller)
        self.streams = streams
        self.n_actions = 0
        dt = qe.BF16 if spec.w_dtype == "bf16" else qe.F32
        fw = qe.E4M3 if spec.fmt_w == "E4M3" else qe.E5M2
        self.w = [upload(spec.weight(u) if weights is None else weights[u], self.d) for u in range(len(spec.shapes))]
        for u, (n, k) in enumerate(spec.shapes):
            rec = qe.SCALING_CURRENT if spec.scaling == "current" else qe.SCALING_DELAYED
            st, idx = self.ctx.qe_layer_register(0, u, n, k, spec.tokens, self.w[u], dt, spec.history, spec.margin,
                                                 fmt_w=fw, scaling=rec)
            assert st == "OK" and idx == u
        self.grad = torch.zeros(spec.grad_elems(), dtype=torch.float32, device=self.d)
        for u, (n, k) in enumerate(spec.shapes):
            for m in range(spec.M):
                assert self.ctx.qe_arena_bind(u, m, self.grad, spec.grad_elems(), spec.offset(u, m),
                                              spec.ld(u)) == "OK"
        self.refs = {}
        self.written = set()
        self.outs = {}

    def _out(self, rows, cols):
        if self.spec.out_dtype == "bf16":
            return torch.zeros((rows, cols), dtype=torch.int16, device=self.d)
        return torch.zeros((rows, cols), dtype=torch.float32, device=self.d)

    def _mode(self, u, m):
        off = self.spec.offset(u, m)
        return self.qe.ACCUM if (u, off) in self.written else self.qe.INIT

    def run(self, schedule, epoch, step):
        for a, m in schedule:
            for u in range(len(self.spec.shapes)):
                if self.streams:
                    s = self.streams[self.n_actions % len(self.streams)]
                    with torch.cuda.stream(s):
                        self._action(a, m, u, epoch, step, s)
                else:
                    self._action(a, m, u, epoch, step, None)
                self.n_actions += 1

    def _action(self, a, m, u, epoch, step, caller):
        qe, spec = self.qe, self.spec
        dt = qe.BF16 if spec.in_dtype == "bf16" else qe.F32
        odt = qe.BF16 if spec.out_dtype == "bf16" else qe.F32
        n, k = spec.shapes[u]
        key = qe.key(epoch, 0, m, u)
        x, dy = spec.inputs(u, m, step)
        if a == "F":
            y = self._out(spec.tokens, n)
            xin = upload(x, self.d)
            if self.x_misaligned:
                buf = torch.empty(xin.numel() + 1, dtype=xin.dtype, device=self.d)
                buf[1:].copy_(xin.reshape(-1))
                xin = buf[1:].view(xin.shape)
                assert xin.data_ptr() % 16 != 0
            st, self.refs[(u, m)] = self.ctx.qe_fp8_linear_fwd(u, key, xin, dt, spec.tokens, y, odt, caller=caller)
            self.written_x = xin  # keep the offset buffer alive until the action has run
            self.outs[("y", u, m, step)] = y
        elif a == "dI":
            dx = self._out(spec.tokens, k)
            st = self.ctx.qe_fp8_linear_dgrad(u, key, self.refs[(u, m)], upload(dy, self.d), dt, dx, odt,
                                             caller=caller)
            self.outs[("dx", u, m, step)] = dx
        elif a == "dW":
            mode = self._mode(u, m)
            st = self.ctx.qe_fp8_linear_wgrad_place(u, key, self.refs[(u, m)], self.grad, spec.offset(u, m),
                                                    spec.ld(u), mode, caller=caller)
            self.written.add((u, spec.offset(u, m)))
        else:
            dx = self._out(spec.tokens, k)
            mode = self._mode(u, m)
            st = self.ctx.qe_fp8_linear_bwd_full(u, key, self.refs[(u, m)], upload(dy, self.d), dt, dx, odt,
                                                 self.grad, spec.offset(u, m), spec.ld(u), mode, caller=caller)
            self.written.add((u, spec.offset(u, m)))
            self.outs[("dx", u, m, step)] = dx
        assert st == "OK", (a, m, u, st)

    def end_step(self, new_weights=None):
        assert self.ctx.qe_arena_finalize() == "OK"
        if new_weights is not None:
            torch.cuda.synchronize()
            for u, w in enumerate(new_weights):
                self.w[u].copy_(upload(w, self.d))
            torch.cuda.synchronize()  # the next actions may run on other streams
        assert self.ctx.qe_optimizer_commit() == "OK"
        self.written = set()

    def fp8_state(self, u):
        H = self.spec.history
        out = {}
        for name, role in (("x", self.qe.ROLE_X), ("w", self.qe.ROLE_W), ("dy", self.qe.ROLE_DY)):
            m = self.ctx.qe_layer_meta(u, role)
            h = dev_f32(m.amax_history, H, self.d)
            s = dev_f32(m.scale, 1, self.d)[0]
            si = dev_f32(m.scale_inv, 1, self.d)[0]
            out[name] = (h, s, si)
        return out

    def slot_codes(self, u, m):
        n, k = self.spec.shapes[u]
        p = self.ctx.qe_layer_slot_payload(u, m)
        t = self.spec.tokens
        xt = dev_bytes(p["x_q_t"], k * p["ld_x_q_t"], self.d).reshape(k, p["ld_x_q_t"])[:, :t]
        dyt = dev_bytes(p["dy_q_t"], n * p["ld_dy_q_t"], self.d).reshape(n, p["ld_dy_q_t"])[:, :t]
        return xt, dyt

    def cache_codes(self, u):
        n, k = self.spec.shapes[u]
        c = self.ctx.qe_layer_cache(u)
        wq = dev_bytes(c["w_q"], n * c["ld_w_q"], self.d).reshape(n, c["ld_w_q"])[:, :k]
        wqt = dev_bytes(c["w_q_t"], k * c["ld_w_q_t"], self.d).reshape(k, c["ld_w_q_t"])[:, :n]
        return wq, wqt


class OracleStage:
    def __init__(self, spec, weights=None):
        """`weights`: the current master weights (workloads.Tensor per layer), default the initial ones."""
        self.spec = spec
        self.st = Stage(spec.M)
        for u, (n, k) in enumerate(spec.shapes):
            w = spec.weight(u) if weights is None else weights[u]
            self.st.add_layer(0, u, w.as_f32(), spec.tokens, spec.history, spec.margin, fmt_w=spec.fmt_w,
                             scaling=spec.scaling)
        self.buf = 1 << 12
        self.st.add_buffer(self.buf, spec.grad_elems())
        for u, (n, k) in enumerate(spec.shapes):
            for m in range(spec.M):
                assert self.st.bind(u, m, self.buf, spec.offset(u, m), spec.ld(u)) == OC.OK
        self.refs = {}
        self.outs = {}

    def _mode(self, u, m):
        b = self.st.contract.bindings[(u, m)]
        init = not any(o.written and o.start() == b.start() for o in self.st.contract.bindings.values())
        return OC.INIT if init else OC.ACCUM

    def run(self, schedule, epoch, step):
        spec = self.spec
        for a, m in schedule:
            for u, (n, k) in enumerate(spec.shapes):
                key = (epoch, 0, m, u, 0)
                x, dy = spec.inputs(u, m, step)
                if a == "F":
                    st, y, self.refs[(u, m)] = self.st.fwd(u, key, x.as_f32())
                    self.outs[("y", u, m, step)] = y
                elif a == "dI":
                    st, self.outs[("dx", u, m, step)] = self.st.dgrad(u, key, self.refs[(u, m)], dy.as_f32())
                elif a == "dW":
                    st = self.st.wgrad_place(u, key, self.refs[(u, m)], self.buf, spec.offset(u, m), spec.ld(u),
                                             self._mode(u, m))
                else:
                    st, self.outs[("dx", u, m, step)] = self.st.bwd_full(u, key, self.refs[(u, m)], dy.as_f32(),
                                                                         self.buf, spec.offset(u, m), spec.ld(u),
                                                                         self._mode(u, m))
                assert st == OC.OK, (a, m, u, st)

    def sgd_weights(self, lr=1e-3):
        """W <- W - lr * sum of the step's gradient views, rounded like the inputs."""
        spec = self.spec
        g = self.st.arena[self.buf]
        new = []
        for u, (n, k) in enumerate(spec.shapes):
            acc = np.zeros((n, k), dtype=np.float64)
            for m in range(1 if spec.shared_view else spec.M):
                o = spec.offset(u, m)
                acc += g[o:o + n * spec.ld(u)].reshape(n, spec.ld(u))[:, :k]
            w = (self.st.layers[u].w.astype(np.float64) - lr * acc).astype(np.float32)
            t = W.Tensor(W.f32_to_bf16_bits(w), "bf16") if spec.w_dtype == "bf16" else W.Tensor(w, "f32")
            new.append(t)
        return new

    def end_step(self, new_weights=None):
        assert self.st.finalize() == OC.OK
        if new_weights is not None:
            for u, w in enumerate(new_weights):
                self.st.set_weight(u, w.as_f32())
        assert self.st.optimizer_commit() == OC.OK
