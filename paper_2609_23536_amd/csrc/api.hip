// C ABI of the FP8 split linear: argument validation, the stage context, the
// stream-ordered executor with HIP-graph capture / replay, and the stateless
// hot-path entry points.
//
// Executor (§4.4 of the paper): every layer action runs on one context-owned
// graph stream.  The graph stream first waits on the caller's stream; the
// action's kernel sequence is then either launched directly (eager) or
// replayed from a graph captured once per (layer, action, slot) (§4.3, eq.
// G_r: G = 3 M L graphs, which qe_prebuild_graphs captures up front); finally
// an event recorded right after the launch is waited on by the caller's
// stream (the two-way handoff of §2.3).  The completion event is recorded by
// hipEventRecord after hipGraphLaunch, never as an event-record node inside
// the graph: on this runtime a stream waiting on an event that a graph node
// records was measured not to wait for the graph's kernels (a consumer on the
// caller's stream saw stale output in most trials), while a record enqueued
// after the launch orders correctly.
//
// Dynamic inputs (§4.4).  Graphs bind the buffers of the call they were
// captured for.  When an action is called with other buffers, the default
// (QE_GRAPH_INPUTS_REBIND) rewrites the arguments of the graph's kernel nodes
// in place (hipGraphExecKernelNodeSetParams): every action's launches are
// recorded on the host first (qe::klaunch in record mode) and compared with
// the ones the graph holds, and only nodes whose argument bytes differ are
// rewritten; a different launch shape (grid, kernel instance) captures the
// graph again.  QE_GRAPH_INPUTS_COPY is the paper's scheme: graphs bind
// library-owned static buffers, and the caller's inputs are copied in before
// the replay and the outputs copied out after it.  QE_GRAPH_INPUTS_RECAPTURE
// captures the graph again on any change (for comparison).
#include <hip/hip_runtime.h>
#include <string.h>

#include <chrono>
#include <map>
#include <mutex>
#include <new>
#include <vector>

#include "../../include/qe.h"
#include "contract.h"
#include "kernels.h"

// Scratch of qe_quantize_fp8_current_noalloc: one amax accumulator
// (kAmaxLines lines, kAmaxStride floats apart: 16 KiB), one copy per device,
// held until the process ends.  In host code this name is a host-side stand-in:
// the device address comes from hipGetSymbolAddress (noalloc_scratch below).
static __device__ __align__(256) float scratch[qe::kAmaxLines * qe::kAmaxStride];

namespace {

int64_t rup16(int64_t v) { return (v + 15) / 16 * 16; }

// Device address of `scratch` on the current device, looked up once per
// device (each device holds its own copy at its own address).
constexpr int kScratchDevices = 64;
std::mutex g_scratch_mu;
float *g_scratch_ptr[kScratchDevices] = {};

float *noalloc_scratch() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kScratchDevices) return nullptr;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void *p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) return nullptr;
    g_scratch_ptr[dev] = static_cast<float *>(p);
  }
  return g_scratch_ptr[dev];
}

// Makes the context's device current for the scope of one call and restores
// the caller's device afterwards.
struct DeviceGuard {
  int prev = -1;
  bool ok = true;
  explicit DeviceGuard(int dev) {
    if (hipGetDevice(&prev) != hipSuccess) {
      prev = -1;
      ok = false;
      return;
    }
    if (prev != dev) ok = hipSetDevice(dev) == hipSuccess;
  }
  ~DeviceGuard() {
    int cur = -1;
    if (prev >= 0 && hipGetDevice(&cur) == hipSuccess && cur != prev) (void)hipSetDevice(prev);
  }
  DeviceGuard(const DeviceGuard &) = delete;
  DeviceGuard &operator=(const DeviceGuard &) = delete;
};

struct Call {
  int32_t kind;  // qe::KernelClass
  int32_t pad;
  union {
    qe::QuantParams q;
    qe::UpdateParams u;
    qe::GemmParams g;
    qe::GradCopyParams c;
    qe::AmaxParams a;
  };
  // KC_QUANT only: a second, independent cast of the same input dtype and
  // FP8 format that runs in the same launch (has_q2 != 0)
  qe::QuantParams q2;
  int32_t has_q2, pad2;
  // KC_GEMM only: a delayed scale update run by extra workgroups of the same
  // launch (has_gu != 0)
  qe::UpdateParams gu;
  int32_t has_gu, pad3;
  Call() { memset(static_cast<void *>(this), 0, sizeof(*this)); }
};
using Plan = std::vector<Call>;

struct SlotDev {
  uint8_t *x_q_t = nullptr;   // [K, ld_t]
  uint8_t *dy_q_t = nullptr;  // [N, ld_t]
  float *x_sinv = nullptr;
  float *dy_sinv = nullptr;
};

struct LayerDev {
  qe_layer_desc desc{};
  float *meta = nullptr;   // hist[3][H] | scale[3] | scale_inv[3]
  float *accum = nullptr;  // amax accumulators of the three roles
  uint8_t *w_q = nullptr, *w_q_t = nullptr;
  float *w_sinv = nullptr;
  uint8_t *x_q = nullptr, *dy_q = nullptr;  // row-wise scratch
  // QE_GRAPH_INPUTS_COPY only: static input / output buffers the graphs bind,
  // sized for max_tokens rows of FP32
  void *x_st = nullptr, *y_st = nullptr, *dy_st = nullptr, *dx_st = nullptr;
  float *grad_stage = nullptr;              // [N, K] FP32, copied-gradient path only
  int64_t ld_wq = 0, ld_wqt = 0, ld_xq = 0, ld_dyq = 0, ld_t = 0;
  std::vector<SlotDev> slots;
  std::vector<void *> allocs;

  qe::MetaRef role(int r) const {
    const int H = desc.history_len;
    qe::MetaRef m{};
    m.hist = meta + size_t(r) * H;
    m.scale = meta + size_t(3) * H + r;
    m.scale_inv = meta + size_t(3) * H + 3 + r;
    m.history_len = H;
    m.margin = desc.margin;
    m.fmt = r == QE_ROLE_X ? desc.fmt_x : (r == QE_ROLE_W ? desc.fmt_w : desc.fmt_dy);
    m.accum = accum ? accum + size_t(r) * qe::kAmaxLines * qe::kAmaxStride : nullptr;
    return m;
  }
};

struct GraphEntry {
  hipGraph_t graph = nullptr;  // kept: its kernel nodes name the nodes of exec
  hipGraphExec_t exec = nullptr;
  hipEvent_t done = nullptr;   // recorded on the launch stream right after every replay
  std::vector<qe::KernelRec> recs;    // the graph's launches as currently bound
  std::vector<hipGraphNode_t> nodes;  // its kernel nodes, in launch order
  bool rebindable = false;            // nodes match recs one to one
  bool launched = false;
};

// A device-to-device copy around a replay (QE_GRAPH_INPUTS_COPY).
struct Copy {
  void *dst;
  const void *src;
  size_t bytes;
};

struct TimedCall {
  int kind;
  hipEvent_t t0, t1;
};

}  // namespace

struct qe_ctx {
  qe_config cfg{};
  qe::Contract contract;
  hipStream_t gs = nullptr;
  hipEvent_t ev_in = nullptr, ev_tail = nullptr;
  // replay_on_caller: an event recorded on each action's stream right after
  // the action; the next action's stream waits on it (no stream handle of
  // the caller is kept, so a caller may destroy its streams between actions)
  bool has_last = false;
  hipEvent_t ev_chain = nullptr;
  // completion event of the last action: its graph's own event, or ev_chain /
  // ev_tail after direct launches
  hipEvent_t last_ev = nullptr;
  long long *d_token = nullptr;
  // qe_prebuild_graphs: the buffer every prebuilt graph binds in place of the
  // caller's X, Y, dY and dX until a call binds its own (so a graph is never
  // replayed on pointers that name no allocation)
  void *placeholder = nullptr;
  std::vector<LayerDev> layers;
  std::map<uint64_t, GraphEntry> graphs;
  qe_ctx_state st{};
  int timing = 0;
  std::vector<TimedCall> timed;
  std::vector<hipEvent_t> event_pool;
  double kc_ms[qe::KC_COUNT] = {};
  int64_t kc_n[qe::KC_COUNT] = {};
  explicit qe_ctx(const qe_config &c) : cfg(c), contract(c.microbatches) {}
};

namespace {

bool valid_dtype(int d) { return d == QE_F32 || d == QE_BF16; }
bool valid_fmt(int f) { return f == QE_E4M3 || f == QE_E5M2; }
bool elem_aligned(const void *p, int dt) { return uintptr_t(p) % (dt == QE_BF16 ? 2 : 4) == 0; }

hipError_t launch(const Call &c, hipStream_t s) {
  switch (c.kind) {
    case qe::KC_QUANT: return c.has_q2 ? qe::launch_quantize_pair(c.q, c.q2, s) : qe::launch_quantize(c.q, s);
    case qe::KC_UPDATE: return qe::launch_scale_update(c.u, s);
    case qe::KC_COPY: return qe::launch_grad_copy(c.c, s);
    case qe::KC_AMAX: return qe::launch_amax(c.a, s);
    default: return qe::launch_gemm(c.g, s, c.has_gu ? &c.gu : nullptr);
  }
}

hipEvent_t pooled_event(qe_ctx *c) {
  if (!c->event_pool.empty()) {
    hipEvent_t e = c->event_pool.back();
    c->event_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

hipError_t enqueue(qe_ctx *c, const Plan &plan, bool timed, hipStream_t s) {
  for (const Call &call : plan) {
    if (timed) {
      TimedCall t{call.kind, pooled_event(c), pooled_event(c)};
      if (!t.t0 || !t.t1) return hipErrorOutOfMemory;
      qe::LaunchTiming lt{t.t0, t.t1, false};
      qe::tl_timing = &lt;
      hipError_t e = launch(call, s);
      qe::tl_timing = nullptr;
      if (e == hipSuccess && !lt.started) {  // the call launched nothing (an empty tensor): a zero-length pair
        e = hipEventRecord(t.t0, s);
        if (e == hipSuccess) e = hipEventRecord(t.t1, s);
      }
      if (e != hipSuccess) {
        if (lt.started) {  // a launch already carries the pair: never hand it out again
          (void)hipEventDestroy(t.t0);
          (void)hipEventDestroy(t.t1);
        } else {           // unused: back to the pool
          c->event_pool.push_back(t.t0);
          c->event_pool.push_back(t.t1);
        }
        return e;
      }
      c->timed.push_back(t);
    } else {
      const hipError_t e = launch(call, s);
      if (e != hipSuccess) return e;
    }
  }
  return hipSuccess;
}

// Wait for every action enqueued so far: the graph stream, and with
// replay_on_caller the chaining event of the last action (earlier actions
// precede it in the chained order).
hipError_t sync_actions(qe_ctx *c) {
  hipError_t e = hipStreamSynchronize(c->gs);
  if (e == hipSuccess && c->has_last && c->last_ev) e = hipEventSynchronize(c->last_ev);
  return e;
}

}  // namespace
namespace qe {
thread_local std::vector<KernelRec> *tl_record = nullptr;
thread_local LaunchTiming *tl_timing = nullptr;
}
namespace {

// The launches `plan` makes, recorded on the host without touching the device.
std::vector<qe::KernelRec> record_plan(qe_ctx *c, const Plan &plan) {
  std::vector<qe::KernelRec> v;
  qe::tl_record = &v;
  (void)enqueue(c, plan, false, nullptr);
  qe::tl_record = nullptr;
  return v;
}

// Kernel nodes of a graph captured from one stream, in launch order: such a
// capture is a chain.  False if the graph is not a chain.
bool chain_kernel_nodes(hipGraph_t g, std::vector<hipGraphNode_t> &out) {
  out.clear();
  size_t n = 0, nr = 0;
  if (hipGraphGetNodes(g, nullptr, &n) != hipSuccess || n == 0) return false;
  if (hipGraphGetRootNodes(g, nullptr, &nr) != hipSuccess || nr != 1) return false;
  hipGraphNode_t cur = nullptr;
  if (hipGraphGetRootNodes(g, &cur, &nr) != hipSuccess) return false;
  for (size_t seen = 1; seen <= n; ++seen) {
    hipGraphNodeType t;
    if (hipGraphNodeGetType(cur, &t) != hipSuccess) return false;
    if (t == hipGraphNodeTypeKernel) out.push_back(cur);
    size_t nd = 0;
    if (hipGraphNodeGetDependentNodes(cur, nullptr, &nd) != hipSuccess || nd > 1) return false;
    if (nd == 0) return seen == n;
    if (hipGraphNodeGetDependentNodes(cur, &cur, &nd) != hipSuccess) return false;
  }
  return false;
}

hipKernelNodeParams node_params(const qe::KernelRec &r, void **argv) {
  hipKernelNodeParams kp;
  memset(&kp, 0, sizeof(kp));
  r.argv(argv);
  kp.func = const_cast<void *>(r.func);
  kp.gridDim = r.grid;
  kp.blockDim = r.block;
  kp.sharedMemBytes = r.shmem;
  kp.kernelParams = argv;
  kp.extra = nullptr;
  return kp;
}

// Capture `plan` into e (replacing what e held).
qe_status capture(qe_ctx *c, GraphEntry &e, const Plan &plan, std::vector<qe::KernelRec> &&recs) {
  const auto t0 = std::chrono::steady_clock::now();
  // the graph being replaced may still be replaying: let that replay finish
  // before its executable (and the argument memory it reads) goes away
  if (e.exec != nullptr && e.launched && hipEventSynchronize(e.done) != hipSuccess) return QE_ERR_HIP;
  if (e.exec != nullptr) (void)hipGraphExecDestroy(e.exec);
  if (e.graph != nullptr) (void)hipGraphDestroy(e.graph);
  e.exec = nullptr;
  e.graph = nullptr;
  e.rebindable = false;
  e.launched = false;
  e.nodes.clear();
  if (e.done == nullptr && hipEventCreateWithFlags(&e.done, hipEventDisableTiming) != hipSuccess) {
    e.done = nullptr;
    return QE_ERR_HIP;
  }
  hipGraph_t graph = nullptr;
  if (hipStreamBeginCapture(c->gs, hipStreamCaptureModeThreadLocal) != hipSuccess) return QE_ERR_HIP;
  const hipError_t le = enqueue(c, plan, false, c->gs);
  const hipError_t ce = hipStreamEndCapture(c->gs, &graph);
  if (le != hipSuccess || ce != hipSuccess || graph == nullptr) {
    if (graph) (void)hipGraphDestroy(graph);
    return QE_ERR_HIP;
  }
  if (hipGraphInstantiate(&e.exec, graph, nullptr, nullptr, 0) != hipSuccess) {
    e.exec = nullptr;
    (void)hipGraphDestroy(graph);
    return QE_ERR_HIP;
  }
  e.graph = graph;
  e.recs = std::move(recs);
  // The nodes can be rewritten in place only if they are the recorded
  // launches, one to one and in order.
  bool ok = chain_kernel_nodes(graph, e.nodes) && e.nodes.size() == e.recs.size();
  for (size_t i = 0; ok && i < e.nodes.size(); ++i) {
    hipKernelNodeParams kp;
    memset(&kp, 0, sizeof(kp));
    const qe::KernelRec &r = e.recs[i];
    ok = hipGraphKernelNodeGetParams(e.nodes[i], &kp) == hipSuccess && kp.func == r.func &&
         kp.gridDim.x == r.grid.x && kp.gridDim.y == r.grid.y && kp.gridDim.z == r.grid.z &&
         kp.blockDim.x == r.block.x && kp.blockDim.y == r.block.y && kp.blockDim.z == r.block.z &&
         kp.sharedMemBytes == r.shmem;
  }
  e.rebindable = ok;
  c->st.captures += 1;
  c->st.capture_ns +=
      std::chrono::duration_cast<std::chrono::nanoseconds>(std::chrono::steady_clock::now() - t0).count();
  return QE_OK;
}

// Bring e's graph to `plan`: nothing if it already matches, the changed
// kernel-node arguments rewritten in place if only arguments differ (the
// graph's previous replay is waited for first, so no replay in flight sees a
// half-written node), else a new capture.
qe_status bind_graph(qe_ctx *c, GraphEntry &e, const Plan &plan) {
  std::vector<qe::KernelRec> recs = record_plan(c, plan);
  const int mode = c->cfg.graph_inputs;
  bool same_shape = e.exec != nullptr && e.recs.size() == recs.size();
  for (size_t i = 0; same_shape && i < recs.size(); ++i) same_shape = recs[i].same_shape(e.recs[i]);
  if (!same_shape) return capture(c, e, plan, std::move(recs));
  std::vector<size_t> diff;
  for (size_t i = 0; i < recs.size(); ++i)
    if (!recs[i].same_args(e.recs[i])) diff.push_back(i);
  if (diff.empty()) return QE_OK;
  if (mode != QE_GRAPH_INPUTS_REBIND || !e.rebindable) return capture(c, e, plan, std::move(recs));
  if (e.launched && hipEventSynchronize(e.done) != hipSuccess) return QE_ERR_HIP;
  for (size_t i : diff) {
    void *argv[qe::kMaxKernelArgs];
    const hipKernelNodeParams kp = node_params(recs[i], argv);
    if (hipGraphExecKernelNodeSetParams(e.exec, e.nodes[i], &kp) != hipSuccess) {
      // the exec may hold a mix of old and new arguments: never replay it
      (void)hipGraphExecDestroy(e.exec);
      e.exec = nullptr;
      return QE_ERR_HIP;
    }
    e.recs[i] = recs[i];
  }
  c->st.rebinds += 1;
  c->st.rebound_nodes += int64_t(diff.size());
  return QE_OK;
}

hipError_t copy_all(const std::vector<Copy> &cs, hipStream_t s) {
  for (const Copy &k : cs)
    if (k.bytes > 0) {
      const hipError_t e = hipMemcpyAsync(k.dst, k.src, k.bytes, hipMemcpyDeviceToDevice, s);
      if (e != hipSuccess) return e;
    }
  return hipSuccess;
}

// One action's kernel sequence, replayed from its graph (one per (layer,
// action, slot)), or launched directly.  Graph-stream executor: the two-way
// handoff around it (§2.3, §4.4).  replay_on_caller: launched on the caller's
// stream, chained to the previous action through that action's completion
// event.  `pre` / `post`: the dynamic-input copies of QE_GRAPH_INPUTS_COPY,
// enqueued after the caller -> graph edge and before the completion event.
qe_status run_plan(qe_ctx *c, const Plan &plan, uint64_t gkey, hipStream_t caller, const std::vector<Copy> &pre = {},
                   const std::vector<Copy> &post = {}) {
  DeviceGuard dg(c->cfg.device);
  if (!dg.ok) return QE_ERR_HIP;
  const bool on_caller = c->cfg.replay_on_caller != 0;
  const hipStream_t s = on_caller ? caller : c->gs;
  if (on_caller) {
    // Stream order covers both directions of the handoff.  The wait on the
    // previous action's event orders actions issued from different streams;
    // on the same stream it is already satisfied by stream order.
    if (c->has_last && hipStreamWaitEvent(caller, c->last_ev, 0) != hipSuccess) return QE_ERR_HIP;
  } else if (caller != c->gs) {
    if (hipEventRecord(c->ev_in, caller) != hipSuccess) return QE_ERR_HIP;
    if (hipStreamWaitEvent(c->gs, c->ev_in, 0) != hipSuccess) return QE_ERR_HIP;
  }
  if (copy_all(pre, s) != hipSuccess) return QE_ERR_HIP;
  hipEvent_t done = on_caller ? c->ev_chain : c->ev_tail;
  if (c->cfg.use_graphs) {
    GraphEntry &e = c->graphs[gkey];
    const qe_status bs = bind_graph(c, e, plan);
    if (bs != QE_OK) return bs;
    if (hipGraphLaunch(e.exec, s) != hipSuccess) return QE_ERR_HIP;
    e.launched = true;
    c->st.replays += 1;
    done = e.done;  // the graph's own event: a rebind waits for exactly this replay
  } else {
    if (enqueue(c, plan, c->timing != 0, s) != hipSuccess) return QE_ERR_HIP;
  }
  if (copy_all(post, s) != hipSuccess) return QE_ERR_HIP;
  if (hipEventRecord(done, s) != hipSuccess) return QE_ERR_HIP;
  c->last_ev = done;
  c->has_last = true;
  if (on_caller) return QE_OK;
  if (!c->cfg.one_way_handoff && caller != c->gs) {
    if (hipStreamWaitEvent(caller, done, 0) != hipSuccess) return QE_ERR_HIP;
  }
  c->st.handoffs += 2;
  return QE_OK;
}

uint64_t graph_key(int layer, int action, uint32_t slot) {
  return (uint64_t(uint32_t(layer)) << 32) | (uint64_t(action) << 24) | uint64_t(slot);
}
enum { ACT_FWD = 1, ACT_FWD_REFRESH = 2, ACT_DGRAD = 3, ACT_WGRAD = 4, ACT_FULL = 5 };

Call quant_call(const void *in, int in_dt, int64_t rows, int64_t cols, const qe::MetaRef &m, uint8_t *q_row,
                int64_t ld_row, uint8_t *q_col, int64_t ld_col, float *snapshot, bool record = true) {
  Call c;
  c.kind = qe::KC_QUANT;
  c.q.in = in;
  c.q.in_bf16 = in_dt == QE_BF16;
  c.q.fmt = m.fmt;
  c.q.rows = rows;
  c.q.cols = cols;
  c.q.scale = m.scale;
  c.q.scale_inv = m.scale_inv;
  c.q.amax_slot = record ? m.hist : nullptr;
  c.q.amax_accum = record ? m.accum : nullptr;
  c.q.q_row = q_row;
  c.q.ld_row = ld_row;
  c.q.q_col = q_col;
  c.q.ld_col = ld_col;
  c.q.snapshot = snapshot;
  return c;
}

// Appends two independent casts; with the same input dtype and FP8 format
// they share one launch.
void push_quant_pair(Plan &p, const Call &a, const Call &b) {
  if (a.q.in_bf16 == b.q.in_bf16 && a.q.fmt == b.q.fmt) {
    Call c = a;
    c.q2 = b.q;
    c.has_q2 = 1;
    p.push_back(c);
  } else {
    p.push_back(a);
    p.push_back(b);
  }
}

Call gemm_call(const uint8_t *a, int fa, int64_t lda, const uint8_t *b, int fb, int64_t ldb, int64_t m, int64_t n,
               int64_t k, const float *sa, const float *sb, void *cptr, int c_dt, int64_t ldc, int mode) {
  Call c;
  c.kind = qe::KC_GEMM;
  c.g.a = a;
  c.g.b = b;
  c.g.lda = lda;
  c.g.ldb = ldb;
  c.g.m = m;
  c.g.n = n;
  c.g.k = k;
  c.g.a_scale_inv = sa;
  c.g.b_scale_inv = sb;
  c.g.c = cptr;
  c.g.ldc = ldc;
  c.g.fmt_a = fa;
  c.g.fmt_b = fb;
  c.g.out = mode == QE_PLACE_ACCUM ? 2 : (c_dt == QE_BF16 ? 1 : 0);
  return c;
}

Call amax_call(const void *in, int in_dt, int64_t numel, const qe::MetaRef &m) {
  Call c;
  c.kind = qe::KC_AMAX;
  c.a = qe::amax_params(in, in_dt == QE_BF16, numel, m.hist, m.accum);
  return c;
}

Call update_call(const LayerDev &L, std::initializer_list<int> roles, long long *token) {
  Call c;
  c.kind = qe::KC_UPDATE;
  int n = 0;
  for (int r : roles) c.u.m[n++] = L.role(r);
  c.u.n = n;
  c.u.token = token;
  return c;
}

// Appends a delayed scale update.  Right after a GEMM it rides on the GEMM's
// launch as extra workgroups: every GEMM of an action reads the scale_inv
// snapshots of the slot and the weight cache, never the live scales, so the
// update may run beside it (one launch less per F and per dI).
void push_update(Plan &p, const Call &u) {
  if (!p.empty() && p.back().kind == qe::KC_GEMM && !p.back().has_gu) {
    p.back().gu = u.u;
    p.back().has_gu = 1;
  } else {
    p.push_back(u);
  }
}

// Plans of the physical actions (the kernel sequences of §3.2).
Plan plan_fwd(qe_ctx *c, const LayerDev &L, uint32_t m, const void *x, int x_dt, int64_t tokens, void *y, int y_dt,
              bool refresh) {
  const qe_layer_desc &d = L.desc;
  const SlotDev &S = L.slots[m];
  Plan p;
  if (d.scaling == QE_SCALING_CURRENT) {  // amax first, then the scales, then the casts
    if (refresh) p.push_back(amax_call(d.w, d.w_dtype, d.n_out * d.k_in, L.role(QE_ROLE_W)));
    p.push_back(amax_call(x, x_dt, tokens * d.k_in, L.role(QE_ROLE_X)));
    p.push_back(refresh ? update_call(L, {QE_ROLE_X, QE_ROLE_W}, c->d_token) : update_call(L, {QE_ROLE_X}, c->d_token));
    const Call qx =
        quant_call(x, x_dt, tokens, d.k_in, L.role(QE_ROLE_X), L.x_q, L.ld_xq, S.x_q_t, L.ld_t, S.x_sinv, false);
    if (refresh)
      push_quant_pair(p, quant_call(d.w, d.w_dtype, d.n_out, d.k_in, L.role(QE_ROLE_W), L.w_q, L.ld_wq, L.w_q_t,
                                    L.ld_wqt, L.w_sinv, false), qx);
    else
      p.push_back(qx);
    p.push_back(gemm_call(L.x_q, d.fmt_x, L.ld_xq, L.w_q, d.fmt_w, L.ld_wq, tokens, d.n_out, d.k_in, S.x_sinv,
                          L.w_sinv, y, y_dt, d.n_out, QE_PLACE_INIT));
    return p;
  }
  const Call qx = quant_call(x, x_dt, tokens, d.k_in, L.role(QE_ROLE_X), L.x_q, L.ld_xq, S.x_q_t, L.ld_t, S.x_sinv);
  if (refresh)
    push_quant_pair(
        p, quant_call(d.w, d.w_dtype, d.n_out, d.k_in, L.role(QE_ROLE_W), L.w_q, L.ld_wq, L.w_q_t, L.ld_wqt, L.w_sinv),
        qx);
  else
    p.push_back(qx);
  p.push_back(gemm_call(L.x_q, d.fmt_x, L.ld_xq, L.w_q, d.fmt_w, L.ld_wq, tokens, d.n_out, d.k_in, S.x_sinv, L.w_sinv,
                        y, y_dt, d.n_out, QE_PLACE_INIT));
  push_update(p, update_call(L, {QE_ROLE_X, QE_ROLE_W}, c->d_token));
  return p;
}

// dI's cast and GEMM.  Under delayed scaling the dY update is appended by the
// caller after the action's last use of the old scale (finish_dgrad).
void append_dgrad(qe_ctx *c, Plan &p, const LayerDev &L, uint32_t m, int64_t tokens, const void *dy, int dy_dt,
                  void *dx, int dx_dt) {
  const qe_layer_desc &d = L.desc;
  const SlotDev &S = L.slots[m];
  const bool current = d.scaling == QE_SCALING_CURRENT;
  if (current) {
    p.push_back(amax_call(dy, dy_dt, tokens * d.n_out, L.role(QE_ROLE_DY)));
    p.push_back(update_call(L, {QE_ROLE_DY}, c->d_token));
  }
  p.push_back(quant_call(dy, dy_dt, tokens, d.n_out, L.role(QE_ROLE_DY), L.dy_q, L.ld_dyq, S.dy_q_t, L.ld_t,
                         S.dy_sinv, !current));
  p.push_back(gemm_call(L.dy_q, d.fmt_dy, L.ld_dyq, L.w_q_t, d.fmt_w, L.ld_wqt, tokens, d.k_in, d.n_out, S.dy_sinv,
                        L.w_sinv, dx, dx_dt, d.k_in, QE_PLACE_INIT));
}

void finish_dgrad(qe_ctx *c, Plan &p, const LayerDev &L) {
  if (L.desc.scaling != QE_SCALING_CURRENT) push_update(p, update_call(L, {QE_ROLE_DY}, c->d_token));
}

void append_wgrad(Plan &p, const LayerDev &L, uint32_t m, int64_t tokens, float *mg, int64_t offset, int64_t ld,
                  int mode) {
  const qe_layer_desc &d = L.desc;
  const SlotDev &S = L.slots[m];
  if (L.grad_stage == nullptr) {  // direct placement: the GEMM epilogue writes the view
    p.push_back(gemm_call(S.dy_q_t, d.fmt_dy, L.ld_t, S.x_q_t, d.fmt_x, L.ld_t, d.n_out, d.k_in, tokens, S.dy_sinv,
                          S.x_sinv, mg + offset, QE_F32, ld, mode));
    return;
  }
  // copied gradients: GEMM into the private buffer, then copy / add into the view
  p.push_back(gemm_call(S.dy_q_t, d.fmt_dy, L.ld_t, S.x_q_t, d.fmt_x, L.ld_t, d.n_out, d.k_in, tokens, S.dy_sinv,
                        S.x_sinv, L.grad_stage, QE_F32, d.k_in, QE_PLACE_INIT));
  Call c;
  c.kind = qe::KC_COPY;
  c.c.src = L.grad_stage;
  c.c.dst = mg + offset;
  c.c.n = d.n_out;
  c.c.k = d.k_in;
  c.c.ld = ld;
  c.c.accumulate = mode == QE_PLACE_ACCUM;
  p.push_back(c);
}

size_t esize(int dt) { return dt == QE_BF16 ? 2 : 4; }

// QE_GRAPH_INPUTS_COPY: graphs bind the layer's static buffers.
bool copy_inputs(const qe_ctx *c) { return c->cfg.use_graphs && c->cfg.graph_inputs == QE_GRAPH_INPUTS_COPY; }

qe_status fail_physical(qe_ctx *c) {
  c->contract.abort_epoch();
  return QE_ERR_HIP;
}

void *dev_alloc(qe_ctx *c, LayerDev &L, size_t bytes, bool *ok) {
  void *p = nullptr;
  if (bytes == 0) bytes = 16;
  if (hipMalloc(&p, bytes) != hipSuccess) {
    *ok = false;
    return nullptr;
  }
  if (hipMemset(p, 0, bytes) != hipSuccess) *ok = false;
  L.allocs.push_back(p);
  c->st.device_bytes += int64_t(bytes);
  return p;
}

bool meta_ok(const qe_fp8_meta *m) {
  return m && m->amax_history && m->scale && m->scale_inv && uintptr_t(m->amax_accum) % 4 == 0 &&
         m->history_len >= 1 &&
         m->history_len <= qe::kMaxHistory && valid_fmt(m->fmt);
}

// ------------------------------------------------------------------ checkpoint payload
constexpr char kCkptMagic[8] = {'Q', 'E', 'C', 'K', 'P', 'T', '0', '1'};
constexpr uint32_t kCkptVersion = 1;

struct CkptHeader {
  char magic[8];
  uint32_t version;
  uint32_t n_layers;
  int32_t microbatches;
  int32_t reserved;
  int64_t e_w;
};
struct CkptLayer {
  uint32_t stage, unit;
  int64_t n_out, k_in, max_tokens;
  int32_t w_dtype, history_len, margin, fmt_x, fmt_w, fmt_dy, scaling, reserved;
};
static_assert(sizeof(CkptHeader) == 32 && sizeof(CkptLayer) == 64, "checkpoint record sizes");

uint64_t fnv1a(const uint8_t *p, size_t n) {
  uint64_t h = 1469598103934665603ull;
  for (size_t i = 0; i < n; ++i) {
    h ^= p[i];
    h *= 1099511628211ull;
  }
  return h;
}

CkptLayer ckpt_layer_of(const qe_layer_desc &d) {
  CkptLayer r;
  memset(&r, 0, sizeof(r));
  r.stage = d.stage;
  r.unit = d.unit;
  r.n_out = d.n_out;
  r.k_in = d.k_in;
  r.max_tokens = d.max_tokens;
  r.w_dtype = d.w_dtype;
  r.history_len = d.history_len;
  r.margin = d.margin;
  r.fmt_x = d.fmt_x;
  r.fmt_w = d.fmt_w;
  r.fmt_dy = d.fmt_dy;
  r.scaling = d.scaling;
  return r;
}

// Payload bytes of the FP8 state of one layer: 3 roles x (H + 2) floats.
size_t ckpt_state_bytes(const qe_layer_desc &d) { return sizeof(float) * 3 * (size_t(d.history_len) + 2); }

int64_t ckpt_size(const std::vector<LayerDev> &layers) {
  size_t n = sizeof(CkptHeader) + sizeof(uint64_t);
  for (const auto &L : layers) n += sizeof(CkptLayer) + ckpt_state_bytes(L.desc);
  return int64_t(n);
}

qe::MetaRef meta_ref(const qe_fp8_meta &m) {
  qe::MetaRef r{};
  r.hist = m.amax_history;
  r.scale = m.scale;
  r.scale_inv = m.scale_inv;
  r.history_len = m.history_len;
  r.margin = m.margin;
  r.fmt = m.fmt;
  r.accum = m.amax_accum;
  return r;
}

}  // namespace

extern "C" {

const char *qe_status_str(qe_status s) {
  switch (s) {
    case QE_OK: return "OK";
    case QE_ERR_INVALID_ARG: return "INVALID_ARG";
    case QE_ERR_STALE_REF: return "STALE_REF";
    case QE_ERR_KEY_MISMATCH: return "KEY_MISMATCH";
    case QE_ERR_KEY_LIVE: return "KEY_LIVE";
    case QE_ERR_POOL_FULL: return "POOL_FULL";
    case QE_ERR_DUPLICATE_CONSUMER: return "DUPLICATE_CONSUMER";
    case QE_ERR_ORDER: return "ORDER";
    case QE_ERR_EPOCH: return "EPOCH";
    case QE_ERR_STALE_CACHE: return "STALE_CACHE";
    case QE_ERR_DEST_MISMATCH: return "DEST_MISMATCH";
    case QE_ERR_DEST_ALIAS: return "DEST_ALIAS";
    case QE_ERR_DUP_WRITE: return "DUP_WRITE";
    case QE_ERR_ARENA_INVALID: return "ARENA_INVALID";
    case QE_ERR_INCOMPLETE: return "INCOMPLETE";
    case QE_ERR_NOT_QUIESCENT: return "NOT_QUIESCENT";
    case QE_ERR_HIP: return "HIP";
    case QE_ERR_UNSUPPORTED: return "UNSUPPORTED";
  }
  return "UNKNOWN";
}

// ------------------------------------------------------------------ stateless hot-path calls
qe_status qe_amax_scale_update(const qe_fp8_meta *metas_host, int32_t n_metas, int64_t *device_token,
                               qe_stream stream) {
  if (metas_host == nullptr || n_metas < 1 || n_metas > qe::kMaxMetas) return QE_ERR_INVALID_ARG;
  qe::UpdateParams p;
  memset(&p, 0, sizeof(p));
  for (int i = 0; i < n_metas; ++i) {
    if (!meta_ok(&metas_host[i])) return QE_ERR_INVALID_ARG;
    p.m[i] = meta_ref(metas_host[i]);
  }
  p.n = n_metas;
  p.token = reinterpret_cast<long long *>(device_token);
  return qe::launch_scale_update(p, static_cast<hipStream_t>(stream)) == hipSuccess ? QE_OK : QE_ERR_HIP;
}

qe_status qe_quantize_fp8(const void *in, qe_dtype in_dtype, int64_t rows, int64_t cols, const qe_fp8_meta *meta_host,
                          uint8_t *q_row, int64_t ld_row, uint8_t *q_col, int64_t ld_col, float *scale_inv_snapshot,
                          qe_stream stream) {
  if (!valid_dtype(in_dtype) || rows < 0 || cols < 0 || !meta_ok(meta_host)) return QE_ERR_INVALID_ARG;
  if (rows > 0 && cols > 0 && in == nullptr) return QE_ERR_INVALID_ARG;
  if (q_row != nullptr && ld_row < cols) return QE_ERR_INVALID_ARG;
  if (q_col != nullptr && ld_col < rows) return QE_ERR_INVALID_ARG;
  if (uintptr_t(in) % (in_dtype == QE_BF16 ? 2 : 4) != 0) return QE_ERR_INVALID_ARG;
  const qe::MetaRef m = meta_ref(*meta_host);
  const Call c = quant_call(in, in_dtype, rows, cols, m, q_row, ld_row, q_col, ld_col, scale_inv_snapshot);
  return qe::launch_quantize(c.q, static_cast<hipStream_t>(stream)) == hipSuccess ? QE_OK : QE_ERR_HIP;
}

qe_status qe_amax(const void *in, qe_dtype in_dtype, int64_t numel, const qe_fp8_meta *meta_host, qe_stream stream) {
  if (!valid_dtype(in_dtype) || numel < 0 || !meta_ok(meta_host)) return QE_ERR_INVALID_ARG;
  if (numel > 0 && in == nullptr) return QE_ERR_INVALID_ARG;
  if (uintptr_t(in) % (in_dtype == QE_BF16 ? 2 : 4) != 0) return QE_ERR_INVALID_ARG;
  const qe::MetaRef m = meta_ref(*meta_host);
  const qe::AmaxParams p = qe::amax_params(in, in_dtype == QE_BF16, numel, m.hist, m.accum);
  return qe::launch_amax(p, static_cast<hipStream_t>(stream)) == hipSuccess ? QE_OK : QE_ERR_HIP;
}

qe_status qe_quantize_fp8_current(const void *in, qe_dtype in_dtype, int64_t rows, int64_t cols,
                                  const qe_fp8_meta *meta_host, uint8_t *q_row, int64_t ld_row, uint8_t *q_col,
                                  int64_t ld_col, float *scale_inv_snapshot, int64_t *device_token,
                                  qe_stream stream) {
  if (!valid_dtype(in_dtype) || rows < 0 || cols < 0 || !meta_ok(meta_host) || meta_host->history_len != 1)
    return QE_ERR_INVALID_ARG;
  if (rows > 0 && cols > 0 && in == nullptr) return QE_ERR_INVALID_ARG;
  if (q_row != nullptr && ld_row < cols) return QE_ERR_INVALID_ARG;
  if (q_col != nullptr && ld_col < rows) return QE_ERR_INVALID_ARG;
  if (uintptr_t(in) % (in_dtype == QE_BF16 ? 2 : 4) != 0) return QE_ERR_INVALID_ARG;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  const qe::MetaRef m = meta_ref(*meta_host);
  const Call a = amax_call(in, in_dtype, rows * cols, m);
  qe::UpdateParams u;
  memset(&u, 0, sizeof(u));
  u.m[0] = m;
  u.n = 1;
  u.token = reinterpret_cast<long long *>(device_token);
  const Call q = quant_call(in, in_dtype, rows, cols, m, q_row, ld_row, q_col, ld_col, scale_inv_snapshot, false);
  if (qe::launch_amax(a.a, s) != hipSuccess || qe::launch_scale_update(u, s) != hipSuccess ||
      qe::launch_quantize(q.q, s) != hipSuccess)
    return QE_ERR_HIP;
  return QE_OK;
}

qe_status qe_quantize_fp8_current_noalloc(const void *in, qe_dtype in_dtype, int64_t rows, int64_t cols,
                                          const qe_fp8_meta *meta_host, uint8_t *q_row, int64_t ld_row,
                                          uint8_t *q_col, int64_t ld_col, float *scale_inv_snapshot,
                                          int64_t *device_token, qe_stream stream) {
  if (!valid_dtype(in_dtype) || rows < 0 || cols < 0 || !meta_ok(meta_host) || meta_host->history_len != 1 ||
      meta_host->amax_accum != nullptr)
    return QE_ERR_INVALID_ARG;
  if (rows > 0 && cols > 0 && in == nullptr) return QE_ERR_INVALID_ARG;
  if (q_row != nullptr && ld_row < cols) return QE_ERR_INVALID_ARG;
  if (q_col != nullptr && ld_col < rows) return QE_ERR_INVALID_ARG;
  if (uintptr_t(in) % (in_dtype == QE_BF16 ? 2 : 4) != 0) return QE_ERR_INVALID_ARG;
  float *acc = noalloc_scratch();
  if (acc == nullptr) return QE_ERR_HIP;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  qe::MetaRef m = meta_ref(*meta_host);
  m.accum = acc;  // the amax pass folds into the scratch accumulator; the update folds and clears it
  const Call a = amax_call(in, in_dtype, rows * cols, m);
  qe::UpdateParams u;
  memset(&u, 0, sizeof(u));
  u.m[0] = m;
  u.n = 1;
  u.token = reinterpret_cast<long long *>(device_token);
  const Call q = quant_call(in, in_dtype, rows, cols, m, q_row, ld_row, q_col, ld_col, scale_inv_snapshot, false);
  // the scratch keeps the last call's contents: cleared first, by a kernel
  if (qe::launch_fill_zero(acc, int64_t(qe::kAmaxLines) * qe::kAmaxStride, s) != hipSuccess ||
      qe::launch_amax(a.a, s) != hipSuccess || qe::launch_scale_update(u, s) != hipSuccess ||
      qe::launch_quantize(q.q, s) != hipSuccess)
    return QE_ERR_HIP;
  return QE_OK;
}

qe_status qe_set_gemm_tile(qe_gemm_tile tile) {
  if (tile < QE_TILE_AUTO || tile > QE_TILE_256x224) return QE_ERR_INVALID_ARG;
  qe::set_gemm_tile_override(int(tile));
  return QE_OK;
}

qe_status qe_fp8_gemm_tn(const uint8_t *a, qe_fp8_fmt fmt_a, int64_t lda, const uint8_t *b, qe_fp8_fmt fmt_b,
                         int64_t ldb, int64_t m, int64_t n, int64_t k, const float *a_scale_inv,
                         const float *b_scale_inv, void *c, qe_dtype c_dtype, int64_t ldc, qe_place_mode mode,
                         qe_stream stream) {
  if (!valid_fmt(fmt_a) || !valid_fmt(fmt_b) || !valid_dtype(c_dtype)) return QE_ERR_INVALID_ARG;
  if (mode != QE_PLACE_INIT && mode != QE_PLACE_ACCUM) return QE_ERR_INVALID_ARG;
  if (mode == QE_PLACE_ACCUM && c_dtype != QE_F32) return QE_ERR_INVALID_ARG;
  if (m < 0 || n < 0 || k < 0 || k >= (int64_t(1) << 31) || ldc < n) return QE_ERR_INVALID_ARG;
  if (m == 0 || n == 0) return QE_OK;
  if (!a || !b || !c || !a_scale_inv || !b_scale_inv) return QE_ERR_INVALID_ARG;
  if (lda % 16 || ldb % 16 || lda < rup16(k) || ldb < rup16(k)) return QE_ERR_INVALID_ARG;
  if (uintptr_t(a) % 16 || uintptr_t(b) % 16) return QE_ERR_INVALID_ARG;
  if (uintptr_t(c) % (c_dtype == QE_F32 ? 4 : 2)) return QE_ERR_INVALID_ARG;
  const Call call = gemm_call(a, fmt_a, lda, b, fmt_b, ldb, m, n, k, a_scale_inv, b_scale_inv, c, c_dtype, ldc, mode);
  return qe::launch_gemm(call.g, static_cast<hipStream_t>(stream)) == hipSuccess ? QE_OK : QE_ERR_HIP;
}

// ------------------------------------------------------------------ context
qe_status qe_ctx_create(const qe_config *cfg_host, qe_ctx **out_host) {
  if (cfg_host == nullptr || out_host == nullptr || cfg_host->microbatches < 1 || cfg_host->microbatches > 4096)
    return QE_ERR_INVALID_ARG;
  // the one-way (testing) handoff only exists for the graph stream
  if (cfg_host->replay_on_caller != 0 && (cfg_host->replay_on_caller != 1 || cfg_host->one_way_handoff != 0))
    return QE_ERR_INVALID_ARG;
  if (cfg_host->graph_inputs < QE_GRAPH_INPUTS_REBIND || cfg_host->graph_inputs > QE_GRAPH_INPUTS_COPY)
    return QE_ERR_INVALID_ARG;
  *out_host = nullptr;
  qe_ctx *c = new (std::nothrow) qe_ctx(*cfg_host);
  if (c == nullptr) return QE_ERR_HIP;
  c->st.device_token = -1;
  c->st.arena_valid = 1;
  if (!c->cfg.null_executor) {
    hipDeviceProp_t prop;
    DeviceGuard dg(c->cfg.device);
    if (!dg.ok || hipGetDeviceProperties(&prop, c->cfg.device) != hipSuccess) {
      delete c;
      return QE_ERR_HIP;
    }
    if (strncmp(prop.gcnArchName, "gfx950", 6) != 0) {
      delete c;
      return QE_ERR_UNSUPPORTED;
    }
    bool ok = hipStreamCreateWithFlags(&c->gs, hipStreamNonBlocking) == hipSuccess;
    // The caller -> graph edge is only ever consumed by kernels on this device,
    // so a device-scope release is enough there (saves ~2 us per action on
    // MI355X).  The graph -> caller edge keeps the system-scope release: after
    // it the caller may hand results to the host or to a copy engine.
    ok = ok && hipEventCreateWithFlags(&c->ev_in, hipEventDisableTiming | hipEventDisableSystemFence) == hipSuccess;
    ok = ok && hipEventCreateWithFlags(&c->ev_tail, hipEventDisableTiming) == hipSuccess;
    ok = ok && hipEventCreateWithFlags(&c->ev_chain, hipEventDisableTiming) == hipSuccess;
    ok = ok && hipMalloc(reinterpret_cast<void **>(&c->d_token), sizeof(long long)) == hipSuccess;
    ok = ok && hipMemset(c->d_token, 0, sizeof(long long)) == hipSuccess;
    if (!ok) {
      qe_ctx_destroy(c);
      return QE_ERR_HIP;
    }
  }
  *out_host = c;
  return QE_OK;
}

void qe_ctx_destroy(qe_ctx *c) {
  if (c == nullptr) return;
  if (!c->cfg.null_executor) {
    DeviceGuard dg(c->cfg.device);
    if (c->gs) (void)sync_actions(c);
    for (auto &kv : c->graphs) {
      if (kv.second.exec) (void)hipGraphExecDestroy(kv.second.exec);
      if (kv.second.graph) (void)hipGraphDestroy(kv.second.graph);
      if (kv.second.done) (void)hipEventDestroy(kv.second.done);
    }
    for (auto &L : c->layers)
      for (void *p : L.allocs) (void)hipFree(p);
    for (auto &t : c->timed) {
      (void)hipEventDestroy(t.t0);
      (void)hipEventDestroy(t.t1);
    }
    for (hipEvent_t e : c->event_pool) (void)hipEventDestroy(e);
    if (c->d_token) (void)hipFree(c->d_token);
    if (c->placeholder) (void)hipFree(c->placeholder);
    if (c->ev_in) (void)hipEventDestroy(c->ev_in);
    if (c->ev_tail) (void)hipEventDestroy(c->ev_tail);
    if (c->ev_chain) (void)hipEventDestroy(c->ev_chain);
    if (c->gs) (void)hipStreamDestroy(c->gs);
  }
  delete c;
}

qe_status qe_layer_register(qe_ctx *c, const qe_layer_desc *d, int32_t *layer_out_host) {
  if (c == nullptr || d == nullptr || layer_out_host == nullptr) return QE_ERR_INVALID_ARG;
  constexpr int64_t kMaxDim = int64_t(1) << 31;  // each is a reduction length of one of the three GEMMs
  if (d->n_out >= kMaxDim || d->k_in >= kMaxDim || d->max_tokens >= kMaxDim) return QE_ERR_INVALID_ARG;
  if (d->n_out < 1 || d->k_in < 1 || d->max_tokens < 0 || d->history_len < 1 || d->history_len > qe::kMaxHistory ||
      d->margin < -126 || d->margin > 252 || !valid_dtype(d->w_dtype) || !valid_fmt(d->fmt_x) ||
      !valid_fmt(d->fmt_w) || !valid_fmt(d->fmt_dy))
    return QE_ERR_INVALID_ARG;
  if (d->scaling != QE_SCALING_DELAYED && d->scaling != QE_SCALING_CURRENT) return QE_ERR_INVALID_ARG;
  if (d->scaling == QE_SCALING_CURRENT && d->history_len != 1) return QE_ERR_INVALID_ARG;
  if (!c->cfg.null_executor && d->w == nullptr) return QE_ERR_INVALID_ARG;
  if (!elem_aligned(d->w, d->w_dtype)) return QE_ERR_INVALID_ARG;
  if (c->contract.has_layer(d->stage, d->unit)) return QE_ERR_INVALID_ARG;
  LayerDev L;
  L.desc = *d;
  const int M = c->cfg.microbatches;
  L.slots.resize(size_t(M));
  L.ld_wq = rup16(d->k_in);
  L.ld_wqt = rup16(d->n_out);
  L.ld_xq = rup16(d->k_in);
  L.ld_dyq = rup16(d->n_out);
  L.ld_t = rup16(d->max_tokens);
  if (!c->cfg.null_executor) {
    DeviceGuard dg(c->cfg.device);
    if (!dg.ok) return QE_ERR_HIP;
    const int64_t bytes_before = c->st.device_bytes;
    bool ok = true;
    const int H = d->history_len;
    L.meta = static_cast<float *>(dev_alloc(c, L, sizeof(float) * (3 * size_t(H) + 6), &ok));
    L.accum = static_cast<float *>(dev_alloc(c, L, sizeof(float) * 3 * qe::kAmaxLines * qe::kAmaxStride, &ok));
    L.w_q = static_cast<uint8_t *>(dev_alloc(c, L, size_t(d->n_out) * L.ld_wq, &ok));
    L.w_q_t = static_cast<uint8_t *>(dev_alloc(c, L, size_t(d->k_in) * L.ld_wqt, &ok));
    L.w_sinv = static_cast<float *>(dev_alloc(c, L, sizeof(float), &ok));
    L.x_q = static_cast<uint8_t *>(dev_alloc(c, L, size_t(d->max_tokens) * L.ld_xq, &ok));
    L.dy_q = static_cast<uint8_t *>(dev_alloc(c, L, size_t(d->max_tokens) * L.ld_dyq, &ok));
    if (c->cfg.copy_gradients)
      L.grad_stage = static_cast<float *>(dev_alloc(c, L, sizeof(float) * size_t(d->n_out) * size_t(d->k_in), &ok));
    if (c->cfg.use_graphs && c->cfg.graph_inputs == QE_GRAPH_INPUTS_COPY) {
      const size_t xb = sizeof(float) * size_t(d->max_tokens) * size_t(d->k_in);
      const size_t yb = sizeof(float) * size_t(d->max_tokens) * size_t(d->n_out);
      L.x_st = dev_alloc(c, L, xb, &ok);
      L.dx_st = dev_alloc(c, L, xb, &ok);
      L.y_st = dev_alloc(c, L, yb, &ok);
      L.dy_st = dev_alloc(c, L, yb, &ok);
    }
    for (auto &S : L.slots) {
      S.x_q_t = static_cast<uint8_t *>(dev_alloc(c, L, size_t(d->k_in) * L.ld_t, &ok));
      S.dy_q_t = static_cast<uint8_t *>(dev_alloc(c, L, size_t(d->n_out) * L.ld_t, &ok));
      S.x_sinv = static_cast<float *>(dev_alloc(c, L, sizeof(float), &ok));
      S.dy_sinv = static_cast<float *>(dev_alloc(c, L, sizeof(float), &ok));
    }
    if (ok) {
      const float ones[6] = {1.f, 1.f, 1.f, 1.f, 1.f, 1.f};
      ok = hipMemcpy(L.meta + 3 * size_t(H), ones, sizeof(ones), hipMemcpyHostToDevice) == hipSuccess;
      ok = ok && hipMemcpy(L.w_sinv, ones, sizeof(float), hipMemcpyHostToDevice) == hipSuccess;
    }
    if (!ok) {
      for (void *p : L.allocs) (void)hipFree(p);
      c->st.device_bytes = bytes_before;
      return QE_ERR_HIP;
    }
  }
  *layer_out_host = c->contract.add_layer(d->stage, d->unit, d->n_out, d->k_in, d->max_tokens);
  c->layers.push_back(L);
  return QE_OK;
}

qe_status qe_layer_meta(const qe_ctx *c, int32_t layer, qe_role role, qe_fp8_meta *out) {
  if (c == nullptr || out == nullptr || layer < 0 || layer >= int(c->layers.size()) || role < 0 || role > 2)
    return QE_ERR_INVALID_ARG;
  const LayerDev &L = c->layers[size_t(layer)];
  memset(out, 0, sizeof(*out));
  out->history_len = L.desc.history_len;
  out->margin = L.desc.margin;
  out->fmt = role == QE_ROLE_X ? L.desc.fmt_x : (role == QE_ROLE_W ? L.desc.fmt_w : L.desc.fmt_dy);
  if (L.meta != nullptr) {
    const qe::MetaRef m = L.role(role);
    out->amax_history = m.hist;
    out->scale = m.scale;
    out->scale_inv = m.scale_inv;
    out->amax_accum = m.accum;
  }
  return QE_OK;
}

qe_status qe_layer_cache(const qe_ctx *c, int32_t layer, const uint8_t **w_q, int64_t *ld_w_q, const uint8_t **w_q_t,
                         int64_t *ld_w_q_t, const float **w_scale_inv) {
  if (c == nullptr || layer < 0 || layer >= int(c->layers.size())) return QE_ERR_INVALID_ARG;
  const LayerDev &L = c->layers[size_t(layer)];
  if (w_q) *w_q = L.w_q;
  if (ld_w_q) *ld_w_q = L.ld_wq;
  if (w_q_t) *w_q_t = L.w_q_t;
  if (ld_w_q_t) *ld_w_q_t = L.ld_wqt;
  if (w_scale_inv) *w_scale_inv = L.w_sinv;
  return QE_OK;
}

qe_status qe_layer_slot_payload(const qe_ctx *c, int32_t layer, int32_t slot, const uint8_t **x_q_t,
                                int64_t *ld_x_q_t, const uint8_t **dy_q_t, int64_t *ld_dy_q_t,
                                const float **x_scale_inv, const float **dy_scale_inv) {
  if (c == nullptr || layer < 0 || layer >= int(c->layers.size()) || slot < 0 || slot >= c->cfg.microbatches)
    return QE_ERR_INVALID_ARG;
  const LayerDev &L = c->layers[size_t(layer)];
  const SlotDev &S = L.slots[size_t(slot)];
  if (x_q_t) *x_q_t = S.x_q_t;
  if (ld_x_q_t) *ld_x_q_t = L.ld_t;
  if (dy_q_t) *dy_q_t = S.dy_q_t;
  if (ld_dy_q_t) *ld_dy_q_t = L.ld_t;
  if (x_scale_inv) *x_scale_inv = S.x_sinv;
  if (dy_scale_inv) *dy_scale_inv = S.dy_sinv;
  return QE_OK;
}

// ------------------------------------------------------------------ actions
qe_status qe_fp8_linear_fwd(qe_ctx *c, int32_t layer, qe_tape_key key, const void *x, qe_dtype x_dtype,
                            int64_t tokens, void *y, qe_dtype y_dtype, qe_tape_ref *ref_out_host, qe_stream caller) {
  if (c == nullptr || ref_out_host == nullptr || !valid_dtype(x_dtype) || !valid_dtype(y_dtype))
    return QE_ERR_INVALID_ARG;
  if (!c->cfg.null_executor && tokens > 0 && (x == nullptr || y == nullptr)) return QE_ERR_INVALID_ARG;
  if (!elem_aligned(x, x_dtype) || !elem_aligned(y, y_dtype)) return QE_ERR_INVALID_ARG;
  bool refresh = false;
  const qe_status st = c->contract.check_fwd(layer, key, tokens, &refresh);
  if (st != QE_OK) return st;
  if (c->contract.physical_fails()) return fail_physical(c);
  if (!c->cfg.null_executor) {
    const LayerDev &L = c->layers[size_t(layer)];
    std::vector<Copy> pre, post;
    const void *xg = x;
    void *yg = y;
    if (copy_inputs(c)) {
      xg = L.x_st;
      yg = L.y_st;
      pre.push_back({L.x_st, x, size_t(tokens) * size_t(L.desc.k_in) * esize(x_dtype)});
      post.push_back({y, L.y_st, size_t(tokens) * size_t(L.desc.n_out) * esize(y_dtype)});
    }
    const Plan p = plan_fwd(c, L, key.microbatch, xg, x_dtype, tokens, yg, y_dtype, refresh);
    if (run_plan(c, p, graph_key(layer, refresh ? ACT_FWD_REFRESH : ACT_FWD, key.microbatch),
                 static_cast<hipStream_t>(caller), pre, post) != QE_OK)
      return fail_physical(c);
  }
  *ref_out_host = c->contract.commit_fwd(layer, key, tokens, refresh);
  return QE_OK;
}

qe_status qe_fp8_linear_dgrad(qe_ctx *c, int32_t layer, qe_tape_key key, qe_tape_ref ref, const void *dy,
                              qe_dtype dy_dtype, void *dx, qe_dtype dx_dtype, qe_stream caller) {
  if (c == nullptr || !valid_dtype(dy_dtype) || !valid_dtype(dx_dtype)) return QE_ERR_INVALID_ARG;
  const qe_status st = c->contract.check_dgrad(layer, key, ref);
  if (st != QE_OK) return st;
  const int64_t tokens = c->contract.layer(layer).slots[ref.slot].tokens;
  if (!c->cfg.null_executor && tokens > 0 && (dy == nullptr || dx == nullptr)) return QE_ERR_INVALID_ARG;
  if (!elem_aligned(dy, dy_dtype) || !elem_aligned(dx, dx_dtype)) return QE_ERR_INVALID_ARG;
  if (c->contract.physical_fails()) return fail_physical(c);
  if (!c->cfg.null_executor) {
    const LayerDev &L = c->layers[size_t(layer)];
    std::vector<Copy> pre, post;
    const void *dyg = dy;
    void *dxg = dx;
    if (copy_inputs(c)) {
      dyg = L.dy_st;
      dxg = L.dx_st;
      pre.push_back({L.dy_st, dy, size_t(tokens) * size_t(L.desc.n_out) * esize(dy_dtype)});
      post.push_back({dx, L.dx_st, size_t(tokens) * size_t(L.desc.k_in) * esize(dx_dtype)});
    }
    Plan p;
    append_dgrad(c, p, L, ref.slot, tokens, dyg, dy_dtype, dxg, dx_dtype);
    finish_dgrad(c, p, L);
    if (run_plan(c, p, graph_key(layer, ACT_DGRAD, ref.slot), static_cast<hipStream_t>(caller), pre, post) !=
        QE_OK)
      return fail_physical(c);
  }
  c->contract.commit_dgrad(layer, ref);
  return QE_OK;
}

qe_status qe_fp8_linear_wgrad_place(qe_ctx *c, int32_t layer, qe_tape_key key, qe_tape_ref ref, float *main_grad,
                                    int64_t offset, int64_t ld, qe_place_mode mode, qe_stream caller) {
  if (c == nullptr) return QE_ERR_INVALID_ARG;
  const qe_status st =
      c->contract.check_wgrad(layer, key, ref, reinterpret_cast<uintptr_t>(main_grad), offset, ld, int(mode));
  if (st != QE_OK) return st;
  if (c->contract.physical_fails()) return fail_physical(c);
  if (!c->cfg.null_executor) {
    const LayerDev &L = c->layers[size_t(layer)];
    const int64_t tokens = c->contract.layer(layer).slots[ref.slot].tokens;
    Plan p;
    append_wgrad(p, L, ref.slot, tokens, main_grad, offset, ld, mode);
    if (run_plan(c, p, graph_key(layer, ACT_WGRAD, ref.slot), static_cast<hipStream_t>(caller)) != QE_OK)
      return fail_physical(c);
  }
  c->contract.commit_wgrad(layer, ref);
  return QE_OK;
}

qe_status qe_fp8_linear_bwd_full(qe_ctx *c, int32_t layer, qe_tape_key key, qe_tape_ref ref, const void *dy,
                                 qe_dtype dy_dtype, void *dx, qe_dtype dx_dtype, float *main_grad, int64_t offset,
                                 int64_t ld, qe_place_mode mode, qe_stream caller) {
  if (c == nullptr || !valid_dtype(dy_dtype) || !valid_dtype(dx_dtype)) return QE_ERR_INVALID_ARG;
  const qe_status st =
      c->contract.check_bwd_full(layer, key, ref, reinterpret_cast<uintptr_t>(main_grad), offset, ld, int(mode));
  if (st != QE_OK) return st;
  const int64_t tokens = c->contract.layer(layer).slots[ref.slot].tokens;
  if (!c->cfg.null_executor && tokens > 0 && (dy == nullptr || dx == nullptr)) return QE_ERR_INVALID_ARG;
  if (!elem_aligned(dy, dy_dtype) || !elem_aligned(dx, dx_dtype)) return QE_ERR_INVALID_ARG;
  if (c->contract.physical_fails()) return fail_physical(c);
  if (!c->cfg.null_executor) {
    const LayerDev &L = c->layers[size_t(layer)];
    std::vector<Copy> pre, post;
    const void *dyg = dy;
    void *dxg = dx;
    if (copy_inputs(c)) {
      dyg = L.dy_st;
      dxg = L.dx_st;
      pre.push_back({L.dy_st, dy, size_t(tokens) * size_t(L.desc.n_out) * esize(dy_dtype)});
      post.push_back({dx, L.dx_st, size_t(tokens) * size_t(L.desc.k_in) * esize(dx_dtype)});
    }
    Plan p;
    append_dgrad(c, p, L, ref.slot, tokens, dyg, dy_dtype, dxg, dx_dtype);
    append_wgrad(p, L, ref.slot, tokens, main_grad, offset, ld, mode);
    finish_dgrad(c, p, L);
    if (run_plan(c, p, graph_key(layer, ACT_FULL, ref.slot), static_cast<hipStream_t>(caller), pre, post) != QE_OK)
      return fail_physical(c);
  }
  c->contract.commit_bwd_full(layer, ref);
  return QE_OK;
}

// ------------------------------------------------------------------ arena / epoch
qe_status qe_arena_bind(qe_ctx *c, int32_t layer, uint32_t microbatch, float *buf, int64_t buf_elems, int64_t offset,
                        int64_t ld) {
  if (c == nullptr) return QE_ERR_INVALID_ARG;
  return c->contract.bind(layer, int64_t(microbatch), reinterpret_cast<uintptr_t>(buf), buf_elems, offset, ld);
}

qe_status qe_prebuild_graphs(qe_ctx *c, const qe_prebuild_desc *d) {
  if (c == nullptr || d == nullptr || d->tokens < 0 || !valid_dtype(d->x_dtype) || !valid_dtype(d->y_dtype) ||
      !valid_dtype(d->dy_dtype) || !valid_dtype(d->dx_dtype))
    return QE_ERR_INVALID_ARG;
  if (!c->cfg.use_graphs) return QE_ERR_INVALID_ARG;
  for (const auto &L : c->layers)
    if (d->tokens > L.desc.max_tokens) return QE_ERR_INVALID_ARG;
  if (c->cfg.null_executor) return QE_OK;
  DeviceGuard dg(c->cfg.device);
  if (!dg.ok) return QE_ERR_HIP;
  const auto t0 = std::chrono::steady_clock::now();
  const bool cp = copy_inputs(c);
  const int M = c->cfg.microbatches;
  if (!cp && c->placeholder == nullptr) {
    size_t bytes = 16;
    for (const auto &L : c->layers) {  // max_tokens rows: enough for any later prebuild too
      const size_t t = size_t(L.desc.max_tokens);
      const size_t w = size_t(L.desc.k_in > L.desc.n_out ? L.desc.k_in : L.desc.n_out);
      bytes = t * w * sizeof(float) > bytes ? t * w * sizeof(float) : bytes;
    }
    if (hipMalloc(&c->placeholder, bytes) != hipSuccess) {
      c->placeholder = nullptr;
      return QE_ERR_HIP;
    }
    c->st.device_bytes += int64_t(bytes);
  }
  for (int l = 0; l < int(c->layers.size()); ++l) {
    const LayerDev &L = c->layers[size_t(l)];
    const qe::LayerBook &B = c->contract.layer(l);
    const int64_t t = d->tokens > 0 ? d->tokens : L.desc.max_tokens;
    // Dynamic buffers are unknown here: the graphs bind the placeholder in
    // their place until the first call binds its own.
    const void *xg = cp ? L.x_st : c->placeholder;
    void *yg = cp ? L.y_st : c->placeholder;
    const void *dyg = cp ? L.dy_st : c->placeholder;
    void *dxg = cp ? L.dx_st : c->placeholder;
    for (int m = 0; m < M; ++m) {
      // F (microbatch 0 refreshes the weight cache: it is the first forward
      // after every optimizer commit), dI, and dW into the bound view
      const bool refresh = m == 0;
      const Plan pf = plan_fwd(c, L, uint32_t(m), xg, d->x_dtype, t, yg, d->y_dtype, refresh);
      qe_status st = bind_graph(c, c->graphs[graph_key(l, refresh ? ACT_FWD_REFRESH : ACT_FWD, uint32_t(m))], pf);
      if (st != QE_OK) return st;
      Plan pd;
      append_dgrad(c, pd, L, uint32_t(m), t, dyg, d->dy_dtype, dxg, d->dx_dtype);
      finish_dgrad(c, pd, L);
      st = bind_graph(c, c->graphs[graph_key(l, ACT_DGRAD, uint32_t(m))], pd);
      if (st != QE_OK) return st;
      const qe::View &V = B.views[size_t(m)];
      if (!V.bound) continue;
      // a microbatch whose view an earlier microbatch shares accumulates
      int mode = QE_PLACE_INIT;
      for (int m2 = 0; m2 < m; ++m2)
        if (B.views[size_t(m2)].bound && B.views[size_t(m2)].start() == V.start()) mode = QE_PLACE_ACCUM;
      Plan pw;
      append_wgrad(pw, L, uint32_t(m), t, reinterpret_cast<float *>(V.buf), V.offset, V.ld, mode);
      st = bind_graph(c, c->graphs[graph_key(l, ACT_WGRAD, uint32_t(m))], pw);
      if (st != QE_OK) return st;
    }
  }
  c->st.prebuild_ns +=
      std::chrono::duration_cast<std::chrono::nanoseconds>(std::chrono::steady_clock::now() - t0).count();
  return QE_OK;
}

qe_status qe_arena_finalize(qe_ctx *c) { return c ? c->contract.finalize() : QE_ERR_INVALID_ARG; }
qe_status qe_optimizer_commit(qe_ctx *c) { return c ? c->contract.optimizer_commit() : QE_ERR_INVALID_ARG; }
qe_status qe_arena_rebuild(qe_ctx *c) { return c ? c->contract.rebuild() : QE_ERR_INVALID_ARG; }

qe_status qe_checkpoint_export(qe_ctx *c, void *buf_host, int64_t capacity, int64_t *size_out_host) {
  if (c == nullptr || size_out_host == nullptr) return QE_ERR_INVALID_ARG;
  const qe_status q = c->contract.checkpoint_check();
  if (q != QE_OK) return q;
  const int64_t size = ckpt_size(c->layers);
  *size_out_host = size;
  if (buf_host == nullptr) return QE_OK;
  if (capacity < size) return QE_ERR_INVALID_ARG;
  DeviceGuard dg(c->cfg.device);
  if (!c->cfg.null_executor && (!dg.ok || sync_actions(c) != hipSuccess)) return QE_ERR_HIP;
  std::vector<uint8_t> out(size_t(size), 0);
  uint8_t *w = out.data();
  CkptHeader h;
  memset(&h, 0, sizeof(h));
  memcpy(h.magic, kCkptMagic, sizeof(h.magic));
  h.version = kCkptVersion;
  h.n_layers = uint32_t(c->layers.size());
  h.microbatches = c->cfg.microbatches;
  h.e_w = c->contract.e_w();
  memcpy(w, &h, sizeof(h));
  w += sizeof(h);
  std::vector<float> meta;
  for (const auto &L : c->layers) {
    const CkptLayer r = ckpt_layer_of(L.desc);
    memcpy(w, &r, sizeof(r));
    w += sizeof(r);
    const size_t H = size_t(L.desc.history_len);
    meta.assign(3 * H + 6, 0.0f);  // hist[3][H] | scale[3] | scale_inv[3]
    if (L.meta != nullptr) {
      if (hipMemcpy(meta.data(), L.meta, sizeof(float) * meta.size(), hipMemcpyDeviceToHost) != hipSuccess)
        return QE_ERR_HIP;
    } else {
      for (int k = 0; k < 6; ++k) meta[3 * H + size_t(k)] = 1.0f;  // null executor: initial state
    }
    for (size_t role = 0; role < 3; ++role) {
      memcpy(w, meta.data() + role * H, sizeof(float) * H);
      w += sizeof(float) * H;
      memcpy(w, meta.data() + 3 * H + role, sizeof(float));
      w += sizeof(float);
      memcpy(w, meta.data() + 3 * H + 3 + role, sizeof(float));
      w += sizeof(float);
    }
  }
  const uint64_t hash = fnv1a(out.data(), size_t(w - out.data()));
  memcpy(w, &hash, sizeof(hash));
  memcpy(buf_host, out.data(), out.size());
  return QE_OK;
}

qe_status qe_checkpoint_import(qe_ctx *c, const void *buf_host, int64_t size) {
  if (c == nullptr || buf_host == nullptr || size != ckpt_size(c->layers)) return QE_ERR_INVALID_ARG;
  const uint8_t *b = static_cast<const uint8_t *>(buf_host);
  uint64_t hash = 0;
  memcpy(&hash, b + size - int64_t(sizeof(hash)), sizeof(hash));
  if (hash != fnv1a(b, size_t(size) - sizeof(hash))) return QE_ERR_INVALID_ARG;
  CkptHeader h;
  memcpy(&h, b, sizeof(h));
  if (memcmp(h.magic, kCkptMagic, sizeof(h.magic)) != 0 || h.version != kCkptVersion ||
      h.n_layers != uint32_t(c->layers.size()) || h.microbatches != c->cfg.microbatches || h.e_w < 0)
    return QE_ERR_INVALID_ARG;
  const uint8_t *r = b + sizeof(h);
  for (const auto &L : c->layers) {  // configuration check before any change
    CkptLayer got;
    memcpy(&got, r, sizeof(got));
    const CkptLayer mine = ckpt_layer_of(L.desc);
    if (memcmp(&got, &mine, sizeof(got)) != 0) return QE_ERR_INVALID_ARG;
    r += sizeof(got) + ckpt_state_bytes(L.desc);
  }
  const qe_status q = c->contract.checkpoint_check();
  if (q != QE_OK) return q;
  if (!c->cfg.null_executor) {
    DeviceGuard dg(c->cfg.device);
    if (!dg.ok || sync_actions(c) != hipSuccess) return QE_ERR_HIP;
    r = b + sizeof(h);
    std::vector<float> meta;
    for (const auto &L : c->layers) {
      r += sizeof(CkptLayer);
      const size_t H = size_t(L.desc.history_len);
      meta.assign(3 * H + 6, 0.0f);
      for (size_t role = 0; role < 3; ++role) {
        memcpy(meta.data() + role * H, r, sizeof(float) * H);
        r += sizeof(float) * H;
        memcpy(meta.data() + 3 * H + role, r, sizeof(float));
        r += sizeof(float);
        memcpy(meta.data() + 3 * H + 3 + role, r, sizeof(float));
        r += sizeof(float);
      }
      if (hipMemcpy(L.meta, meta.data(), sizeof(float) * meta.size(), hipMemcpyHostToDevice) != hipSuccess ||
          hipMemset(L.accum, 0, sizeof(float) * 3 * qe::kAmaxLines * qe::kAmaxStride) != hipSuccess)
        return QE_ERR_HIP;
    }
  }
  return c->contract.restore(h.e_w);
}

qe_status qe_abort_epoch(qe_ctx *c) {
  if (c == nullptr) return QE_ERR_INVALID_ARG;
  c->contract.abort_epoch();
  return QE_OK;
}

qe_status qe_sync(qe_ctx *c) {
  if (c == nullptr) return QE_ERR_INVALID_ARG;
  if (c->cfg.null_executor) return QE_OK;
  DeviceGuard dg(c->cfg.device);
  if (!dg.ok || sync_actions(c) != hipSuccess) return QE_ERR_HIP;
  long long tok = 0;
  if (hipMemcpy(&tok, c->d_token, sizeof(tok), hipMemcpyDeviceToHost) != hipSuccess) return QE_ERR_HIP;
  c->st.device_token = tok;
  return QE_OK;
}

qe_status qe_get_state(const qe_ctx *c, qe_ctx_state *out) {
  if (c == nullptr || out == nullptr) return QE_ERR_INVALID_ARG;
  *out = c->st;
  out->e_w = c->contract.e_w();
  out->token = c->contract.token();
  out->arena_valid = c->contract.arena_valid();
  out->finalized = c->contract.finalized();
  out->graphs = int64_t(c->graphs.size());
  out->arena_bytes = c->contract.arena_bytes();
  return QE_OK;
}

qe_status qe_get_layer_state(const qe_ctx *c, int32_t layer, qe_layer_state *out) {
  if (c == nullptr || out == nullptr || layer < 0 || layer >= c->contract.num_layers()) return QE_ERR_INVALID_ARG;
  const qe::LayerBook &L = c->contract.layer(layer);
  memset(out, 0, sizeof(*out));
  out->e_c = L.e_c;
  out->refreshes = L.refreshes;
  out->n_slots = int32_t(L.slots.size());
  return QE_OK;
}

qe_status qe_get_slot_state(const qe_ctx *c, int32_t layer, int32_t slot, qe_slot_state *out) {
  if (c == nullptr || out == nullptr || layer < 0 || layer >= c->contract.num_layers() || slot < 0 ||
      slot >= c->cfg.microbatches)
    return QE_ERR_INVALID_ARG;
  const qe::LayerBook &L = c->contract.layer(layer);
  const qe::SlotState &S = L.slots[size_t(slot)];
  const qe::View &V = L.views[size_t(slot)];
  memset(out, 0, sizeof(*out));
  out->live = S.live;
  out->generation = S.generation;
  out->bits = S.bits;
  out->key = S.key;
  out->tokens = S.tokens;
  out->bound = V.bound;
  out->written = V.written;
  out->view_offset = V.offset;
  out->view_ld = V.ld;
  out->view_buf = reinterpret_cast<const float *>(V.buf);
  return QE_OK;
}

qe_status qe_inject_fault(qe_ctx *c, int32_t n) {
  if (c == nullptr || n < 0) return QE_ERR_INVALID_ARG;
  c->contract.inject_fault(n);
  return QE_OK;
}

qe_status qe_set_kernel_timing(qe_ctx *c, int32_t enable) {
  if (c == nullptr) return QE_ERR_INVALID_ARG;
  c->timing = enable != 0;
  return QE_OK;
}

qe_status qe_get_kernel_timing(qe_ctx *c, int32_t kernel_class, double *total_ms_host, int64_t *launches_host) {
  if (c == nullptr || kernel_class < 0 || kernel_class >= qe::KC_COUNT || !total_ms_host || !launches_host)
    return QE_ERR_INVALID_ARG;
  if (!c->cfg.null_executor && !c->timed.empty()) {
    DeviceGuard dg(c->cfg.device);
    if (!dg.ok || sync_actions(c) != hipSuccess) return QE_ERR_HIP;
    // read every pair first, so that a failure leaves the totals and the
    // pending pairs as they were (a later call reads them again)
    std::vector<float> ms(c->timed.size(), 0.f);
    for (size_t i = 0; i < c->timed.size(); ++i)
      if (hipEventElapsedTime(&ms[i], c->timed[i].t0, c->timed[i].t1) != hipSuccess) return QE_ERR_HIP;
    for (size_t i = 0; i < c->timed.size(); ++i) {
      const TimedCall &t = c->timed[i];
      c->kc_ms[t.kind] += ms[i];
      c->kc_n[t.kind] += 1;
      c->event_pool.push_back(t.t0);
      c->event_pool.push_back(t.t1);
    }
    c->timed.clear();
  }
  *total_ms_host = c->kc_ms[kernel_class];
  *launches_host = c->kc_n[kernel_class];
  return QE_OK;
}

}  // extern "C"
