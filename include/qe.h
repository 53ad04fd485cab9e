/*
 * qe.h -- C ABI of the MI355X (gfx950) FP8 delayed-scaling linear layer with
 * split backward.
 *
 * The paper ("Explicit State and Resource Contracts for Low-Precision
 * Pipeline Parallel Training under Captured Graphs") splits a pipeline stage
 * into three checked actions, forward (F), input gradient (dI) and deferred
 * weight gradient (dW), with the state transition of §3.2:
 *     (Y_m, S1, T_m) = F(X_m, W, S0);  (dX_m, B_m, S2, Q_m) = dI(dY_m, T_m, S1);
 *     dW_m = dW(Q_m)
 * where S is the delayed-scaling FP8 state.  This library implements that
 * path for FP8 linear layers: per-tensor amax and the scale update from a
 * rolling amax history, FP8 quantization with a fused transpose, the three
 * FP8 GEMMs, and direct placement of dW into a flat FP32 main-gradient buffer
 * (§3.4).  The bookkeeping of §3.1-§3.6 and Algorithm 1 (§4.1) guards the
 * actions, and the per-action kernel sequence can be replayed through HIP
 * graphs on one stream-ordered executor with a two-way stream handoff (§4.4).
 *
 * Conventions for every call:
 *  - Pointers are DEVICE pointers unless the parameter name ends in _host.
 *    The library never takes ownership of a caller pointer.
 *  - `stream` / `caller` is a hipStream_t passed as void* (0 = the null
 *    stream).  All device work is asynchronous with respect to the host and
 *    ordered on that stream (or, for the layer actions, on the context's
 *    graph stream behind a two-way handoff with `caller`).
 *  - Matrices are row-major.  A "leading dimension" is the distance in
 *    elements between consecutive rows.
 *  - Every call validates its arguments first.  A call that returns anything
 *    other than QE_OK enqueued no device work and changed no state, except
 *    QE_ERR_HIP from a layer action, which aborts the epoch (see
 *    qe_abort_epoch).
 *  - A context is used by one host thread at a time.
 */
#ifndef QE_H
#define QE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef void *qe_stream; /* a hipStream_t */

typedef enum {
  QE_OK = 0,
  QE_ERR_INVALID_ARG = 1,        /* bad pointer, size, layout, index or enum */
  QE_ERR_STALE_REF = 2,          /* TapeRef names a free slot or an older generation (§3.1) */
  QE_ERR_KEY_MISMATCH = 3,       /* TapeKey differs from the key bound to the slot / layer */
  QE_ERR_KEY_LIVE = 4,           /* forward of a key whose tape is still live */
  QE_ERR_POOL_FULL = 5,          /* the microbatch's slot holds another live key */
  QE_ERR_DUPLICATE_CONSUMER = 6, /* dI or dW already ran on this tape (§3.1) */
  QE_ERR_ORDER = 7,              /* dW before dI, or INIT/ACCUM against the view's state */
  QE_ERR_EPOCH = 8,              /* key epoch differs from the weight version e_W (§3.3) */
  QE_ERR_STALE_CACHE = 9,        /* non-first forward while e_C != e_W (§3.3) */
  QE_ERR_DEST_MISMATCH = 10,     /* dW destination differs from the bound view (§3.4) */
  QE_ERR_DEST_ALIAS = 11,        /* bound view overlaps another layer's / another view */
  QE_ERR_DUP_WRITE = 12,         /* the view was already written this epoch */
  QE_ERR_ARENA_INVALID = 13,     /* arena flagged unusable after an abort (§4.5) */
  QE_ERR_INCOMPLETE = 14,        /* finalize / commit with a bound view unwritten */
  QE_ERR_NOT_QUIESCENT = 15,     /* commit with a live tape (Invariant 4) */
  QE_ERR_HIP = 16,               /* a HIP runtime call failed; the epoch is aborted */
  QE_ERR_UNSUPPORTED = 17        /* no gfx950 device, or library built without it */
} qe_status;

typedef enum { QE_E4M3 = 0, QE_E5M2 = 1 } qe_fp8_fmt;   /* OCP FP8 formats (max 448 / 57344) */
typedef enum { QE_F32 = 0, QE_BF16 = 1 } qe_dtype;
typedef enum { QE_PLACE_INIT = 0, QE_PLACE_ACCUM = 1 } qe_place_mode;
typedef enum { QE_ROLE_X = 0, QE_ROLE_W = 1, QE_ROLE_DY = 2 } qe_role;
/* Scaling recipe of a layer: delayed (scales from the amax history, §2.1) or
 * current / dynamic (each tensor's scale from its own amax, the kind of
 * output boundary §4.2 allows at the last stage). */
typedef enum { QE_SCALING_DELAYED = 0, QE_SCALING_CURRENT = 1 } qe_scaling;

/* TapeKey K = (e, s, m, u, i): optimizer epoch, pipeline stage, microbatch,
 * sub-layer unit, invocation counter (§3.1). */
typedef struct {
  uint32_t epoch, stage, microbatch, unit, invocation;
} qe_tape_key;

/* TapeRef R = (p, g_p): slot and its generation at allocation (§3.1). */
typedef struct {
  uint32_t slot, generation;
} qe_tape_ref;

/* Amax accumulator: QE_AMAX_LINES floats spaced QE_AMAX_STRIDE floats
 * (256 bytes) apart, QE_AMAX_LINES * QE_AMAX_STRIDE floats (16 KiB) in all,
 * zero-initialised.  Its value is the max over the lines.  Producers fold a
 * workgroup's max into line (workgroup % QE_AMAX_LINES), so concurrent
 * workgroups never contend for one cache line: device-scope atomics on one
 * line serialise at the memory side (about 11 ns each on MI355X), which a
 * single accumulator float would pay once per workgroup. */
#define QE_AMAX_LINES 64
#define QE_AMAX_STRIDE 64

/* Delayed-scaling state of one tensor role (§2.1): all device pointers.
 * amax_history[history_len]; scale and scale_inv are single floats;
 * amax_accum is an optional amax accumulator (NULL: amaxes are folded into
 * amax_history[0] directly).  Initial state: history and accumulator all
 * zero, scale = scale_inv = 1. */
typedef struct {
  float *amax_history;
  float *scale;
  float *scale_inv;
  int32_t history_len;
  int32_t margin;
  int32_t fmt; /* qe_fp8_fmt */
  int32_t reserved;
  float *amax_accum;
} qe_fp8_meta;

/* ------------------------------------------------------------------------
 * Hot-path primitives (stateless; device pointers; stream-ordered)
 * ------------------------------------------------------------------------ */

/* Delayed scale update (§2.1; the S0->S1 / S1->S2 transitions of §3.2) for
 * n_metas roles in one launch.  For each meta: if amax_accum is set, its
 * value is first folded into amax_history[0] (max) and its lines cleared;
 * then a = max(amax_history[0..H-1])
 * (NaN propagates); if a is finite and > 0, e = floor(log2(fmax/a)) - margin
 * clamped to [-126, 126], scale = 2^e, scale_inv = 2^-e, else scale is kept;
 * then the history rotates one place towards index 0 (index 0 moves to H-1)
 * and index 0 is cleared.  `metas_host` is a host array; 1 <= n_metas <= 8;
 * 1 <= history_len <= 8192.  If device_token is non-null, one int64 at that
 * device address is incremented once per call (the effect token of §3.2).
 * Errors: QE_ERR_INVALID_ARG for null pointers / bad sizes; QE_ERR_HIP. */
qe_status qe_amax_scale_update(const qe_fp8_meta *metas_host, int32_t n_metas, int64_t *device_token,
                               qe_stream stream);

/* FP8 quantization with fused transpose and amax (§2.1, §3.2).
 * in: [rows, cols] row-major, QE_F32 or QE_BF16, leading dimension cols.
 * Writes q_row[r * ld_row + c] = Q(in[r][c] * scale) and
 *        q_col[c * ld_col + r] = the same code (the transpose),
 * where Q rounds to nearest even and saturates to +-fmax (NaN -> 0x7F|sign).
 * Either output may be NULL.  max|in| (unscaled) is folded with a max (NaN
 * propagates) into meta->amax_accum if set (it then reaches amax_history[0]
 * at the next qe_amax_scale_update), else into meta->amax_history[0].  If scale_inv_snapshot
 * is non-null the scale_inv paired with the scale used is copied there.
 * Layout rules: ld_row >= cols, ld_col >= rows.  rows or cols may be 0.
 * Errors: QE_ERR_INVALID_ARG; QE_ERR_HIP. */
qe_status qe_quantize_fp8(const void *in, qe_dtype in_dtype, int64_t rows, int64_t cols, const qe_fp8_meta *meta_host,
                          uint8_t *q_row, int64_t ld_row, uint8_t *q_col, int64_t ld_col, float *scale_inv_snapshot,
                          qe_stream stream);

/* Amax of a tensor (§2.1): max |in[i]| over the numel contiguous elements of
 * in (QE_F32 or QE_BF16), computed exactly, folded with a max (NaN
 * propagates) into the role's amax slot: meta->amax_accum if set, else
 * meta->amax_history[0].  numel may be 0.  in must be aligned to its element
 * size.  Errors: QE_ERR_INVALID_ARG; QE_ERR_HIP. */
qe_status qe_amax(const void *in, qe_dtype in_dtype, int64_t numel, const qe_fp8_meta *meta_host, qe_stream stream);

/* Current (dynamic) scaling cast: the scale is set from the amax of `in`
 * itself, then `in` is cast with it (the dynamic alternative to delayed
 * scaling, §2.1; a last-stage boundary in §4.2).  Three launches on `stream`:
 * qe_amax into the role's amax slot, the scale update of
 * qe_amax_scale_update (so e = floor(log2(fmax / amax)) - margin, an amax of
 * 0, inf or NaN keeps the previous scale, and the slot is cleared again),
 * then the cast of qe_quantize_fp8 without recording an amax.  The meta must
 * have history_len == 1 and a clear amax slot on entry (as initialised and
 * as every call leaves it).  Other arguments as for qe_quantize_fp8;
 * device_token as for qe_amax_scale_update.
 * Errors: QE_ERR_INVALID_ARG (also for history_len != 1); QE_ERR_HIP. */
qe_status qe_quantize_fp8_current(const void *in, qe_dtype in_dtype, int64_t rows, int64_t cols,
                                  const qe_fp8_meta *meta_host, uint8_t *q_row, int64_t ld_row, uint8_t *q_col,
                                  int64_t ld_col, float *scale_inv_snapshot, int64_t *device_token,
                                  qe_stream stream);

/* Allocation-free variant of qe_quantize_fp8_current, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc): the same cast with the same results, but
 * the amax accumulator (the per-line partial maxima the amax pass folds its
 * workgroups into) is a scratch array inside the library, 16 KiB per device
 * and held by each device the library runs on until the process ends,
 * instead of one the caller brings in meta_host->amax_accum, which must be
 * NULL here.  The call allocates nothing (no hipMalloc, hipFree or allocating
 * library routine); the first call on a device looks up that device's copy of
 * the scratch.  Four launches on `stream`: a kernel clears the scratch, then
 * qe_quantize_fp8_current's amax pass, scale update and cast.  The scratch
 * size does not depend on the tensor (any number of workgroups folds into its
 * 64 lines), so every size qe_quantize_fp8_current accepts is accepted.
 * Every call on one device shares that device's scratch: calls that overlap
 * on one device (on different streams, or from different host threads
 * without ordering) race and give undefined results; calls ordered on one
 * stream are independent.  Other arguments and errors as for
 * qe_quantize_fp8_current; QE_ERR_INVALID_ARG also when
 * meta_host->amax_accum is set; QE_ERR_HIP if the scratch cannot be found. */
qe_status qe_quantize_fp8_current_noalloc(const void *in, qe_dtype in_dtype, int64_t rows, int64_t cols,
                                          const qe_fp8_meta *meta_host, uint8_t *q_row, int64_t ld_row,
                                          uint8_t *q_col, int64_t ld_col, float *scale_inv_snapshot,
                                          int64_t *device_token, qe_stream stream);

/* FP8 GEMM in "TN" form (both operands contiguous along the reduction axis):
 *     D[i][j] = (a_scale_inv * b_scale_inv) * sum_r A[i][r] * B[j][r]
 * A: m x k codes of format fmt_a, row stride lda bytes.  B: n x k codes of
 * format fmt_b, stride ldb.  a_scale_inv / b_scale_inv: one device float each.
 * FP32 accumulation.  mode QE_PLACE_INIT stores D into c (QE_F32 or QE_BF16);
 * QE_PLACE_ACCUM adds it in FP32 (c must be QE_F32): c = fl32(c + D).  Only
 * the m x n view c[i * ldc + j] is read or written.  F (Y = X W^T), dI
 * (dX = dY W) and dW (dW = dY^T X) of §3.2 are all this call on the codes and
 * transposed codes of qe_quantize_fp8.
 * Layout rules: a, b 16-byte aligned; lda, ldb multiples of 16 and >= k
 * rounded up to 16; ldc >= n; c 4-byte aligned (QE_F32) or 2-byte (QE_BF16);
 * k < 2^31.  Operands of 2 GiB or more are run as several launches over
 * row blocks of A (or of B), with the same per-element results.
 * Errors: QE_ERR_INVALID_ARG; QE_ERR_HIP. */
qe_status qe_fp8_gemm_tn(const uint8_t *a, qe_fp8_fmt fmt_a, int64_t lda, const uint8_t *b, qe_fp8_fmt fmt_b,
                         int64_t ldb, int64_t m, int64_t n, int64_t k, const float *a_scale_inv,
                         const float *b_scale_inv, void *c, qe_dtype c_dtype, int64_t ldc, qe_place_mode mode,
                         qe_stream stream);

/* Macro-tile shape of every FP8 GEMM the library launches (qe_fp8_gemm_tn and
 * the layer actions).  QE_TILE_AUTO picks, per call, the shape that needs the
 * fewest rounds of workgroups over the device's compute units (256 on
 * MI355X, read from the device properties), weighted by a
 * measured per-round cost; the others force one shape (for tests and
 * measurements).  Process-wide; it applies to launches enqueued afterwards
 * (a graph captured earlier keeps the shapes it was captured with).  The
 * five shapes give the same bits: the same 16x16x128 MFMA with the same
 * reduction bytes per lane, the same order along K, no split reduction.
 * Errors: QE_ERR_INVALID_ARG for a value outside the enum. */
typedef enum {
  QE_TILE_AUTO = 0,
  QE_TILE_256x256 = 1,
  QE_TILE_256x192 = 2,
  QE_TILE_192x256 = 3,
  QE_TILE_256x128 = 4,
  QE_TILE_256x224 = 5
} qe_gemm_tile;
qe_status qe_set_gemm_tile(qe_gemm_tile tile);

/* ------------------------------------------------------------------------
 * Stage context: layers, tape slots, versions, arena, executor
 * ------------------------------------------------------------------------ */

typedef struct qe_ctx qe_ctx;

typedef struct {
  int32_t device;        /* HIP device ordinal */
  int32_t microbatches;  /* M: tape slots per layer, slot p = microbatch m */
  int32_t use_graphs;    /* 1: capture each (layer, action, slot) sequence once and replay it */
  int32_t null_executor; /* 1: run the contract only, no HIP call at all (host-only testing) */
  int32_t one_way_handoff; /* testing only: skip the caller's wait on the graph tail (§2.3) */
  int32_t copy_gradients;  /* 1: dW goes to a private FP32 buffer, then is copied into the bound view
                              (the copied-gradient path of §3.4, an ablation baseline); 0: direct */
  int32_t replay_on_caller; /* 0 (default): every action runs on the library's graph stream behind the
                              two-way handoff of §2.3 / §4.4 (the graph stream waits on the caller's
                              event, the caller waits on the graph's tail event).  1: every action's
                              graph (or kernels) is launched on the caller's stream itself, so stream
                              order gives both directions of the handoff; every action's stream
                              first waits on an event recorded right after the previous action (on
                              its stream), so actions issued from different streams stay in one
                              total order, as on one graph stream (on the same stream the wait is
                              already satisfied).  No caller stream handle is kept between actions.
                              The same ordering contract, without the two cross-stream waits per
                              action of the graph-stream executor. */
  int32_t graph_inputs;     /* how a replayed graph meets the buffers of each call (§4.4, dynamic
                              inputs); use_graphs only.  QE_GRAPH_INPUTS_REBIND (0, default): the
                              graph's kernel nodes are rewritten in place with the call's pointers
                              when they differ from the ones it holds (the host first waits for that
                              graph's previous replay to finish); a different launch shape (token
                              count, dtype, alignment class) captures it again.
                              QE_GRAPH_INPUTS_RECAPTURE (1): captured again on any change.
                              QE_GRAPH_INPUTS_COPY (2): the paper's scheme: graphs bind static
                              library buffers (max_tokens rows of FP32 for X, Y, dY, dX per layer);
                              each call copies X (F) or dY (dI) in after the caller -> graph edge
                              and Y or dX out before the completion event. */
} qe_config;

enum {
  QE_GRAPH_INPUTS_REBIND = 0,
  QE_GRAPH_INPUTS_RECAPTURE = 1,
  QE_GRAPH_INPUTS_COPY = 2
};

typedef struct {
  uint32_t stage, unit;  /* with microbatch/epoch/invocation, forms the TapeKey of every action */
  int64_t n_out, k_in;   /* W is [n_out, k_in] */
  int64_t max_tokens;    /* largest microbatch (rows of X) the slots can hold */
  const void *w;         /* master weights, caller-owned, fixed address, updated in place by the caller */
  int32_t w_dtype;       /* qe_dtype */
  int32_t history_len;   /* amax history length H (all roles) */
  int32_t margin;        /* scale margin (all roles) */
  int32_t fmt_x, fmt_w, fmt_dy; /* qe_fp8_fmt per role */
  int32_t scaling;       /* qe_scaling; QE_SCALING_CURRENT requires history_len == 1 */
} qe_layer_desc;

/* Create a context: one pipeline stage's executor and contract state (§4.1,
 * Algorithm 1, whose state starts at e_W = 0, token 0, every slot free at
 * generation 0; §4.4 for the one stream-ordered graph stream).  Allocates the
 * graph stream and events (unless null_executor, the host-only mode of the
 * CPU fault injections of §5.2).  Errors: QE_ERR_INVALID_ARG (also
 * replay_on_caller outside {0, 1}, or together with one_way_handoff, or
 * graph_inputs outside its enum), QE_ERR_UNSUPPORTED, QE_ERR_HIP. */
qe_status qe_ctx_create(const qe_config *cfg_host, qe_ctx **out_host);
/* Destroy a context: waits for its device work, then frees its graphs,
 * events, streams and every allocation of its layers.  NULL is a no-op. */
void qe_ctx_destroy(qe_ctx *ctx);

/* Register a linear layer: one sub-layer unit u of the stage, the (s, u)
 * part of every TapeKey of its actions (§3.1), with the delayed-scaling state
 * S of its three tensor roles (§2.1, §3.2), its weight cache and version
 * e_C (§3.3) and one tape slot per configured microbatch (§4.3: static
 * binding, one slot per microbatch).  Allocates its FP8 state (three roles),
 * its quantized-weight cache W_q [N,K] and W_q^T [K,N], one tape payload per
 * slot (X_q^T [K, tokens], dY_q^T [N, tokens] and the two scale_inv
 * snapshots: the retained Q_m of §3.2), and scratch for the row-wise X_q /
 * dY_q.  (stage, unit) must be unique (QE_ERR_INVALID_ARG); so must be the
 * bounds: 1 <= history_len <= 8192, n_out, k_in and max_tokens below 2^31
 * (each is the reduction length of one of the three products), formats and
 * dtypes in their enums.
 * With desc->scaling == QE_SCALING_CURRENT every cast below takes its scale
 * from the amax of the tensor it casts (qe_quantize_fp8_current's sequence)
 * instead of from the history; nothing else about the actions changes. */
qe_status qe_layer_register(qe_ctx *ctx, const qe_layer_desc *desc_host, int32_t *layer_out_host);

/* Device pointers of a role's FP8 state S (§2.1: amax history, scale,
 * scale_inv; §3.5: the part of the state a checkpoint persists), for
 * inspection.  Errors: QE_ERR_INVALID_ARG for a bad layer or role. */
qe_status qe_layer_meta(const qe_ctx *ctx, int32_t layer, qe_role role, qe_fp8_meta *out_host);

/* Device pointers of the quantized-weight cache (§3.3) and a slot's tape
 * payload Q_m (§3.2), for inspection.  Row strides in bytes are returned in
 * ld_*; any out pointer may be NULL.  Errors: QE_ERR_INVALID_ARG. */
qe_status qe_layer_cache(const qe_ctx *ctx, int32_t layer, const uint8_t **w_q, int64_t *ld_w_q,
                         const uint8_t **w_q_t, int64_t *ld_w_q_t, const float **w_scale_inv);
qe_status qe_layer_slot_payload(const qe_ctx *ctx, int32_t layer, int32_t slot, const uint8_t **x_q_t,
                                int64_t *ld_x_q_t, const uint8_t **dy_q_t, int64_t *ld_dy_q_t,
                                const float **x_scale_inv, const float **dy_scale_inv);

/* F (§3.2, Algorithm 1): check that key.epoch = e_W, the microbatch's slot is
 * free, and the weight cache is current (only microbatch 0 may refresh it,
 * setting e_C <- e_W; §3.3).  Device work: [refresh: quantize W into the
 * cache, record amax(W)]; quantize X into the slot's X_q^T (+ row-wise
 * scratch), record amax(X), snapshot scale_inv(X); Y = X W^T in FP8; update
 * the X and W scales.  Then the slot's generation is advanced, the key bound
 * and the effect token advanced; *ref_out_host receives (slot, generation).
 * Current scaling: amax(X) [and amax(W) on refresh] first, then the X [and
 * W] scale update, then the casts without recording, then the GEMM.
 * x: [tokens, K] (QE_F32/QE_BF16); y: [tokens, N] (QE_F32/QE_BF16). */
qe_status qe_fp8_linear_fwd(qe_ctx *ctx, int32_t layer, qe_tape_key key, const void *x, qe_dtype x_dtype,
                            int64_t tokens, void *y, qe_dtype y_dtype, qe_tape_ref *ref_out_host,
                            qe_stream caller);

/* dI (§3.2): resolve ref (live slot, equal generation, equal key, epoch) and
 * require dI not yet run.  Device work: quantize dY once (the slot's dY_q^T +
 * row-wise scratch), record amax(dY), snapshot scale_inv(dY); dX = dY W in
 * FP8 using the cached W_q^T; update the dY scale.  Marks dI done, advances the
 * effect token.  Current scaling: amax(dY), the dY scale update, then the
 * cast without recording, then the GEMM.  dy: [tokens, N]; dx: [tokens, K]. */
qe_status qe_fp8_linear_dgrad(qe_ctx *ctx, int32_t layer, qe_tape_key key, qe_tape_ref ref, const void *dy,
                              qe_dtype dy_dtype, void *dx, qe_dtype dx_dtype, qe_stream caller);

/* Deferred dW with direct placement (§3.2, §3.4, §4.3): resolve ref, require
 * dI done and dW not, a valid arena, and a destination equal to the view bound
 * by qe_arena_bind for (layer, key.microbatch) that is unwritten this epoch.
 * mode QE_PLACE_INIT is legal only while no binding sharing the view has
 * written this epoch, QE_PLACE_ACCUM only after one has (else QE_ERR_ORDER).
 * Device work: main_grad[offset + n*ld + k] (=, or +=)
 *   scale_inv(dY)_slot * scale_inv(X)_slot * sum_t dY_q^T[n][t] X_q^T[k][t]
 * using the snapshots kept in the slot, never the live scales; no FP8 state
 * update, no token advance.  With qe_config.copy_gradients the GEMM writes a
 * private [N, K] FP32 buffer and a second kernel copies (or adds) it into
 * the view; the bits are the same as with direct placement.  Marks dW done and the view written; the slot is
 * released (payload dropped, generation kept) once dI and dW have both run. */
qe_status qe_fp8_linear_wgrad_place(qe_ctx *ctx, int32_t layer, qe_tape_key key, qe_tape_ref ref,
                                    float *main_grad, int64_t offset, int64_t ld, qe_place_mode mode,
                                    qe_stream caller);

/* Full backward: dI immediately followed by dW on the same tape, in one
 * action (the non-split baseline the paper compares against, §5.2).  Checks
 * are the union of both; the dW bits equal those of the split path. */
qe_status qe_fp8_linear_bwd_full(qe_ctx *ctx, int32_t layer, qe_tape_key key, qe_tape_ref ref, const void *dy,
                                 qe_dtype dy_dtype, void *dx, qe_dtype dx_dtype, float *main_grad,
                                 int64_t offset, int64_t ld, qe_place_mode mode, qe_stream caller);

/* Bind the dW destination of (layer, microbatch): the [N, K] view with row
 * stride ld at `offset` elements into the flat FP32 buffer `buf` of buf_elems
 * elements (§3.4; one view per matrix parameter and configured microbatch,
 * §4.3).  Views of one layer may be shared by several microbatches (the first
 * write initialises, later ones accumulate); any other overlap is
 * QE_ERR_DEST_ALIAS.  Requires ld >= K and offset + (N-1)*ld + K <= buf_elems;
 * a view already written this epoch cannot be rebound (QE_ERR_DUP_WRITE). */
qe_status qe_arena_bind(qe_ctx *ctx, int32_t layer, uint32_t microbatch, float *buf, int64_t buf_elems,
                        int64_t offset, int64_t ld);

/* Static binding (§4.3, eq. G_r = 3 M L_r): capture, before the first step,
 * the graph of every action the stage will replay: for each registered layer
 * and each microbatch m < M, F (m = 0 with the weight-cache refresh, since
 * microbatch 0 is the first forward after every commit), dI, and dW into the
 * view bound to (layer, m) (QE_PLACE_ACCUM when an earlier microbatch's view
 * of the layer starts at the same address, else QE_PLACE_INIT; unbound
 * (layer, m) pairs get no dW graph).  The graphs are built for `tokens` rows
 * (0: each layer's max_tokens) and the given dtypes; the caller's X, Y, dY, dX
 * buffers are not known yet, so every call binds them into its graph
 * (qe_config.graph_inputs) without a new capture when the tokens and dtypes
 * match.  Capture and instantiation time is added to qe_ctx_state.capture_ns
 * and prebuild_ns, the graphs to .captures.  Requires use_graphs.  No device
 * work is enqueued.  Errors: QE_ERR_INVALID_ARG (no graphs, a bad dtype,
 * tokens above a layer's max_tokens); QE_ERR_HIP. */
typedef struct {
  int64_t tokens;
  int32_t x_dtype, y_dtype;   /* qe_dtype of F's input and output */
  int32_t dy_dtype, dx_dtype; /* qe_dtype of dI's input and output */
} qe_prebuild_desc;
qe_status qe_prebuild_graphs(qe_ctx *ctx, const qe_prebuild_desc *desc_host);

/* Arena finalization (§3.4, §4.5; Algorithm 1 before the optimizer step):
 * every bound view written exactly once this epoch (else QE_ERR_INCOMPLETE,
 * Table "faults": finalize with a missing dW), arena valid (else
 * QE_ERR_ARENA_INVALID).  Changes nothing when refused. */
qe_status qe_arena_finalize(qe_ctx *ctx);

/* Optimizer commit (Algorithm 1, §4.5): requires no live tape
 * (QE_ERR_NOT_QUIESCENT), a valid and, if any view is bound, finalized arena.
 * Advances e_W, so the next microbatch-0 forward refreshes every cache.  The
 * caller updates the master weights in place between finalize and commit. */
qe_status qe_optimizer_commit(qe_ctx *ctx);

/* Abort the epoch (§4.5): purge the live tapes of e_W (generations kept) and
 * flag the arena unusable until qe_arena_rebuild (Table "faults": a write
 * after an aborted write is refused with QE_ERR_ARENA_INVALID). */
qe_status qe_abort_epoch(qe_ctx *ctx);
/* Rebuild the arena after an abort (§4.5): views stay bound, written marks
 * and finalization are cleared, the arena is valid again. */
qe_status qe_arena_rebuild(qe_ctx *ctx);

/* Quiescent checkpoint (§3.5, Invariant 4).  A checkpoint holds the
 * persistent part of the stage: the logical optimizer epoch e_W, every
 * registered layer's static configuration and precision recipe, and the FP8
 * state (amax history, scale, scale_inv) of its three roles.  Tapes, slot
 * generations, the effect token, graphs, events, arena bindings and the
 * weight caches are process-local and are not in it.
 *
 * Payload (host bytes, little-endian, version 1): a 32-byte header {char
 * magic[8] = "QECKPT01"; uint32 version; uint32 n_layers; int32 microbatches;
 * int32 reserved; int64 e_w}; per layer a 64-byte record {uint32 stage, unit;
 * int64 n_out, k_in, max_tokens; int32 w_dtype, history_len, margin, fmt_x,
 * fmt_w, fmt_dy, scaling, reserved} followed, for the roles X, W, dY in that
 * order, by history_len history floats, the scale and the scale_inv; then an
 * 8-byte FNV-1a hash of all preceding bytes.
 *
 * Export: allowed only at a quiescent point: no live tape, and no arena write
 * or finalize since the last qe_optimizer_commit (else QE_ERR_NOT_QUIESCENT;
 * Table "faults": a checkpoint with live work is withheld), and a valid arena
 * (else QE_ERR_ARENA_INVALID); nothing changes when refused.  It waits for
 * the graph stream, then writes the payload.  *size_out_host always receives
 * the payload size; with buf_host == NULL only the size is returned;
 * capacity < size is QE_ERR_INVALID_ARG.  With null_executor the FP8 state
 * written is the initial one (history 0, scales 1). */
qe_status qe_checkpoint_export(qe_ctx *ctx, void *buf_host, int64_t capacity, int64_t *size_out_host);

/* Import (restart): into a context whose layers were registered in the same
 * order with the same configuration (stage, unit, n_out, k_in, max_tokens,
 * w_dtype, history_len, margin, formats, scaling) and the same microbatch
 * count, at a quiescent point.  Loads the FP8 state (clearing the amax
 * accumulators), sets e_W to the saved epoch and marks every weight cache
 * stale, so the first forward of the epoch (microbatch 0) re-quantizes W with
 * the restored W scale; the token and generations stay this process's.
 * Errors, with nothing changed: QE_ERR_INVALID_ARG (bad size, magic, version,
 * hash, or a configuration that differs), QE_ERR_NOT_QUIESCENT /
 * QE_ERR_ARENA_INVALID as for export.  QE_ERR_HIP: the device copy failed and
 * the FP8 state is undefined; discard the context. */
qe_status qe_checkpoint_import(qe_ctx *ctx, const void *buf_host, int64_t size);

/* Block until all device work of the context's actions has finished (the
 * graph stream, and the completion event of the last action, which every
 * earlier action precedes), then read back the device effect token: the
 * token of §3.2 / Invariant 1, which advances once per F and per dI, so a
 * caller can check that the device ran exactly the state-mutating actions the
 * host committed (qe_ctx_state.device_token == .token).  Errors: QE_ERR_HIP. */
qe_status qe_sync(qe_ctx *ctx);

typedef struct {
  int64_t e_w;               /* weight version */
  int64_t token;             /* host effect token: +1 per F and per dI */
  int64_t device_token;      /* last value read back by qe_sync (-1 if never) */
  int32_t arena_valid, finalized;
  int64_t graphs;            /* graph executables held */
  int64_t captures;          /* captures performed (prebuilt ones, first uses and re-captures) */
  int64_t replays;           /* graph launches */
  int64_t handoffs;          /* caller<->graph stream handoffs (2 per action; 0 with replay_on_caller) */
  int64_t capture_ns;        /* host time spent capturing + instantiating */
  int64_t arena_bytes;       /* bytes covered by bound views */
  int64_t device_bytes;      /* bytes the library allocated */
  int64_t rebinds;           /* replays whose graph had kernel-node arguments rewritten first */
  int64_t rebound_nodes;     /* kernel nodes rewritten by those rebinds */
  int64_t prebuild_ns;       /* host time of qe_prebuild_graphs (captures + instantiations) */
} qe_ctx_state;

typedef struct {
  int64_t e_c;               /* cache version (-1: never filled) */
  int64_t refreshes;
  int32_t n_slots;
  int32_t reserved;
} qe_layer_state;

typedef struct {
  int32_t live;
  uint32_t generation;
  uint32_t bits;             /* 1 = dI done, 2 = dW done */
  uint32_t reserved;
  qe_tape_key key;           /* valid when live */
  int64_t tokens;            /* valid when live */
  int32_t bound, written;    /* arena view of (layer, slot) */
  int64_t view_offset, view_ld;
  const float *view_buf;
} qe_slot_state;

/* Host snapshots of the contract state (§3.1-§3.6: e_W, the effect token,
 * arena validity and finalization; per layer e_C and refreshes; per slot
 * liveness, generation g_p, consumer bits, bound key and view) and of the
 * executor's counters (graphs, captures, rebinds, replays, handoffs, §4.3 /
 * §4.4).  Pure reads; no device work.  Errors: QE_ERR_INVALID_ARG. */
qe_status qe_get_state(const qe_ctx *ctx, qe_ctx_state *out_host);
qe_status qe_get_layer_state(const qe_ctx *ctx, int32_t layer, qe_layer_state *out_host);
qe_status qe_get_slot_state(const qe_ctx *ctx, int32_t layer, int32_t slot, qe_slot_state *out_host);

/* Testing hook (host only), the fault injection of §5.2 and Table "faults"
 * (a physical failure after the checks): the n-th next layer action that
 * passes its checks fails as if its device work could not be enqueued
 * (QE_ERR_HIP; the epoch is aborted, §4.5).  n = 0 disarms. */
qe_status qe_inject_fault(qe_ctx *ctx, int32_t n);

/* Kernel timing (measurement support; the paper times whole steps after
 * warm-up and capture, §5.1): when enabled (eager mode only; replayed graphs
 * are not timed), every launch the context makes is timed by a pair of HIP
 * events that its kernels carry (hipExtLaunchKernel: from the start of its
 * first kernel to the end of its last), and counted under its kernel class:
 * 0 quantize (a paired weight-and-input cast is one launch), 1 stand-alone
 * scale update, 2 GEMM (with any scale update that runs in its extra
 * workgroups), 3 gradient copy, 4 amax pass.  qe_get_kernel_timing waits for
 * the context's actions and returns the running totals of one class since
 * the context was created (milliseconds, launches); kernel_class outside
 * 0..4 is QE_ERR_INVALID_ARG. */
qe_status qe_set_kernel_timing(qe_ctx *ctx, int32_t enable);
qe_status qe_get_kernel_timing(qe_ctx *ctx, int32_t kernel_class, double *total_ms_host, int64_t *launches_host);

const char *qe_status_str(qe_status s);

#ifdef __cplusplus
}
#endif
#endif /* QE_H */
