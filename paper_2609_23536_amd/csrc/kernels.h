// Internal launch interface of the gfx950 kernels (not part of the C ABI).
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <string.h>

#include <vector>

namespace qe {

// One kernel launch: function, launch shape and argument bytes.  The launch
// functions below go through klaunch(), which either launches the kernel on a
// stream or, while a recording list is installed on the calling thread,
// appends the launch to it without touching the device.  The executor records
// an action's launches to compare them with the kernel nodes of the graph it
// captured earlier and to rewrite the arguments of those nodes in place when
// only the arguments differ (hipGraphExecKernelNodeSetParams).
constexpr int kMaxKernelArgs = 8;
constexpr int kKernelArgBytes = 1024;
struct KernelRec {
  const void *func;
  dim3 grid, block;
  uint32_t shmem;
  uint32_t nargs;
  uint32_t used;  // bytes of blob in use
  uint16_t off[kMaxKernelArgs];
  alignas(16) uint8_t blob[kKernelArgBytes];
  KernelRec() { memset(static_cast<void *>(this), 0, sizeof(*this)); }
  // argument pointers for hipLaunchKernel / kernel-node parameters
  void argv(void **out) const {
    for (uint32_t i = 0; i < nargs; ++i) out[i] = const_cast<uint8_t *>(blob) + off[i];
  }
  bool same_shape(const KernelRec &o) const {
    return func == o.func && grid.x == o.grid.x && grid.y == o.grid.y && grid.z == o.grid.z &&
           block.x == o.block.x && block.y == o.block.y && block.z == o.block.z && shmem == o.shmem &&
           nargs == o.nargs && used == o.used && memcmp(off, o.off, sizeof(off)) == 0;
  }
  bool same_args(const KernelRec &o) const { return memcmp(blob, o.blob, used) == 0; }
};

// Installed by the executor on the calling thread while it records a plan.
extern thread_local std::vector<KernelRec> *tl_record;

// Kernel timing of one executor call, installed on the calling thread while
// the call launches: the launches carry the events in their own dispatch
// (hipExtLaunchKernel), so `start` takes the start of the first kernel and
// `stop` the end of each, i.e. of the last: the pair spans the call's kernels
// and nothing queued around them.
struct LaunchTiming {
  hipEvent_t start, stop;
  bool started;
};
extern thread_local LaunchTiming *tl_timing;

template <typename T>
inline void pack_arg(KernelRec &r, const T &v) {
  static_assert(sizeof(T) <= 512, "kernel argument too large");
  uint32_t o = (r.used + uint32_t(alignof(T)) - 1) & ~(uint32_t(alignof(T)) - 1);
  memcpy(r.blob + o, &v, sizeof(T));
  r.off[r.nargs++] = uint16_t(o);
  r.used = o + uint32_t(sizeof(T));
}

template <typename... P, typename... A>
hipError_t klaunch(void (*f)(P...), dim3 grid, dim3 block, size_t shmem, hipStream_t s, const A &...a) {
  static_assert(sizeof...(P) == sizeof...(A) && sizeof...(P) <= kMaxKernelArgs, "kernel arguments");
  KernelRec r;
  r.func = reinterpret_cast<const void *>(f);
  r.grid = grid;
  r.block = block;
  r.shmem = uint32_t(shmem);
  (pack_arg<P>(r, P(a)), ...);
  if (tl_record != nullptr) {
    tl_record->push_back(r);
    return hipSuccess;
  }
  void *argv[kMaxKernelArgs];
  r.argv(argv);
  if (tl_timing != nullptr) {
    hipEvent_t first = tl_timing->started ? nullptr : tl_timing->start;
    tl_timing->started = true;
    return hipExtLaunchKernel(r.func, grid, block, argv, shmem, s, first, tl_timing->stop, 0);
  }
  return hipLaunchKernel(r.func, grid, block, argv, shmem, s);
}

constexpr int kMaxMetas = 8;
constexpr int kMaxHistory = 8192;
constexpr int kAmaxLines = 64;   // amax accumulator: lines per role
constexpr int kAmaxStride = 64;  // floats between lines (256 bytes)

struct MetaRef {
  float *hist;
  float *scale;
  float *scale_inv;
  int32_t history_len;
  int32_t margin;
  int32_t fmt;
  int32_t pad;
  float *accum;  // amax accumulator or null
};

// Fold a workgroup's max |x| (a float32 bit pattern, NaN above inf) into the
// role's amax slot: line (workgroup % kAmaxLines) of the accumulator when
// there is one, else the single float.  Called by one lane.
__device__ __forceinline__ void fold_amax(float *accum, float *slot, uint32_t a) {
  if (a == 0u) return;
  if (accum != nullptr)
    atomicMax(reinterpret_cast<unsigned int *>(accum + (blockIdx.x % kAmaxLines) * kAmaxStride), a);
  else if (slot != nullptr)
    atomicMax(reinterpret_cast<unsigned int *>(slot), a);
}

// Delayed scale update of n roles in one launch (one workgroup per role).
struct UpdateParams {
  MetaRef m[kMaxMetas];
  int32_t n;
  int32_t pad;
  long long *token;  // incremented once per launch when non-null
};

// Cast (+transpose) + amax of one [rows, cols] tensor.
struct QuantParams {
  const void *in;
  int32_t in_bf16;  // 0: float32, 1: bfloat16 bits
  int32_t fmt;      // 0: E4M3, 1: E5M2
  int64_t rows, cols;
  const float *scale;
  const float *scale_inv;
  float *amax_slot;   // history[0] of the role; null (with amax_accum null): nothing recorded
  float *amax_accum;  // the role's amax accumulator, used instead of amax_slot when set
  uint8_t *q_row;
  int64_t ld_row;
  uint8_t *q_col;
  int64_t ld_col;
  float *snapshot;
};

// D = 2^(ea+eb) * sum_r A[i][r] B[j][r];  out = D (INIT) or out + D (ACCUM).
struct GemmParams {
  const uint8_t *a;
  const uint8_t *b;
  int64_t lda, ldb;
  int64_t m, n, k;
  const float *a_scale_inv;
  const float *b_scale_inv;
  void *c;
  int64_t ldc;
  int32_t fmt_a, fmt_b;
  int32_t out;  // 0: f32 store, 1: bf16 store, 2: f32 accumulate
  int32_t pad;
};

// dst[n * ld + k] (=, or +=) src[n * k + k'] for the copied-gradient path.
struct GradCopyParams {
  const float *src;  // [n, k] dense
  float *dst;        // [n, ld] view
  int64_t n, k, ld;
  int32_t accumulate;
  int32_t pad;
};

// *amax = max(*amax, max |in|) over numel contiguous elements (current scaling).
// The tensor is split into `head` single elements before the first 16-byte
// boundary, nvec 16-byte vectors from in + body_offset bytes, and `tail`
// single elements from element tail_start (built by amax_params).
struct AmaxParams {
  const void *in;
  float *amax;   // single float slot (used when accum is null)
  float *accum;  // amax accumulator
  int64_t body_offset, nvec, tail_start;
  int32_t head, tail;
  int32_t in_bf16;
  int32_t pad;
};

enum KernelClass { KC_QUANT = 0, KC_UPDATE = 1, KC_GEMM = 2, KC_COPY = 3, KC_AMAX = 4, KC_COUNT = 5 };

hipError_t launch_scale_update(const UpdateParams &p, hipStream_t s);
hipError_t launch_quantize(const QuantParams &p, hipStream_t s);
// Two independent casts with the same input dtype and FP8 format in one launch.
hipError_t launch_quantize_pair(const QuantParams &a, const QuantParams &b, hipStream_t s);
// `fused`, if non-null, is a delayed scale update (n >= 1 roles) run in extra
// workgroups of the same launch (or in a launch of its own right after it when
// the GEMM is empty or uses the 8-wave kernel); the GEMM must not read the
// live scales it writes.
hipError_t launch_gemm(const GemmParams &p, hipStream_t s, const UpdateParams *fused = nullptr);
// 0: tile shape from the cost model; 1..4: force 256x256, 256x192, 192x256, 256x128
void set_gemm_tile_override(int tile);
hipError_t launch_grad_copy(const GradCopyParams &p, hipStream_t s);
hipError_t launch_amax(const AmaxParams &p, hipStream_t s);
// p[0..n) = 0 with a kernel (no memset node when captured into a graph)
hipError_t launch_fill_zero(float *p, int64_t n, hipStream_t s);
AmaxParams amax_params(const void *in, bool bf16, int64_t numel, float *amax, float *accum);

}  // namespace qe
