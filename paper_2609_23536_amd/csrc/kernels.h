// Internal launch interface of the gfx950 kernels (not part of the C ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace qe {

constexpr int kMaxMetas = 8;
constexpr int kMaxHistory = 8192;

struct MetaRef {
  float *hist;
  float *scale;
  float *scale_inv;
  int32_t history_len;
  int32_t margin;
  int32_t fmt;
  int32_t pad;
};

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
  float *amax_slot;  // history[0] of the role
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

enum KernelClass { KC_QUANT = 0, KC_UPDATE = 1, KC_GEMM = 2, KC_COPY = 3, KC_COUNT = 4 };

hipError_t launch_scale_update(const UpdateParams &p, hipStream_t s);
hipError_t launch_quantize(const QuantParams &p, hipStream_t s);
hipError_t launch_gemm(const GemmParams &p, hipStream_t s);
hipError_t launch_grad_copy(const GradCopyParams &p, hipStream_t s);

}  // namespace qe
