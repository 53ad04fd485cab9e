// Copied-gradient placement (the ablation baseline of direct placement).
//
// §3.4 of the paper contrasts direct placement of dW into stable arena views
// with the conservative path, which materialises the gradient in a buffer of
// its own and copies it into the destination afterwards.  This kernel is that
// copy: dst[n * ld + k] = src[n * K + k] (INIT) or dst[...] += src[...]
// (ACCUM, one FP32 add, the same operation the GEMM epilogue performs when it
// places directly, so both paths give identical bits).  HBM-bound: 8 bytes
// per element (12 for ACCUM).  One 256-lane workgroup per 4 rows x 1024
// columns; 16-byte accesses when rows are 16-byte aligned.
#include "kernels.h"

namespace qe {
namespace {

constexpr int kThreads = 256;
constexpr int kCols = 1024;  // columns per workgroup (4 floats per lane)
constexpr int kRows = 4;

template <bool ACCUM, bool VEC>
__global__ __launch_bounds__(kThreads) void grad_copy_kernel(GradCopyParams p, int64_t col_blocks) {
  const int64_t b = blockIdx.x;
  const int64_t r0 = (b / col_blocks) * kRows;
  const int64_t c0 = (b % col_blocks) * kCols + int64_t(threadIdx.x) * 4;
#pragma unroll
  for (int r = 0; r < kRows; ++r) {
    const int64_t row = r0 + r;
    if (row >= p.n) break;
    const float *s = p.src + row * p.k;
    float *d = p.dst + row * p.ld;
    if (VEC && c0 + 4 <= p.k) {
      const float4 v = *reinterpret_cast<const float4 *>(s + c0);
      float4 *dp = reinterpret_cast<float4 *>(d + c0);
      if constexpr (ACCUM) {
        const float4 o = *dp;
        *dp = make_float4(o.x + v.x, o.y + v.y, o.z + v.z, o.w + v.w);
      } else {
        *dp = v;
      }
    } else {
      for (int t = 0; t < 4; ++t) {
        const int64_t c = c0 + t;
        if (c >= p.k) break;
        if constexpr (ACCUM)
          d[c] = d[c] + s[c];
        else
          d[c] = s[c];
      }
    }
  }
}

}  // namespace

hipError_t launch_grad_copy(const GradCopyParams &p, hipStream_t s) {
  if (p.n <= 0 || p.k <= 0) return hipSuccess;
  const int64_t col_blocks = (p.k + kCols - 1) / kCols;
  const int64_t blocks = ((p.n + kRows - 1) / kRows) * col_blocks;
  const bool vec = (p.k % 4 == 0) && (p.ld % 4 == 0) && (reinterpret_cast<uintptr_t>(p.src) % 16 == 0) &&
                   (reinterpret_cast<uintptr_t>(p.dst) % 16 == 0);
  const dim3 grid(static_cast<unsigned>(blocks)), block(kThreads);
  if (p.accumulate)
    return vec ? klaunch(grad_copy_kernel<true, true>, grid, block, 0, s, p, col_blocks)
               : klaunch(grad_copy_kernel<true, false>, grid, block, 0, s, p, col_blocks);
  return vec ? klaunch(grad_copy_kernel<false, true>, grid, block, 0, s, p, col_blocks)
             : klaunch(grad_copy_kernel<false, false>, grid, block, 0, s, p, col_blocks);
}

}  // namespace qe
