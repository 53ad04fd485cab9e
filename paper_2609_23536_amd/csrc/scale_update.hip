// Delayed scale update from a rolling amax history (gfx950): one workgroup
// per role, the history staged in LDS so the rotation is a plain read-all /
// barrier / write-all.  Latency-bound (a few KB).  The update itself is
// scale_update_role (scale_update.h), which a GEMM launch can also run in
// extra workgroups of its own grid.
#include "scale_update.h"

namespace qe {
namespace {

__global__ __launch_bounds__(kUpdateThreads) void scale_update_kernel(UpdateParams p) {
  extern __shared__ uint32_t hist_sh[];
  __shared__ uint32_t red[kUpdateThreads / 64];
  scale_update_role(p.m[blockIdx.x], blockIdx.x == 0 ? p.token : nullptr, hist_sh, red);
}

}  // namespace

hipError_t launch_scale_update(const UpdateParams &p, hipStream_t s) {
  int hmax = 0;
  for (int i = 0; i < p.n; ++i) hmax = p.m[i].history_len > hmax ? p.m[i].history_len : hmax;
  size_t lds = size_t(hmax) * sizeof(uint32_t);
  return klaunch(scale_update_kernel, dim3(p.n), dim3(kUpdateThreads), lds, s, p);
}

}  // namespace qe
