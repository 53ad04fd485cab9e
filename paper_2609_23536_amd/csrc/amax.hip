// Amax pass of current (dynamic) scaling (gfx950).
//
// Current scaling sets a tensor's scale from the amax of that same tensor
// (the dynamic alternative to delayed scaling, §2.1 of the paper), so the
// amax must be known before the cast: this read-only pass folds max |x| over
// the whole tensor into the role's amax slot with a max (NaN propagates), the
// scale update then turns it into a scale, and the cast runs last.
//
// HBM-bound: reads 2 or 4 bytes per element and writes nothing but one atomic
// per workgroup (into one of the accumulator's lines, see fold_amax).  Each
// lane keeps several independent 16-byte loads in flight over a grid-stride
// loop; |x| is taken on the bit patterns (sign cleared),
// which order like the values with NaN above inf, so the max is an unsigned
// integer max and exact.  Elements before the first 16-byte boundary and after
// the last whole vector (at most 7 + 7) are read one by one by workgroup 0.
// A tensor that fits in the 256 MB memory-side cache is read with ordinary
// cached loads (16 per lane in flight), so that the cast that follows re-reads
// it from that cache; a larger one cannot stay there, and is streamed with
// non-temporal loads (4 per lane in flight, up to 64 workgroups per CU), which
// read faster on MI355X (measured on a cold 940 MB bf16 tensor: 6.2 TB/s
// against 3.8 TB/s).  That
// cache is write-back:
// when earlier kernels left it dirty, this pass also pays for their write-back
// to HBM (measured: a cold 235 MB read takes 47 us clean and 100 us right
// after a 470 MB write), so its own bandwidth figure understates the bytes
// HBM moves while it runs.
#include "kernels.h"

namespace qe {
namespace {

constexpr int kThreads = 256;
constexpr int kUnroll = 16;            // 256 bytes per lane in flight per batch (cached loads)
constexpr int kUnrollNT = 4;           // 64 bytes (non-temporal loads)
constexpr int64_t kNTBytes = int64_t(256) << 20;  // the memory-side cache of MI355X
constexpr int64_t kMaxBlocks = 4096;     // cached loads: 16 workgroups per CU
constexpr int64_t kMaxBlocksNT = 16384;  // non-temporal loads: 64 workgroups per CU

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint32_t umax(uint32_t a, uint32_t b) { return a > b ? a : b; }

// |x| of the one or two values in a 32-bit word, as float32 bit patterns.
template <bool BF16>
__device__ __forceinline__ uint32_t word_abs(uint32_t w) {
  if constexpr (BF16) return umax((w << 16) & 0x7fff0000u, w & 0x7fff0000u);
  return w & 0x7fffffffu;
}

template <bool BF16, bool NT>
__global__ __launch_bounds__(kThreads) void amax_kernel(AmaxParams p) {
  constexpr int kU = NT ? kUnrollNT : kUnroll;
  const int tid = threadIdx.x;
  const u32x4 *v = reinterpret_cast<const u32x4 *>(static_cast<const char *>(p.in) + p.body_offset);
  const int64_t stride = int64_t(gridDim.x) * kThreads;
  int64_t i = int64_t(blockIdx.x) * kThreads + tid;
  uint32_t m = 0;
  for (; i + (kU - 1) * stride < p.nvec; i += kU * stride) {
    u32x4 r[kU];
#pragma unroll
    for (int u = 0; u < kU; ++u) r[u] = NT ? __builtin_nontemporal_load(v + i + u * stride) : v[i + u * stride];
#pragma unroll
    for (int u = 0; u < kU; ++u)
      m = umax(m, umax(umax(word_abs<BF16>(r[u].x), word_abs<BF16>(r[u].y)),
                       umax(word_abs<BF16>(r[u].z), word_abs<BF16>(r[u].w))));
  }
  for (; i < p.nvec; i += stride) {
    const u32x4 r = NT ? __builtin_nontemporal_load(v + i) : v[i];
    m = umax(m, umax(umax(word_abs<BF16>(r.x), word_abs<BF16>(r.y)), umax(word_abs<BF16>(r.z), word_abs<BF16>(r.w))));
  }
  if (blockIdx.x == 0 && tid < p.head + p.tail) {
    const int64_t e = tid < p.head ? int64_t(tid) : p.tail_start + (tid - p.head);
    if constexpr (BF16) {
      m = umax(m, (uint32_t(static_cast<const uint16_t *>(p.in)[e]) << 16) & 0x7fff0000u);
    } else {
      m = umax(m, static_cast<const uint32_t *>(p.in)[e] & 0x7fffffffu);
    }
  }

  __shared__ uint32_t red[kThreads / 64];
  for (int off = 32; off > 0; off >>= 1) m = umax(m, uint32_t(__shfl_xor(int(m), off, 64)));
  if ((tid & 63) == 0) red[tid >> 6] = m;
  __syncthreads();
  if (tid == 0) {
    uint32_t a = red[0];
#pragma unroll
    for (int w = 1; w < kThreads / 64; ++w) a = umax(a, red[w]);
    fold_amax(p.accum, p.amax, a);
  }
}

__global__ __launch_bounds__(kThreads) void fill_zero_kernel(float *p, int64_t n) {
  for (int64_t i = int64_t(blockIdx.x) * kThreads + threadIdx.x; i < n; i += int64_t(gridDim.x) * kThreads)
    p[i] = 0.0f;
}

}  // namespace

hipError_t launch_fill_zero(float *p, int64_t n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  int64_t blocks = (n + kThreads - 1) / kThreads;
  if (blocks > 1024) blocks = 1024;
  return klaunch(fill_zero_kernel, dim3(unsigned(blocks)), dim3(kThreads), 0, s, p, n);
}

hipError_t launch_amax(const AmaxParams &p, hipStream_t s) {
  if (p.nvec == 0 && p.head + p.tail == 0) return hipSuccess;  // empty tensor: amax 0, nothing to fold
  const bool nt = p.nvec * 16 > kNTBytes;
  const int64_t per = int64_t(kThreads) * (nt ? kUnrollNT : kUnroll);
  int64_t blocks = (p.nvec + per - 1) / per;
  if (blocks > (nt ? kMaxBlocksNT : kMaxBlocks)) blocks = nt ? kMaxBlocksNT : kMaxBlocks;
  if (blocks < 1) blocks = 1;
  const dim3 grid(static_cast<unsigned>(blocks)), block(kThreads);
  if (nt)
    return p.in_bf16 ? klaunch(amax_kernel<true, true>, grid, block, 0, s, p) : klaunch(amax_kernel<false, true>, grid, block, 0, s, p);
  return p.in_bf16 ? klaunch(amax_kernel<true, false>, grid, block, 0, s, p) : klaunch(amax_kernel<false, false>, grid, block, 0, s, p);
}

AmaxParams amax_params(const void *in, bool bf16, int64_t numel, float *amax, float *accum) {
  AmaxParams p;
  memset(&p, 0, sizeof(p));  // padding too: recorded launches are compared bytewise
  p.in = in;
  p.in_bf16 = bf16 ? 1 : 0;
  p.amax = amax;
  p.accum = accum;
  const int64_t es = bf16 ? 2 : 4;
  const uintptr_t addr = reinterpret_cast<uintptr_t>(in);
  int64_t head = int64_t((16 - addr % 16) % 16) / es;  // elements before the first 16-byte boundary
  if (head > numel) head = numel;
  const int64_t rest = numel - head;
  p.head = int32_t(head);
  p.body_offset = head * es;
  p.nvec = rest * es / 16;
  p.tail_start = head + p.nvec * (16 / es);
  p.tail = int32_t(numel - p.tail_start);
  return p;
}

}  // namespace qe
