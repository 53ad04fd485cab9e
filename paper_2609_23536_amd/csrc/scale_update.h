// Delayed scale update of one tensor role, as a device function: the body of
// scale_update_kernel, and of the extra workgroups a GEMM launch can carry
// (the update then runs beside the GEMM's tiles, which read only the
// scale_inv snapshots the cast wrote, never the live scale).
//
// The paper's delayed scaling (§2.1) derives each tensor role's scale from a
// moving window of past amaxes; §3.2 fixes that F updates the forward roles
// once and dI the gradient role once, and dW never.  Reading of the formula:
//   a = max(history)  (NaN propagates)
//   if a is finite and > 0:  e = floor(log2(fmax / a)) - margin, clamped to
//                            [-126, 126]; scale = 2^e; scale_inv = 2^-e
//   history rotates one place towards index 0 (index 0 -> H-1); index 0 = 0.
// floor(log2(fmax/a)) is evaluated exactly on the bit pattern of a: with
// a = m * 2^E, m in [1,2), and fmax = 1.75 * 2^Emax, it is Emax - E, minus one
// when m > 1.75.  A float log2 would round 7 - tiny up to 7.
#pragma once

#include "kernels.h"

namespace qe {

constexpr int kUpdateThreads = 256;

__device__ __forceinline__ uint32_t update_wave_max(uint32_t v) {
  for (int off = 32; off > 0; off >>= 1) {
    uint32_t o = __shfl_xor(v, off, 64);
    v = o > v ? o : v;
  }
  return v;
}

// One workgroup of kUpdateThreads lanes updates role m.  hist_sh: LDS for
// history_len words; red: LDS for kUpdateThreads / 64 words.  `token`, if
// non-null, is incremented by this workgroup (pass it to one workgroup only).
__device__ __forceinline__ void scale_update_role(const MetaRef &m, long long *token, uint32_t *hist_sh,
                                                  uint32_t *red) {
  const int H = m.history_len;
  const int tid = threadIdx.x;

  // amax values are >= +0 or a positive-signed NaN, so their bit patterns order
  // like the values, and every NaN pattern sorts above +inf.
  // The role's amax accumulator (if any) is folded into history[0] and cleared.
  // All global reads are issued before the first store (the accumulator's
  // clear), so they overlap instead of paying two memory latencies in a row.
  const bool has_acc = m.accum != nullptr && tid < kAmaxLines;
  uint32_t acc = has_acc ? __float_as_uint(m.accum[tid * kAmaxStride]) & 0x7fffffffu : 0u;
  constexpr int kPre = 4;  // history elements per lane read up front (H <= 1024)
  uint32_t pre[kPre];
#pragma unroll
  for (int k = 0; k < kPre; ++k) {
    const int i = tid + k * kUpdateThreads;
    pre[k] = i < H ? __float_as_uint(m.hist[i]) & 0x7fffffffu : 0u;
  }
  acc = update_wave_max(acc);  // wave 0 holds the accumulator's value, the other waves 0
  if (has_acc) m.accum[tid * kAmaxStride] = 0.0f;

  uint32_t mx = 0;
#pragma unroll
  for (int k = 0; k < kPre; ++k) {
    const int i = tid + k * kUpdateThreads;
    uint32_t b = pre[k];
    if (i == 0) b = b > acc ? b : acc;  // i == 0 only on lane 0 of wave 0
    if (i < H) hist_sh[i] = b;
    mx = b > mx ? b : mx;
  }
  for (int i = tid + kPre * kUpdateThreads; i < H; i += kUpdateThreads) {
    const uint32_t b = __float_as_uint(m.hist[i]) & 0x7fffffffu;
    hist_sh[i] = b;
    mx = b > mx ? b : mx;
  }
  mx = update_wave_max(mx);
  if ((tid & 63) == 0) red[tid >> 6] = mx;
  __syncthreads();

  if (tid == 0) {
    uint32_t a = red[0];
    for (int w = 1; w < kUpdateThreads / 64; ++w) a = red[w] > a ? red[w] : a;
    if (a != 0u && a < 0x7f800000u) {
      int E;
      bool above;  // mantissa m > 1.75
      if (a >= 0x00800000u) {
        E = int(a >> 23) - 127;
        above = (a & 0x007fffffu) > 0x00600000u;
      } else {  // subnormal: a = f * 2^-149
        int pbit = 31 - __clz(a);
        E = pbit - 149;
        above = (uint64_t(a) << 2) > (uint64_t(7) << pbit);
      }
      const int emax = m.fmt == 0 ? 8 : 15;
      int e = emax - E - (above ? 1 : 0) - m.margin;
      e = e < -126 ? -126 : (e > 126 ? 126 : e);
      *m.scale = __uint_as_float(uint32_t(e + 127) << 23);
      *m.scale_inv = __uint_as_float(uint32_t(127 - e) << 23);
    }
    // the effect token: an atomic add whose result is not used, so the lane
    // does not wait for the old value
    if (token != nullptr) __hip_atomic_fetch_add(token, 1ll, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  // Rotate: new[i] = old[i+1] (i < H-1), new[H-1] = old[0], then new[0] = 0.
  for (int i = tid; i < H; i += kUpdateThreads) {
    float v;
    if (i == 0)
      v = 0.0f;
    else
      v = __uint_as_float(i == H - 1 ? hist_sh[0] : hist_sh[i + 1]);
    m.hist[i] = v;
  }
}

}  // namespace qe
