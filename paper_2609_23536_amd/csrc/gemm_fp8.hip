// FP8 GEMM for the three products of the split linear (gfx950 MFMA).
//
// §3.2 of the paper: F computes Y = X W^T, dI computes dX = dY W, and the
// deferred dW computes dW = dY^T X, each on FP8-quantized operands.  With the
// quantizer writing every operand both row-wise and transposed, all three are
// the same "TN" product with both operands contiguous along the reduction:
//     D[i][j] = 2^(ea + eb) * sum_r A[i][r] B[j][r]
// where 2^ea, 2^eb are the operands' scale inverses (powers of two, so the
// rescale is one exact ldexp).  The epilogue stores D (FP32 or BF16), or adds
// it to an FP32 destination in place: the direct placement of dW into its
// slice of the flat main-gradient buffer (§3.4), with no staging copy.
//
// Kernel: BM x BN x 128 macro-tile per workgroup, 64-wide waves on a WM x WN
// grid, each wave owning a (BM/WM) x (BN/WN) sub-tile accumulated with
// v_mfma_f32_16x16x128_f8f6f4 (operand formats chosen per call: E4M3 or
// E5M2).  K tiles are staged through LDS, double-buffered, loaded with
// 16-byte global loads into registers one tile ahead of the MFMA work.  LDS
// rows are 128 bytes; their 16-byte chunks are XOR-swizzled by (row/2) mod 8
// so the 16 rows read by one fragment load hit all 64 banks once.
//
// MFMA operand order: the B fragment is passed as source A and the A fragment
// as source B, so each lane ends up holding four consecutive output columns of
// one output row and the epilogue stores 16 bytes per lane.  Within a lane the
// 32 reduction bytes of a fragment come from the same positions for A and B,
// so any fixed assignment of reduction indices to MFMA slots gives the same
// dot products.
//
// Determinism: no atomics and no split reduction; the same inputs produce the
// same bits, which the split-vs-full-backward check relies on.
#include "kernels.h"

namespace qe {
namespace {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v4f __attribute__((ext_vector_type(4)));

constexpr int BK = 128;
constexpr int kGroupM = 8;

__device__ __forceinline__ uint32_t lds_off(int row, int chunk) {
  return uint32_t(row) * BK + (uint32_t((chunk ^ (row >> 1)) & 7) << 4);
}

__device__ __forceinline__ uint4 mask_tail(uint4 v, int64_t valid) {
  // keep bytes [0, valid), zero the rest (valid in [0, 16])
  if (valid >= 16) return v;
  uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int64_t lo = 4 * q;
    if (valid <= lo)
      w[q] = 0u;
    else if (valid < lo + 4)
      w[q] &= (1u << (8 * (valid - lo))) - 1u;
  }
  return make_uint4(w[0], w[1], w[2], w[3]);
}

__device__ __forceinline__ uint32_t f32_to_bf16_bits(float f) {
  const uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (u >> 16) | 0x40u;
  return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
}

__device__ __forceinline__ int pow2_exponent(const float *p) { return int((__float_as_uint(*p) >> 23) & 0xffu) - 127; }

// Workgroups are dealt to the 8 XCDs round-robin; renumber so that each XCD
// gets a contiguous range of tiles (shared A rows / B columns stay in one L2).
__device__ __forceinline__ int xcd_remap(int wg, int total) {
  const int per = total / 8, rem = total % 8;
  const int xcd = wg % 8, idx = wg / 8;
  return xcd < rem ? xcd * (per + 1) + idx : rem * (per + 1) + (xcd - rem) * per + idx;
}

template <int BM, int BN, int WM, int WN, int FA, int FB, int OUT>
__global__ __launch_bounds__(WM *WN * 64) void gemm_tn_kernel(GemmParams g, int tiles_m, int tiles_n, int vec_ok) {
  constexpr int NT = WM * WN * 64;
  constexpr int TM = BM / WM, TN = BN / WN;
  constexpr int FI = TM / 16, FJ = TN / 16;
  constexpr int ACH = BM * (BK / 16) / NT;
  constexpr int BCH = BN * (BK / 16) / NT;
  static_assert(ACH * NT == BM * (BK / 16) && BCH * NT == BN * (BK / 16), "tile / thread mismatch");

  __shared__ __attribute__((aligned(16))) uint8_t sA[2][BM * BK];
  __shared__ __attribute__((aligned(16))) uint8_t sB[2][BN * BK];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;

  // tile coordinates: XCD-contiguous, then grouped along M
  const int pid = xcd_remap(blockIdx.x, tiles_m * tiles_n);
  const int in_group = kGroupM * tiles_n;
  const int group = pid / in_group;
  const int first_m = group * kGroupM;
  const int gsize = min(tiles_m - first_m, kGroupM);
  const int tm = first_m + (pid % in_group) % gsize;
  const int tn = (pid % in_group) / gsize;
  const int64_t m0 = int64_t(tm) * BM, n0 = int64_t(tn) * BN;

  const int64_t M = g.m, N = g.n, K = g.k;
  const uint8_t *__restrict__ A = g.a;
  const uint8_t *__restrict__ B = g.b;
  const bool mfull = m0 + BM <= M, nfull = n0 + BN <= N;
  const int KT = int((K + BK - 1) / BK);

  v4f acc[FI][FJ];
#pragma unroll
  for (int i = 0; i < FI; ++i)
#pragma unroll
    for (int j = 0; j < FJ; ++j) acc[i][j] = v4f{0.f, 0.f, 0.f, 0.f};

  uint4 ra[ACH], rb[BCH];

  auto gload = [&](int kt) {
    const int64_t k0 = int64_t(kt) * BK;
    const bool kfull = k0 + BK <= K;
#pragma unroll
    for (int c = 0; c < ACH; ++c) {
      const int q = c * NT + tid, row = q >> 3, ch = q & 7;
      const int64_t gr = m0 + row, gk = k0 + ch * 16;
      if ((mfull || gr < M) && (kfull || gk < K)) {
        uint4 v = *reinterpret_cast<const uint4 *>(A + gr * g.lda + gk);
        ra[c] = kfull ? v : mask_tail(v, K - gk);
      } else {
        ra[c] = make_uint4(0u, 0u, 0u, 0u);
      }
    }
#pragma unroll
    for (int c = 0; c < BCH; ++c) {
      const int q = c * NT + tid, row = q >> 3, ch = q & 7;
      const int64_t gr = n0 + row, gk = k0 + ch * 16;
      if ((nfull || gr < N) && (kfull || gk < K)) {
        uint4 v = *reinterpret_cast<const uint4 *>(B + gr * g.ldb + gk);
        rb[c] = kfull ? v : mask_tail(v, K - gk);
      } else {
        rb[c] = make_uint4(0u, 0u, 0u, 0u);
      }
    }
  };

  auto sstore = [&](int buf) {
#pragma unroll
    for (int c = 0; c < ACH; ++c) {
      const int q = c * NT + tid, row = q >> 3, ch = q & 7;
      *reinterpret_cast<uint4 *>(&sA[buf][lds_off(row, ch)]) = ra[c];
    }
#pragma unroll
    for (int c = 0; c < BCH; ++c) {
      const int q = c * NT + tid, row = q >> 3, ch = q & 7;
      *reinterpret_cast<uint4 *>(&sB[buf][lds_off(row, ch)]) = rb[c];
    }
  };

  auto frag = [&](const uint8_t *base, int row) -> v8i {
    const int gq = lane >> 4;
    const uint4 lo = *reinterpret_cast<const uint4 *>(base + lds_off(row, 2 * gq));
    const uint4 hi = *reinterpret_cast<const uint4 *>(base + lds_off(row, 2 * gq + 1));
    return v8i{int(lo.x), int(lo.y), int(lo.z), int(lo.w), int(hi.x), int(hi.y), int(hi.z), int(hi.w)};
  };

  auto compute = [&](int buf) {
    v8i bfr[FJ];
#pragma unroll
    for (int j = 0; j < FJ; ++j) bfr[j] = frag(sB[buf], wn * TN + j * 16 + (lane & 15));
#pragma unroll
    for (int i = 0; i < FI; ++i) {
      const v8i afr = frag(sA[buf], wm * TM + i * 16 + (lane & 15));
#pragma unroll
      for (int j = 0; j < FJ; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(bfr[j], afr, acc[i][j], FB, FA, 0, 0, 0, 0);
    }
  };

  if (KT > 0) {
    gload(0);
    sstore(0);
    __syncthreads();
    for (int kt = 0; kt < KT; ++kt) {
      if (kt + 1 < KT) gload(kt + 1);
      compute(kt & 1);
      if (kt + 1 < KT) sstore((kt + 1) & 1);
      __syncthreads();
    }
  }

  // epilogue: lane holds rows (lane & 15), columns 4*(lane >> 4) .. +3 of each 16x16 block
  const int e = pow2_exponent(g.a_scale_inv) + pow2_exponent(g.b_scale_inv);
#pragma unroll
  for (int i = 0; i < FI; ++i) {
    const int64_t row = m0 + wm * TM + i * 16 + (lane & 15);
    if (!(mfull || row < M)) continue;
#pragma unroll
    for (int j = 0; j < FJ; ++j) {
      const int64_t col = n0 + wn * TN + j * 16 + 4 * (lane >> 4);
      float v[4];
#pragma unroll
      for (int t = 0; t < 4; ++t) v[t] = __builtin_ldexpf(acc[i][j][t], e);
      if (vec_ok && (nfull || col + 4 <= N)) {
        if constexpr (OUT == 0) {
          *reinterpret_cast<float4 *>(static_cast<float *>(g.c) + row * g.ldc + col) = make_float4(v[0], v[1], v[2], v[3]);
        } else if constexpr (OUT == 1) {
          const uint32_t lo = f32_to_bf16_bits(v[0]) | (f32_to_bf16_bits(v[1]) << 16);
          const uint32_t hi = f32_to_bf16_bits(v[2]) | (f32_to_bf16_bits(v[3]) << 16);
          *reinterpret_cast<uint2 *>(static_cast<uint16_t *>(g.c) + row * g.ldc + col) = make_uint2(lo, hi);
        } else {
          float4 *dst = reinterpret_cast<float4 *>(static_cast<float *>(g.c) + row * g.ldc + col);
          const float4 o = *dst;
          *dst = make_float4(o.x + v[0], o.y + v[1], o.z + v[2], o.w + v[3]);
        }
      } else {
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          if (col + t >= N) break;
          if constexpr (OUT == 0) {
            static_cast<float *>(g.c)[row * g.ldc + col + t] = v[t];
          } else if constexpr (OUT == 1) {
            static_cast<uint16_t *>(g.c)[row * g.ldc + col + t] = uint16_t(f32_to_bf16_bits(v[t]));
          } else {
            float *dst = static_cast<float *>(g.c) + row * g.ldc + col + t;
            *dst = *dst + v[t];
          }
        }
      }
    }
  }
}

template <int BM, int BN, int WM, int WN, int FA, int FB>
hipError_t launch_out(const GemmParams &g, hipStream_t s) {
  const int tiles_m = int((g.m + BM - 1) / BM), tiles_n = int((g.n + BN - 1) / BN);
  const uintptr_t cp = reinterpret_cast<uintptr_t>(g.c);
  const int vec_ok = (g.out == 1) ? (g.ldc % 4 == 0 && cp % 8 == 0) : (g.ldc % 4 == 0 && cp % 16 == 0);
  const dim3 grid(unsigned(tiles_m) * unsigned(tiles_n)), block(WM * WN * 64);
  switch (g.out) {
    case 0: hipLaunchKernelGGL((gemm_tn_kernel<BM, BN, WM, WN, FA, FB, 0>), grid, block, 0, s, g, tiles_m, tiles_n, vec_ok); break;
    case 1: hipLaunchKernelGGL((gemm_tn_kernel<BM, BN, WM, WN, FA, FB, 1>), grid, block, 0, s, g, tiles_m, tiles_n, vec_ok); break;
    default: hipLaunchKernelGGL((gemm_tn_kernel<BM, BN, WM, WN, FA, FB, 2>), grid, block, 0, s, g, tiles_m, tiles_n, vec_ok); break;
  }
  return hipGetLastError();
}

template <int BM, int BN, int WM, int WN>
hipError_t launch_fmts(const GemmParams &g, hipStream_t s) {
  if (g.fmt_a == 0 && g.fmt_b == 0) return launch_out<BM, BN, WM, WN, 0, 0>(g, s);
  if (g.fmt_a == 1 && g.fmt_b == 0) return launch_out<BM, BN, WM, WN, 1, 0>(g, s);
  if (g.fmt_a == 0 && g.fmt_b == 1) return launch_out<BM, BN, WM, WN, 0, 1>(g, s);
  return launch_out<BM, BN, WM, WN, 1, 1>(g, s);
}

}  // namespace

hipError_t launch_gemm(const GemmParams &g, hipStream_t s) {
  if (g.m <= 0 || g.n <= 0) return hipSuccess;
  return launch_fmts<256, 256, 2, 2>(g, s);
}

}  // namespace qe
