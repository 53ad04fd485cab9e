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

constexpr int kCUs = 256;  // MI355X compute units; one 128 KB-LDS workgroup each

__device__ __forceinline__ uint32_t lds_off(int row, int chunk) {
  return uint32_t(row) * BK + (uint32_t((chunk ^ (row >> 1)) & 7) << 4);
}

__device__ __forceinline__ uint4 mask_tail(uint4 v, int64_t valid) {
  // keep bytes [0, valid), zero the rest; branch-free
  uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int64_t nb = valid - 4 * q;  // bytes of this dword to keep
    const int k = nb <= 0 ? 0 : (nb >= 4 ? 4 : int(nb));
    w[q] &= uint32_t((uint64_t(1) << (8 * k)) - 1u);
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
  const int KT = int(K / BK);              // full K tiles
  const int64_t ktail = K - int64_t(KT) * BK;
  const int T = KT + (ktail > 0 ? 1 : 0);  // K iterations

  // Per-thread 16-byte chunks of the A and B tiles, as 32-bit byte offsets
  // from the operand base (the host keeps every operand below 2 GiB).  Rows
  // past M / N are clamped to the last row: they feed accumulators that are
  // never stored.  Chunk c of a thread sits RS rows below chunk 0 and, the
  // swizzle depending only on row / 2 mod 8, RS * BK bytes further in LDS.
  constexpr int RS = NT / 8;
  const int r0 = tid >> 3, ch0 = tid & 7;
  uint32_t oa[ACH], ob[BCH];
#pragma unroll
  for (int c = 0; c < ACH; ++c) oa[c] = uint32_t(min(m0 + c * RS + r0, M - 1) * g.lda) + ch0 * 16;
#pragma unroll
  for (int c = 0; c < BCH; ++c) ob[c] = uint32_t(min(n0 + c * RS + r0, N - 1) * g.ldb) + ch0 * 16;
  const uint32_t l0 = lds_off(r0, ch0);

  v4f acc[FI][FJ];
#pragma unroll
  for (int i = 0; i < FI; ++i)
#pragma unroll
    for (int j = 0; j < FJ; ++j) acc[i][j] = v4f{0.f, 0.f, 0.f, 0.f};

  uint4 ra[ACH], rb[BCH];
  const uint8_t *__restrict__ A = g.a;
  const uint8_t *__restrict__ B = g.b;

  // full K tile: no bounds checks at all
  auto gload = [&](int kt) {
    const uint32_t k0 = uint32_t(kt) * BK;
#pragma unroll
    for (int c = 0; c < ACH; ++c) ra[c] = *reinterpret_cast<const uint4 *>(A + (oa[c] + k0));
#pragma unroll
    for (int c = 0; c < BCH; ++c) rb[c] = *reinterpret_cast<const uint4 *>(B + (ob[c] + k0));
  };
  // the last, partial K tile: bytes at or past K are zero
  auto gload_tail = [&]() {
    const uint32_t k0 = uint32_t(KT) * BK;
    const int64_t gk = int64_t(k0) + ch0 * 16;
#pragma unroll
    for (int c = 0; c < ACH; ++c)
      ra[c] = gk < K ? mask_tail(*reinterpret_cast<const uint4 *>(A + (oa[c] + k0)), K - gk) : make_uint4(0u, 0u, 0u, 0u);
#pragma unroll
    for (int c = 0; c < BCH; ++c)
      rb[c] = gk < K ? mask_tail(*reinterpret_cast<const uint4 *>(B + (ob[c] + k0)), K - gk) : make_uint4(0u, 0u, 0u, 0u);
  };
  auto load = [&](int t) {
    if (t < KT)
      gload(t);
    else
      gload_tail();
  };

  auto sstore = [&](int buf) {
#pragma unroll
    for (int c = 0; c < ACH; ++c) *reinterpret_cast<uint4 *>(&sA[buf][l0 + c * RS * BK]) = ra[c];
#pragma unroll
    for (int c = 0; c < BCH; ++c) *reinterpret_cast<uint4 *>(&sB[buf][l0 + c * RS * BK]) = rb[c];
  };

  // Fragment reads.  Lane l of a 16-row fragment reads row (l & 15) of it,
  // 16-byte chunks 2(l >> 4) and 2(l >> 4) + 1.  Fragment rows start at
  // multiples of 16, so the swizzle term (row >> 1) & 7 depends on l only and
  // fragment f of a wave sits exactly 16 * 128 * f bytes after fragment 0:
  // two per-lane base offsets (low / high chunk) serve every fragment.
  const int fr = lane & 15, fq = lane >> 4;
  const uint32_t f_lo = uint32_t(fr) * BK + (uint32_t((2 * fq) ^ (fr >> 1)) & 7) * 16;
  const uint32_t f_hi = uint32_t(fr) * BK + (uint32_t((2 * fq + 1) ^ (fr >> 1)) & 7) * 16;
  auto frag = [&](const uint8_t *base) -> v8i {
    const uint4 lo = *reinterpret_cast<const uint4 *>(base + f_lo);
    const uint4 hi = *reinterpret_cast<const uint4 *>(base + f_hi);
    return v8i{int(lo.x), int(lo.y), int(lo.z), int(lo.w), int(hi.x), int(hi.y), int(hi.z), int(hi.w)};
  };

  // A fragments are read one step ahead of the MFMAs that consume them, so the
  // LDS latency of fragment i+1 hides behind the FJ MFMAs of fragment i.
  auto compute = [&](int buf) {
    const uint8_t *a_s = &sA[buf][wm * TM * BK];
    const uint8_t *b_s = &sB[buf][wn * TN * BK];
    v8i bfr[FJ];
#pragma unroll
    for (int j = 0; j < FJ; ++j) bfr[j] = frag(b_s + j * 16 * BK);
    v8i acur = frag(a_s);
#pragma unroll
    for (int i = 0; i < FI; ++i) {
      v8i anext = acur;
      if (i + 1 < FI) anext = frag(a_s + (i + 1) * 16 * BK);
#pragma unroll
      for (int j = 0; j < FJ; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(bfr[j], acur, acc[i][j], FB, FA, 0, 0, 0, 0);
      acur = anext;
    }
  };

  if (T > 0) {
    load(0);
    sstore(0);
    __syncthreads();
    for (int t = 0; t < T; ++t) {
      if (t + 1 < T) load(t + 1);
      compute(t & 1);
      if (t + 1 < T) sstore((t + 1) & 1);
      __syncthreads();
    }
  }

  // epilogue: lane holds rows (lane & 15), columns 4*(lane >> 4) .. +3 of each 16x16 block
  const int e = pow2_exponent(g.a_scale_inv) + pow2_exponent(g.b_scale_inv);
  const bool mfull = m0 + BM <= M, nfull = n0 + BN <= N;
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
  // The kernel addresses each operand with 32-bit offsets: split any operand
  // of 2 GiB or more into row blocks (independent GEMMs on disjoint outputs).
  constexpr int64_t kLim = int64_t(1) << 31;
  const int64_t cbytes = g.out == 1 ? 2 : 4;
  if (g.m * g.lda >= kLim) {
    const int64_t rows = (kLim - 1) / g.lda / 256 * 256;
    for (int64_t r = 0; r < g.m; r += rows) {
      GemmParams sub = g;
      sub.a = g.a + r * g.lda;
      sub.m = g.m - r < rows ? g.m - r : rows;
      sub.c = static_cast<char *>(g.c) + r * g.ldc * cbytes;
      const hipError_t e = launch_gemm(sub, s);
      if (e != hipSuccess) return e;
    }
    return hipSuccess;
  }
  if (g.n * g.ldb >= kLim) {
    const int64_t cols = (kLim - 1) / g.ldb / 256 * 256;
    for (int64_t c0 = 0; c0 < g.n; c0 += cols) {
      GemmParams sub = g;
      sub.b = g.b + c0 * g.ldb;
      sub.n = g.n - c0 < cols ? g.n - c0 : cols;
      sub.c = static_cast<char *>(g.c) + c0 * cbytes;
      const hipError_t e = launch_gemm(sub, s);
      if (e != hipSuccess) return e;
    }
    return hipSuccess;
  }
  // Tile choice by wave quantization: each CU runs one workgroup at a time, so
  // a grid costs ceil(tiles / CUs) rounds of one tile's time.  A 256 x 128
  // tile takes ~0.57 of a 256 x 256 tile (measured on MI355X; it is less
  // efficient per FLOP), so it wins when the 256 x 256 grid leaves the last
  // round mostly empty (e.g. N = 6144: 384 tiles, 1.5 rounds).
  const int64_t t256 = ((g.m + 255) / 256) * ((g.n + 255) / 256);
  const int64_t t128 = ((g.m + 255) / 256) * ((g.n + 127) / 128);
  const double c256 = double((t256 + kCUs - 1) / kCUs);
  const double c128 = 0.57 * double((t128 + kCUs - 1) / kCUs);
  if (c128 < c256) return launch_fmts<256, 128, 4, 2>(g, s);
  return launch_fmts<256, 256, 2, 4>(g, s);
}

}  // namespace qe
