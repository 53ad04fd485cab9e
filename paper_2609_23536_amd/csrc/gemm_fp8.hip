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
// Two kernels share the scheme below; both use v_mfma_f32_16x16x128_f8f6f4
// with the same assignment of reduction bytes to lanes, so every tile shape
// accumulates each output element in the same order and gives the same bits.
//  * gemm_tn_w4_kernel, 256 x 256 x 128 tiles (and 256 x 224, 256 x 192,
//    192 x 256): four waves (one per SIMD) on a 2 x 2 grid, each a 128 x 128 sub-tile of
//    8 x 8 MFMA blocks.  A K tile's 64 MFMAs run in two phases; every fragment
//    read or LDS-bound load is issued right after an MFMA, in a fixed order
//    (sched_barrier), so the MFMA pipe stays busy in the single wave, and the
//    LDS-bound loads are branch-free (two instructions each) because a single
//    wave issues at most one instruction per four cycles, eight per MFMA.
//    The K loop is rotated so that its back-edge sits at the stage barrier,
//    where all LDS reads have completed; the compiler can then wait for
//    fragment reads one by one instead of draining them at the loop head.
//    The epilogue goes through LDS so every store instruction writes whole
//    row runs (512-byte FP32 runs; BF16 values are rounded first and go as
//    256-byte runs).  Larger wave tiles mean less LDS traffic per FLOP than
//    eight waves.
//  * gemm_tn_kernel, 256 x 128 x 128 tiles: eight waves (two per SIMD) on a
//    4 x 2 grid; used when it quantizes better onto the compute units.
// Operand formats (E4M3 or E5M2) are chosen per call.  K tiles are
// double-buffered in LDS and filled by LDS-bound global loads
// (global_load_lds_dwordx4: no register staging, no LDS store instructions)
// issued a K tile ahead; each wave waits for its own loads and a barrier
// publishes the stage.  The 4-wave kernel splits a K tile's loads: the B part
// goes into a stage's B half as soon as every wave holds the B fragments of
// the tile that stage held (during phase A, a K step and a half before it is
// read), the A part in the first half of phase B; a second barrier per K step
// marks the B half free.  (Measured on MI355X: against all loads spread over
// phase B, the Llama-3-70B stage's GEMMs 4% faster, products whose operands
// stream from HBM up to 8%.)  LDS rows are 128 bytes; their 16-byte chunks are
// XOR-swizzled by (row/2) mod 8 so a fragment read hits the 64 banks evenly,
// and since fragments start on multiples of 16 rows, every fragment of a wave
// is one base address plus a constant.  The LDS-bound loads are inline
// assembly: the compiler's own form makes it wait for them before every LDS
// read, serialising the loads with the MFMA work.  Rows past M / N are
// clamped to the last row (their results are never stored), so only the last,
// partial K tile needs masking; it goes through registers.
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
#include "scale_update.h"

#include <atomic>

namespace qe {
namespace {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v2i __attribute__((ext_vector_type(2)));
typedef float v4f __attribute__((ext_vector_type(4)));

constexpr int BK = 128;
// Tiles are numbered down groups of kGroupM row tiles, column after column,
// and each XCD takes a contiguous range of that order, so a round's 32 tiles
// on one XCD are 4 row tiles x 8 column tiles sharing their operand slabs in
// its L2.  Measured on MI355X over the Llama-3-70B stage's twelve products:
// 4 rows 1.2% faster than 8 (two runs), 2 rows 1.8% slower, 16 rows 5%
// slower; the 8B stage's products are level between 4, 6 and 8.
constexpr int kGroupM = 4;


// Cache policy of the epilogue's output traffic (stores, and the destination
// reads of the accumulate mode): non-temporal.  The output is written once
// and not read again by this kernel, so keeping it out of the L2 leaves the L2
// to the operand rows and columns that later tiles of the grid re-read;
// measured on MI355X over the Llama-3-8B stage's twelve products: -3.7% time
// with FP32 / BF16 stores, -5% in accumulate mode, most on the seven-round
// shapes.
constexpr int kNT = 2;  // the buffer instructions' nt bit

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

// Two floats to two bf16 (round to nearest even, NaN stays a quiet NaN with
// its sign and top payload bits) with the gfx950 packed conversion; bit-equal
// to the integer form (u + 0x7fff + ((u >> 16) & 1)) >> 16 on every input,
// which was checked on MI355X over all exponents, boundaries, denormals and NaNs.
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t bf16x2_bits(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{lo, hi}, bf16x2_t));
}
__device__ __forceinline__ uint16_t bf16_bits(float f) { return uint16_t(bf16x2_bits(f, 0.0f)); }

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

  __shared__ __attribute__((aligned(16))) uint8_t smem[2 * (BM + BN) * BK];
  constexpr int NW = WM * WN;
  constexpr int STAGE = (BM + BN) * BK;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;

  const int pid = xcd_remap(blockIdx.x, tiles_m * tiles_n);
  const int in_group = kGroupM * tiles_n;
  const int group = pid / in_group;
  const int first_m = group * kGroupM;
  const int gsize = min(tiles_m - first_m, kGroupM);
  const int tm = first_m + (pid % in_group) % gsize;
  const int tn = (pid % in_group) / gsize;
  const int64_t m0 = int64_t(tm) * BM, n0 = int64_t(tn) * BN;

  const int64_t M = g.m, N = g.n, K = g.k;
  const int KT = int(K / BK);
  const int64_t ktail = K - int64_t(KT) * BK;
  const int T = KT + (ktail > 0 ? 1 : 0);

  // LDS-bound loads: each wave instruction fills one contiguous 1 KB block
  // (8 rows x 128 B), lane l writing bytes 16l..16l+15; lane l fetches the
  // global chunk that the swizzle puts at row 8b + l/8, physical chunk l % 8.
  const int lrow = lane >> 3;
  uint32_t oa[ACH], ob[BCH];
#pragma unroll
  for (int c = 0; c < ACH; ++c) {
    const int row = 8 * (wave + NW * c) + lrow;
    const int lch = (lane & 7) ^ ((row >> 1) & 7);
    oa[c] = uint32_t(min(m0 + row, M - 1) * g.lda) + lch * 16;
  }
#pragma unroll
  for (int c = 0; c < BCH; ++c) {
    const int row = 8 * (wave + NW * c) + lrow;
    const int lch = (lane & 7) ^ ((row >> 1) & 7);
    ob[c] = uint32_t(min(n0 + row, N - 1) * g.ldb) + lch * 16;
  }
  const uint32_t lds_base = uint32_t(reinterpret_cast<uintptr_t>(smem));
  const uint32_t wblk = __builtin_amdgcn_readfirstlane(lds_base + uint32_t(wave) * 1024u);

  v4f acc[FI][FJ];
#pragma unroll
  for (int i = 0; i < FI; ++i)
#pragma unroll
    for (int j = 0; j < FJ; ++j) acc[i][j] = v4f{0.f, 0.f, 0.f, 0.f};

  auto issue_full = [&](int kt, int buf) {
    const uint8_t *ga = g.a + int64_t(kt) * BK;
    const uint8_t *gb = g.b + int64_t(kt) * BK;
    const uint32_t sa = wblk + uint32_t(buf * STAGE);
    const uint32_t sb = sa + uint32_t(BM * BK);
#pragma unroll
    for (int c = 0; c < ACH; ++c)
      asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(oa[c]), "s"(ga),
                   "s"(sa + uint32_t(c * NW * 1024)) : "memory", "m0");
#pragma unroll
    for (int c = 0; c < BCH; ++c)
      asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(ob[c]), "s"(gb),
                   "s"(sb + uint32_t(c * NW * 1024)) : "memory", "m0");
  };
  auto issue_tail = [&](int buf) {
    uint8_t *dA = smem + buf * STAGE;
    uint8_t *dB = dA + BM * BK;
    const uint32_t k0 = uint32_t(KT) * BK;
#pragma unroll
    for (int c = 0; c < ACH; ++c) {
      const int row = 8 * (wave + NW * c) + lrow;
      const int64_t gk = int64_t(k0) + (((lane & 7) ^ ((row >> 1) & 7)) * 16);
      const uint4 v = gk < K ? mask_tail(*reinterpret_cast<const uint4 *>(g.a + (oa[c] + k0)), K - gk) : make_uint4(0u, 0u, 0u, 0u);
      *reinterpret_cast<uint4 *>(dA + (wave + NW * c) * 1024 + lane * 16) = v;
    }
#pragma unroll
    for (int c = 0; c < BCH; ++c) {
      const int row = 8 * (wave + NW * c) + lrow;
      const int64_t gk = int64_t(k0) + (((lane & 7) ^ ((row >> 1) & 7)) * 16);
      const uint4 v = gk < K ? mask_tail(*reinterpret_cast<const uint4 *>(g.b + (ob[c] + k0)), K - gk) : make_uint4(0u, 0u, 0u, 0u);
      *reinterpret_cast<uint4 *>(dB + (wave + NW * c) * 1024 + lane * 16) = v;
    }
  };
  auto issue = [&](int t, int buf) {
    if (t < KT)
      issue_full(t, buf);
    else
      issue_tail(buf);
  };

  const int fr = lane & 15, fq = lane >> 4;
  const uint32_t f_lo = uint32_t(fr) * BK + (uint32_t((2 * fq) ^ (fr >> 1)) & 7) * 16;
  const uint32_t f_hi = uint32_t(fr) * BK + (uint32_t((2 * fq + 1) ^ (fr >> 1)) & 7) * 16;
  auto frag = [&](const uint8_t *base) -> v8i {
    const uint4 lo = *reinterpret_cast<const uint4 *>(base + f_lo);
    const uint4 hi = *reinterpret_cast<const uint4 *>(base + f_hi);
    return v8i{int(lo.x), int(lo.y), int(lo.z), int(lo.w), int(hi.x), int(hi.y), int(hi.z), int(hi.w)};
  };

  auto compute = [&](int buf) {
    const uint8_t *a_s = smem + buf * STAGE + wm * TM * BK;
    const uint8_t *b_s = smem + buf * STAGE + BM * BK + wn * TN * BK;
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

  auto stage_sync = [&]() {
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
  };

  if (T > 0) {
    issue(0, 0);
    stage_sync();
    for (int t = 0; t < T; ++t) {
      if (t + 1 < T) issue(t + 1, (t + 1) & 1);
      compute(t & 1);
      stage_sync();
    }
  }

  // epilogue: lane holds rows (lane & 15), columns 4*(lane >> 4) .. +3 of each 16x16 block
  const int e = pow2_exponent(g.a_scale_inv) + pow2_exponent(g.b_scale_inv);
  const bool mfull = m0 + BM <= M, nfull = n0 + BN <= N;
  // Full tile, vector-aligned destination: buffer stores (and accumulate
  // loads) at a scalar block offset plus one fixed per-lane offset, with no
  // bounds checks; every offset stays below 2^31.  Edge tiles take the checked
  // path below.
  constexpr int ES = OUT == 1 ? 2 : 4;  // output element bytes
  if (vec_ok && mfull && nfull && g.ldc * ES * (BM + 1) < (int64_t(1) << 31)) {
    const int wu = __builtin_amdgcn_readfirstlane(wave);
    const int wmu = wu / WN, wnu = wu % WN;
    const __amdgpu_buffer_rsrc_t crs = __builtin_amdgcn_make_buffer_rsrc(
        static_cast<char *>(g.c) + (m0 * g.ldc + n0) * ES, short(0), 0x7fffffff, 0x00020000);
    const uint32_t voff = uint32_t((lane & 15) * g.ldc + 4 * (lane >> 4)) * uint32_t(ES);
    const int rstep = int(g.ldc) * ES;
#pragma unroll
    for (int i = 0; i < FI; ++i)
#pragma unroll
      for (int j = 0; j < FJ; ++j) {
        const int so = (wmu * TM + i * 16) * rstep + (wnu * TN + j * 16) * ES;
        float v[4];
#pragma unroll
        for (int t = 0; t < 4; ++t) v[t] = __builtin_ldexpf(acc[i][j][t], e);
        if constexpr (OUT == 0) {
          const v4i w = {__builtin_bit_cast(int, v[0]), __builtin_bit_cast(int, v[1]), __builtin_bit_cast(int, v[2]),
                         __builtin_bit_cast(int, v[3])};
          __builtin_amdgcn_raw_buffer_store_b128(w, crs, voff, so, kNT);
        } else if constexpr (OUT == 1) {
          const v2i w = {int(bf16x2_bits(v[0], v[1])), int(bf16x2_bits(v[2], v[3]))};
          __builtin_amdgcn_raw_buffer_store_b64(w, crs, voff, so, kNT);
        } else {
          const float4 o = __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(crs, voff, so, kNT));
          const float4 r = make_float4(o.x + v[0], o.y + v[1], o.z + v[2], o.w + v[3]);
          __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(v4i, r), crs, voff, so, kNT);
        }
      }
    return;
  }
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
          const uint32_t lo = bf16x2_bits(v[0], v[1]);
          const uint32_t hi = bf16x2_bits(v[2], v[3]);
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
            static_cast<uint16_t *>(g.c)[row * g.ldc + col + t] = bf16_bits(v[t]);
          } else {
            float *dst = static_cast<float *>(g.c) + row * g.ldc + col + t;
            *dst = *dst + v[t];
          }
        }
      }
    }
  }
}

// 256 x 256 x 128 tile (also 256 x 224, 256 x 192 and 192 x 256), four waves
// (one per SIMD) on a 2 x 2 grid, each wave a TM x TN sub-tile of 16 x 16 blocks of
// v_mfma_f32_16x16x128_f8f6f4, one MFMA per block per K tile.  (On random FP8
// operands this MFMA sustains about a third more throughput than the 32 x 32 x
// 64 one on MI355X, which draws more power per FLOP; with constant operands
// the two are equal.)
// A K tile's MFMAs run in two phases of I/2 block rows each:
//   phase A (block rows 0 .. I/2-1, column-major): uses A fragments
//     0 .. I/2-1 and every B fragment; reads A fragments I/2 .. I-1 of the
//     same tile; issues the B part of the LDS-bound loads of the tile two K
//     tiles ahead into this stage's B half;
//   phase B (block rows I/2 .. I-1, column-major): each B fragment's last use
//     is followed by the read of the next tile's B fragment into the same
//     registers, and the next tile's A fragments 0 .. I/2-1 are read too; the
//     A part of the loads of the tile after next is issued in its first half.
// So all of tile t is read by the end of its phase A, where the stage barrier
// sits: it frees tile t's A half for the A part of tile t+2 and publishes tile
// t+1.  A second barrier, after phase B, marks the B half of tile t+1's stage
// free once every wave holds tile t+1's B fragments, so phase A of tile t+1
// loads tile t+3's B part there: a K step and a half of latency budget for
// the B part, about a phase for the A part.  Fragment registers: I + J
// fragments of 8 VGPRs, no second set.  The K loop is rotated (phase B of tile t, then phase A of tile t+1)
// so its back-edge sits at the barrier, where every LDS read has completed;
// the waits for fragment reads inside an iteration can then be partial.
template <int FA, int FB, int OUT, int BM, int BN>
__global__ __launch_bounds__(256) void gemm_tn_w4_kernel(GemmParams g, int tiles_m, int tiles_n, int vec_ok,
                                                         UpdateParams upd) {
  static_assert((BM == 256 || BM == 192) && (BN == 256 || BN == 224 || BN == 192), "tile sizes");
  constexpr int NW = 4, TM = BM / 2, TN = BN / 2;
  constexpr int I = TM / 16, J = TN / 16;    // 16 x 16 MFMA blocks per wave sub-tile
  constexpr int IA = I / 2, IB = I - IA;     // block rows of phase A and phase B
  constexpr int QA = IA * J, QB = IB * J;    // MFMAs per phase
  constexpr int CHA = BM / 32, CHB = BN / 32;  // 16-byte LDS-bound loads per lane per K tile
  constexpr int ND = CHA + CHB;              // LDS-bound loads per K tile
  constexpr int STAGE = (BM + BN) * BK;
  constexpr int EP = TN + 4;                 // epilogue staging row, in floats (padded)
  static_assert(NW * 32 * EP * 4 <= 2 * STAGE, "epilogue staging fits in the stages");
  static_assert(CHA * NW * 1024 == BM * BK, "LDS-bound load d of a tile lands at stage + 4096 d");
  // two K stages, then one 1 KB block per wave that absorbs the loads issued
  // past the last full K tile (so the loop issues them unconditionally)
  __shared__ __attribute__((aligned(16))) uint8_t smem[2 * STAGE + NW * 1024];
  static_assert(sizeof(smem) >= (kMaxHistory + kUpdateThreads / 64) * 4, "history staging fits in the stages");

  // Workgroups past the tiles (dispatched last) run the delayed scale update
  // of the action's roles beside the tiles: the tiles read the scale_inv
  // snapshots, never the live scales this update writes.
  if (int(blockIdx.x) >= tiles_m * tiles_n) {
    const int r = int(blockIdx.x) - tiles_m * tiles_n;
    uint32_t *hs = reinterpret_cast<uint32_t *>(smem);
    scale_update_role(upd.m[r], r == 0 ? upd.token : nullptr, hs, hs + kMaxHistory);
    return;
  }

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;

  const int pid = xcd_remap(blockIdx.x, tiles_m * tiles_n);
  const int in_group = kGroupM * tiles_n;
  const int group = pid / in_group;
  const int first_m = group * kGroupM;
  const int gsize = min(tiles_m - first_m, kGroupM);
  const int tm = first_m + (pid % in_group) % gsize;
  const int tn = (pid % in_group) / gsize;
  const int64_t m0 = int64_t(tm) * BM, n0 = int64_t(tn) * BN;

  const int64_t M = g.m, N = g.n, K = g.k;
  const int KT = int(K / BK);
  const int64_t ktail = K - int64_t(KT) * BK;
  const int T = KT + (ktail > 0 ? 1 : 0);

  const int lrow = lane >> 3;
  uint32_t oa[CHA], ob[CHB];
#pragma unroll
  for (int c = 0; c < CHA; ++c) {
    const int row = 8 * (wave + NW * c) + lrow;
    const int lch = (lane & 7) ^ ((row >> 1) & 7);
    oa[c] = uint32_t(min(m0 + row, M - 1) * g.lda) + lch * 16;
  }
#pragma unroll
  for (int c = 0; c < CHB; ++c) {
    const int row = 8 * (wave + NW * c) + lrow;
    const int lch = (lane & 7) ^ ((row >> 1) & 7);
    ob[c] = uint32_t(min(n0 + row, N - 1) * g.ldb) + lch * 16;
  }
  const uint32_t lds_base = uint32_t(reinterpret_cast<uintptr_t>(smem));
  const uint32_t wblk = __builtin_amdgcn_readfirstlane(lds_base + uint32_t(wave) * 1024u);
  const uint32_t wdummy = __builtin_amdgcn_readfirstlane(lds_base + uint32_t(2 * STAGE) + uint32_t(wave) * 1024u);

  auto issue = [&](int kt, int buf) {
    if (kt < KT) {
      const uint8_t *ga = g.a + int64_t(kt) * BK;
      const uint8_t *gb = g.b + int64_t(kt) * BK;
      const uint32_t sa = wblk + uint32_t(buf * STAGE);
      const uint32_t sb = sa + uint32_t(BM * BK);
#pragma unroll
      for (int c = 0; c < CHA; ++c)
        asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(oa[c]), "s"(ga),
                     "s"(sa + uint32_t(c * NW * 1024)) : "memory", "m0");
#pragma unroll
      for (int c = 0; c < CHB; ++c)
        asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(ob[c]), "s"(gb),
                     "s"(sb + uint32_t(c * NW * 1024)) : "memory", "m0");
    } else {  // the last, partial K tile, through registers: bytes at or past K are zero
      uint8_t *dA = smem + buf * STAGE;
      uint8_t *dB = dA + BM * BK;
      const uint32_t k0 = uint32_t(KT) * BK;
#pragma unroll
      for (int c = 0; c < CHA; ++c) {
        const int row = 8 * (wave + NW * c) + lrow;
        const int64_t gk = int64_t(k0) + (((lane & 7) ^ ((row >> 1) & 7)) * 16);
        const uint4 va = gk < K ? mask_tail(*reinterpret_cast<const uint4 *>(g.a + (oa[c] + k0)), K - gk) : make_uint4(0u, 0u, 0u, 0u);
        *reinterpret_cast<uint4 *>(dA + (wave + NW * c) * 1024 + lane * 16) = va;
      }
#pragma unroll
      for (int c = 0; c < CHB; ++c) {
        const int row = 8 * (wave + NW * c) + lrow;
        const int64_t gk = int64_t(k0) + (((lane & 7) ^ ((row >> 1) & 7)) * 16);
        const uint4 vb = gk < K ? mask_tail(*reinterpret_cast<const uint4 *>(g.b + (ob[c] + k0)), K - gk) : make_uint4(0u, 0u, 0u, 0u);
        *reinterpret_cast<uint4 *>(dB + (wave + NW * c) * 1024 + lane * 16) = vb;
      }
    }
  };

  // 16-row fragments: lane l reads row (l & 15), the 32 bytes 32 (l >> 4) .. +31
  // of the K tile, i.e. logical chunks 2 (l >> 4) and the next.  The swizzle
  // term depends on (l & 15) only, so every fragment is base + constant.
  const int fr = lane & 15, fq = lane >> 4;
  const uint32_t f_lo = uint32_t(fr) * BK + (uint32_t((2 * fq) ^ (fr >> 1)) & 7) * 16;
  const uint32_t f_hi = uint32_t(fr) * BK + (uint32_t((2 * fq + 1) ^ (fr >> 1)) & 7) * 16;
  auto frag = [&](const uint8_t *base) -> v8i {
    const uint4 lo = *reinterpret_cast<const uint4 *>(base + f_lo);
    const uint4 hi = *reinterpret_cast<const uint4 *>(base + f_hi);
    return v8i{int(lo.x), int(lo.y), int(lo.z), int(lo.w), int(hi.x), int(hi.y), int(hi.z), int(hi.w)};
  };
  auto read_a = [&](int buf, int i, v8i (&fa)[I]) { fa[i] = frag(smem + buf * STAGE + (wm * TM + i * 16) * BK); };
  auto read_b = [&](int buf, int j, v8i (&fb)[J]) {
    fb[j] = frag(smem + buf * STAGE + (BM + wn * TN + j * 16) * BK);
  };

  v4f acc[I][J];
#pragma unroll
  for (int i = 0; i < I; ++i)
#pragma unroll
    for (int j = 0; j < J; ++j) acc[i][j] = v4f{0.f, 0.f, 0.f, 0.f};

  auto mfma = [&](int i, int j, const v8i (&fa)[I], const v8i (&fb)[J]) {
    acc[i][j] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(fb[j], fa[i], acc[i][j], FB, FA, 0, 0, 0, 0);
  };
  // LDS-bound loads inside the K loop, two instructions each: load d of a K
  // tile lands at stage + 4096 d, so M0 steps by a uniform stride, and the
  // step is issued before an MFMA and the load after it (the MFMA is the wait
  // state M0 needs).  Past the last full K tile the loads still run, from
  // tile 0 into the wave's dummy block with stride 0: no branch per load.
  auto dma_m0 = [&](int d, uint32_t base, uint32_t stride) {
    if (d == 0)
      asm volatile("s_mov_b32 m0, %0" ::"s"(base) : "m0");
    else
      asm volatile("s_add_u32 m0, m0, %0" ::"s"(stride) : "m0", "scc");
  };
  auto dma_load = [&](int d, const uint8_t *ga, const uint8_t *gb) {
    if (d < CHA)
      asm volatile("global_load_lds_dwordx4 %0, %1" ::"v"(oa[d]), "s"(ga) : "memory");
    else
      asm volatile("global_load_lds_dwordx4 %0, %1" ::"v"(ob[d - CHA]), "s"(gb) : "memory");
  };

  // Phase A of a tile from stage `buf`: column-major MFMAs over block rows
  // 0 .. IA-1 (B fragment j is first needed at MFMA j * IA, so the fragments
  // read last in the previous phase B are needed last); A fragments IA .. I-1
  // of the same tile are read after the first MFMAs (one per even slot), long
  // before phase B needs them.  The tile's B fragments are all in registers
  // by now, so the same stage's B half already takes the B part of the tile
  // two K tiles ahead (`kt3`), spread over the phase: a K step and a half
  // before it is read.
  auto b_slot = [](int q, int k) { return (k * QA) / CHB + 1 == q; };
  auto phase_a = [&](int buf, bool dmab, int kt3, v8i (&fa)[I], v8i (&fb)[J]) {
    const uint8_t *gb = dmab ? g.b + int64_t(kt3) * BK : g.b;
    const uint32_t base = dmab ? wblk + uint32_t(buf * STAGE + BM * BK) : wdummy;
    const uint32_t stride = dmab ? uint32_t(NW * 1024) : 0u;
#pragma unroll
    for (int q = 0; q < QA; ++q) {
      int d = -1;  // the B-part load of this slot (folds to a constant once unrolled)
#pragma unroll
      for (int k = 0; k < CHB; ++k) d = b_slot(q, k) ? k : d;
      __builtin_amdgcn_sched_barrier(0);
      if (d >= 0) dma_m0(d, base, stride);
      __builtin_amdgcn_sched_barrier(0);
      mfma(q % IA, q / IA, fa, fb);
      __builtin_amdgcn_sched_barrier(0);
      if (d >= 0) dma_load(CHA + d, g.a, gb);
      if (q % 2 == 0 && q / 2 < IB) read_a(buf, IA + q / 2, fa);
    }
    __builtin_amdgcn_sched_barrier(0);
  };
  // Phase B of a tile: column-major MFMAs over block rows IA .. I-1.  After
  // the last use of B fragment j, the next tile's B fragment j is read from
  // stage `nbuf` into the same registers; the next tile's A fragments
  // 0 .. IA-1 are read in the first slots (their registers are free since
  // phase A).  `dma` issues the A part of tile `kt2` into stage `buf`.
  // Slots of phase B, one kind of memory instruction each where possible: the
  // next tile's A fragments after MFMAs 0, 4, 8, ..; LDS-bound loads after
  // MFMAs q = 1, 2 (mod 4), so the A part is issued in the first half of the
  // phase; B fragments after the last use of each (q = 3 (mod 4) when IB =
  // 4).  Loads that do not fit go to the latest q = 0 (mod 4) slots past the A
  // reads.  (Measured: the A part spread over all of phase B instead, equal;
  // the B part packed into the first half of phase A, 0.5% slower.)
  auto load_slot = [](int q) -> bool {
    constexpr int n12 = (QB / 4) * 2;
    if (q % 4 == 1 || q % 4 == 2) return (q / 4) * 2 + (q % 4 - 1) < CHA;
    if (q % 4 == 0 && CHA > n12) return q / 4 >= IA && QB / 4 - 1 - q / 4 < CHA - n12;
    return false;
  };
  auto phase_b = [&](int nbuf, bool dma, int kt2, int buf, v8i (&fa)[I], v8i (&fb)[J]) {
    static_assert(QB % 4 == 0, "phase B slots come in fours");
    const uint8_t *ga = dma ? g.a + int64_t(kt2) * BK : g.a;
    const uint8_t *gb = dma ? g.b + int64_t(kt2) * BK : g.b;
    const uint32_t base = dma ? wblk + uint32_t(buf * STAGE) : wdummy;
    const uint32_t stride = dma ? uint32_t(NW * 1024) : 0u;
#pragma unroll
    for (int q = 0; q < QB; ++q) {
      const int j = q / IB, i = IA + q % IB;
      const bool ld = load_slot(q);
      int d = 0;  // loads in earlier slots (folds to a constant once unrolled)
#pragma unroll
      for (int r = 0; r < q; ++r) d += load_slot(r) ? 1 : 0;
      __builtin_amdgcn_sched_barrier(0);
      if (ld) dma_m0(d, base, stride);
      __builtin_amdgcn_sched_barrier(0);  // M0 is written before the MFMA, never next to the load
      mfma(i, j, fa, fb);
      __builtin_amdgcn_sched_barrier(0);
      if (ld) dma_load(d, ga, gb);
      if (q % 4 == 0 && q / 4 < IA) read_a(nbuf, q / 4, fa);
      if (q % IB == IB - 1) read_b(nbuf, j, fb);  // last use of B fragment j was this MFMA
    }
    __builtin_amdgcn_sched_barrier(0);
  };

  if (T > 0) {
    v8i fa[I], fb[J];
    issue(0, 0);
    if (KT > 1) {
      // both first K tiles are full: tile 1's LDS-bound loads stay in flight
      // while the wave waits for its tile-0 loads (the ND most recent ones
      // are tile 1's; the counter completes in order)
      issue(1, 1);
      asm volatile("s_waitcnt vmcnt(%0)" ::"n"(ND) : "memory");
    } else {
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < J; ++j) read_b(0, j, fb);
#pragma unroll
    for (int i = 0; i < IA; ++i) read_a(0, i, fa);
    if (T > 1 && KT <= 1) issue(1, 1);  // tile 1 is the partial tail: through registers
    __syncthreads();                       // every wave holds tile 0's B fragments: stage 0's B half is free
    phase_a(0, 2 < KT, 2, fa, fb);         // and takes tile 2's B part
    // tile 1 complete; the CHB most recent loads (tile 2's B part) may still
    // be in flight: the counter completes in order
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(CHB) : "memory");
    __syncthreads();                       // tile 1 published; tile 0 fully read
    for (int t = 0; t < T; ++t) {
      const int buf = t & 1;
      const bool dma = t + 2 < KT;
      if (t + 2 < T && !dma) issue(t + 2, buf);
      // phase B of tile t, with tile t+2's A part; reads of tile t+1 (in the
      // last iteration they read a stale stage that is never used: always in
      // bounds, and branch-free here)
      phase_b(buf ^ 1, dma, t + 2, buf, fa, fb);
      if (t + 1 < T) {
        __syncthreads();                   // tile t+1's B fragments read by every wave
        phase_a(buf ^ 1, t + 3 < KT, t + 3, fa, fb);  // with tile t+3's B part
        asm volatile("s_waitcnt vmcnt(%0)" ::"n"(CHB) : "memory");
        __syncthreads();                   // tile t+2 published; tile t+1 fully read
      }
    }
  }

  // Epilogue through LDS: the MFMA layout gives each lane one row and a column
  // quad per 16 x 16 block, so store instructions would touch 16 rows x 64 B.
  // Each wave instead writes one 32-row block of its sub-tile (32 x TN FP32,
  // rows padded to TN + 4 floats) into LDS, then reads it back row-contiguous:
  // 32 lanes x 16 B cover one 512-byte output row run per store instruction.
  __syncthreads();  // every wave is done reading the last stage
  float *ep = reinterpret_cast<float *>(smem) + wave * 32 * EP;
  const int e = pow2_exponent(g.a_scale_inv) + pow2_exponent(g.b_scale_inv);
  const bool nfull = n0 + BN <= N;
  // Full tile with a vector-aligned destination (the common case): no bounds
  // checks, every store address is a uniform row base (scalar registers) plus
  // one per-lane offset, and LDS addresses are one base plus immediates.  With
  // one wave per SIMD the epilogue runs at instruction latency, so its
  // instruction count is its time.  Other tiles take the checked path.
  constexpr int ES = OUT == 1 ? 2 : 4;  // output element bytes
  // (buffer instructions: the row offset is a scalar operand; every offset of
  // the wave's TM x TN block stays below 2^31)
  const bool fast = vec_ok && nfull && m0 + BM <= M && g.ldc * ES * (TM + 2) < (int64_t(1) << 31);
  const bool has_col = (lane & 31) * 4 < TN;  // TN = 112 or 96: 28 or 24 of each 32 lanes hold a column quad
  const int wu = __builtin_amdgcn_readfirstlane(wave);
  const uint32_t voff = uint32_t((lane >> 5) * g.ldc + (lane & 31) * 4) * uint32_t(ES);
  char *cbase = static_cast<char *>(g.c) + ((m0 + (wu >> 1) * TM) * g.ldc + n0 + (wu & 1) * TN) * ES;
  const __amdgpu_buffer_rsrc_t crs = __builtin_amdgcn_make_buffer_rsrc(cbase, short(0), 0x7fffffff, 0x00020000);
  const int rstep = int(g.ldc) * ES;  // bytes per output row
  float *ew = ep + (lane & 15) * EP + 4 * (lane >> 4);
  const float *er = ep + (lane >> 5) * EP + (lane & 31) * 4;
#pragma unroll
  for (int i = 0; i < TM / 32; ++i) {
    // accumulate: read this block's destination first, so the loads are in
    // flight during the LDS round trip instead of one dependent load per row
    float4 pre[16];
    if constexpr (OUT == 2) {
      if (fast) {
#pragma unroll
        for (int it = 0; it < 16; ++it)
          if (has_col) pre[it] = __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(crs, voff, (i * 32 + 2 * it) * rstep, kNT));
      } else {
#pragma unroll
        for (int it = 0; it < 16; ++it) {
          const int64_t row = m0 + wm * TM + i * 32 + 2 * it + (lane >> 5);
          const int64_t col = n0 + wn * TN + (lane & 31) * 4;
          pre[it] = make_float4(0.f, 0.f, 0.f, 0.f);
          if (has_col && row < M && vec_ok && (nfull || col + 4 <= N))
            pre[it] = *reinterpret_cast<const float4 *>(static_cast<const float *>(g.c) + row * g.ldc + col);
        }
      }
    }
    if constexpr (OUT == 1) {
      if (fast) {
        // BF16 output: rounded before the LDS round trip, which then moves
        // half the bytes (rows of TN values padded to TN + 8), and every store
        // instruction writes four 2 * TN-byte row runs, 16 bytes per lane.
        // The same round-to-nearest-even of the same FP32 value, so the same
        // bits; measured 0.3-0.5% faster per stage step on MI355X.
        constexpr int EPH = TN + 8;
        uint16_t *eh = reinterpret_cast<uint16_t *>(ep);
        uint16_t *ehw = eh + (lane & 15) * EPH + 4 * (lane >> 4);
#pragma unroll
        for (int h = 0; h < 2; ++h)
#pragma unroll
          for (int j = 0; j < J; ++j) {
            const v4f a = acc[2 * i + h][j];
            *reinterpret_cast<uint2 *>(ehw + h * 16 * EPH + j * 16) =
                make_uint2(bf16x2_bits(__builtin_ldexpf(a[0], e), __builtin_ldexpf(a[1], e)),
                           bf16x2_bits(__builtin_ldexpf(a[2], e), __builtin_ldexpf(a[3], e)));
          }
        const uint16_t *ehr = eh + (lane >> 4) * EPH + (lane & 15) * 8;
        const uint32_t voffh = uint32_t((lane >> 4) * g.ldc + (lane & 15) * 8) * 2u;
#pragma unroll
        for (int it = 0; it < 8; ++it) {
          if ((lane & 15) * 8 >= TN) continue;
          const uint4 v = *reinterpret_cast<const uint4 *>(ehr + it * 4 * EPH);
          __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(v4i, v), crs, voffh, (i * 32 + 4 * it) * rstep, kNT);
        }
        continue;
      }
    }
    // block rows 2i and 2i+1: lane holds row (lane & 15) of each, four
    // consecutive columns 16 j + 4 (lane >> 4) .. +3 of every column block j
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int j = 0; j < J; ++j)
        *reinterpret_cast<float4 *>(ew + h * 16 * EP + j * 16) =
            make_float4(__builtin_ldexpf(acc[2 * i + h][j][0], e), __builtin_ldexpf(acc[2 * i + h][j][1], e),
                        __builtin_ldexpf(acc[2 * i + h][j][2], e), __builtin_ldexpf(acc[2 * i + h][j][3], e));
    // same wave writes then reads its own LDS rows: LDS operations of one wave
    // complete in order
    if (fast) {
#pragma unroll
      for (int it = 0; it < 16; ++it) {
        if (!has_col) continue;
        const float4 v4 = *reinterpret_cast<const float4 *>(er + it * 2 * EP);
        const int so = (i * 32 + 2 * it) * rstep;
        if constexpr (OUT == 0) {
          __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(v4i, v4), crs, voff, so, kNT);
        } else if constexpr (OUT == 1) {
          const v2i w = {int(bf16x2_bits(v4.x, v4.y)), int(bf16x2_bits(v4.z, v4.w))};
          __builtin_amdgcn_raw_buffer_store_b64(w, crs, voff, so, kNT);
        } else {
          const float4 o = pre[it];
          const float4 r = make_float4(o.x + v4.x, o.y + v4.y, o.z + v4.z, o.w + v4.w);
          __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(v4i, r), crs, voff, so, kNT);
        }
      }
      continue;
    }
#pragma unroll
    for (int it = 0; it < 16; ++it) {
      const int r = 2 * it + (lane >> 5);
      const int64_t row = m0 + wm * TM + i * 32 + r;
      const int cl = (lane & 31) * 4;
      const int64_t col = n0 + wn * TN + cl;
      if (!has_col) continue;
      const float4 v4 = *reinterpret_cast<const float4 *>(ep + r * EP + cl);
      if (row >= M) continue;
      const float v[4] = {v4.x, v4.y, v4.z, v4.w};
      if (vec_ok && (nfull || col + 4 <= N)) {
        if constexpr (OUT == 0) {
          *reinterpret_cast<float4 *>(static_cast<float *>(g.c) + row * g.ldc + col) = v4;
        } else if constexpr (OUT == 1) {
          const uint32_t lo = bf16x2_bits(v[0], v[1]);
          const uint32_t hi = bf16x2_bits(v[2], v[3]);
          *reinterpret_cast<uint2 *>(static_cast<uint16_t *>(g.c) + row * g.ldc + col) = make_uint2(lo, hi);
        } else {
          const float4 o = pre[it];
          *reinterpret_cast<float4 *>(static_cast<float *>(g.c) + row * g.ldc + col) =
              make_float4(o.x + v[0], o.y + v[1], o.z + v[2], o.w + v[3]);
        }
      } else {
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          if (col + t >= N) break;
          if constexpr (OUT == 0) {
            static_cast<float *>(g.c)[row * g.ldc + col + t] = v[t];
          } else if constexpr (OUT == 1) {
            static_cast<uint16_t *>(g.c)[row * g.ldc + col + t] = bf16_bits(v[t]);
          } else {
            float *dst = static_cast<float *>(g.c) + row * g.ldc + col + t;
            *dst = *dst + v[t];
          }
        }
      }
    }
  }
}

template <int FA, int FB, int BM, int BN>
hipError_t launch_w4(const GemmParams &g, hipStream_t s, const UpdateParams &u) {
  const int tiles_m = int((g.m + BM - 1) / BM), tiles_n = int((g.n + BN - 1) / BN);
  const uintptr_t cp = reinterpret_cast<uintptr_t>(g.c);
  const int vec_ok = (g.out == 1) ? (g.ldc % 4 == 0 && cp % 8 == 0) : (g.ldc % 4 == 0 && cp % 16 == 0);
  const dim3 grid(unsigned(tiles_m) * unsigned(tiles_n) + unsigned(u.n)), block(256);
  switch (g.out) {
    case 0: return klaunch(gemm_tn_w4_kernel<FA, FB, 0, BM, BN>, grid, block, 0, s, g, tiles_m, tiles_n, vec_ok, u);
    case 1: return klaunch(gemm_tn_w4_kernel<FA, FB, 1, BM, BN>, grid, block, 0, s, g, tiles_m, tiles_n, vec_ok, u);
    default: return klaunch(gemm_tn_w4_kernel<FA, FB, 2, BM, BN>, grid, block, 0, s, g, tiles_m, tiles_n, vec_ok, u);
  }
}

template <int BM, int BN>
hipError_t launch_w4_fmts(const GemmParams &g, hipStream_t s, const UpdateParams &u) {
  if (g.fmt_a == 0 && g.fmt_b == 0) return launch_w4<0, 0, BM, BN>(g, s, u);
  if (g.fmt_a == 1 && g.fmt_b == 0) return launch_w4<1, 0, BM, BN>(g, s, u);
  if (g.fmt_a == 0 && g.fmt_b == 1) return launch_w4<0, 1, BM, BN>(g, s, u);
  return launch_w4<1, 1, BM, BN>(g, s, u);
}

template <int BM, int BN, int WM, int WN, int FA, int FB>
hipError_t launch_out(const GemmParams &g, hipStream_t s) {
  const int tiles_m = int((g.m + BM - 1) / BM), tiles_n = int((g.n + BN - 1) / BN);
  const uintptr_t cp = reinterpret_cast<uintptr_t>(g.c);
  const int vec_ok = (g.out == 1) ? (g.ldc % 4 == 0 && cp % 8 == 0) : (g.ldc % 4 == 0 && cp % 16 == 0);
  const dim3 grid(unsigned(tiles_m) * unsigned(tiles_n)), block(WM * WN * 64);
  switch (g.out) {
    case 0: return klaunch(gemm_tn_kernel<BM, BN, WM, WN, FA, FB, 0>, grid, block, 0, s, g, tiles_m, tiles_n, vec_ok);
    case 1: return klaunch(gemm_tn_kernel<BM, BN, WM, WN, FA, FB, 1>, grid, block, 0, s, g, tiles_m, tiles_n, vec_ok);
    default: return klaunch(gemm_tn_kernel<BM, BN, WM, WN, FA, FB, 2>, grid, block, 0, s, g, tiles_m, tiles_n, vec_ok);
  }
}

template <int BM, int BN, int WM, int WN>
hipError_t launch_fmts(const GemmParams &g, hipStream_t s) {
  if (g.fmt_a == 0 && g.fmt_b == 0) return launch_out<BM, BN, WM, WN, 0, 0>(g, s);
  if (g.fmt_a == 1 && g.fmt_b == 0) return launch_out<BM, BN, WM, WN, 1, 0>(g, s);
  if (g.fmt_a == 0 && g.fmt_b == 1) return launch_out<BM, BN, WM, WN, 0, 1>(g, s);
  return launch_out<BM, BN, WM, WN, 1, 1>(g, s);
}

}  // namespace

// Relative cost of a round of tiles against a round of 256 x 256 ones at the
// same K, measured on MI355X (K = 4096, one round of each shape, bf16 out):
// 256 x 192 0.89, 192 x 256 0.86 (0.75 of the MFMA work at a lower
// efficiency per FLOP), the 8-wave 256 x 128 kernel 0.905; 256 x 224 0.978
// (bf16 out) and 0.972 (FP32 out), two rounds against two.  Rounded up, so
// a tie keeps the larger tile.
constexpr double kCost192 = 0.90;
constexpr double kCost128 = 0.92;
constexpr double kCost224 = 0.98;

static std::atomic<int> g_tile_override{0};

// Compute units of the current device (one 128 KB-LDS workgroup each at a
// time), read once per device from its properties; 256 on MI355X.
static int cu_count() {
  constexpr int kMaxDevices = 64;
  static std::atomic<int> cache[kMaxDevices];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return 256;
  int n = cache[dev].load(std::memory_order_relaxed);
  if (n > 0) return n;
  if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
  cache[dev].store(n, std::memory_order_relaxed);
  return n;
}

hipError_t launch_gemm(const GemmParams &g, hipStream_t s, const UpdateParams *fused) {
  UpdateParams none;
  memset(&none, 0, sizeof(none));
  const UpdateParams &u = fused != nullptr ? *fused : none;
  if (g.m <= 0 || g.n <= 0) return u.n > 0 ? launch_scale_update(u, s) : hipSuccess;
  // The kernel addresses each operand with 32-bit offsets: split any operand
  // of 2 GiB or more into row blocks (independent GEMMs on disjoint outputs),
  // whole 256-row tiles per block where a tile's rows fit in 2 GiB, else as
  // many rows as fit (at least one: its offsets are then 0 plus the K offset,
  // which stays below 2^31 because K does).
  constexpr int64_t kLim = int64_t(1) << 31;
  if (g.k >= kLim) return hipErrorInvalidValue;
  auto block_rows = [](int64_t ld) -> int64_t {
    const int64_t r = (kLim - 1) / ld;
    return r >= 256 ? r / 256 * 256 : (r > 0 ? r : 1);
  };
  const int64_t cbytes = g.out == 1 ? 2 : 4;
  if (g.m * g.lda >= kLim) {
    const int64_t rows = block_rows(g.lda);
    for (int64_t r = 0; r < g.m; r += rows) {
      GemmParams sub = g;
      sub.a = g.a + r * g.lda;
      sub.m = g.m - r < rows ? g.m - r : rows;
      sub.c = static_cast<char *>(g.c) + r * g.ldc * cbytes;
      const hipError_t e = launch_gemm(sub, s, r + rows >= g.m ? fused : nullptr);  // the update rides on the last
      if (e != hipSuccess) return e;
    }
    return hipSuccess;
  }
  if (g.n * g.ldb >= kLim) {
    const int64_t cols = block_rows(g.ldb);
    for (int64_t c0 = 0; c0 < g.n; c0 += cols) {
      GemmParams sub = g;
      sub.b = g.b + c0 * g.ldb;
      sub.n = g.n - c0 < cols ? g.n - c0 : cols;
      sub.c = static_cast<char *>(g.c) + c0 * cbytes;
      const hipError_t e = launch_gemm(sub, s, c0 + cols >= g.n ? fused : nullptr);
      if (e != hipSuccess) return e;
    }
    return hipSuccess;
  }
  // Tile choice by wave quantization: each CU runs one workgroup at a time, so
  // a grid costs ceil(tiles / CUs) rounds of one tile's time; the smaller tiles
  // win where the 256 x 256 grid leaves its last round mostly empty (N = 6144:
  // 384 tiles = 1.5 rounds, against 512 tiles of 256 x 192 = 2 rounds of 0.89;
  // N = 14336: 896 tiles = 3.5 rounds, against 1024 of 256 x 224 = 4 of 0.98).
  const int64_t cus = cu_count();
  auto rounds = [&](int64_t bm, int64_t bn) {
    const int64_t t = ((g.m + bm - 1) / bm) * ((g.n + bn - 1) / bn);
    return double((t + cus - 1) / cus);
  };
  const int force = g_tile_override.load(std::memory_order_relaxed);
  const double c256 = rounds(256, 256);
  const double c128 = kCost128 * rounds(256, 128);
  const double cn192 = kCost192 * rounds(256, 192);
  const double cm192 = kCost192 * rounds(192, 256);
  const double cn224 = kCost224 * rounds(256, 224);
  // the 8-wave kernel has 512 lanes per workgroup: its update runs as a launch of its own
  auto eight_wave = [&]() {
    const hipError_t e = launch_fmts<256, 128, 4, 2>(g, s);
    return e != hipSuccess || u.n == 0 ? e : launch_scale_update(u, s);
  };
  if (force == 1) return launch_w4_fmts<256, 256>(g, s, u);
  if (force == 2) return launch_w4_fmts<256, 192>(g, s, u);
  if (force == 3) return launch_w4_fmts<192, 256>(g, s, u);
  if (force == 4) return eight_wave();
  if (force == 5) return launch_w4_fmts<256, 224>(g, s, u);
  double best = c256;
  int pick = 1;
  if (cn224 < best) { best = cn224; pick = 5; }
  if (cn192 < best) { best = cn192; pick = 2; }
  if (cm192 < best) { best = cm192; pick = 3; }
  if (c128 < best) { best = c128; pick = 4; }
  if (pick == 2) return launch_w4_fmts<256, 192>(g, s, u);
  if (pick == 3) return launch_w4_fmts<192, 256>(g, s, u);
  if (pick == 4) return eight_wave();
  if (pick == 5) return launch_w4_fmts<256, 224>(g, s, u);
  return launch_w4_fmts<256, 256>(g, s, u);
}

void set_gemm_tile_override(int tile) { g_tile_override.store(tile, std::memory_order_relaxed); }

}  // namespace qe
