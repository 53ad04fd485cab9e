// FP8 quantization with fused transpose and amax recording (gfx950).
//
// Delayed scaling (§2.1 of the paper): a tensor is cast with the scale the
// previous update produced, and its amax is recorded for later updates.  The
// split backward (§3.2) needs each operand both row-wise (for F / dI) and
// column-wise (for the deferred dW), so one pass writes both:
//   q_row[r][c] = Q(x[r][c] * scale),  q_col[c][r] = the same code,
//   history[0]  = max(history[0], max |x|)      (unscaled, NaN propagates)
// Q rounds to nearest even and saturates to +-fmax; NaN becomes 0x7F with the
// input's sign bit.  Formats: OCP E4M3 (max 448) and E5M2 (max 57344).
//
// Layout: one workgroup of 256 lanes per 128 x 128 tile.  Phase 1: every load
// instruction is one contiguous 16-byte piece per lane along a row (16 lanes
// per bf16 row, 32 per fp32 row); each lane converts its 8 (or 4) values and
// stores the codes row-wise and into an LDS tile whose 16-byte chunks are
// XOR-swizzled by row block.
// Phase 2: each lane gathers a 16-row x 4-column block of codes from LDS and
// writes four 16-byte column segments; eight consecutive lanes complete one
// 128-byte run of a transposed row.  amax: a max over the |x| bit patterns
// (which order like the values, NaN above inf) per lane, a wave shuffle
// reduction, then one atomicMax per workgroup into one of the 64 lines of the
// role's amax accumulator (same-line atomics serialise).  HBM-bound: per element it
// moves 2 or 4 bytes in and 2 bytes out.
#include "kernels.h"

namespace qe {
namespace {

constexpr int kTile = 128;
constexpr int kThreads = 256;

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// Four scaled values -> four FP8 codes, byte i = value i.  The hardware
// conversion rounds to nearest even but neither saturates (it overflows to
// NaN / inf) nor keeps the sign of a NaN, so values are clamped first with
// med3, which maps NaN to -fmax; NaN inputs are repaired separately.
template <int FMT>
__device__ __forceinline__ uint32_t enc4(float a, float b, float c, float d) {
  constexpr float fm = FMT == 0 ? 448.0f : 57344.0f;
  const float ca = __builtin_amdgcn_fmed3f(a, -fm, fm);
  const float cb = __builtin_amdgcn_fmed3f(b, -fm, fm);
  const float cc = __builtin_amdgcn_fmed3f(c, -fm, fm);
  const float cd = __builtin_amdgcn_fmed3f(d, -fm, fm);
  int r;
  if constexpr (FMT == 0) {
    r = __builtin_amdgcn_cvt_pk_fp8_f32(ca, cb, 0, false);
    r = __builtin_amdgcn_cvt_pk_fp8_f32(cc, cd, r, true);
  } else {
    r = __builtin_amdgcn_cvt_pk_bf8_f32(ca, cb, 0, false);
    r = __builtin_amdgcn_cvt_pk_bf8_f32(cc, cd, r, true);
  }
  return uint32_t(r);
}

// NaN -> 0x7F with the input's sign bit, for the rare thread that saw one.
__device__ __forceinline__ uint32_t nan_fix(uint32_t u, int byte, float v) {
  if (v != v) {
    const uint32_t code = 0x7fu | ((__float_as_uint(v) >> 24) & 0x80u);
    u = (u & ~(0xffu << (8 * byte))) | (code << (8 * byte));
  }
  return u;
}

__device__ __forceinline__ float bf16_to_f32(uint32_t bits16) { return __uint_as_float(bits16 << 16); }

__device__ __forceinline__ uint32_t abs_bits(float v) { return __float_as_uint(v) & 0x7fffffffu; }

__device__ __forceinline__ uint32_t lds_chunk_offset(int row, int chunk) {
  return uint32_t(row) * kTile + (uint32_t((chunk ^ (row >> 4)) & 7) << 4);
}

__device__ __forceinline__ uint32_t byte_of(uint32_t w, int j) { return (w >> (8 * j)) & 0xffu; }

// E values of one 16-byte input load (8 bf16 or 4 fp32), as floats
template <bool BF16>
__device__ __forceinline__ void unpack16(const uint4 &v, float *f) {
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
  if constexpr (BF16) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      f[2 * e] = bf16_to_f32(w[e] & 0xffffu);
      f[2 * e + 1] = __uint_as_float(w[e] & 0xffff0000u);
    }
  } else {
#pragma unroll
    for (int e = 0; e < 4; ++e) f[e] = __uint_as_float(w[e]);
  }
}

// One launch casts one tensor, or two independent ones (the forward's weight
// refresh and input cast) whose tiles follow each other in one grid, so the
// second tensor's tiles fill the first one's tail instead of a second launch
// ramping up after it.
struct QuantJob {
  QuantParams p;
  int64_t tiles, tiles_c;
  int32_t aligned, pad;
};
struct QuantPair {
  QuantJob j[2];
  int32_t n, pad;
};

template <bool BF16, int FMT>
__global__ __launch_bounds__(kThreads) void quantize_kernel(QuantPair pp) {
  __shared__ __attribute__((aligned(16))) uint8_t tile[kTile * kTile];
  __shared__ uint32_t red[kThreads / 64];
  // Phase 1 mapping: one 16-byte load per lane per step, consecutive lanes on
  // consecutive 16 bytes of a row (LPR lanes per 128-element row).
  constexpr int EPL = BF16 ? 8 : 4;          // elements per load
  constexpr int LPR = kTile / EPL;           // lanes per tile row
  constexpr int NLD = kTile * kTile / (EPL * kThreads);  // loads per lane
  const int tid = threadIdx.x;
  const bool second = pp.n > 1 && int64_t(blockIdx.x) >= pp.j[0].tiles;  // uniform per workgroup
  const QuantJob &job = second ? pp.j[1] : pp.j[0];
  const QuantParams &p = job.p;
  const int64_t tiles_c = job.tiles_c;
  const int aligned = job.aligned;
  const int64_t t = second ? int64_t(blockIdx.x) - pp.j[0].tiles : int64_t(blockIdx.x);
  const int64_t r0 = (t / tiles_c) * kTile;
  const int64_t c0 = (t % tiles_c) * kTile;
  const float scale = *p.scale;
  if (t == 0 && tid == 0 && p.snapshot != nullptr) *p.snapshot = *p.scale_inv;
  const bool full = aligned && r0 + kTile <= p.rows && c0 + kTile <= p.cols;
  uint32_t amax = 0;

  if (full) {
    uint4 raw[NLD];
#pragma unroll
    for (int it = 0; it < NLD; ++it) {
      const int q = it * kThreads + tid, row = q / LPR, cl = q % LPR;
      const int64_t eoff = (r0 + row) * p.cols + c0 + cl * EPL;
      const u32x4 x = __builtin_nontemporal_load(
          reinterpret_cast<const u32x4 *>(static_cast<const char *>(p.in) + eoff * (BF16 ? 2 : 4)));
      raw[it] = make_uint4(x.x, x.y, x.z, x.w);
    }
    uint32_t codes[NLD][EPL / 4];
#pragma unroll
    for (int it = 0; it < NLD; ++it) {
      float f[EPL];
      unpack16<BF16>(raw[it], f);
#pragma unroll
      for (int e = 0; e < EPL; ++e) {
        const uint32_t b = abs_bits(f[e]);
        amax = b > amax ? b : amax;
      }
#pragma unroll
      for (int w = 0; w < EPL / 4; ++w)
        codes[it][w] = enc4<FMT>(f[4 * w] * scale, f[4 * w + 1] * scale, f[4 * w + 2] * scale, f[4 * w + 3] * scale);
    }
    if (__builtin_expect(amax > 0x7f800000u, 0)) {  // this lane saw a NaN
#pragma unroll
      for (int it = 0; it < NLD; ++it) {
        float f[EPL];
        unpack16<BF16>(raw[it], f);
#pragma unroll
        for (int e = 0; e < EPL; ++e) codes[it][e / 4] = nan_fix(codes[it][e / 4], e % 4, f[e]);
      }
    }
#pragma unroll
    for (int it = 0; it < NLD; ++it) {
      const int q = it * kThreads + tid, row = q / LPR, cl = q % LPR;
      const int col = cl * EPL;
      const uint32_t lofs = lds_chunk_offset(row, col >> 4) + (col & 15);
      if constexpr (BF16) {
        if (p.q_row != nullptr)
          *reinterpret_cast<uint2 *>(p.q_row + (r0 + row) * p.ld_row + c0 + col) = make_uint2(codes[it][0], codes[it][1]);
        *reinterpret_cast<uint2 *>(tile + lofs) = make_uint2(codes[it][0], codes[it][1]);
      } else {
        if (p.q_row != nullptr) *reinterpret_cast<uint32_t *>(p.q_row + (r0 + row) * p.ld_row + c0 + col) = codes[it][0];
        *reinterpret_cast<uint32_t *>(tile + lofs) = codes[it][0];
      }
    }
  } else {
    for (int it = 0; it < 4; ++it) {
      const int q = it * kThreads + tid, row = q >> 3, cc = q & 7;
      const int64_t r = r0 + row;
      float f[16];
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int64_t c = c0 + cc * 16 + e;
        float v = 0.0f;
        if (r < p.rows && c < p.cols) {
          if constexpr (BF16)
            v = bf16_to_f32(static_cast<const uint16_t *>(p.in)[r * p.cols + c]);
          else
            v = static_cast<const float *>(p.in)[r * p.cols + c];
        }
        f[e] = v;
        const uint32_t b = abs_bits(v);
        amax = b > amax ? b : amax;
      }
      uint32_t w[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        w[k] = enc4<FMT>(f[4 * k] * scale, f[4 * k + 1] * scale, f[4 * k + 2] * scale, f[4 * k + 3] * scale);
#pragma unroll
        for (int e = 0; e < 4; ++e) w[k] = nan_fix(w[k], e, f[4 * k + e]);
      }
      if (p.q_row != nullptr && r < p.rows) {
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int64_t c = c0 + cc * 16 + e;
          if (c < p.cols) p.q_row[r * p.ld_row + c] = uint8_t(byte_of(w[e >> 2], e & 3));
        }
      }
      *reinterpret_cast<uint4 *>(tile + lds_chunk_offset(row, cc)) = make_uint4(w[0], w[1], w[2], w[3]);
    }
  }

  // amax: wave shuffle reduction, then one atomic per workgroup
  for (int off = 32; off > 0; off >>= 1) {
    uint32_t o = __shfl_xor(amax, off, 64);
    amax = o > amax ? o : amax;
  }
  if ((tid & 63) == 0) red[tid >> 6] = amax;
  __syncthreads();
  if (tid == 0) {
    uint32_t a = red[0];
    for (int w = 1; w < kThreads / 64; ++w) a = red[w] > a ? red[w] : a;
    fold_amax(p.amax_accum, p.amax_slot, a);
  }

  if (p.q_col == nullptr) return;
  // Phase 2: lane (rb, cq) transposes rows rb*16..+16 x columns 4cq..4cq+3.
  const int rb = tid & 7, cq = tid >> 3;
  uint32_t d[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int R = rb * 16 + i;
    d[i] = *reinterpret_cast<const uint32_t *>(tile + lds_chunk_offset(R, cq >> 2) + ((cq & 3) << 2));
  }
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    uint32_t w[4];
#pragma unroll
    for (int q = 0; q < 4; ++q)
      w[q] = byte_of(d[4 * q], j) | (byte_of(d[4 * q + 1], j) << 8) | (byte_of(d[4 * q + 2], j) << 16) |
             (byte_of(d[4 * q + 3], j) << 24);
    const int64_t col = c0 + 4 * cq + j;
    const int64_t rbase = r0 + rb * 16;
    if (full) {
      *reinterpret_cast<uint4 *>(p.q_col + col * p.ld_col + rbase) = make_uint4(w[0], w[1], w[2], w[3]);
    } else if (col < p.cols) {
#pragma unroll
      for (int e = 0; e < 16; ++e)
        if (rbase + e < p.rows) p.q_col[col * p.ld_col + rbase + e] = uint8_t(byte_of(w[e >> 2], e & 3));
    }
  }
}

template <bool BF16>
hipError_t launch_fmt(const QuantPair &pp, int fmt, hipStream_t s) {
  int64_t tiles = 0;
  for (int i = 0; i < pp.n; ++i) tiles += pp.j[i].tiles;
  if (fmt == 0) return klaunch(quantize_kernel<BF16, 0>, dim3(unsigned(tiles)), dim3(kThreads), 0, s, pp);
  return klaunch(quantize_kernel<BF16, 1>, dim3(unsigned(tiles)), dim3(kThreads), 0, s, pp);
}

QuantJob make_job(const QuantParams &p) {
  QuantJob j;
  memset(&j, 0, sizeof(j));  // padding too: recorded launches are compared bytewise
  j.p = p;
  const int64_t tiles_r = (p.rows + kTile - 1) / kTile;
  const int64_t tiles_c = (p.cols + kTile - 1) / kTile;
  j.tiles = tiles_r * tiles_c;
  if (j.tiles < 1) j.tiles = 1;  // still writes the scale_inv snapshot
  j.tiles_c = tiles_c < 1 ? 1 : tiles_c;
  const int64_t esize = p.in_bf16 ? 2 : 4;
  const bool in_al = (reinterpret_cast<uintptr_t>(p.in) % 16 == 0) && ((p.cols * esize) % 16 == 0);
  const bool row_al = p.q_row == nullptr || ((reinterpret_cast<uintptr_t>(p.q_row) % 16 == 0) && p.ld_row % 16 == 0);
  const bool col_al = p.q_col == nullptr || ((reinterpret_cast<uintptr_t>(p.q_col) % 16 == 0) && p.ld_col % 16 == 0);
  j.aligned = (in_al && row_al && col_al) ? 1 : 0;
  return j;
}

hipError_t launch_pair(const QuantPair &pp, hipStream_t s) {
  return pp.j[0].p.in_bf16 ? launch_fmt<true>(pp, pp.j[0].p.fmt, s) : launch_fmt<false>(pp, pp.j[0].p.fmt, s);
}

}  // namespace

hipError_t launch_quantize(const QuantParams &p, hipStream_t s) {
  QuantPair pp;
  memset(&pp, 0, sizeof(pp));
  pp.j[0] = make_job(p);
  pp.n = 1;
  return launch_pair(pp, s);
}

hipError_t launch_quantize_pair(const QuantParams &a, const QuantParams &b, hipStream_t s) {
  if (a.in_bf16 != b.in_bf16 || a.fmt != b.fmt) {  // different kernel instances: two launches
    const hipError_t e = launch_quantize(a, s);
    return e != hipSuccess ? e : launch_quantize(b, s);
  }
  QuantPair pp;
  memset(&pp, 0, sizeof(pp));
  pp.j[0] = make_job(a);
  pp.j[1] = make_job(b);
  pp.n = 2;
  return launch_pair(pp, s);
}

}  // namespace qe
