// Rank-r products of the low-rank term (bf16), Section 3.3's U (V^T x)
// evaluated for a batch of tokens:
//
//   T_lr = X V^T   V is r x K row-major: B read as [n][k]   (BKN = false)
//   S    = dY U    U is N x r row-major: B read as [k][n]   (BKN = true)
//
// C[M x r] = A[M x K] . op(B) with r small (a multiple of the block size).
// These products stream A once and are bound by that read; the block-sparse
// tile kernels would need a split of K with fp32 partials and a second pass
// to keep the chip busy at this width.  Here one workgroup owns 32 token rows
// x 64 output columns and its NW waves (4, or 8 for long K) split the K range
// among themselves (wave w takes the 64-wide K steps w, w + NW, ...), each
// accumulating the whole 32 x 64 tile; the NW tiles are summed through LDS
// in wave order (deterministic) and stored once.
//
// Operands reach the MFMA straight from global memory where they can: the
// contraction does not care in which order k is visited as long as both
// operands agree, so 16-wide slice c of the MFMA takes k = c * 16 + (l / 32)
// * 8 .. + 7 of the step in lane l, one 16-byte load.  The two lane halves
// then read 32 adjacent bytes of a row per load, which halves the L1
// requests of a lane-per-row load against giving each half its own 32-k
// run.  That serves A and a [n][k] B directly.  A [k][n] B (U) is staged per
// wave in a private 64 x 64 LDS tile and read back with the gfx950
// transpose read, which hands each lane 4 consecutive k of one column.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "pf_launch.h"

namespace pf {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef short s16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef uint16_t bf16_t;
typedef __amdgpu_buffer_rsrc_t rsrc_t;

constexpr int SK_TM = 32;   // token rows per workgroup
constexpr int SK_TN = 64;   // output columns per workgroup
constexpr int SK_BK = 64;   // K per step
constexpr int SK_NT = SK_TN / 32;

__device__ __forceinline__ rsrc_t make_rsrc(const void *p, int64_t bytes) {
  const int64_t b = bytes < 0 ? 0 : (bytes > 0x7fffffff ? 0x7fffffff : bytes);
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(p), (short)0, (int)b, 0x00020000);
}
__device__ __forceinline__ u32x4 bload(rsrc_t r, uint32_t voff, uint32_t soff) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, (int)voff, (int)soff, 0);
}
__device__ __forceinline__ int xcd_remap(int bid, int n) {
  constexpr int X = 8;
  const int q = n / X, rem = n % X, x = bid % X, slot = bid / X;
  return x * q + min(x, rem) + slot;
}
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)lo) |
         ((uint32_t)__builtin_bit_cast(uint16_t, (__bf16)hi) << 16);
}
__device__ __forceinline__ bf16x8 as_frag(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

// One step's operands in registers: A (4 chunks of 8 k) and B (SK_NT tiles x
// 4 chunks for [n][k]; 8 row chunks of the 64 x 64 tile for [k][n]).
struct SkStage {
  u32x4 a[4];
  u32x4 b[8];
};

// Byte offset of element (k, n) of a wave's 64 x 64 [k][n] LDS tile: 128-byte
// k rows whose 16-byte chunks are XOR-swizzled by bit 1 of k, so that the
// four k rows one 16-lane group of a transpose read covers fall in distinct
// banks.
__device__ __forceinline__ uint32_t sk_lds_off(int k, int n) {
  return (uint32_t)(k * 128 + ((((n >> 3) ^ (((k >> 1) & 1) << 2)) << 4) | ((n & 7) << 1)));
}

template <bool BKN, int NW>
__global__ __launch_bounds__(64 * NW) void skinny_kernel(SkinnyArgs a) {
  __shared__ __attribute__((aligned(16))) uint8_t smem[NW * 64 * 128 > NW * SK_NT * 16 * 64 * 4
                                                           ? NW * 64 * 128
                                                           : NW * SK_NT * 16 * 64 * 4];
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int ncol_tiles = (a.ncols + SK_TN - 1) / SK_TN;
  const int bid = xcd_remap(blockIdx.x, gridDim.x);
  const int tt = bid / ncol_tiles, ct = bid % ncol_tiles;  // column tiles of a token tile adjacent
  const int64_t t0 = (int64_t)tt * SK_TM;
  const int n0 = ct * SK_TN;
  const int ksteps = (a.K + SK_BK - 1) / SK_BK;
  const int h = lane >> 5, r32 = lane & 31;

  // A: the workgroup's 32 rows only, rows past M read as zero (range); a k
  // slice past K is pointed out of range (the host keeps 32 rows of A and
  // all of B below that offset).  Step s adds s * 128 bytes through the
  // scalar offset.
  const int64_t a_rows = a.M - t0 < SK_TM ? a.M - t0 : SK_TM;
  const rsrc_t rA = make_rsrc((const bf16_t *)a.A + t0 * a.lda, a_rows * a.lda * 2);
  const uint32_t voffA = (uint32_t)(r32 * a.lda * 2 + h * 16);
  const uint32_t OUT = 0x7ffffff0u;
  rsrc_t rB;
  uint32_t voffB[8];
  if constexpr (!BKN) {
    // V rows n0 .. n0 + 63 (rows past r read as zero).
    rB = make_rsrc((const bf16_t *)a.B + (int64_t)n0 * a.ldb, (int64_t)(a.ncols - n0) * a.ldb * 2);
#pragma unroll
    for (int j = 0; j < SK_NT; ++j) voffB[j] = (uint32_t)((j * 32 + r32) * a.ldb * 2 + h * 16);
  } else {
    // U rows (k) of the step, columns n0 .. n0 + 63: chunk q = lane + 64 i is
    // row q / 8, 8 columns at (q % 8) * 8; columns past r are pointed out of
    // range, rows past K fall outside the buffer.
    rB = make_rsrc(a.B, (int64_t)a.K * a.ldb * 2);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int q = lane + 64 * i, row = q >> 3, col = n0 + (q & 7) * 8;
      voffB[i] = col < a.ncols ? (uint32_t)(row * a.ldb * 2 + col * 2) : OUT;
    }
  }

  // Steps past the end (s * SK_BK >= K) read zeros: A and [n][k] B are
  // pointed out of range, [k][n] B rows fall outside the buffer.  The step's
  // byte offset goes through the scalar offset; readfirstlane makes it a
  // scalar (else each load is wrapped in a per-lane loop).
  auto load = [&](int s, SkStage &st) __attribute__((always_inline)) {
    const uint32_t soff = (uint32_t)__builtin_amdgcn_readfirstlane(s * 128);
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      // K is a multiple of 32, so a 16-k slice is wholly inside or outside.
      const bool kin = s * SK_BK + c * 16 < a.K;
      st.a[c] = bload(rA, kin ? voffA + c * 32 : OUT, soff);
    }
    if constexpr (!BKN) {
#pragma unroll
      for (int j = 0; j < SK_NT; ++j)
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          const bool kin = s * SK_BK + c * 16 < a.K;
          st.b[j * 4 + c] = bload(rB, kin ? voffB[j] + c * 32 : OUT, soff);
        }
    } else {
      // The step's row offset goes into the per-lane offset, which the
      // buffer range check covers, so rows past K read as zero.
      const uint32_t rows = (uint32_t)(s * SK_BK) * (uint32_t)(a.ldb * 2);
#pragma unroll
      for (int i = 0; i < 8; ++i) st.b[i] = bload(rB, voffB[i] == OUT ? OUT : voffB[i] + rows, 0);
    }
  };

  uint8_t *const tile = smem + w * (64 * 128);  // this wave's [k][n] tile (BKN)
  f32x16 acc[SK_NT];
#pragma unroll
  for (int j = 0; j < SK_NT; ++j)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[j][e] = 0.f;

  auto compute = [&](SkStage &st) __attribute__((always_inline)) {
    if constexpr (BKN) {
      // Stage the 64 x 64 U tile; a wave's LDS accesses complete in order,
      // so its reads below see these writes (no barrier: the tile is private).
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int q = lane + 64 * i;
        *(u32x4 *)(tile + sk_lds_off(q >> 3, (q & 7) * 8)) = st.b[i];
      }
    }
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const bf16x8 af = as_frag(st.a[c]);
#pragma unroll
      for (int j = 0; j < SK_NT; ++j) {
        bf16x8 bfr;
        if constexpr (!BKN) {
          bfr = as_frag(st.b[j * 4 + c]);
        } else {
          // Transpose read: within each 16-lane group, lanes 4m..4m+3 address
          // k row m and lane i receives column (group base + i); rows
          // c*16 + h*8 + 0..3, then + 4..7, match the k of A's slice c.
          const int g16 = lane >> 4, i = lane & 15;
          const int n = j * 32 + (g16 & 1) * 16 + (i & 3) * 4;
          const int k = c * 16 + (g16 >> 1) * 8 + (i >> 2);
          typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
          const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)(tile + sk_lds_off(k, n)));
          const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)(tile + sk_lds_off(k + 4, n)));
          const s16x8 v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
          bfr = __builtin_bit_cast(bf16x8, v);
        }
        // D rows = output columns, D columns = tokens: lane l ends with token
        // l % 32 and columns (e / 4) * 8 + (l / 32) * 4 + e % 4 of tile j.
        acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bfr, af, acc[j], 0, 0, 0);
      }
    }
  };

  // Three register stages: this wave's next two steps are in flight while
  // the current one is computed (the chain of a wave is up to K / (64 NW)
  // steps long, each a memory round trip if not overlapped).  The loop body
  // has no branches around its loads, so the wait before each compute
  // leaves the two younger stages in flight; the step count is rounded up
  // to whole rounds of three, the extra steps reading zeros.
  SkStage s0, s1, s2;
  const int n = ksteps > w ? (ksteps - w + NW - 1) / NW : 0;  // this wave's steps
  const int n3 = (n + 2) / 3 * 3;
  auto step_of = [&](int i) { return w + i * NW; };
  load(step_of(0), s0);
  load(step_of(1), s1);
  for (int i = 0; i < n3; i += 3) {
    load(step_of(i + 2), s2);
    compute(s0);
    load(step_of(i + 3), s0);
    compute(s1);
    load(step_of(i + 4), s1);
    compute(s2);
  }

  // Sum the waves' tiles in wave order through LDS (fp32, lane-major:
  // float index (j * 16 + e) * 64 + lane of wave w).
  __syncthreads();
  float *const red = (float *)smem;
#pragma unroll
  for (int j = 0; j < SK_NT; ++j)
#pragma unroll
    for (int e = 0; e < 16; ++e) red[((w * SK_NT + j) * 16 + e) * 64 + lane] = acc[j][e];
  __syncthreads();
  // Thread -> (j, e-group g, lane) items: 4 consecutive output columns of one
  // token row each.
  for (int item = threadIdx.x; item < SK_NT * 4 * 64; item += 64 * NW) {
    const int l = item & 63, g = (item >> 6) & 3, j = item >> 8;
    float v[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      float x = 0.f;
#pragma unroll
      for (int ww = 0; ww < NW; ++ww) x += red[((ww * SK_NT + j) * 16 + g * 4 + q) * 64 + l];
      v[q] = x;
    }
    const int64_t t = t0 + (l & 31);
    const int col = n0 + j * 32 + g * 8 + (l >> 5) * 4;
    if (t < a.M && col < a.ncols) {
      bf16_t *dst = (bf16_t *)a.C + t * a.ldc + col;
      *(uint2 *)dst = uint2{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])};
    }
  }
}

}  // namespace

hipError_t launch_skinny(bool b_kn, const SkinnyArgs &a, hipStream_t s) {
  const int64_t tiles = ((a.M + SK_TM - 1) / SK_TM) * ((a.ncols + SK_TN - 1) / SK_TN);
  if (tiles <= 0 || tiles > 0x7fffffff) return hipErrorInvalidValue;
  // Eight waves once each of four would have 16 or more steps (measured:
  // at 48 steps four waves were faster than eight).
#ifndef PF_SKINNY_WIDE_STEPS
#define PF_SKINNY_WIDE_STEPS 64
#endif
  const bool wide = (a.K + SK_BK - 1) / SK_BK >= PF_SKINNY_WIDE_STEPS;
  if (b_kn) {
    if (wide) launch_kernel(skinny_kernel<true, 8>, dim3((unsigned)tiles), dim3(512), s, a);
    else launch_kernel(skinny_kernel<true, 4>, dim3((unsigned)tiles), dim3(256), s, a);
  } else {
    if (wide) launch_kernel(skinny_kernel<false, 8>, dim3((unsigned)tiles), dim3(512), s, a);
    else launch_kernel(skinny_kernel<false, 4>, dim3((unsigned)tiles), dim3(256), s, a);
  }
  return hipGetLastError();
}

}  // namespace pf
