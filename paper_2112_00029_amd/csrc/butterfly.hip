// Product form of the block butterfly (Section 3.2: a product of factors,
// each a matrix on the support of I + B_k; appendix on benchmarking the
// butterfly multiply), applied to a batch of token rows in one launch.
//
// The product of the factors with strides 2 .. k is block-diagonal in groups
// of k blocks, so a workgroup owns TM token rows x one group of k blocks
// (k * 32 features): it loads that activation tile into LDS once, applies the
// L = log2 k factors to it in place, one after another, and writes the
// result.  A factor of stride 2^(f+1) maps each block pair (p, p + h),
// h = 2^f, onto itself:
//     forward        y_p = x_p W(p,p)^T + x_q W(p,q)^T,  q = p + h (and y_q alike)
//     backward-data  g'_p = g_p F(p,p) + g_q F(q,p)              (and g'_q alike)
// so the waves take disjoint pairs, read both input blocks into registers,
// run the four 32 x 32 block products on MFMA and write both output blocks
// back; a barrier separates factors.  Each pair's four weight blocks
// (8 KiB) are loaded into registers one pair ahead and staged in a private
// LDS region per wave (the backward reads them transposed with the gfx950
// transpose read).  Optionally the input of every factor (forward) or the
// gradient at every factor's output (backward) is written out, token-major
// as [T][L][n], for the weight gradient.
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
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
typedef uint16_t bf16_t;

constexpr int BB = kBflyBlock;  // block size (32)
constexpr int TM = 32;          // token rows per workgroup
constexpr int NW = 4;           // waves
constexpr int BLK_BYTES = BB * BB * 2;
constexpr int ACT_BYTES = TM * kBflyMaxGroupCols * 2;

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)lo) |
         ((uint32_t)__builtin_bit_cast(uint16_t, (__bf16)hi) << 16);
}

__device__ __forceinline__ s16x4 tr16(const uint8_t *p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4 *)(p));
}

// One pair's four weight blocks in registers: lane l holds the 16-byte
// chunks l + 64 j (j = 0..7) of the 8 KiB [W(p,p) W(p,q) W(q,p) W(q,q)].
struct WReg {
  u32x4 r[8];
};

template <bool BWD>
__global__ __launch_bounds__(256, 1) void bfly_kernel(BflyArgs a) {
  __shared__ __attribute__((aligned(16))) uint8_t act_s[ACT_BYTES];
  __shared__ __attribute__((aligned(16))) uint8_t wst_s[NW * 4 * BLK_BYTES];

  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int k = a.k;                    // blocks per group
  const int cpr = k * BB * 2 / 16;      // 16-byte chunks per activation row
  const int swm = (cpr < 16 ? cpr : 16) - 1;
  const int ngroups = a.nb / k;
  const int tt = blockIdx.x / ngroups, grp = blockIdx.x % ngroups;
  const int64_t t0 = (int64_t)tt * TM;
  const int64_t col0 = (int64_t)grp * k * BB;
  const int rows = (int)min<int64_t>(TM, a.T - t0);

  // Activation tile: row m (token t0 + m) holds the group's k * 32 features;
  // chunk c of row m sits at chunk c XOR (m & swm), so that the 32 rows one
  // fragment read touches spread over the banks.
  auto act = [&](int m, int c) __attribute__((always_inline)) -> uint8_t * {
    return act_s + m * (cpr * 16) + ((c ^ (m & swm)) << 4);
  };
  const bf16_t *in = (const bf16_t *)a.in;
  for (int idx = threadIdx.x; idx < TM * cpr; idx += 256) {
    const int m = idx / cpr, c = idx % cpr;
    u32x4 v = {0u, 0u, 0u, 0u};
    if (m < rows) v = *(const u32x4 *)(in + (t0 + m) * a.n + col0 + c * 8);
    *(u32x4 *)act(m, c) = v;
  }
  // Copy of the tile to dst (row stride ld elements, column offset off).
  auto copy_out = [&](bf16_t *dst, int64_t ld, int64_t off) __attribute__((always_inline)) {
    for (int idx = threadIdx.x; idx < TM * cpr; idx += 256) {
      const int m = idx / cpr, c = idx % cpr;
      if (m < rows) *(u32x4 *)(dst + (t0 + m) * ld + off + col0 + c * 8) = *(const u32x4 *)act(m, c);
    }
  };

  // This wave's work: pairs q = w, w + 4, ... of every factor (each factor
  // has k / 2 pairs).
  const int nper = k / 2 > w ? (k / 2 - w + NW - 1) / NW : 0;
  const int L = a.nfac;
  const bf16_t *F = (const bf16_t *)a.F;
  uint8_t *const wst = wst_s + w * (4 * BLK_BYTES);

  // Block row p of the group (p & h == 0) of pair q of factor f.
  auto pair_row = [&](int f, int q) __attribute__((always_inline)) -> int {
    return ((q >> f) << (f + 1)) | (q & ((1 << f) - 1));
  };
  auto wload = [&](int f, int q, WReg &W) __attribute__((always_inline)) {
    const int h = 1 << f;
    const int64_t P = (int64_t)grp * k + pair_row(f, q);
    // The two kept blocks of a block row are contiguous (ascending column).
    const bf16_t *rp = F + ((int64_t)f * a.nb + P) * 2 * BB * BB;
    const bf16_t *rq = F + ((int64_t)f * a.nb + P + h) * 2 * BB * BB;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int idx = lane + 64 * j;
      W.r[j] = *(const u32x4 *)(j < 4 ? rp + idx * 8 : rq + (idx - 256) * 8);
    }
  };
  // Stage into this wave's region: block i (0..3) as 32 rows of 64 bytes;
  // the forward reads rows (chunk XOR (row / 4) % 4 spreads a fragment
  // read's 32 rows over the banks), the backward reads columns with the
  // transpose read, which needs no swizzle at this row length.
  auto wstage = [&](const WReg &W) __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int idx = lane + 64 * j;
      const int blk = idx >> 7, row = (idx >> 2) & 31, c = idx & 3;
      const int sc = BWD ? c : (c ^ ((row >> 2) & 3));
      *(u32x4 *)(wst + blk * BLK_BYTES + row * 64 + (sc << 4)) = W.r[j];
    }
  };
  // MFMA operand (rows = 32 output features, 16 k of slice ks) of staged block blk.
  auto wfrag = [&](int blk, int ks) __attribute__((always_inline)) -> bf16x8 {
    const uint8_t *base = wst + blk * BLK_BYTES;
    if constexpr (!BWD) {
      // W(o, i) stored [n][k]: lane l reads row l % 32, 8 k at ks * 16 + (l / 32) * 8.
      const int r = lane & 31, c = ks * 2 + (lane >> 5);
      return *(const bf16x8 *)(base + r * 64 + ((c ^ ((r >> 2) & 3)) << 4));
    } else {
      // F(i, o) stored [k][n]: transpose read (lanes 4m..4m+3 of a 16-lane
      // group address k row m; lane j receives the 4 k of column j).
      const int g16 = lane >> 4, i = lane & 15;
      const int n = (g16 & 1) * 16 + (i & 3) * 4;
      const int kk = ks * 16 + (g16 >> 1) * 8 + (i >> 2);
      const int c = n >> 3, half = ((n >> 2) & 1) << 3;
      const s16x4 lo = tr16(base + kk * 64 + (c << 4) + half);
      const s16x4 hi = tr16(base + (kk + 4) * 64 + (c << 4) + half);
      const s16x8 v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
      return __builtin_bit_cast(bf16x8, v);
    }
  };
  // Token operand (rows = 32 tokens) of group-local block i, slice ks.
  auto xfrag = [&](int i, int ks) __attribute__((always_inline)) -> bf16x8 {
    return *(const bf16x8 *)act(lane & 31, i * 4 + ks * 2 + (lane >> 5));
  };
  // Accumulator of output block o (lane l: token l % 32, features 8 (e / 4)
  // + 4 (l / 32) + e % 4) to the activation tile, bf16.
  auto put = [&](int o, const f32x16 &acc) __attribute__((always_inline)) {
    const int m = lane & 31;
#pragma unroll
    for (int e4 = 0; e4 < 4; ++e4) {
      const u32x2 v = {pack_bf16x2(acc[4 * e4 + 0], acc[4 * e4 + 1]),
                       pack_bf16x2(acc[4 * e4 + 2], acc[4 * e4 + 3])};
      *(u32x2 *)(act(m, o * 4 + e4) + (lane >> 5) * 8) = v;
    }
  };
  auto process = [&](int f, int q, const WReg &W) __attribute__((always_inline)) {
    const int p = pair_row(f, q), qq = p + (1 << f);
    wstage(W);
    bf16x8 x[2][2];
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      x[0][ks] = xfrag(p, ks);
      x[1][ks] = xfrag(qq, ks);
    }
    f32x16 acc[2];
#pragma unroll
    for (int o = 0; o < 2; ++o) {
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[o][e] = 0.f;
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
          // Staged block order: W(p,p) W(p,q) W(q,p) W(q,q).  Forward output
          // o from input i uses W(o, i); backward output o from input i uses
          // F(i, o).
          const int blk = BWD ? 2 * i + o : 2 * o + i;
          acc[o] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wfrag(blk, ks), x[i][ks], acc[o], 0, 0, 0);
        }
    }
    put(p, acc[0]);
    put(qq, acc[1]);
  };

  bf16_t *save = (bf16_t *)a.save;
  const int64_t sld = (int64_t)L * a.n;
  const int total = L * nper;
  WReg WA, WB;
  auto factor_of = [&](int item) __attribute__((always_inline)) -> int {
    const int fi = item / nper;
    return BWD ? L - 1 - fi : fi;
  };
  if (total > 0) wload(factor_of(0), w, WA);
  __syncthreads();
  int item = 0;
  for (int fi = 0; fi < L; ++fi) {
    const int f = BWD ? L - 1 - fi : fi;
    if (save) {
      // Forward: the input of factor f; backward: the gradient at its output.
      copy_out(save, sld, (int64_t)f * a.n);
      __syncthreads();
    }
    for (int j = 0; j < nper; ++j, ++item) {
      const int q = w + NW * j;
      const bool more = item + 1 < total;
      const int fn = more ? factor_of(item + 1) : 0, qn = more ? w + NW * ((item + 1) % nper) : 0;
      if ((item & 1) == 0) {
        if (more) wload(fn, qn, WB);
        process(f, q, WA);
      } else {
        if (more) wload(fn, qn, WA);
        process(f, q, WB);
      }
    }
    __syncthreads();
  }
  copy_out((bf16_t *)a.out, a.n, 0);
}

}  // namespace

hipError_t launch_bfly(bool bwd, const BflyArgs &a, hipStream_t s) {
  if (a.k < 2 || a.k * BB > kBflyMaxGroupCols || a.nb % a.k || a.T < 1) return hipErrorInvalidValue;
  const int64_t grid = ((a.T + TM - 1) / TM) * (a.nb / a.k);
  if (grid <= 0 || grid > 0x7fffffff) return hipErrorInvalidValue;
  if (bwd)
    launch_kernel(bfly_kernel<true>, dim3((unsigned)grid), dim3(256), s, a);
  else
    launch_kernel(bfly_kernel<false>, dim3((unsigned)grid), dim3(256), s, a);
  return hipGetLastError();
}

}  // namespace pf
