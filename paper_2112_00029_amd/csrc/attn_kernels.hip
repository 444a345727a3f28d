// Block-sparse softmax attention for gfx950: 64 x 64 score blocks on the
// flat block butterfly mask, head dim 64, bf16 I/O, fp32 softmax/accumulate.
//
// Workgroup = 4 waves over one 64-row block (of queries for the forward and
// dQ, of keys for dK/dV); each wave owns 16 rows.  Everything is computed in
// transposed form so that each lane owns ONE row (its softmax statistics are
// per-lane scalars) and the probability tile feeds the next MFMA straight
// from registers:
//   forward : S^T = K_j Q_w^T (16x16x32 MFMA), online softmax per query,
//             O^T += V_j^T P^T.
//   dQ      : recompute S^T, P^T; dP^T = V_j dO_w^T; dS^T = P^T o (dP^T -
//             delta); dQ^T += K_j^T dS^T.
//   dK, dV  : S = Q_i K_w^T, P, dP = dO_i V_w^T, dS; dV^T += dO_i^T P,
//             dK^T += Q_i^T dS.
// The register tile of P (rows = 16 keys per MFMA output, 4 per lane) is
// used as a K-operand with keys in the order {16c + 4*(l/16) + 0..3} for two
// consecutive c; the matching operand is read from LDS with the transpose
// read in that same key order, so the contraction pairs up correctly.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <mutex>

#include "pf_launch.h"

namespace pf {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef short s16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint16_t bf16_t;
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));

constexpr int D = 64;       // head dim
constexpr int BQ = 64;      // block size
constexpr int LDK = D + 8;  // LDS row stride (elements)
constexpr int LDV = D + 16;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// 2^x on the hardware exponential unit (v_exp_f32): results below 2^-126
// flush toward zero, which a softmax probability can afford; saves the
// range-reduction sequence the library exp2f adds for denormal outputs.
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Wait for every global load of this wave (vmcnt 0; LDS counter too).
// Placed before a block loop whose first MFMAs use operands loaded ahead of
// it: otherwise the compiler's wait analysis, joining that path with the
// loop's back edge, can wait for the next tile's loads just issued at the
// top of the loop as well.
__device__ __forceinline__ void wait_loads() { __builtin_amdgcn_s_waitcnt(0x70); }

// x combined with the value of lane l ^ 16 (l ^ 32) by max or +: the two
// swaps exchange rows of 16 (halves of 32) lanes inside the VALU, where a
// lane shuffle would make a round trip through the LDS.  Each lane gets its
// own and its partner's value in some order, so max and + give the same bits
// in both lanes and as the shuffle form.
__device__ __forceinline__ float max_xor16(float x) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float max_xor32(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float add_xor16(float x) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float add_xor32(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

__device__ __forceinline__ float bf2f_a(bf16_t h) { return __uint_as_float(((uint32_t)h) << 16); }
__device__ __forceinline__ bf16_t f2bf_a(float f) { return __builtin_bit_cast(bf16_t, (__bf16)f); }

__device__ __forceinline__ int xcd_remap_a(int bid, int n) {
  constexpr int X = 8;
  int q = n / X, rem = n % X, x = bid % X, slot = bid / X;
  return x * q + min(x, rem) + slot;
}

__device__ __forceinline__ s16x4 tr16a(const bf16_t *p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) s16x4 *)(p));
}

// A-operand of a 16x16x32 MFMA, A[m][k] = tile[k][m] (tile stored [k][m],
// m contiguous), with k in the permuted order {kb + 4*(l/16) + 0..3} then
// {kb + 16 + 4*(l/16) + 0..3}; m = m0 + l % 16.
__device__ __forceinline__ bf16x8 fragA_tr_perm(const bf16_t *tile, int ld, int kb, int m0, int lane) {
  const int g = lane >> 4, i = lane & 15;
  const bf16_t *p = tile + (kb + g * 4 + (i >> 2)) * ld + m0 + (i & 3) * 4;
  s16x4 lo = tr16a(p), hi = tr16a(p + 16 * ld);
  s16x8 v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
  return __builtin_bit_cast(bf16x8, v);
}

// Operand of a 16x16x32 MFMA from a [row][k] tile: row r0 + l % 16,
// k = kb + (l/16)*8 + 0..7 (16-byte read).
__device__ __forceinline__ bf16x8 frag_rows(const bf16_t *tile, int ld, int r0, int kb, int lane) {
  return *(const bf16x8 *)(tile + (r0 + (lane & 15)) * ld + kb + (lane >> 4) * 8);
}

// Same from global memory.
__device__ __forceinline__ bf16x8 frag_rows_g(const bf16_t *p, int r0, int kb, int lane) {
  return *(const bf16x8 *)(p + (int64_t)(r0 + (lane & 15)) * D + kb + (lane >> 4) * 8);
}

// Pack a register tile (two 16-row MFMA outputs c0, c1) as the permuted
// K-operand.
__device__ __forceinline__ bf16x8 pack_perm(const f32x4 &c0, const f32x4 &c1) {
  bf16x8 v;
  v[0] = (__bf16)c0[0]; v[1] = (__bf16)c0[1]; v[2] = (__bf16)c0[2]; v[3] = (__bf16)c0[3];
  v[4] = (__bf16)c1[0]; v[5] = (__bf16)c1[1]; v[6] = (__bf16)c1[2]; v[7] = (__bf16)c1[3];
  return v;
}

#define MFMA16(a, b, c) __builtin_amdgcn_mfma_f32_16x16x32_bf16((a), (b), (c), 0, 0, 0)

// Cooperative load of a 64 x 64 bf16 tile (row stride D in global) into
// registers: 512 chunks of 16 bytes, two per thread.
struct Tile64 {
  u32x4 r0, r1;  // named fields: never addressed with a run-time index
  __device__ __forceinline__ void load(const bf16_t *g, int tid) {
    const int row = tid >> 3, c = (tid & 7) * 8;
    r0 = *(const u32x4 *)(g + row * D + c);
    r1 = *(const u32x4 *)(g + (row + 32) * D + c);
  }
  __device__ __forceinline__ void store(bf16_t *s, int ld, int tid) const {
    const int row = tid >> 3, c = (tid & 7) * 8;
    *(u32x4 *)(s + row * ld + c) = r0;
    *(u32x4 *)(s + (row + 32) * ld + c) = r1;
  }
};

// ---------------------------------------------------------------------------
// Work order: (head, block) of logical id L.  Block rows (or, for dK/dV,
// block columns) below nlong are the global stripes of the mask, which keep
// every block of the other side: they go first, over all heads, so that the
// long workgroups do not trail the launch; the rest follow head by head.
__device__ __forceinline__ void attn_order(int L, int BH, int nb, int nlong, int &bh, int &blk) {
  if (L < nlong * BH) {
    blk = L / BH;
    bh = L % BH;
  } else {
    const int r = L - nlong * BH, m = nb - nlong;
    bh = r / m;
    blk = nlong + r % m;
  }
}

// Forward
// ---------------------------------------------------------------------------
// NG groups of 4 waves share one 64-query block: group g takes the row's
// kept blocks g, g + NG, ... (each group has its own double-buffered K/V
// tiles; all groups run the same number of iterations so every barrier is
// reached by the whole workgroup) and the groups' softmax states (reference,
// sum, unnormalised O) are merged through LDS in group order at the end.
// NG = 1 is the plain kernel; NG = 4 serves the long rows of global stripes.
template <int NG>
__global__ __launch_bounds__(256 * NG) void attn_fwd_kernel(AttnArgs a) {
  __shared__ __attribute__((aligned(16))) bf16_t Ks[NG][2][BQ * LDK];
  __shared__ __attribute__((aligned(16))) bf16_t Vs[NG][2][BQ * LDV];

  const int tid = threadIdx.x & 255, lane = tid & 63, wave = tid >> 6;
  const int grp = NG > 1 ? __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 8) : 0;
  const int bid = xcd_remap_a(blockIdx.x, gridDim.x) + a.first;
  int bh, qb;
  attn_order(bid, a.BH, a.nbq, a.nlong, bh, qb);
  const int64_t head = (int64_t)bh * a.S * D;
  const bf16_t *Q = (const bf16_t *)a.Q + head;
  const bf16_t *K = (const bf16_t *)a.K + head;
  const bf16_t *V = (const bf16_t *)a.V + head;
  const int q0 = qb * BQ + wave * 16;
  const float c = a.scale * kLog2e;

  bf16x8 qf[2];
  qf[0] = frag_rows_g(Q, q0, 0, lane);
  qf[1] = frag_rows_g(Q, q0, 32, lane);

  const int p0 = a.row_ptr[qb], p1 = a.row_ptr[qb + 1];
  const int iters = (p1 - p0 + NG - 1) / NG;
  float m_run = -INFINITY, l_run = 0.f;
  f32x4 o[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) o[i] = f32x4{0.f, 0.f, 0.f, 0.f};

  Tile64 tk, tv;
  if (p0 + grp < p1) {
    tk.load(K + (int64_t)a.col_idx[p0 + grp] * BQ * D, tid);
    tv.load(V + (int64_t)a.col_idx[p0 + grp] * BQ * D, tid);
    tk.store(Ks[grp][0], LDK, tid);
    tv.store(Vs[grp][0], LDV, tid);
  }
  // Block column of this group's next tile, loaded one iteration ahead so
  // that the tile loads do not wait on it (clamped into the row, which is
  // never empty; unused past its end).
  int cn = a.col_idx[min(p0 + grp + NG, p1 - 1)];
  wait_loads();
  __syncthreads();

  for (int it = 0; it < iters; ++it) {
    const int cur = it & 1;
    const int p = p0 + it * NG + grp;
    const bool valid = p < p1, next = p + NG < p1;
    if (next) {
      tk.load(K + (int64_t)cn * BQ * D, tid);
      tv.load(V + (int64_t)cn * BQ * D, tid);
    }
    cn = a.col_idx[min(p + 2 * NG, p1 - 1)];
    if (valid) {
      // S^T[key][query] for 64 keys x this wave's 16 queries.
      f32x4 s[4];
#pragma unroll
      for (int mt = 0; mt < 4; ++mt) {
        s[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
        s[mt] = MFMA16(frag_rows(Ks[grp][cur], LDK, mt * 16, 0, lane), qf[0], s[mt]);
        s[mt] = MFMA16(frag_rows(Ks[grp][cur], LDK, mt * 16, 32, lane), qf[1], s[mt]);
      }
      float bmax = -INFINITY;
#pragma unroll
      for (int mt = 0; mt < 4; ++mt)
#pragma unroll
        for (int j = 0; j < 4; ++j) bmax = fmaxf(bmax, s[mt][j]);
      bmax = max_xor32(max_xor16(bmax));
      // The softmax reference m_run moves only when some row's maximum grew
      // by more than 8 (log2 units): until then the probabilities stay below
      // 2^8 and the rescale of O and l, a wave-uniform branch, is skipped.
      const float m_cand = fmaxf(m_run, bmax * c);
      if (__builtin_amdgcn_ballot_w64(m_cand > m_run + 8.0f)) {
        const float alpha = fast_exp2(m_run - m_cand);
        m_run = m_cand;
        l_run *= alpha;
#pragma unroll
        for (int dt = 0; dt < 4; ++dt)
#pragma unroll
          for (int j = 0; j < 4; ++j) o[dt][j] *= alpha;
      }
      float rs = 0.f;
#pragma unroll
      for (int mt = 0; mt < 4; ++mt)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          float e = fast_exp2(s[mt][j] * c - m_run);
          s[mt][j] = e;
          rs += e;
        }
      rs = add_xor32(add_xor16(rs));
      l_run += rs;
      // O^T[dim][query] += V^T[dim][key] P^T[key][query]
      const bf16x8 pb0 = pack_perm(s[0], s[1]), pb1 = pack_perm(s[2], s[3]);
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) {
        o[dt] = MFMA16(fragA_tr_perm(Vs[grp][cur], LDV, 0, dt * 16, lane), pb0, o[dt]);
        o[dt] = MFMA16(fragA_tr_perm(Vs[grp][cur], LDV, 32, dt * 16, lane), pb1, o[dt]);
      }
    }
    if (next) {
      tk.store(Ks[grp][cur ^ 1], LDK, tid);
      tv.store(Vs[grp][cur ^ 1], LDV, tid);
    }
    __syncthreads();
  }

  if constexpr (NG > 1) {
    // Merge: groups 1.. leave (m, l, o) per lane in their K tiles (18 floats
    // x 64 lanes x 4 waves = exactly one group's K tiles), group 0 combines
    // them relative to the largest reference.  A group without blocks has
    // m = -inf and contributes 0.
    float *mrg = (float *)&Ks[grp][0][0] + wave * (18 * 64) + lane;
    if (grp > 0) {
      mrg[0] = m_run;
      mrg[64] = l_run;
#pragma unroll
      for (int dt = 0; dt < 4; ++dt)
#pragma unroll
        for (int j = 0; j < 4; ++j) mrg[(2 + dt * 4 + j) * 64] = o[dt][j];
    }
    __syncthreads();
    if (grp > 0) return;
    float m = m_run;
#pragma unroll
    for (int g = 1; g < NG; ++g) m = fmaxf(m, ((float *)&Ks[g][0][0])[wave * (18 * 64) + lane]);
    const float s0 = fast_exp2(m_run - m);
    l_run *= s0;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
      for (int j = 0; j < 4; ++j) o[dt][j] *= s0;
#pragma unroll
    for (int g = 1; g < NG; ++g) {
      const float *src = (const float *)&Ks[g][0][0] + wave * (18 * 64) + lane;
      const float sg = src[0] == -INFINITY ? 0.f : fast_exp2(src[0] - m);
      l_run += src[64] * sg;
#pragma unroll
      for (int dt = 0; dt < 4; ++dt)
#pragma unroll
        for (int j = 0; j < 4; ++j) o[dt][j] += src[(2 + dt * 4 + j) * 64] * sg;
    }
    m_run = m;
  }

  const float inv = 1.f / l_run;
  const int q = q0 + (lane & 15);
  bf16_t *O = (bf16_t *)a.Oout + head + (int64_t)q * D;
#pragma unroll
  for (int dt = 0; dt < 4; ++dt) {
    u32x2 w;
    w[0] = (uint32_t)f2bf_a(o[dt][0] * inv) | ((uint32_t)f2bf_a(o[dt][1] * inv) << 16);
    w[1] = (uint32_t)f2bf_a(o[dt][2] * inv) | ((uint32_t)f2bf_a(o[dt][3] * inv) << 16);
    *(u32x2 *)(O + dt * 16 + (lane >> 4) * 4) = w;
  }
  if (lane < 16) a.lse[(int64_t)bh * a.S + q] = (m_run + __log2f(l_run)) * kLn2;
}

// ---------------------------------------------------------------------------
// Backward, pass 1: delta and dQ (one workgroup per query block)
// ---------------------------------------------------------------------------
// NG groups of 4 waves split the row's kept blocks as in the forward; their
// dQ partial sums are added through LDS in group order.
template <int NG>
__global__ __launch_bounds__(256 * NG) void attn_bwd_dq_kernel(AttnArgs a) {
  __shared__ __attribute__((aligned(16))) bf16_t Ks[NG][2][BQ * LDK];
  __shared__ __attribute__((aligned(16))) bf16_t Vs[NG][2][BQ * LDK];

  const int tid = threadIdx.x & 255, lane = tid & 63, wave = tid >> 6;
  const int grp = NG > 1 ? __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 8) : 0;
  const int bid = xcd_remap_a(blockIdx.x, gridDim.x) + a.first;
  int bh, qb;
  attn_order(bid, a.BH, a.nbq, a.nlong, bh, qb);
  const int64_t head = (int64_t)bh * a.S * D;
  const bf16_t *Q = (const bf16_t *)a.Q + head;
  const bf16_t *K = (const bf16_t *)a.K + head;
  const bf16_t *V = (const bf16_t *)a.V + head;
  const bf16_t *O = (const bf16_t *)a.O + head;
  const bf16_t *dO = (const bf16_t *)a.dO + head;
  const int q0 = qb * BQ + wave * 16;
  const int q = q0 + (lane & 15);
  const float c = a.scale * kLog2e;

  bf16x8 qf[2], dof[2];
  qf[0] = frag_rows_g(Q, q0, 0, lane);
  qf[1] = frag_rows_g(Q, q0, 32, lane);
  dof[0] = frag_rows_g(dO, q0, 0, lane);
  dof[1] = frag_rows_g(dO, q0, 32, lane);

  // delta = rowsum(dO o O): lane covers dims (l/16)*16 .. +15 of query q.
  float delta = 0.f;
  {
    const bf16_t *po = O + (int64_t)q * D + (lane >> 4) * 16;
    const bf16_t *pd = dO + (int64_t)q * D + (lane >> 4) * 16;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const u32x4 vo = *(const u32x4 *)(po + h * 8), vd = *(const u32x4 *)(pd + h * 8);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        delta += __uint_as_float(vo[e] << 16) * __uint_as_float(vd[e] << 16);
        delta += __uint_as_float(vo[e] & 0xffff0000u) * __uint_as_float(vd[e] & 0xffff0000u);
      }
    }
    delta += __shfl_xor(delta, 16);
    delta += __shfl_xor(delta, 32);
  }
  if (lane < 16 && grp == 0) a.delta[(int64_t)bh * a.S + q] = delta;
  const float lse2 = a.lse_in[(int64_t)bh * a.S + q] * kLog2e;

  const int p0 = a.row_ptr[qb], p1 = a.row_ptr[qb + 1];
  const int iters = (p1 - p0 + NG - 1) / NG;
  f32x4 dq[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) dq[i] = f32x4{0.f, 0.f, 0.f, 0.f};

  Tile64 tk, tv;
  if (p0 + grp < p1) {
    tk.load(K + (int64_t)a.col_idx[p0 + grp] * BQ * D, tid);
    tv.load(V + (int64_t)a.col_idx[p0 + grp] * BQ * D, tid);
    tk.store(Ks[grp][0], LDK, tid);
    tv.store(Vs[grp][0], LDK, tid);
  }
  // Next block column one iteration ahead, as in the forward.
  int cn = a.col_idx[min(p0 + grp + NG, p1 - 1)];
  __syncthreads();

  for (int it = 0; it < iters; ++it) {
    const int cur = it & 1;
    const int p = p0 + it * NG + grp;
    const bool valid = p < p1, next = p + NG < p1;
    if (next) {
      tk.load(K + (int64_t)cn * BQ * D, tid);
      tv.load(V + (int64_t)cn * BQ * D, tid);
    }
    cn = a.col_idx[min(p + 2 * NG, p1 - 1)];
    if (valid) {
    f32x4 s[4], dp[4];
#pragma unroll
    for (int mt = 0; mt < 4; ++mt) {
      s[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
      s[mt] = MFMA16(frag_rows(Ks[grp][cur], LDK, mt * 16, 0, lane), qf[0], s[mt]);
      s[mt] = MFMA16(frag_rows(Ks[grp][cur], LDK, mt * 16, 32, lane), qf[1], s[mt]);
      dp[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
      dp[mt] = MFMA16(frag_rows(Vs[grp][cur], LDK, mt * 16, 0, lane), dof[0], dp[mt]);
      dp[mt] = MFMA16(frag_rows(Vs[grp][cur], LDK, mt * 16, 32, lane), dof[1], dp[mt]);
    }
#pragma unroll
    for (int mt = 0; mt < 4; ++mt)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        float pr = fast_exp2(s[mt][j] * c - lse2);
        s[mt][j] = pr * (dp[mt][j] - delta);  // dS^T
      }
    const bf16x8 d0 = pack_perm(s[0], s[1]), d1 = pack_perm(s[2], s[3]);
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) {
      dq[dt] = MFMA16(fragA_tr_perm(Ks[grp][cur], LDK, 0, dt * 16, lane), d0, dq[dt]);
      dq[dt] = MFMA16(fragA_tr_perm(Ks[grp][cur], LDK, 32, dt * 16, lane), d1, dq[dt]);
    }
    }
    if (next) {
      tk.store(Ks[grp][cur ^ 1], LDK, tid);
      tv.store(Vs[grp][cur ^ 1], LDK, tid);
    }
    __syncthreads();
  }

  if constexpr (NG > 1) {
    // Groups 1.. leave their 16 partial sums per lane in their K tiles;
    // group 0 adds them in group order.
    float *mrg = (float *)&Ks[grp][0][0] + wave * (16 * 64) + lane;
    if (grp > 0) {
#pragma unroll
      for (int dt = 0; dt < 4; ++dt)
#pragma unroll
        for (int j = 0; j < 4; ++j) mrg[(dt * 4 + j) * 64] = dq[dt][j];
    }
    __syncthreads();
    if (grp > 0) return;
#pragma unroll
    for (int g = 1; g < NG; ++g) {
      const float *src = (const float *)&Ks[g][0][0] + wave * (16 * 64) + lane;
#pragma unroll
      for (int dt = 0; dt < 4; ++dt)
#pragma unroll
        for (int j = 0; j < 4; ++j) dq[dt][j] += src[(dt * 4 + j) * 64];
    }
  }

  bf16_t *dQ = (bf16_t *)a.dQ + head + (int64_t)q * D;
#pragma unroll
  for (int dt = 0; dt < 4; ++dt) {
    u32x2 w;
    w[0] = (uint32_t)f2bf_a(dq[dt][0] * a.scale) | ((uint32_t)f2bf_a(dq[dt][1] * a.scale) << 16);
    w[1] = (uint32_t)f2bf_a(dq[dt][2] * a.scale) | ((uint32_t)f2bf_a(dq[dt][3] * a.scale) << 16);
    *(u32x2 *)(dQ + dt * 16 + (lane >> 4) * 4) = w;
  }
}

// ---------------------------------------------------------------------------
// Backward, pass 2: dK and dV (one workgroup per key block)
// ---------------------------------------------------------------------------
// NG groups of 4 waves split the column's kept blocks as in the forward;
// their dK and dV partial sums are added through LDS in group order.
template <int NG>
__global__ __launch_bounds__(256 * NG) void attn_bwd_dkv_kernel(AttnArgs a) {
  __shared__ __attribute__((aligned(16))) bf16_t Qs[NG][2][BQ * LDK];
  __shared__ __attribute__((aligned(16))) bf16_t dOs[NG][2][BQ * LDK];
  __shared__ float ls[NG][2][BQ], ds[NG][2][BQ];

  const int tid = threadIdx.x & 255, lane = tid & 63, wave = tid >> 6;
  const int grp = NG > 1 ? __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 8) : 0;
  const int bid = xcd_remap_a(blockIdx.x, gridDim.x) + a.first;
  int bh, kb;
  attn_order(bid, a.BH, a.nbq, a.nlong, bh, kb);
  const int64_t head = (int64_t)bh * a.S * D;
  const bf16_t *Q = (const bf16_t *)a.Q + head;
  const bf16_t *K = (const bf16_t *)a.K + head;
  const bf16_t *V = (const bf16_t *)a.V + head;
  const bf16_t *dO = (const bf16_t *)a.dO + head;
  const float *lse = a.lse_in + (int64_t)bh * a.S;
  const float *dl = a.delta + (int64_t)bh * a.S;
  const int k0 = kb * BQ + wave * 16;
  const float c = a.scale * kLog2e;

  bf16x8 kf[2], vf[2];
  kf[0] = frag_rows_g(K, k0, 0, lane);
  kf[1] = frag_rows_g(K, k0, 32, lane);
  vf[0] = frag_rows_g(V, k0, 0, lane);
  vf[1] = frag_rows_g(V, k0, 32, lane);

  const int p0 = a.col_ptr[kb], p1 = a.col_ptr[kb + 1];
  f32x4 dk[4], dv[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    dk[i] = f32x4{0.f, 0.f, 0.f, 0.f};
    dv[i] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  if (p0 < p1) {  // a key block no query attends keeps zero gradients

  Tile64 tq, td;
  float rl = 0.f, rd = 0.f;
  auto gload = [&](int p) {
    const int64_t qrow = (int64_t)a.row_idx[p] * BQ;
    tq.load(Q + qrow * D, tid);
    td.load(dO + qrow * D, tid);
    // Raw values: scaling here would make the wave wait for the load.
    if (tid < BQ) { rl = lse[qrow + tid]; rd = dl[qrow + tid]; }
  };
  auto sstore = [&](int buf) {
    tq.store(Qs[grp][buf], LDK, tid);
    td.store(dOs[grp][buf], LDK, tid);
    if (tid < BQ) { ls[grp][buf][tid] = rl * kLog2e; ds[grp][buf][tid] = rd; }
  };
  const int iters = (p1 - p0 + NG - 1) / NG;
  if (p0 + grp < p1) {
    gload(p0 + grp);
    sstore(0);
  }
  __syncthreads();

  for (int it = 0; it < iters; ++it) {
    const int cur = it & 1;
    const int p = p0 + it * NG + grp;
    const bool valid = p < p1, next = p + NG < p1;
    if (next) gload(p + NG);
    if (valid) {
    // S[query][key], dP[query][key] for 64 queries x this wave's 16 keys.
    f32x4 s[4], dp[4];
#pragma unroll
    for (int mt = 0; mt < 4; ++mt) {
      s[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
      s[mt] = MFMA16(frag_rows(Qs[grp][cur], LDK, mt * 16, 0, lane), kf[0], s[mt]);
      s[mt] = MFMA16(frag_rows(Qs[grp][cur], LDK, mt * 16, 32, lane), kf[1], s[mt]);
      dp[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
      dp[mt] = MFMA16(frag_rows(dOs[grp][cur], LDK, mt * 16, 0, lane), vf[0], dp[mt]);
      dp[mt] = MFMA16(frag_rows(dOs[grp][cur], LDK, mt * 16, 32, lane), vf[1], dp[mt]);
    }
#pragma unroll
    for (int mt = 0; mt < 4; ++mt)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int qi = mt * 16 + (lane >> 4) * 4 + j;
        const float pr = fast_exp2(s[mt][j] * c - ls[grp][cur][qi]);
        s[mt][j] = pr;
        dp[mt][j] = pr * (dp[mt][j] - ds[grp][cur][qi]);  // dS
      }
    const bf16x8 pb0 = pack_perm(s[0], s[1]), pb1 = pack_perm(s[2], s[3]);
    const bf16x8 sb0 = pack_perm(dp[0], dp[1]), sb1 = pack_perm(dp[2], dp[3]);
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) {
      dv[dt] = MFMA16(fragA_tr_perm(dOs[grp][cur], LDK, 0, dt * 16, lane), pb0, dv[dt]);
      dv[dt] = MFMA16(fragA_tr_perm(dOs[grp][cur], LDK, 32, dt * 16, lane), pb1, dv[dt]);
      dk[dt] = MFMA16(fragA_tr_perm(Qs[grp][cur], LDK, 0, dt * 16, lane), sb0, dk[dt]);
      dk[dt] = MFMA16(fragA_tr_perm(Qs[grp][cur], LDK, 32, dt * 16, lane), sb1, dk[dt]);
    }
    }
    if (next) sstore(cur ^ 1);
    __syncthreads();
  }
  }

  if constexpr (NG > 1) {
    // Groups 1.. leave their 32 partial sums per lane in their Q and dO
    // tiles; group 0 adds them in group order.  (The key block's kept-block
    // count is workgroup-uniform, so every thread reaches this barrier.)
    float *mk = (float *)&Qs[grp][0][0] + wave * (16 * 64) + lane;
    float *mv = (float *)&dOs[grp][0][0] + wave * (16 * 64) + lane;
    if (grp > 0) {
#pragma unroll
      for (int dt = 0; dt < 4; ++dt)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          mk[(dt * 4 + j) * 64] = dk[dt][j];
          mv[(dt * 4 + j) * 64] = dv[dt][j];
        }
    }
    __syncthreads();
    if (grp > 0) return;
#pragma unroll
    for (int g = 1; g < NG; ++g) {
      const float *sk = (const float *)&Qs[g][0][0] + wave * (16 * 64) + lane;
      const float *sv = (const float *)&dOs[g][0][0] + wave * (16 * 64) + lane;
#pragma unroll
      for (int dt = 0; dt < 4; ++dt)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          dk[dt][j] += sk[(dt * 4 + j) * 64];
          dv[dt][j] += sv[(dt * 4 + j) * 64];
        }
    }
  }

  const int key = k0 + (lane & 15);
  bf16_t *dK = (bf16_t *)a.dK + head + (int64_t)key * D;
  bf16_t *dV = (bf16_t *)a.dV + head + (int64_t)key * D;
#pragma unroll
  for (int dt = 0; dt < 4; ++dt) {
    u32x2 w;
    w[0] = (uint32_t)f2bf_a(dk[dt][0] * a.scale) | ((uint32_t)f2bf_a(dk[dt][1] * a.scale) << 16);
    w[1] = (uint32_t)f2bf_a(dk[dt][2] * a.scale) | ((uint32_t)f2bf_a(dk[dt][3] * a.scale) << 16);
    *(u32x2 *)(dK + dt * 16 + (lane >> 4) * 4) = w;
    w[0] = (uint32_t)f2bf_a(dv[dt][0]) | ((uint32_t)f2bf_a(dv[dt][1]) << 16);
    w[1] = (uint32_t)f2bf_a(dv[dt][2]) | ((uint32_t)f2bf_a(dv[dt][3]) << 16);
    *(u32x2 *)(dV + dt * 16 + (lane >> 4) * 4) = w;
  }
}

// Launchers.  part 0: every block row (column) with the plain kernel;
// part 1: the nlong global rows (columns) of every head with the grouped
// kernel; part 2: the remaining rows with the plain kernel.
namespace {
template <typename F1, typename FG>
hipError_t attn_launch(F1 plain, FG grouped, int ng, AttnArgs a, int part, hipStream_t s) {
  int64_t grid;
  if (part == 1) {
    grid = (int64_t)a.BH * a.nlong;
    a.first = 0;
  } else if (part == 2) {
    grid = (int64_t)a.BH * (a.nbq - a.nlong);
    a.first = a.BH * a.nlong;
  } else {
    grid = (int64_t)a.BH * a.nbq;
    a.first = 0;
  }
  if (grid <= 0 || grid > 0x7fffffff) return hipErrorInvalidValue;
  if (part == 1)
    launch_kernel(grouped, dim3((unsigned)grid), dim3(256 * ng), s, a);
  else
    launch_kernel(plain, dim3((unsigned)grid), dim3(256), s, a);
  return hipGetLastError();
}
}  // namespace

hipError_t launch_attn_fwd(const AttnArgs &a, int part, hipStream_t s) {
  return attn_launch(attn_fwd_kernel<1>, attn_fwd_kernel<4>, 4, a, part, s);
}

hipError_t launch_attn_bwd_dq(const AttnArgs &a, int part, hipStream_t s) {
  return attn_launch(attn_bwd_dq_kernel<1>, attn_bwd_dq_kernel<4>, 4, a, part, s);
}

hipError_t launch_attn_bwd_dkv(const AttnArgs &a, int part, hipStream_t s) {
  return attn_launch(attn_bwd_dkv_kernel<1>, attn_bwd_dkv_kernel<2>, 2, a, part, s);
}

// Scratch of the allocation-free attention backward: the row terms delta,
// one float per query row of the call (kAttnScratchRows at most).  Each GPU
// the library runs on holds its own copy until the process ends.  In host
// code `scratch` names a host-side stand-in, not device memory: only the
// address attn_scratch returns may reach a kernel.
static __device__ __align__(256) float scratch[kAttnScratchRows];

hipError_t attn_scratch(float **ptr) {
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static void *addr[kMaxDevices] = {};
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lk(mu);
  if (!addr[dev]) {
    // Once per device, with that device current: its copy of the array.
    void *p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    addr[dev] = p;
  }
  *ptr = (float *)addr[dev];
  return hipSuccess;
}

}  // namespace pf
