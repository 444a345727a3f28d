// Block-sparse GEMM kernels for gfx950 (CDNA4): bf16 (or fp32) operands,
// fp32 accumulation on MFMA.
//
//  nt_kernel  C[T x n] = A[T x k] . B^T restricted to kept blocks, plus an
//             optional low-rank term L . R^T fused into the same K-loop.
//             Forward:        A = X,  B = packed W blocks (stored [n][k]),
//                             low-rank T_lr . U^T.
//             Backward-data:  A = dY, B = packed W blocks read as [k][n]
//                             (the transposed layout), low-rank S . V.
//             Dense mode (comparator and the skinny rank-r products): the
//             K-steps run over every block of a dense B.
//  tn_kernel  out = A^T . B reduced over tokens, only for kept blocks
//             (weight gradient restricted to the mask) plus dense regions
//             (dU = dY^T T_lr, dV = S^T X).  Token range may be split across
//             workgroups; partials are combined in split order by the last
//             workgroup to finish an item (deterministic).
//
// Tiles: 256 threads = 4 waves of 64.  Operands stream global -> registers
// -> LDS (double-buffered, one barrier per K-step of 32).  MFMA fragments
// are read from LDS with 16-byte reads ([row][k] tiles) or with the gfx950
// transpose read ds_read_b64_tr_b16 ([k][row] tiles): within each group of
// 16 lanes, lanes 4m..4m+3 address row m (4 x 16-bit each) of a 4 x 16
// tile and lane j receives column j, i.e. 4 consecutive k of one row.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>
#include <type_traits>

#include "pf_internal.h"

namespace pf {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef short s16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

typedef uint16_t bf16_t;  // bfloat16 storage
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));  // 16-byte chunk

__device__ unsigned int g_tn_counters[kMaxCounters];

__device__ __forceinline__ float bf2f(bf16_t h) {
  return __uint_as_float(((uint32_t)h) << 16);
}
__device__ __forceinline__ bf16_t f2bf(float f) {
  __bf16 h = (__bf16)f;  // round to nearest even
  return __builtin_bit_cast(bf16_t, h);
}
template <typename T>
__device__ __forceinline__ float to_f(T v) {
  if constexpr (std::is_same<T, float>::value) return v; else return bf2f(v);
}
template <typename T>
__device__ __forceinline__ T from_f(float v) {
  if constexpr (std::is_same<T, float>::value) return v; else return f2bf(v);
}

__device__ __forceinline__ float gelu_f(float x) {
  return 0.5f * x * (1.0f + erff(x * 0.70710678118654752f));
}
__device__ __forceinline__ float gelu_grad_f(float x) {
  float Phi = 0.5f * (1.0f + erff(x * 0.70710678118654752f));
  float phi = 0.39894228040143268f * __expf(-0.5f * x * x);
  return Phi + x * phi;
}

// Workgroups are dispatched round-robin over the 8 XCDs; remap so that
// consecutive logical ids run on the same XCD (and share its L2).
__device__ __forceinline__ int xcd_remap(int bid, int n) {
  constexpr int X = 8;
  int q = n / X, rem = n % X, x = bid % X, slot = bid / X;
  return x * q + min(x, rem) + slot;
}

__device__ __forceinline__ s16x4 tr16(const bf16_t *p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) s16x4 *)(p));
}

__device__ __forceinline__ bf16x8 cat8(s16x4 lo, s16x4 hi) {
  s16x8 v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
  return __builtin_bit_cast(bf16x8, v);
}

// MFMA fragment of a 32-row operand stored [k][row] in LDS (row
// contiguous): lane l gets row (l % 32), k = ks*16 + (l / 32)*8 + 0..7.
__device__ __forceinline__ bf16x8 frag_kmajor(const bf16_t *base, int ld,
                                              int ks, int row0, int lane) {
  int g16 = lane >> 4, i = lane & 15;
  int n0 = (g16 & 1) * 16, kb = (g16 >> 1) * 8;
  const bf16_t *p = base + (ks * 16 + kb + (i >> 2)) * ld + row0 + n0 + (i & 3) * 4;
  return cat8(tr16(p), tr16(p + 4 * ld));
}

// MFMA fragment of a 32-row operand stored [row][k] in LDS.
__device__ __forceinline__ bf16x8 frag_rmajor(const bf16_t *base, int ld,
                                              int ks, int row0, int lane) {
  return *(const bf16x8 *)(base + (row0 + (lane & 31)) * ld + ks * 16 +
                           (lane >> 5) * 8);
}

// Compile-time loop: f(std::integral_constant<int, i>) for i in [0, N), so
// that register arrays are indexed by constants from the start.
template <int I, int N, typename F>
__device__ __forceinline__ void static_for_impl(F &&f) {
  if constexpr (I < N) {
    f(std::integral_constant<int, I>{});
    static_for_impl<I + 1, N>(f);
  }
}
template <int N, typename F>
__device__ __forceinline__ void static_for(F &&f) {
  static_for_impl<0, N>(f);
}

__device__ __forceinline__ int uniform(int v) { return __builtin_amdgcn_readfirstlane(v); }

// Up to 8 staged 16-byte chunks in named registers (struct fields, unlike
// array elements, cannot be addressed with a run-time index, so they always
// stay in VGPRs).
struct Stage8 {
  u32x4 r0, r1, r2, r3, r4, r5, r6, r7;
  template <int I>
  __device__ __forceinline__ u32x4 &at() {
    static_assert(I >= 0 && I < 8, "stage index");
    if constexpr (I == 0) return r0;
    else if constexpr (I == 1) return r1;
    else if constexpr (I == 2) return r2;
    else if constexpr (I == 3) return r3;
    else if constexpr (I == 4) return r4;
    else if constexpr (I == 5) return r5;
    else if constexpr (I == 6) return r6;
    else return r7;
  }
};

// ---------------------------------------------------------------------------
// NT kernel
// ---------------------------------------------------------------------------
template <typename T, int BLK, int G, bool BKN>
__global__ __launch_bounds__(256) void nt_kernel(NTArgs a) {
  constexpr bool BF = std::is_same<T, bf16_t>::value;
  constexpr int BM = 128, BK = 32, BN = G * BLK;
  constexpr int KSUB = BLK / BK;
  constexpr int VEC = 16 / (int)sizeof(T);
  constexpr int PADA = BF ? 8 : 4;
  constexpr int LDA_S = BK + PADA;
  constexpr int LDB_S = BKN ? (BN + (BF ? 16 : 4)) : (BK + PADA);
  constexpr int A_ELEMS = BM * LDA_S;
  constexpr int B_ELEMS = BKN ? BK * LDB_S : BN * LDB_S;
  constexpr int WN = BN >= 64 ? 2 : 1, WM = 4 / WN;
  constexpr int WTM = BM / WM, WTN = BN / WN;
  constexpr int TM = WTM / 32, TN = WTN / 32;
  constexpr int A_CH = BM * BK / VEC;
  constexpr int CPB = BLK * BK / VEC;  // 16-byte chunks of one block's K-slice
  constexpr int B_CH = G * CPB;
  constexpr int A_LD = A_CH / 256, B_LD = (B_CH + 255) / 256;
  static_assert(A_CH % 256 == 0, "A tile chunks");
  static_assert(CPB % 64 == 0, "a wave's chunks must lie in one block");
  static_assert(TM >= 1 && TN >= 1, "wave tile");

  __shared__ __attribute__((aligned(16))) T smem[2 * (A_ELEMS + B_ELEMS)];

  const T *__restrict__ A = (const T *)a.A;
  const T *__restrict__ B = (const T *)a.B;
  const T *__restrict__ L = (const T *)a.L;
  const T *__restrict__ R = (const T *)a.R;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = uniform(tid >> 6);
  const int wm = wave / WN, wn = wave % WN;
  const int ntn = a.ntiles;
  const int bid = xcd_remap(blockIdx.x, gridDim.x);
  const int mt = bid / ntn, nt = bid % ntn;
  const int64_t m0 = (int64_t)mt * BM;

  int g_valid, nsteps, kcol_off = 0, blk_off = 0;
  const NTTile *tile = a.dense ? nullptr : a.tiles + nt;
  if (a.dense) {
    g_valid = min(G, a.dense_nblk - nt * G);
    nsteps = a.dense_nsteps;
  } else {
    g_valid = tile->g;
    nsteps = tile->nsteps;
    kcol_off = tile->kcol_off;
    blk_off = tile->blk_off;
  }
  // Output block of tile row g (g wave-uniform).
  auto out_blk = [&](int g) __attribute__((always_inline)) -> int {
    return a.dense ? nt * G + min(g, g_valid - 1) : tile->out_blk[g];
  };
  const int total = (nsteps + a.nlr) * KSUB;

  // Base pointer of the B operand slice of step s for tile row g.
  auto b_base = [&](int s, int g, int64_t &ldb_s) __attribute__((always_inline)) -> const T * {
    const int c = s / KSUB, kk = (s % KSUB) * BK;
    if (c < nsteps) {
      if (a.dense) {
        ldb_s = a.ldb;
        const int64_t ob = out_blk(g);
        return BKN ? B + ((int64_t)c * BLK + kk) * a.ldb + ob * BLK
                   : B + (ob * BLK) * a.ldb + (int64_t)c * BLK + kk;
      }
      ldb_s = BLK;
      const int64_t blk = a.blks[blk_off + c * G + g];
      return B + blk * (BLK * BLK) + (BKN ? kk * BLK : kk);
    }
    const int cr = c - nsteps;
    const int64_t ob = out_blk(g);
    ldb_s = a.ldr;
    return BKN ? R + ((int64_t)cr * BLK + kk) * a.ldr + ob * BLK
               : R + (ob * BLK) * a.ldr + (int64_t)cr * BLK + kk;
  };
  auto a_base = [&](int s, int64_t &lda_s) __attribute__((always_inline)) -> const T * {
    const int c = s / KSUB, kk = (s % KSUB) * BK;
    if (c < nsteps) {
      const int kcol = a.dense ? c : a.kcols[kcol_off + c];
      lda_s = a.lda;
      return A + (int64_t)kcol * BLK + kk;
    }
    lda_s = a.ldl;
    return L + (int64_t)(c - nsteps) * BLK + kk;
  };

  static_assert(A_LD <= 8 && B_LD <= 8, "staging registers");
  Stage8 ra, rb;
  auto gload = [&](int s) __attribute__((always_inline)) {
    int64_t lda_s;
    const T *ap = a_base(s, lda_s);
    static_for<A_LD>([&](auto i) __attribute__((always_inline)) {
      const int id = tid + i * 256;
      const int row = id / (BK / VEC), cv = id % (BK / VEC);
      const int64_t gm = m0 + row;
      ra.template at<i>() = gm < a.M ? *(const u32x4 *)(ap + gm * lda_s + cv * VEC) : u32x4{0u, 0u, 0u, 0u};
    });
    static_for<B_LD>([&](auto i) __attribute__((always_inline)) {
      const int id = tid + i * 256;
      if (i * 256 + 256 <= B_CH || id < B_CH) {
        const int g = uniform(id / CPB), r = id % CPB;
        int64_t ldb_s;
        const T *bp = b_base(s, g, ldb_s);
        if (!BKN) {
          const int n = r / (BK / VEC), cv = r % (BK / VEC);
          rb.template at<i>() = *(const u32x4 *)(bp + (int64_t)n * ldb_s + cv * VEC);
        } else {
          const int k = r / (BLK / VEC), nv = r % (BLK / VEC);
          rb.template at<i>() = *(const u32x4 *)(bp + (int64_t)k * ldb_s + nv * VEC);
        }
      }
    });
  };
  auto sstore = [&](int buf) __attribute__((always_inline)) {
    T *As = smem + buf * (A_ELEMS + B_ELEMS);
    T *Bs = As + A_ELEMS;
    static_for<A_LD>([&](auto i) __attribute__((always_inline)) {
      const int id = tid + i * 256;
      const int row = id / (BK / VEC), cv = id % (BK / VEC);
      *(u32x4 *)(As + row * LDA_S + cv * VEC) = ra.template at<i>();
    });
    static_for<B_LD>([&](auto i) __attribute__((always_inline)) {
      const int id = tid + i * 256;
      if (i * 256 + 256 <= B_CH || id < B_CH) {
        const int g = id / CPB, r = id % CPB;
        if (!BKN) {
          const int n = r / (BK / VEC), cv = r % (BK / VEC);
          *(u32x4 *)(Bs + (g * BLK + n) * LDB_S + cv * VEC) = rb.template at<i>();
        } else {
          const int k = r / (BLK / VEC), nv = r % (BLK / VEC);
          *(u32x4 *)(Bs + k * LDB_S + g * BLK + nv * VEC) = rb.template at<i>();
        }
      }
    });
  };

  f32x16 acc[TM][TN];
  static_for<TM>([&](auto i) __attribute__((always_inline)) {
    static_for<TN>([&](auto j) __attribute__((always_inline)) {
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;
    });
  });

  if (total > 0) {
    gload(0);
    sstore(0);
    __syncthreads();
    for (int s = 0; s < total; ++s) {
      const int cur = s & 1;
      if (s + 1 < total) gload(s + 1);
      const T *As = smem + cur * (A_ELEMS + B_ELEMS);
      const T *Bs = As + A_ELEMS;
      if constexpr (BF) {
        static_for<BK / 16>([&](auto ks) __attribute__((always_inline)) {
          bf16x8 af[TM], bfg[TN];
          static_for<TM>([&](auto tm) __attribute__((always_inline)) {
            af[tm] = frag_rmajor((const bf16_t *)As, LDA_S, ks, wm * WTM + tm * 32, lane);
          });
          static_for<TN>([&](auto tn) __attribute__((always_inline)) {
            bfg[tn] = BKN ? frag_kmajor((const bf16_t *)Bs, LDB_S, ks, wn * WTN + tn * 32, lane)
                          : frag_rmajor((const bf16_t *)Bs, LDB_S, ks, wn * WTN + tn * 32, lane);
          });
          static_for<TM>([&](auto tm) __attribute__((always_inline)) {
            static_for<TN>([&](auto tn) __attribute__((always_inline)) {
              acc[tm][tn] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[tm], bfg[tn], acc[tm][tn], 0, 0, 0);
            });
          });
        });
      } else {
        static_for<BK / 2>([&](auto ks) __attribute__((always_inline)) {
          float af[TM], bfg[TN];
          const int kq = ks * 2 + (lane >> 5);
          static_for<TM>([&](auto tm) __attribute__((always_inline)) {
            af[tm] = As[(wm * WTM + tm * 32 + (lane & 31)) * LDA_S + kq];
          });
          static_for<TN>([&](auto tn) __attribute__((always_inline)) {
            const int n = wn * WTN + tn * 32 + (lane & 31);
            bfg[tn] = BKN ? Bs[kq * LDB_S + n] : Bs[n * LDB_S + kq];
          });
          static_for<TM>([&](auto tm) __attribute__((always_inline)) {
            static_for<TN>([&](auto tn) __attribute__((always_inline)) {
              acc[tm][tn] = __builtin_amdgcn_mfma_f32_32x32x2f32(af[tm], bfg[tn], acc[tm][tn], 0, 0, 0);
            });
          });
        });
      }
      if (s + 1 < total) sstore(cur ^ 1);
      __syncthreads();
    }
  }

  // Epilogue: lane holds column (lane % 32) and rows (j/4)*8 + (lane/32)*4
  // + j%4 of each 32 x 32 accumulator tile.
  T *C = (T *)a.C;
  static_for<TN>([&](auto tn) __attribute__((always_inline)) {
    const int g = (wn * WTN + tn * 32) / BLK;  // wave-uniform
    if (g < g_valid) {
      const int64_t col = (int64_t)out_blk(g) * BLK + ((wn * WTN + tn * 32) % BLK) + (lane & 31);
      static_for<TM>([&](auto tm) __attribute__((always_inline)) {
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          const int64_t row = m0 + wm * WTM + tm * 32 + (j >> 2) * 8 + (lane >> 5) * 4 + (j & 3);
          if (row < a.M) {
            float v = acc[tm][tn][j];
            const int64_t o = row * a.ldc + col;
            if (a.epi == 1) {
              if (a.C2) {  // forward GELU: keep the pre-activation
                ((T *)a.C2)[o] = from_f<T>(v);
                v = gelu_f(v);
              } else {     // backward GELU: scale by gelu'(pre-activation)
                v *= gelu_grad_f(to_f<T>(((const T *)a.aux)[o]));
              }
            }
            C[o] = from_f<T>(v);
          }
        }
      });
    }
  });
}

// ---------------------------------------------------------------------------
// TN kernel: 128 x 128 output tiles, reduction over tokens.
// ---------------------------------------------------------------------------
template <typename T, int BLK>
__global__ __launch_bounds__(256) void tn_kernel(TNArgs a) {
  constexpr bool BF = std::is_same<T, bf16_t>::value;
  constexpr int GT = 128 / BLK;  // blocks per tile side
  constexpr int BKT = 32, TILE = 128;
  constexpr int VEC = 16 / (int)sizeof(T);
  constexpr int LDS_S = TILE + (BF ? 16 : 4);
  constexpr int OP_ELEMS = BKT * LDS_S;
  constexpr int CPB = BKT * BLK / VEC;  // chunks of one block column slab
  constexpr int CH = GT * CPB, LD = CH / 256;
  constexpr int TM = 2, TN = 2;  // 4 waves as 2 x 2, 64 x 64 each
  static_assert(CH % 256 == 0 && CPB % 64 == 0, "chunking");

  __shared__ __attribute__((aligned(16))) T smem[2 * 2 * OP_ELEMS];
  __shared__ int s_last;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = uniform(tid >> 6);
  const int wm = wave >> 1, wn = wave & 1;
  const int n_dense_items0 = a.n_dense > 0
      ? ((a.dr[0].na_blk + GT - 1) / GT) * ((a.dr[0].nb_blk + GT - 1) / GT) : 0;
  const int n_dense_items1 = a.n_dense > 1
      ? ((a.dr[1].na_blk + GT - 1) / GT) * ((a.dr[1].nb_blk + GT - 1) / GT) : 0;
  const int items_total = a.n_items + n_dense_items0 + n_dense_items1;
  const int bid = xcd_remap(blockIdx.x, gridDim.x);
  const int split = bid / items_total, item = bid % items_total;

  // Decode the item.
  const bool sparse = item < a.n_items;
  const TNItem *it = sparse ? a.items + item : nullptr;
  const T *Ab, *Bb;
  int64_t lda, ldb, ldo = 0;
  int na, nb, ag = 0, bg = 0;
  T *dout = nullptr;
  if (sparse) {
    Ab = (const T *)a.A; lda = a.lda;
    Bb = (const T *)a.B; ldb = a.ldb;
    na = it->na; nb = it->nb;
  } else {
    int q = item - a.n_items, r = 0;
    if (q >= n_dense_items0) { q -= n_dense_items0; r = 1; }
    const TNDense &d = a.dr[r];
    const int nbg = (d.nb_blk + GT - 1) / GT;
    ag = q / nbg; bg = q % nbg;
    Ab = (const T *)d.A; lda = d.lda;
    Bb = (const T *)d.B; ldb = d.ldb;
    na = min(GT, d.na_blk - ag * GT);
    nb = min(GT, d.nb_blk - bg * GT);
    dout = (T *)d.out;
    ldo = d.ldo;
  }
  // Column blocks and kept-ness (arguments wave-uniform).
  auto acol = [&](int g) __attribute__((always_inline)) -> int { return sparse ? it->a_col[g] : ag * GT + min(g, na - 1); };
  auto bcol = [&](int g) __attribute__((always_inline)) -> int { return sparse ? it->b_col[g] : bg * GT + min(g, nb - 1); };
  auto oblk = [&](int ga, int gb) __attribute__((always_inline)) -> int {
    return sparse ? it->out_blk[ga * kTNMax + gb] : ((ga < na && gb < nb) ? 0 : -1);
  };

  bool live[TM][TN];
  static_for<TM>([&](auto tm) __attribute__((always_inline)) {
    static_for<TN>([&](auto tn) __attribute__((always_inline)) {
      live[tm][tn] = oblk((wm * 64 + tm * 32) / BLK, (wn * 64 + tn * 32) / BLK) >= 0;
    });
  });

  const int64_t t_begin = (int64_t)split * a.chunk;
  const int64_t t_end = min(a.T, t_begin + a.chunk);
  const int nsteps = t_end > t_begin ? (int)((t_end - t_begin + BKT - 1) / BKT) : 0;

  static_assert(LD <= 8, "staging registers");
  Stage8 ra, rb;
  auto gload = [&](int s) __attribute__((always_inline)) {
    static_for<LD>([&](auto i) __attribute__((always_inline)) {
      const int id = tid + i * 256;
      const int g = uniform(id / CPB), r = id % CPB;
      const int t = r / (BLK / VEC), cv = r % (BLK / VEC);
      const int64_t gt = t_begin + (int64_t)s * BKT + t;
      if (gt < t_end) {
        ra.template at<i>() = *(const u32x4 *)(Ab + gt * lda + (int64_t)acol(g) * BLK + cv * VEC);
        rb.template at<i>() = *(const u32x4 *)(Bb + gt * ldb + (int64_t)bcol(g) * BLK + cv * VEC);
      } else {
        ra.template at<i>() = u32x4{0u, 0u, 0u, 0u};
        rb.template at<i>() = u32x4{0u, 0u, 0u, 0u};
      }
    });
  };
  auto sstore = [&](int buf) __attribute__((always_inline)) {
    T *As = smem + buf * 2 * OP_ELEMS;
    T *Bs = As + OP_ELEMS;
    static_for<LD>([&](auto i) __attribute__((always_inline)) {
      const int id = tid + i * 256;
      const int g = id / CPB, r = id % CPB;
      const int t = r / (BLK / VEC), cv = r % (BLK / VEC);
      *(u32x4 *)(As + t * LDS_S + g * BLK + cv * VEC) = ra.template at<i>();
      *(u32x4 *)(Bs + t * LDS_S + g * BLK + cv * VEC) = rb.template at<i>();
    });
  };

  f32x16 acc[TM][TN];
  static_for<TM>([&](auto i) __attribute__((always_inline)) {
    static_for<TN>([&](auto j) __attribute__((always_inline)) {
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;
    });
  });

  if (nsteps > 0) {
    gload(0);
    sstore(0);
    __syncthreads();
    for (int s = 0; s < nsteps; ++s) {
      const int cur = s & 1;
      if (s + 1 < nsteps) gload(s + 1);
      const T *As = smem + cur * 2 * OP_ELEMS;
      const T *Bs = As + OP_ELEMS;
      if constexpr (BF) {
        static_for<BKT / 16>([&](auto ks) __attribute__((always_inline)) {
          bf16x8 af[TM], bfg[TN];
          static_for<TM>([&](auto tm) __attribute__((always_inline)) {
            af[tm] = frag_kmajor((const bf16_t *)As, LDS_S, ks, wm * 64 + tm * 32, lane);
          });
          static_for<TN>([&](auto tn) __attribute__((always_inline)) {
            bfg[tn] = frag_kmajor((const bf16_t *)Bs, LDS_S, ks, wn * 64 + tn * 32, lane);
          });
          static_for<TM>([&](auto tm) __attribute__((always_inline)) {
            static_for<TN>([&](auto tn) __attribute__((always_inline)) {
              if (live[tm][tn])
                acc[tm][tn] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[tm], bfg[tn], acc[tm][tn], 0, 0, 0);
            });
          });
        });
      } else {
        static_for<BKT / 2>([&](auto ks) __attribute__((always_inline)) {
          float af[TM], bfg[TN];
          const int kq = ks * 2 + (lane >> 5);
          static_for<TM>([&](auto tm) __attribute__((always_inline)) { af[tm] = As[kq * LDS_S + wm * 64 + tm * 32 + (lane & 31)]; });
          static_for<TN>([&](auto tn) __attribute__((always_inline)) { bfg[tn] = Bs[kq * LDS_S + wn * 64 + tn * 32 + (lane & 31)]; });
          static_for<TM>([&](auto tm) __attribute__((always_inline)) {
            static_for<TN>([&](auto tn) __attribute__((always_inline)) {
              if (live[tm][tn])
                acc[tm][tn] = __builtin_amdgcn_mfma_f32_32x32x2f32(af[tm], bfg[tn], acc[tm][tn], 0, 0, 0);
            });
          });
        });
      }
      if (s + 1 < nsteps) sstore(cur ^ 1);
      __syncthreads();
    }
  }

  if (a.nsplit > 1) {
    // Partial sums in a lane-contiguous order: [wave][tm][tn][j][lane].
    float *part = a.partials + ((int64_t)item * a.nsplit) * (TILE * TILE);
    auto pidx = [&](int tm, int tn, int j) __attribute__((always_inline)) {
      return (((wave * TM + tm) * TN + tn) * 16 + j) * 64 + lane;
    };
    static_for<TM>([&](auto tm) __attribute__((always_inline)) {
      static_for<TN>([&](auto tn) __attribute__((always_inline)) {
        if (live[tm][tn]) {
#pragma unroll
          for (int j = 0; j < 16; ++j)
            part[(int64_t)split * (TILE * TILE) + pidx(tm, tn, j)] = acc[tm][tn][j];
        }
      });
    });
    __threadfence();
    __syncthreads();
    if (tid == 0) {
      unsigned prev = atomicAdd(&g_tn_counters[item], 1u);
      s_last = (prev == (unsigned)(a.nsplit - 1));
    }
    __syncthreads();
    if (!s_last) return;
    __threadfence();
    static_for<TM>([&](auto tm) __attribute__((always_inline)) {
      static_for<TN>([&](auto tn) __attribute__((always_inline)) {
        if (live[tm][tn]) {
#pragma unroll
          for (int j = 0; j < 16; ++j) {
            float v = 0.f;
            for (int sp = 0; sp < a.nsplit; ++sp)
              v += (sp == split) ? acc[tm][tn][j]
                                 : __builtin_nontemporal_load(&part[(int64_t)sp * (TILE * TILE) + pidx(tm, tn, j)]);
            acc[tm][tn][j] = v;
          }
        }
      });
    });
    if (tid == 0) atomicExch(&g_tn_counters[item], 0u);
  }

  // Store kept blocks.
  static_for<TM>([&](auto tm) __attribute__((always_inline)) {
    static_for<TN>([&](auto tn) __attribute__((always_inline)) {
      if (live[tm][tn]) {
        const int rl0 = wm * 64 + tm * 32, cl0 = wn * 64 + tn * 32;
        const int ga = rl0 / BLK, gb = cl0 / BLK;
        const int cl = cl0 % BLK + (lane & 31);
        if (sparse) {
          T *o = (T *)a.Wout + (int64_t)oblk(ga, gb) * (BLK * BLK) + cl;
#pragma unroll
          for (int j = 0; j < 16; ++j) {
            const int rl = rl0 % BLK + (j >> 2) * 8 + (lane >> 5) * 4 + (j & 3);
            o[rl * BLK] = from_f<T>(acc[tm][tn][j]);
          }
        } else {
          T *o = dout + ((int64_t)acol(ga) * BLK) * ldo + (int64_t)bcol(gb) * BLK + cl;
#pragma unroll
          for (int j = 0; j < 16; ++j) {
            const int rl = rl0 % BLK + (j >> 2) * 8 + (lane >> 5) * 4 + (j & 3);
            o[(int64_t)rl * ldo] = from_f<T>(acc[tm][tn][j]);
          }
        }
      }
    });
  });
}

// ---------------------------------------------------------------------------
// GELU backward (standalone elementwise form)
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(256) void gelu_bwd_kernel(int64_t n, const T *dH, const T *Hpre, T *out) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256)
    out[i] = from_f<T>(to_f<T>(dH[i]) * gelu_grad_f(to_f<T>(Hpre[i])));
}

// ---------------------------------------------------------------------------
// Launchers
// ---------------------------------------------------------------------------
template <typename T, int BLK, int G, bool BKN>
static hipError_t nt_go(const NTArgs &a, hipStream_t s) {
  const int64_t mtiles = (a.M + 127) / 128;
  const int64_t grid = mtiles * a.ntiles;
  if (grid <= 0 || grid > 0x7fffffff) return hipErrorInvalidValue;
  hipLaunchKernelGGL((nt_kernel<T, BLK, G, BKN>), dim3((unsigned)grid), dim3(256), 0, s, a);
  return hipGetLastError();
}

template <typename T, int BLK, bool BKN>
static hipError_t nt_dispatch_g(int G, const NTArgs &a, hipStream_t s) {
  switch (G) {
    case 1: return nt_go<T, BLK, 1, BKN>(a, s);
    case 2: return nt_go<T, BLK, 2, BKN>(a, s);
    case 4:
      if constexpr (BLK <= 64) return nt_go<T, BLK, 4, BKN>(a, s);
      else return hipErrorInvalidValue;
    default: return hipErrorInvalidValue;
  }
}

template <typename T, bool BKN>
static hipError_t nt_dispatch_b(int blk, int G, const NTArgs &a, hipStream_t s) {
  switch (blk) {
    case 32: return nt_dispatch_g<T, 32, BKN>(G, a, s);
    case 64: return nt_dispatch_g<T, 64, BKN>(G, a, s);
    case 128: return nt_dispatch_g<T, 128, BKN>(G, a, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_nt(int dtype, int blk, int G, bool b_kn, const NTArgs &a, hipStream_t s) {
  if (dtype == 0)
    return b_kn ? nt_dispatch_b<bf16_t, true>(blk, G, a, s) : nt_dispatch_b<bf16_t, false>(blk, G, a, s);
  return b_kn ? nt_dispatch_b<float, true>(blk, G, a, s) : nt_dispatch_b<float, false>(blk, G, a, s);
}

int tn_items_total(const TNArgs &a, int blk) {
  const int GT = 128 / blk;
  int n = a.n_items;
  for (int r = 0; r < a.n_dense; ++r)
    n += ((a.dr[r].na_blk + GT - 1) / GT) * ((a.dr[r].nb_blk + GT - 1) / GT);
  return n;
}

template <typename T, int BLK>
static hipError_t tn_go(const TNArgs &a, hipStream_t s) {
  const int64_t grid = (int64_t)tn_items_total(a, BLK) * a.nsplit;
  if (grid <= 0 || grid > 0x7fffffff) return hipErrorInvalidValue;
  hipLaunchKernelGGL((tn_kernel<T, BLK>), dim3((unsigned)grid), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_tn(int dtype, int blk, const TNArgs &a, hipStream_t s) {
  if (dtype == 0) {
    switch (blk) {
      case 32: return tn_go<bf16_t, 32>(a, s);
      case 64: return tn_go<bf16_t, 64>(a, s);
      case 128: return tn_go<bf16_t, 128>(a, s);
    }
  } else {
    switch (blk) {
      case 32: return tn_go<float, 32>(a, s);
      case 64: return tn_go<float, 64>(a, s);
      case 128: return tn_go<float, 128>(a, s);
    }
  }
  return hipErrorInvalidValue;
}

hipError_t launch_gelu_bwd(int dtype, int64_t n, const void *dH, const void *Hpre, void *out, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  int64_t blocks = std::min<int64_t>((n + 255) / 256, 256 * 64);
  if (dtype == 0)
    hipLaunchKernelGGL((gelu_bwd_kernel<bf16_t>), dim3((unsigned)blocks), dim3(256), 0, s, n,
                       (const bf16_t *)dH, (const bf16_t *)Hpre, (bf16_t *)out);
  else
    hipLaunchKernelGGL((gelu_bwd_kernel<float>), dim3((unsigned)blocks), dim3(256), 0, s, n,
                       (const float *)dH, (const float *)Hpre, (float *)out);
  return hipGetLastError();
}

}  // namespace pf
