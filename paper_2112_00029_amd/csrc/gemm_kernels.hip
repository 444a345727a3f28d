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
//             K-steps run over every block of a dense B; the K range may be
//             split over workgroups that write fp32 partial outputs, summed
//             in split order by reduce_rows_kernel (deterministic).
//  tn_kernel  out = A^T . B reduced over tokens, only for kept blocks
//             (weight gradient restricted to the mask) plus dense regions
//             (dU = dY^T T_lr, dV = S^T X).  The token range may be split
//             over workgroups; tn_reduce_kernel sums the partials in split
//             order (deterministic).
//
// Mainloop: 256 threads = 4 waves of 64.  The K dimension advances in steps
// of 64 (bf16) / 32 (fp32).  Operands stream global -> registers -> LDS with
// two register stages (the loads of step s+2 are issued before step s is
// computed) and a double-buffered LDS tile, one barrier per step.  MFMA
// fragments are read from LDS with 16-byte reads ([row][k] tiles) or with
// the gfx950 transpose read ds_read_b64_tr_b16 ([k][row] tiles): within each
// group of 16 lanes, lanes 4m..4m+3 address row m (4 x 16-bit each) of a
// 4 x 16 tile and lane j receives column j, i.e. 4 consecutive k of one row.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>
#include <type_traits>

#include "pf_launch.h"

// Part of this file an object holds (see the launchers at the end).
#ifndef PF_GK_PART
#define PF_GK_PART -1
#endif
#define PF_GK_HAS(p) (PF_GK_PART < 0 || PF_GK_PART == (p))

namespace pf {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef short s16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint16_t bf16_t;  // bfloat16 storage
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));  // 16-byte chunk

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

// MFMA (32x32x16) fragment of a 32-row operand stored [k][row] in LDS (row
// contiguous): lane l gets row (l % 32), k = ks*16 + (l / 32)*8 + 0..7.
__device__ __forceinline__ bf16x8 frag_kmajor(const bf16_t *base, int ld,
                                              int ks, int row0, int lane) {
  int g16 = lane >> 4, i = lane & 15;
  int n0 = (g16 & 1) * 16, kb = (g16 >> 1) * 8;
  const bf16_t *p = base + (ks * 16 + kb + (i >> 2)) * ld + row0 + n0 + (i & 3) * 4;
  return cat8(tr16(p), tr16(p + 4 * ld));
}

// Same fragment from an unpadded [k][128] tile (256-byte k rows) whose
// 16-byte chunks are XOR-swizzled by k: chunk c of k row k sits at chunk
// c ^ ((k & 3) << 2).  The four k rows one 16-lane group reads then fall in
// four different 64-byte bank groups (no LDS bank conflicts).
__device__ __forceinline__ int swz128(int k, int col) {
  return k * 128 + ((((col >> 3) ^ ((k & 3) << 2)) << 3) | (col & 7));
}
__device__ __forceinline__ bf16x8 frag_kmajor_swz(const bf16_t *base, int ks, int row0, int lane) {
  const int g16 = lane >> 4, i = lane & 15;
  const int k = ks * 16 + (g16 >> 1) * 8 + (i >> 2);
  const int col = row0 + (g16 & 1) * 16 + (i & 3) * 4;
  return cat8(tr16(base + swz128(k, col)), tr16(base + swz128(k + 4, col)));
}

// MFMA (32x32x16) fragment of a 32-row operand stored [row][k] in LDS.
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

// Pipeline driver: load(s, ra, rb) issues the global loads of step s into a
// register stage, store(ra, rb, buf) writes a register stage to LDS buffer
// buf, compute(buf, s) runs the MFMAs of step s held in buf.  Four register
// stages rotate over the steps and two LDS buffers alternate; the loads of
// step s+3 are issued right after step s is stored, so three steps' loads
// are in flight while one is computed (a step is a few hundred MFMA cycles,
// well short of a loaded HBM round trip).  One barrier per step suffices:
// buffer s % 2 is rewritten at step s only after every wave has passed the
// barrier of step s-1, i.e. finished computing step s-2.
//
// Loads are issued for up to three steps past the end (load must accept any
// s < total + 3: its reads stay inside the operands or read zeros); only
// compute stops at total.  The loop runs whole groups of four steps with no
// branch around a load, so every entry to its body has the same three
// stages in flight, oldest first, and the wait before each store leaves the
// two younger ones outstanding; up to three remaining steps follow it.
template <typename Load, typename Store, typename Compute>
__device__ __forceinline__ void pipeline4(int total, Stage8 &ra0, Stage8 &rb0, Stage8 &ra1,
                                          Stage8 &rb1, Stage8 &ra2, Stage8 &rb2, Stage8 &ra3,
                                          Stage8 &rb3, Load &&load, Store &&store,
                                          Compute &&compute) {
  if (total <= 0) return;
  load(0, ra0, rb0);
  load(1, ra1, rb1);
  load(2, ra2, rb2);
  auto step = [&](int s, Stage8 &ra, Stage8 &rb, Stage8 &na, Stage8 &nb,
                  int buf) __attribute__((always_inline)) {
    store(ra, rb, buf);
    __syncthreads();
    load(s + 3, na, nb);
    compute(buf, s);
  };
  const int quads = total >> 2;
  for (int p = 0; p < quads; ++p) {
    const int s = 4 * p;
    step(s, ra0, rb0, ra3, rb3, 0);
    step(s + 1, ra1, rb1, ra0, rb0, 1);
    step(s + 2, ra2, rb2, ra1, rb1, 0);
    step(s + 3, ra3, rb3, ra2, rb2, 1);
  }
  const int rem = total & 3, s = 4 * quads;
  if (rem > 0) {
    store(ra0, rb0, 0);
    __syncthreads();
    compute(0, s);
  }
  if (rem > 1) {
    store(ra1, rb1, 1);
    __syncthreads();
    compute(1, s + 1);
  }
  if (rem > 2) {
    store(ra2, rb2, 0);
    __syncthreads();
    compute(0, s + 2);
  }
}

// The same with two register stages (loads one step ahead), for the fp32
// kernels, whose fragments leave no room for four stages: loads may run
// two steps past the end; whole pairs of steps in the loop, an odd last
// step after it.
template <typename Load, typename Store, typename Compute>
__device__ __forceinline__ void pipeline2(int total, Stage8 &ra0, Stage8 &rb0, Stage8 &ra1,
                                          Stage8 &rb1, Load &&load, Store &&store,
                                          Compute &&compute) {
  if (total <= 0) return;
  load(0, ra0, rb0);
  load(1, ra1, rb1);
  const int pairs = total >> 1;
  for (int p = 0; p < pairs; ++p) {
    const int s = 2 * p;
    store(ra0, rb0, 0);
    __syncthreads();
    load(s + 2, ra0, rb0);
    compute(0, s);
    store(ra1, rb1, 1);
    __syncthreads();
    load(s + 3, ra1, rb1);
    compute(1, s + 1);
  }
  if (total & 1) {
    store(ra0, rb0, 0);
    __syncthreads();
    compute(0, total - 1);
  }
}

// ---------------------------------------------------------------------------
// Buffer-resource loads: raw buffer loads return zeros outside [0, bytes),
// which covers ragged token tiles and the zero padding of the K range
// without per-lane branches.
// ---------------------------------------------------------------------------
typedef __amdgpu_buffer_rsrc_t rsrc_t;
__device__ __forceinline__ rsrc_t make_rsrc(const void *p, int64_t bytes) {
  const int64_t b = bytes < 0 ? 0 : (bytes > 0x7fffffff ? 0x7fffffff : bytes);
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(p), (short)0, (int)b, 0x00020000);
}
__device__ __forceinline__ u32x4 bload(rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, 0);
}

// ---------------------------------------------------------------------------
// NT kernel
// ---------------------------------------------------------------------------
// EPI: 0 plain store, 1 forward GELU (also store the pre-activation),
// 2 backward GELU (scale by gelu' of the pre-activation a.aux).
template <typename T, int BLK, int G, bool BKN, int BM, bool DENSE, int EPI>
__global__ __launch_bounds__(256, 2) void nt_kernel(NTArgs a_arg) {
  const NTArgs a = a_arg;  // local copy: lambdas below capture it by reference
  constexpr bool BF = std::is_same<T, bf16_t>::value;
  constexpr int ES = (int)sizeof(T);
  constexpr int BK = BF ? 64 : 32;           // K per pipeline step
  constexpr int BN = G * BLK;
  constexpr int VEC = 16 / ES;               // elements per 16-byte chunk
  constexpr int KW = BK < BLK ? BK : BLK;    // K width of one sub-block
  constexpr int NH = BK / KW;                // sub-blocks per step (2: bf16, b = 32)
  constexpr int PADA = BF ? 8 : 4;
  constexpr int LDA_S = BK + PADA;
  // B read as [k][n]: a 32-column bf16 tile keeps unpadded 64-byte k rows
  // (the four k rows of each 16-lane transpose read, and the two 16-lane
  // groups of a half-wave, then cover distinct banks); wider tiles pad.
  constexpr int LDB_S = BKN ? (BN + (BF ? (BN == 32 ? 0 : 16) : 4)) : (BK + PADA);
  constexpr int A_ELEMS = BM * LDA_S;
  constexpr int B_ELEMS = BKN ? BK * LDB_S : BN * LDB_S;
  constexpr int WNN = BN == 32 ? 1 : 2;      // waves along N
  constexpr int WMM = 4 / WNN;               // waves along M
  constexpr int WTM = BM / WMM, WTN = BN / WNN;
  constexpr int TM = WTM / 32, TN = WTN / 32;
  // A tile: NH sub-blocks of BM rows x KW columns; B tile: G x NH pieces
  // (tile row g, sub-block h) of BLK x KW.
  constexpr int A_CPR = KW / VEC, A_CPH = BM * A_CPR, A_IPH = A_CPH / 256;
  constexpr int A_LD = NH * A_IPH;
  constexpr int B_CPP = BLK * KW / VEC;
  constexpr int B_LD = G * NH * B_CPP / 256;
  static_assert(A_CPH % 256 == 0 && B_CPP % 64 == 0 && (G * NH * B_CPP) % 256 == 0, "chunking");
  static_assert(A_LD <= 8 && B_LD <= 8, "staging registers");
  static_assert(TM >= 1 && TN >= 1 && WTM % 32 == 0 && WTN % 32 == 0, "wave tile");

  __shared__ __attribute__((aligned(16))) T smem[2 * (A_ELEMS + B_ELEMS)];

  const T *__restrict__ A = (const T *)a.A;
  const T *__restrict__ B = (const T *)a.B;
  const T *__restrict__ L = (const T *)a.L;
  const T *__restrict__ R = (const T *)a.R;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WNN, wn = wave % WNN;
  const int ntn = a.ntiles;
  const int mtiles = (int)((a.M + BM - 1) / BM);
  const int bid = xcd_remap(blockIdx.x, gridDim.x);
  // Grouped order: consecutive ids (the workgroups resident on one XCD)
  // cover GM m-tiles x a run of n-tiles, so both the token rows and the
  // weight blocks they read are re-used from that XCD's L2.  Four token
  // tiles (twice as many n-tiles per group as with eight): the 32-wide
  // backward-data tiles of neighbouring block columns share most of their
  // dY block rows (16384 x 4096 b = 32: 481 -> 459 us; 768 -> 3072: 20.7
  // -> 18.8 us).
  constexpr int GM = 4;
  const int split = bid / (mtiles * ntn);
  const int lin = bid % (mtiles * ntn);
  const int first_m = (lin / (GM * ntn)) * GM;
  const int gsz = min(GM, mtiles - first_m);
  const int within = lin - first_m * ntn;
  const int mt = first_m + within % gsz, nt = within / gsz;
  const int64_t m0 = (int64_t)mt * BM;

  int g_valid, nsteps, kcol_off = 0, blk_off = 0;
  const NTTile *tile = DENSE ? nullptr : a.tiles + nt;
  if constexpr (DENSE) {
    g_valid = min(G, a.dense_nblk - nt * G);
    nsteps = a.dense_nsteps;
  } else {
    g_valid = tile->g;
    nsteps = tile->nsteps;
    kcol_off = tile->kcol_off;
    blk_off = tile->blk_off;
  }
  auto out_blk = [&](int g) __attribute__((always_inline)) -> int {
    if constexpr (DENSE) return nt * G + min(g, g_valid - 1);
    else return tile->out_blk[g];
  };
  // Virtual K: the kept blocks, then the low-rank blocks, then zero padding.
  const int vblocks = nsteps + a.nlr;
  const int total_all = (vblocks * BLK + BK - 1) / BK;
  const int per_split = (total_all + a.nsplit - 1) / a.nsplit;
  const int s_begin = split * per_split;
  const int total = max(0, min(total_all, s_begin + per_split) - s_begin);

  // Operand sources as (base, byte range); buffer resources are built at
  // the point of use.  A byte range of 0 yields zeros (K padding).
  const T *const a_base = A + m0 * a.lda;
  const int64_t a_bytes = (a.M - m0) * a.lda * ES;
  const T *const l_base = DENSE ? A : L + m0 * a.ldl;
  const int64_t l_bytes = DENSE ? 0 : (a.M - m0) * a.ldl * ES;
  constexpr int64_t BIG = 0x7fffffff;

  // Sub-block h of step s (all arguments wave-uniform): A base, byte range,
  // row stride and column offset in bytes.  Branch-free: the index tables
  // are read at a clamped position and the phase (kept block, low-rank
  // block, zero padding) is applied with selects.
  auto a_src = [&](int s, int h, const T *&base, int64_t &bytes, uint32_t &ldb,
                   uint32_t &colb) __attribute__((always_inline)) {
    const int k0 = (s_begin + s) * BK + h * KW, c = k0 / BLK, kk = k0 % BLK;
    const bool sp = c < nsteps;
    const int kcol = DENSE ? c : a.kcols[kcol_off + max(min(c, nsteps - 1), 0)];
    base = sp ? a_base : l_base;
    // Steps past this split's range (the pipeline loads ahead) read zeros.
    bytes = s >= total ? 0 : (sp ? a_bytes : (c < vblocks ? l_bytes : 0));
    ldb = (uint32_t)((sp ? a.lda : a.ldl) * ES);
    colb = (uint32_t)(((sp ? kcol : c - nsteps) * BLK + kk) * ES);
  };
  // Piece (g, h) of step s: B base at the piece, byte range, row stride.
  auto b_src = [&](int s, int g, int h, const T *&base, int64_t &bytes,
                   uint32_t &ldb) __attribute__((always_inline)) {
    const int k0 = (s_begin + s) * BK + h * KW, c = k0 / BLK, kk = k0 % BLK;
    const int64_t ob = out_blk(g);
    if constexpr (DENSE) {
      ldb = (uint32_t)(a.ldb * ES);
      base = BKN ? B + ((int64_t)c * BLK + kk) * a.ldb + ob * BLK
                 : B + (ob * BLK) * a.ldb + (int64_t)c * BLK + kk;
      bytes = (c < nsteps && s < total) ? BIG : 0;
    } else {
      const bool sp = c < nsteps;
      const int64_t blk = a.blks[blk_off + max(min(c, nsteps - 1), 0) * G + g];
      const int cr = c - nsteps;
      const T *sp_base = B + blk * (BLK * BLK) + (BKN ? kk * BLK : kk);
      const T *lr_base = BKN ? R + ((int64_t)cr * BLK + kk) * a.ldr + ob * BLK
                             : R + (ob * BLK) * a.ldr + (int64_t)cr * BLK + kk;
      base = sp ? sp_base : lr_base;
      bytes = ((sp || c < vblocks) && s < total) ? BIG : 0;
      ldb = (uint32_t)(sp ? BLK * ES : a.ldr * ES);
    }
  };

  auto load = [&](int s, Stage8 &ra, Stage8 &rb) __attribute__((always_inline)) {
    static_for<NH>([&](auto h) __attribute__((always_inline)) {
      const T *base;
      int64_t bytes;
      uint32_t ldb, colb;
      a_src(s, h, base, bytes, ldb, colb);
      const rsrc_t r = make_rsrc(base, bytes);
      static_for<A_IPH>([&](auto j) __attribute__((always_inline)) {
        const int id = tid + j * 256;
        const uint32_t off = (uint32_t)(id / A_CPR) * ldb + colb + (uint32_t)(id % A_CPR) * 16;
        ra.template at<h * A_IPH + j>() = bload(r, off);
      });
    });
    static_for<B_LD>([&](auto i) __attribute__((always_inline)) {
      const int id = tid + i * 256;
      const int piece = B_CPP % 256 == 0 ? (i * 256) / B_CPP
                                         : __builtin_amdgcn_readfirstlane(id / B_CPP);
      const int rr = id % B_CPP;
      const T *base;
      int64_t bytes;
      uint32_t ldb;
      b_src(s, piece / NH, piece % NH, base, bytes, ldb);
      const rsrc_t r = make_rsrc(base, bytes);
      uint32_t off;
      if constexpr (!BKN) off = (uint32_t)(rr / (KW / VEC)) * ldb + (uint32_t)(rr % (KW / VEC)) * 16;
      else off = (uint32_t)(rr / (BLK / VEC)) * ldb + (uint32_t)(rr % (BLK / VEC)) * 16;
      rb.template at<i>() = bload(r, off);
    });
  };
  auto store = [&](Stage8 &ra, Stage8 &rb, int buf) __attribute__((always_inline)) {
    T *As = smem + buf * (A_ELEMS + B_ELEMS);
    T *Bs = As + A_ELEMS;
    static_for<A_LD>([&](auto i) __attribute__((always_inline)) {
      constexpr int h = i / A_IPH;
      const int id = tid + (i % A_IPH) * 256;
      *(u32x4 *)(As + (id / A_CPR) * LDA_S + h * KW + (id % A_CPR) * VEC) = ra.template at<i>();
    });
    static_for<B_LD>([&](auto i) __attribute__((always_inline)) {
      const int id = tid + i * 256;
      const int piece = id / B_CPP, g = piece / NH, h = piece % NH, rr = id % B_CPP;
      if constexpr (!BKN) {
        *(u32x4 *)(Bs + (g * BLK + rr / (KW / VEC)) * LDB_S + h * KW + (rr % (KW / VEC)) * VEC) =
            rb.template at<i>();
      } else {
        *(u32x4 *)(Bs + (h * KW + rr / (BLK / VEC)) * LDB_S + g * BLK + (rr % (BLK / VEC)) * VEC) =
            rb.template at<i>();
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

  // Mixing weight: scale the kept-block sums once, at the first low-rank
  // K-block (the virtual K index nsteps * BLK).
  const int kswitch = nsteps * BLK;
  auto mix_switch = [&](int k) __attribute__((always_inline)) {
    if (a.mix && k == kswitch) {
      static_for<TM>([&](auto tm) __attribute__((always_inline)) {
        static_for<TN>([&](auto tn) __attribute__((always_inline)) {
#pragma unroll
          for (int e = 0; e < 16; ++e) acc[tm][tn][e] *= a.mix_ratio;
        });
      });
    }
  };
  // MIX: whether this instantiation checks for the mixing switch; the
  // check is a branch per K slice, which keeps the scheduler from moving the
  // next slice's LDS reads under the current MFMAs, so calls without the
  // mixing weight run an instantiation without it.
  auto compute_m = [&](int buf, int s, auto mix) __attribute__((always_inline)) {
    constexpr bool MIX = decltype(mix)::value;
    const T *As = smem + buf * (A_ELEMS + B_ELEMS);
    const T *Bs = As + A_ELEMS;
    if constexpr (BF) {
      static_for<BK / 16>([&](auto ks) __attribute__((always_inline)) {
        if constexpr (MIX) mix_switch((s_begin + s) * BK + ks * 16);
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
        if constexpr (MIX) mix_switch((s_begin + s) * BK + ks * 2);
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
  };

  Stage8 ra0, rb0, ra1, rb1, ra2, rb2, ra3, rb3;
  auto run = [&](auto mix) __attribute__((always_inline)) {
    auto compute = [&](int buf, int s) __attribute__((always_inline)) { compute_m(buf, s, mix); };
    if constexpr (BF) pipeline4(total, ra0, rb0, ra1, rb1, ra2, rb2, ra3, rb3, load, store, compute);
    else pipeline2(total, ra0, rb0, ra1, rb1, load, store, compute);
  };
  if (a.mix) run(std::true_type{});
  else run(std::false_type{});

  // Epilogue.  The accumulators (lane: column lane % 32, rows (j/4)*8 +
  // (lane/32)*4 + j%4 of each 32 x 32 tile) go to an fp32 tile in LDS, then
  // each thread writes 8 consecutive columns of one row (16-byte stores).
  constexpr int CS = BN + 4;
  static_assert(BM * CS * 4 <= (int)sizeof(smem), "epilogue tile");
  float *Cs = (float *)smem;
  __syncthreads();
  static_for<TM>([&](auto tm) __attribute__((always_inline)) {
    static_for<TN>([&](auto tn) __attribute__((always_inline)) {
      const int col = wn * WTN + tn * 32 + (lane & 31);
#pragma unroll
      for (int j = 0; j < 16; ++j)
        Cs[(wm * WTM + tm * 32 + (j >> 2) * 8 + (lane >> 5) * 4 + (j & 3)) * CS + col] = acc[tm][tn][j];
    });
  });
  __syncthreads();
  int ob[G];
  static_for<G>([&](auto g) __attribute__((always_inline)) { ob[g] = out_blk(g); });
  T *C = (T *)a.C;
  constexpr int RCH = BN / 8;  // 8-column chunks per row
  static_for<(BM * RCH) / 256>([&](auto it) __attribute__((always_inline)) {
    const int q = tid + it * 256;
    const int row = q / RCH, c8 = (q % RCH) * 8;
    const int g = c8 / BLK;
    int obg = ob[0];
    static_for<G>([&](auto gg) __attribute__((always_inline)) { if (g == gg) obg = ob[gg]; });
    const int64_t gm = m0 + row;
    if (gm < a.M && g < g_valid) {
      const int64_t col = (int64_t)obg * BLK + (c8 % BLK);
      const f32x4 lo = *(const f32x4 *)(Cs + row * CS + c8);
      const f32x4 hi = *(const f32x4 *)(Cs + row * CS + c8 + 4);
      float v[8] = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
      if (a.nsplit > 1) {
        float *P = a.partials + ((int64_t)split * a.M + gm) * a.ldp + col;
        *(f32x4 *)P = lo;
        *(f32x4 *)(P + 4) = hi;
        return;
      }
      if (a.mix) {
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] *= a.mix_out;
      }
      const int64_t o = gm * a.ldc + col;
      if constexpr (EPI == 1) {  // forward GELU: keep the pre-activation
        if constexpr (BF) {
          u32x4 w;
#pragma unroll
          for (int e = 0; e < 4; ++e)
            w[e] = (uint32_t)f2bf(v[2 * e]) | ((uint32_t)f2bf(v[2 * e + 1]) << 16);
          *(u32x4 *)((T *)a.C2 + o) = w;
        } else {
          *(f32x4 *)((T *)a.C2 + o) = f32x4{v[0], v[1], v[2], v[3]};
          *(f32x4 *)((T *)a.C2 + o + 4) = f32x4{v[4], v[5], v[6], v[7]};
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = gelu_f(v[e]);
      } else if constexpr (EPI == 2) {  // backward GELU: scale by gelu'(pre-activation)
        const T *ax = (const T *)a.aux + o;
        if constexpr (BF) {
          const u32x4 w = *(const u32x4 *)ax;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            v[2 * e] *= gelu_grad_f(__uint_as_float(w[e] << 16));
            v[2 * e + 1] *= gelu_grad_f(__uint_as_float(w[e] & 0xffff0000u));
          }
        } else {
#pragma unroll
          for (int e = 0; e < 8; ++e) v[e] *= gelu_grad_f(ax[e]);
        }
      }
      if constexpr (BF) {
        u32x4 w;
#pragma unroll
        for (int e = 0; e < 4; ++e)
          w[e] = (uint32_t)f2bf(v[2 * e]) | ((uint32_t)f2bf(v[2 * e + 1]) << 16);
        *(u32x4 *)(C + o) = w;
      } else {
        *(f32x4 *)(C + o) = f32x4{v[0], v[1], v[2], v[3]};
        *(f32x4 *)(C + o + 4) = f32x4{v[4], v[5], v[6], v[7]};
      }
    }
  });
}

// Sum of split partials, in split order: C[row][col] = sum_s P[s][row][col].
template <typename T>
__global__ __launch_bounds__(256) void reduce_rows_kernel(int nsplit, const float *__restrict__ P,
                                                          int64_t M, int64_t ncols, T *C,
                                                          int64_t ldc) {
  const int64_t n4 = M * ncols / 4;  // ncols is a multiple of 32
  for (int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x; q < n4; q += (int64_t)gridDim.x * 256) {
    // Splits in batches of 4 (loads issued together, added in split order).
    f32x4 v = *(const f32x4 *)(P + q * 4);
    for (int s0 = 1; s0 < nsplit; s0 += 4) {
      f32x4 t[4];
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (s0 + u < nsplit) t[u] = *(const f32x4 *)(P + (int64_t)(s0 + u) * M * ncols + q * 4);
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (s0 + u < nsplit) v += t[u];
    }
    const int64_t e = q * 4, row = e / ncols, col = e % ncols;
    T *o = C + row * ldc + col;
#pragma unroll
    for (int i = 0; i < 4; ++i) o[i] = from_f<T>(v[i]);
  }
}

// ---------------------------------------------------------------------------
// TN kernel: 128 x 128 output tiles, reduction over tokens.
// ---------------------------------------------------------------------------
template <typename T, int BLK>
struct TNItemView {
  static constexpr int GT = 128 / BLK;
  bool sparse;
  const TNItem *it;
  int na, nb, ag, bg;
  const T *Ab, *Bb;
  int64_t lda, ldb, ldo;
  T *dout;

  __device__ __forceinline__ void decode(const TNArgs &a, int item) {
    const int n0 = a.n_dense > 0 ? ((a.dr[0].na_blk + GT - 1) / GT) * ((a.dr[0].nb_blk + GT - 1) / GT) : 0;
    sparse = item < a.n_items;
    it = sparse ? a.items + item : nullptr;
    ag = bg = 0;
    dout = nullptr;
    ldo = 0;
    if (sparse) {
      Ab = (const T *)a.A; lda = a.lda;
      Bb = (const T *)a.B; ldb = a.ldb;
      na = it->na; nb = it->nb;
    } else {
      int q = item - a.n_items, r = 0;
      if (q >= n0) { q -= n0; r = 1; }
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
  }
  __device__ __forceinline__ int acol(int g) const { return sparse ? it->a_col[g] : ag * GT + min(g, na - 1); }
  __device__ __forceinline__ int bcol(int g) const { return sparse ? it->b_col[g] : bg * GT + min(g, nb - 1); }
  __device__ __forceinline__ int oblk(int ga, int gb) const {
    return sparse ? it->out_blk[ga * kTNMax + gb] : ((ga < na && gb < nb) ? 0 : -1);
  }
};

__device__ __forceinline__ int tn_items_total_dev(const TNArgs &a, int GT) {
  int n = a.n_items;
  for (int r = 0; r < a.n_dense; ++r)
    n += ((a.dr[r].na_blk + GT - 1) / GT) * ((a.dr[r].nb_blk + GT - 1) / GT);
  return n;
}

// Sum of one float per thread over a 256-thread workgroup in a fixed order
// (wave butterflies, then the four wave sums in wave order); every thread
// must call it.  red: 4 floats of LDS.
__device__ __forceinline__ float block_sum256(float x, float *red) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o, 64);
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = x;
  __syncthreads();
  return ((red[0] + red[1]) + red[2]) + red[3];
}

// Partial-sum index of (wave, tm, tn, j, lane): lane-contiguous.
__device__ __forceinline__ int tn_pidx(int wave, int tm, int tn, int j, int lane) {
  return (((wave * 2 + tm) * 2 + tn) * 16 + j) * 64 + lane;
}

template <typename T, int BLK>
__global__ __launch_bounds__(256, 2) void tn_kernel(TNArgs a_arg) {
  const TNArgs a = a_arg;  // local copy: lambdas below capture it by reference
  constexpr bool BF = std::is_same<T, bf16_t>::value;
  constexpr int GT = 128 / BLK;  // blocks per tile side
  constexpr int BKT = BF ? 64 : 32, TILE = 128;
  constexpr int VEC = 16 / (int)sizeof(T);
  constexpr int LDS_S = TILE + (BF ? 0 : 4);  // bf16: unpadded, chunk-swizzled rows
  constexpr int OP_ELEMS = BKT * LDS_S;
  constexpr int CPB = BKT * BLK / VEC;  // chunks of one block column slab
  constexpr int CH = GT * CPB, LD = CH / 256;
  constexpr int TM = 2, TN = 2;  // 4 waves as 2 x 2, 64 x 64 each
  static_assert(CPB % 256 == 0 && LD <= 8, "chunking");

  // Two stages of both operands; the fp32 epilogue tile (128 x 132) reuses
  // the same memory.
  constexpr int SMEM_ELEMS = 2 * 2 * OP_ELEMS > TILE * (TILE + 4) * 4 / (int)sizeof(T)
                                 ? 2 * 2 * OP_ELEMS
                                 : TILE * (TILE + 4) * 4 / (int)sizeof(T);
  __shared__ __attribute__((aligned(16))) T smem[SMEM_ELEMS];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 1, wn = wave & 1;
  const int items_total = tn_items_total_dev(a, GT);
  const int bid = xcd_remap(blockIdx.x, gridDim.x);
  const int split = bid / items_total, pos = bid % items_total;
  // The launch order comes straight from the kernel arguments (a_arg): the
  // local copy keeps the scalar fields only.
  const int item = a.n_order > 0 ? (int)a_arg.order[pos] : pos;

  TNItemView<T, BLK> v;
  v.decode(a, item);

  bool live[TM][TN];
  static_for<TM>([&](auto tm) __attribute__((always_inline)) {
    static_for<TN>([&](auto tn) __attribute__((always_inline)) {
      live[tm][tn] = v.oblk((wm * 64 + tm * 32) / BLK, (wn * 64 + tn * 32) / BLK) >= 0;
    });
  });

  const int64_t t_begin = (int64_t)split * a.chunk;
  const int64_t t_end = min(a.T, t_begin + a.chunk);
  const int nsteps = t_end > t_begin ? (int)((t_end - t_begin + BKT - 1) / BKT) : 0;

  // Token rows past t_end read as zeros (buffer range).  Column offsets of
  // each chunk are fixed for the whole loop.
  const T *const a_base = v.Ab + t_begin * v.lda, *const b_base = v.Bb + t_begin * v.ldb;
  const int64_t a_bytes = (t_end - t_begin) * v.lda * (int64_t)sizeof(T);
  const int64_t b_bytes = (t_end - t_begin) * v.ldb * (int64_t)sizeof(T);
  const uint32_t lda_b = (uint32_t)(v.lda * sizeof(T)), ldb_b = (uint32_t)(v.ldb * sizeof(T));
  uint32_t offA[LD], offB[LD];
  static_for<LD>([&](auto i) __attribute__((always_inline)) {
    constexpr int g = (i * 256) / CPB;
    const int r = (tid + i * 256) % CPB;
    const uint32_t t = r / (BLK / VEC), cb = (r % (BLK / VEC)) * 16;
    offA[i] = t * lda_b + (uint32_t)(v.acol(g) * BLK * sizeof(T)) + cb;
    offB[i] = t * ldb_b + (uint32_t)(v.bcol(g) * BLK * sizeof(T)) + cb;
  });
  auto load = [&](int s, Stage8 &ra, Stage8 &rb) __attribute__((always_inline)) {
    const rsrc_t rA = make_rsrc(a_base, a_bytes), rB = make_rsrc(b_base, b_bytes);
    const uint32_t sa = (uint32_t)(s * BKT) * lda_b, sb = (uint32_t)(s * BKT) * ldb_b;
    static_for<LD>([&](auto i) __attribute__((always_inline)) {
      ra.template at<i>() = bload(rA, sa + offA[i]);
      rb.template at<i>() = bload(rB, sb + offB[i]);
    });
  };
  auto store = [&](Stage8 &ra, Stage8 &rb, int buf) __attribute__((always_inline)) {
    T *As = smem + buf * 2 * OP_ELEMS;
    T *Bs = As + OP_ELEMS;
    static_for<LD>([&](auto i) __attribute__((always_inline)) {
      constexpr int g = (i * 256) / CPB;
      const int r = (tid + i * 256) % CPB;
      const int t = r / (BLK / VEC), c = g * BLK + (r % (BLK / VEC)) * VEC;
      const int o = BF ? swz128(t, c) : t * LDS_S + c;
      *(u32x4 *)(As + o) = ra.template at<i>();
      *(u32x4 *)(Bs + o) = rb.template at<i>();
    });
  };

  f32x16 acc[TM][TN];
  static_for<TM>([&](auto i) __attribute__((always_inline)) {
    static_for<TN>([&](auto j) __attribute__((always_inline)) {
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;
    });
  });

  auto compute = [&](int buf, int) __attribute__((always_inline)) {
    const T *As = smem + buf * 2 * OP_ELEMS;
    const T *Bs = As + OP_ELEMS;
    if constexpr (BF) {
      static_for<BKT / 16>([&](auto ks) __attribute__((always_inline)) {
        bf16x8 af[TM], bfg[TN];
        static_for<TM>([&](auto tm) __attribute__((always_inline)) {
          af[tm] = frag_kmajor_swz((const bf16_t *)As, ks, wm * 64 + tm * 32, lane);
        });
        static_for<TN>([&](auto tn) __attribute__((always_inline)) {
          bfg[tn] = frag_kmajor_swz((const bf16_t *)Bs, ks, wn * 64 + tn * 32, lane);
        });
        // All four sub-tiles, live or not: a branch per MFMA splits the step
        // into blocks the scheduler cannot overlap (the next slice's LDS reads
        // then wait behind every MFMA), and MFMA time is not what bounds this
        // kernel.  A dead sub-tile reads clamped, valid fragments and is
        // never stored.
        static_for<TM>([&](auto tm) __attribute__((always_inline)) {
          static_for<TN>([&](auto tn) __attribute__((always_inline)) {
            acc[tm][tn] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[tm], bfg[tn], acc[tm][tn], 0, 0, 0);
          });
        });
      });
    } else {
      static_for<BKT / 2>([&](auto ks) __attribute__((always_inline)) {
        float af[TM], bfg[TN];
        const int kq = ks * 2 + (lane >> 5);
        static_for<TM>([&](auto tm) __attribute__((always_inline)) {
          af[tm] = As[kq * LDS_S + wm * 64 + tm * 32 + (lane & 31)];
        });
        static_for<TN>([&](auto tn) __attribute__((always_inline)) {
          bfg[tn] = Bs[kq * LDS_S + wn * 64 + tn * 32 + (lane & 31)];
        });
        // fp32 MFMAs are long (the kernel is MFMA-bound at these sizes):
        // sub-tiles without a kept block are skipped (a wave-uniform branch).
        static_for<TM>([&](auto tm) __attribute__((always_inline)) {
          static_for<TN>([&](auto tn) __attribute__((always_inline)) {
            if (live[tm][tn])
              acc[tm][tn] = __builtin_amdgcn_mfma_f32_32x32x2f32(af[tm], bfg[tn], acc[tm][tn], 0, 0, 0);
          });
        });
      });
    }
  };

  Stage8 ra0, rb0, ra1, rb1, ra2, rb2, ra3, rb3;
  if constexpr (BF) pipeline4(nsteps, ra0, rb0, ra1, rb1, ra2, rb2, ra3, rb3, load, store, compute);
  else pipeline2(nsteps, ra0, rb0, ra1, rb1, load, store, compute);

  if (a.nsplit > 1) {
    float *part = a.partials + ((int64_t)item * a.nsplit + split) * (TILE * TILE);
    static_for<TM>([&](auto tm) __attribute__((always_inline)) {
      static_for<TN>([&](auto tn) __attribute__((always_inline)) {
        if (live[tm][tn]) {
#pragma unroll
          for (int j = 0; j < 16; ++j) part[tn_pidx(wave, tm, tn, j, lane)] = acc[tm][tn][j];
        }
      });
    });
    return;
  }
  // Stage the 128 x 128 tile in LDS (fp32), then write each kept b x b block
  // with 16-byte stores of 8 consecutive columns.
  constexpr int CS = TILE + 4;
  static_assert(TILE * CS * 4 <= (int)sizeof(smem), "epilogue tile");
  float *Cs = (float *)smem;
  __syncthreads();
  static_for<TM>([&](auto tm) __attribute__((always_inline)) {
    static_for<TN>([&](auto tn) __attribute__((always_inline)) {
      const int col = wn * 64 + tn * 32 + (lane & 31);
#pragma unroll
      for (int j = 0; j < 16; ++j)
        Cs[(wm * 64 + tm * 32 + (j >> 2) * 8 + (lane >> 5) * 4 + (j & 3)) * CS + col] = acc[tm][tn][j];
    });
  });
  __syncthreads();
  constexpr int RCH = BLK / 8;  // 8-column chunks per block row
  const float sc = v.sparse ? a.scale_w : a.scale_lr;
  float wd = 0.f;  // mixing weight: sum of (unscaled sum) x W over stored kept elements
  static_for<GT * GT>([&](auto q) __attribute__((always_inline)) {
    constexpr int ga = q / GT, gb = q % GT;
    const int blk = v.oblk(ga, gb);
    if (blk >= 0) {
      for (int c = tid; c < BLK * RCH; c += 256) {
        const int rl = c / RCH, c8 = (c % RCH) * 8;
        const float *src = Cs + (ga * BLK + rl) * CS + gb * BLK + c8;
        f32x4 lo = *(const f32x4 *)src, hi = *(const f32x4 *)(src + 4);
        if (a.wdot && v.sparse) {
          const T *wp = (const T *)a.wdot + (int64_t)blk * (BLK * BLK) + rl * BLK + c8;
#pragma unroll
          for (int e = 0; e < 4; ++e) wd += lo[e] * to_f<T>(wp[e]) + hi[e] * to_f<T>(wp[4 + e]);
        }
        lo *= sc;
        hi *= sc;
        T *dst = v.sparse ? (T *)a.Wout + (int64_t)blk * (BLK * BLK) + rl * BLK + c8
                          : v.dout + ((int64_t)v.acol(ga) * BLK + rl) * v.ldo + (int64_t)v.bcol(gb) * BLK + c8;
        if constexpr (BF) {
          u32x4 w;
          w[0] = (uint32_t)f2bf(lo[0]) | ((uint32_t)f2bf(lo[1]) << 16);
          w[1] = (uint32_t)f2bf(lo[2]) | ((uint32_t)f2bf(lo[3]) << 16);
          w[2] = (uint32_t)f2bf(hi[0]) | ((uint32_t)f2bf(hi[1]) << 16);
          w[3] = (uint32_t)f2bf(hi[2]) | ((uint32_t)f2bf(hi[3]) << 16);
          *(u32x4 *)dst = w;
        } else {
          *(f32x4 *)dst = lo;
          *(f32x4 *)(dst + 4) = hi;
        }
      }
    }
  });
  if (a.wdot) {
    __shared__ float red[4];
    const float tot = block_sum256(wd, red);
    if (tid == 0) a.wdot_out[item] = tot;
  }
}

// Second pass of a split TN product: sum the split partials in split order
// and store the kept blocks.  Workgroup (item, part): 16 parts of 1024
// partial sums per item; each thread takes 4 consecutive partial sums
// (4 consecutive columns of one output row in the lane-contiguous order).
template <typename T, int BLK>
__global__ __launch_bounds__(256) void tn_reduce_kernel(TNArgs a_arg) {
  const TNArgs a = a_arg;
  const int bid = xcd_remap(blockIdx.x, gridDim.x);
  const int item = bid / 16, part = bid % 16;
  TNItemView<T, BLK> v;
  v.decode(a, item);
  const int q = (part * 256 + threadIdx.x) * 4;  // partial index
  const int lane = q % 64, j = (q / 64) % 16, tn = (q / 1024) % 2, tm = (q / 2048) % 2, wave = q / 4096;
  const int rl = (wave >> 1) * 64 + tm * 32 + (j >> 2) * 8 + (lane >> 5) * 4 + (j & 3);
  const int cl = (wave & 1) * 64 + tn * 32 + (lane & 31);
  const int ga = rl / BLK, gb = cl / BLK;
  const int blk = v.oblk(ga, gb);
  float wd = 0.f;
  if (blk >= 0) {
    // Splits in batches of 4 (loads issued together, added in split order).
    const float *part_p = a.partials + (int64_t)item * a.nsplit * (128 * 128) + q;
    f32x4 acc = *(const f32x4 *)part_p;
    for (int s0 = 1; s0 < a.nsplit; s0 += 4) {
      f32x4 t[4];
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (s0 + u < a.nsplit) t[u] = *(const f32x4 *)(part_p + (int64_t)(s0 + u) * (128 * 128));
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (s0 + u < a.nsplit) acc += t[u];
    }
    const int64_t po = (int64_t)blk * (BLK * BLK) + (rl % BLK) * BLK + (cl % BLK);
    if (a.wdot && v.sparse) {
      const T *wp = (const T *)a.wdot + po;
      wd = ((acc[0] * to_f<T>(wp[0]) + acc[1] * to_f<T>(wp[1])) + acc[2] * to_f<T>(wp[2])) +
           acc[3] * to_f<T>(wp[3]);
    }
    acc *= v.sparse ? a.scale_w : a.scale_lr;
    T *dst = v.sparse ? (T *)a.Wout + po
                      : v.dout + ((int64_t)v.acol(ga) * BLK + (rl % BLK)) * v.ldo + (int64_t)v.bcol(gb) * BLK + (cl % BLK);
    if constexpr (std::is_same<T, bf16_t>::value) {
      uint2 w;
      w.x = (uint32_t)f2bf(acc[0]) | ((uint32_t)f2bf(acc[1]) << 16);
      w.y = (uint32_t)f2bf(acc[2]) | ((uint32_t)f2bf(acc[3]) << 16);
      *(uint2 *)dst = w;
    } else {
      *(f32x4 *)dst = acc;
    }
  }
  if (a.wdot) {
    __shared__ float red[4];
    const float tot = block_sum256(wd, red);
    if (threadIdx.x == 0) a.wdot_out[item * 16 + part] = tot;
  }
}

// ---------------------------------------------------------------------------
// dgamma of the mixing weight: <S, T_lr> in kMixDotParts fixed partials, then
// one workgroup: sum of the kept-block dot partials minus the S.T_lr ones.
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(256) void mix_dot_kernel(const T *__restrict__ S,
                                                      const T *__restrict__ Tl, int64_t n,
                                                      float *__restrict__ out) {
  float x = 0.f;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)kMixDotParts * 256)
    x += to_f<T>(S[i]) * to_f<T>(Tl[i]);
  __shared__ float red[4];
  const float tot = block_sum256(x, red);
  if (threadIdx.x == 0) out[blockIdx.x] = tot;
}

#if PF_GK_HAS(0)
__global__ __launch_bounds__(256) void mix_final_kernel(const float *__restrict__ wparts, int nw,
                                                        const float *__restrict__ sparts, int ns,
                                                        float *__restrict__ dgamma) {
  float x = 0.f;
  for (int i = threadIdx.x; i < nw; i += 256) x += wparts[i];
  for (int i = threadIdx.x; i < ns; i += 256) x -= sparts[i];
  __shared__ float red[4];
  const float tot = block_sum256(x, red);
  if (threadIdx.x == 0) *dgamma = tot;
}

hipError_t launch_mix_dgamma(int dtype, const void *S, const void *T_lr, int64_t n,
                             const float *wparts, int nw, float *sparts, float *dgamma,
                             hipStream_t s) {
  if (n > 0) {
    if (dtype == 0)
      launch_kernel(mix_dot_kernel<bf16_t>, dim3(kMixDotParts), dim3(256), s, (const bf16_t *)S,
                    (const bf16_t *)T_lr, n, sparts);
    else
      launch_kernel(mix_dot_kernel<float>, dim3(kMixDotParts), dim3(256), s, (const float *)S,
                    (const float *)T_lr, n, sparts);
  }
  launch_kernel(mix_final_kernel, dim3(1), dim3(256), s, wparts, nw, (const float *)sparts,
                n > 0 ? kMixDotParts : 0, dgamma);
  return hipGetLastError();
}
#endif

// ---------------------------------------------------------------------------
// GELU backward (standalone elementwise form)
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(256) void gelu_bwd_kernel(int64_t n, const T *dH, const T *Hpre, T *out) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256)
    out[i] = from_f<T>(to_f<T>(dH[i]) * gelu_grad_f(to_f<T>(Hpre[i])));
}

// ---------------------------------------------------------------------------
// Launchers.  The build compiles this file once per part (PF_GK_PART): 0
// holds the small kernels and the dispatch, 1-4 the NT kernel for (bf16 |
// fp32) x (B as [n][k] | [k][n]), 5-6 the TN kernel for bf16 | fp32, so that
// the template instantiations compile in parallel.  Without PF_GK_PART the
// file holds everything.
// ---------------------------------------------------------------------------

template <typename T, int BLK, int G, bool BKN, int BM, bool DENSE>
static hipError_t nt_go(const NTArgs &a, hipStream_t s) {
  const int64_t mtiles = (a.M + BM - 1) / BM;
  const int64_t grid = mtiles * a.ntiles * std::max(1, a.nsplit);
  if (grid <= 0 || grid > 0x7fffffff) return hipErrorInvalidValue;
  // Epilogue variants: the forward takes the GELU-forward one, the
  // backward-data (B read as [k][n]) the GELU-backward one.
  if (!DENSE && a.epi == 1) {
    if constexpr (!DENSE) {
      if constexpr (BKN) launch_kernel(nt_kernel<T, BLK, G, BKN, BM, DENSE, 2>,
                                       dim3((unsigned)grid), dim3(256), s, a);
      else launch_kernel(nt_kernel<T, BLK, G, BKN, BM, DENSE, 1>,
                         dim3((unsigned)grid), dim3(256), s, a);
    }
  } else {
    launch_kernel(nt_kernel<T, BLK, G, BKN, BM, DENSE, 0>, dim3((unsigned)grid), dim3(256), s, a);
  }
  return hipGetLastError();
}

// Instantiated tiles: sparse tiles with BM = 128 and G * b <= 128; dense
// tiles (comparator, skinny rank-r products) with G * b = 128 and BM = 128
// or 64.
template <typename T, int BLK, bool BKN>
static hipError_t nt_dispatch_g(int G, int bm, bool dense, const NTArgs &a, hipStream_t s) {
  constexpr int GMAX = 128 / BLK;
  if (dense) {
    // fp32 rank-r products narrower than 128 columns run one block wide
    // (32-column tiles need 128 token rows: one 32-row MFMA tile per wave).
    if constexpr (std::is_same<T, float>::value && GMAX > 1) {
      if (G == 1) {
        if constexpr (BLK == 32) return nt_go<T, BLK, 1, BKN, 128, true>(a, s);
        else return bm == 64 ? nt_go<T, BLK, 1, BKN, 64, true>(a, s) : nt_go<T, BLK, 1, BKN, 128, true>(a, s);
      }
    }
    if (G != GMAX) return hipErrorInvalidValue;
    return bm == 64 ? nt_go<T, BLK, GMAX, BKN, 64, true>(a, s) : nt_go<T, BLK, GMAX, BKN, 128, true>(a, s);
  }
  if (bm != 128) return hipErrorInvalidValue;
  if (G == 1) return nt_go<T, BLK, 1, BKN, 128, false>(a, s);
  if constexpr (GMAX >= 2)
    if (G == 2) return nt_go<T, BLK, 2, BKN, 128, false>(a, s);
  if constexpr (GMAX >= 4)
    if (G == 4) return nt_go<T, BLK, 4, BKN, 128, false>(a, s);
  return hipErrorInvalidValue;
}

template <typename T, bool BKN>
hipError_t launch_nt_tb(int blk, int G, int bm, bool dense, const NTArgs &a, hipStream_t s) {
  switch (blk) {
    case 32: return nt_dispatch_g<T, 32, BKN>(G, bm, dense, a, s);
    case 64: return nt_dispatch_g<T, 64, BKN>(G, bm, dense, a, s);
    case 128: return nt_dispatch_g<T, 128, BKN>(G, bm, dense, a, s);
    default: return hipErrorInvalidValue;
  }
}
#if PF_GK_HAS(1)
template hipError_t launch_nt_tb<bf16_t, false>(int, int, int, bool, const NTArgs &, hipStream_t);
#endif
#if PF_GK_HAS(2)
template hipError_t launch_nt_tb<bf16_t, true>(int, int, int, bool, const NTArgs &, hipStream_t);
#endif
#if PF_GK_HAS(3)
template hipError_t launch_nt_tb<float, false>(int, int, int, bool, const NTArgs &, hipStream_t);
#endif
#if PF_GK_HAS(4)
template hipError_t launch_nt_tb<float, true>(int, int, int, bool, const NTArgs &, hipStream_t);
#endif

template <typename T, int BLK>
static hipError_t tn_go(const TNArgs &a, hipStream_t s) {
  const int64_t grid = (int64_t)tn_items_total(a, BLK) * a.nsplit;
  if (grid <= 0 || grid > 0x7fffffff) return hipErrorInvalidValue;
  launch_kernel(tn_kernel<T, BLK>, dim3((unsigned)grid), dim3(256), s, a);
  return hipGetLastError();
}

template <typename T, int BLK>
static hipError_t tn_reduce_go(const TNArgs &a, hipStream_t s) {
  const int64_t items = tn_items_total(a, BLK);
  if (items <= 0 || items * 16 > 0x7fffffff) return hipErrorInvalidValue;
  launch_kernel(tn_reduce_kernel<T, BLK>, dim3((unsigned)(items * 16)), dim3(256), s, a);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_tn_t(int blk, const TNArgs &a, hipStream_t s) {
  switch (blk) {
    case 32: return tn_go<T, 32>(a, s);
    case 64: return tn_go<T, 64>(a, s);
    case 128: return tn_go<T, 128>(a, s);
  }
  return hipErrorInvalidValue;
}
template <typename T>
hipError_t launch_tn_reduce_t(int blk, const TNArgs &a, hipStream_t s) {
  switch (blk) {
    case 32: return tn_reduce_go<T, 32>(a, s);
    case 64: return tn_reduce_go<T, 64>(a, s);
    case 128: return tn_reduce_go<T, 128>(a, s);
  }
  return hipErrorInvalidValue;
}
#if PF_GK_HAS(5)
template hipError_t launch_tn_t<bf16_t>(int, const TNArgs &, hipStream_t);
template hipError_t launch_tn_reduce_t<bf16_t>(int, const TNArgs &, hipStream_t);
#endif
#if PF_GK_HAS(6)
template hipError_t launch_tn_t<float>(int, const TNArgs &, hipStream_t);
template hipError_t launch_tn_reduce_t<float>(int, const TNArgs &, hipStream_t);
#endif

#if PF_GK_HAS(0)
hipError_t launch_nt(int dtype, int blk, int G, bool b_kn, int bm, const NTArgs &a, hipStream_t s) {
  const bool dense = a.dense != 0;
  if (dtype == 0)
    return b_kn ? launch_nt_tb<bf16_t, true>(blk, G, bm, dense, a, s)
                : launch_nt_tb<bf16_t, false>(blk, G, bm, dense, a, s);
  return b_kn ? launch_nt_tb<float, true>(blk, G, bm, dense, a, s)
              : launch_nt_tb<float, false>(blk, G, bm, dense, a, s);
}

hipError_t launch_reduce_rows(int dtype, int nsplit, const float *P, int64_t M, int64_t ncols,
                              void *C, int64_t ldc, hipStream_t s) {
  const int64_t n4 = M * ncols / 4;
  const int64_t blocks = std::max<int64_t>(1, std::min<int64_t>((n4 + 255) / 256, 4096));
  if (dtype == 0)
    launch_kernel(reduce_rows_kernel<bf16_t>,
                  dim3((unsigned)blocks), dim3(256), s, nsplit, P, M, ncols, (bf16_t *)C, ldc);
  else
    launch_kernel(reduce_rows_kernel<float>,
                  dim3((unsigned)blocks), dim3(256), s, nsplit, P, M, ncols, (float *)C, ldc);
  return hipGetLastError();
}

hipError_t launch_tn(int dtype, int blk, const TNArgs &a, hipStream_t s) {
  return dtype == 0 ? launch_tn_t<bf16_t>(blk, a, s) : launch_tn_t<float>(blk, a, s);
}

hipError_t launch_tn_reduce(int dtype, int blk, const TNArgs &a, hipStream_t s) {
  return dtype == 0 ? launch_tn_reduce_t<bf16_t>(blk, a, s) : launch_tn_reduce_t<float>(blk, a, s);
}

hipError_t launch_gelu_bwd(int dtype, int64_t n, const void *dH, const void *Hpre, void *out, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  int64_t blocks = std::min<int64_t>((n + 255) / 256, 256 * 64);
  if (dtype == 0)
    launch_kernel(gelu_bwd_kernel<bf16_t>,
                  dim3((unsigned)blocks), dim3(256), s, n, (const bf16_t *)dH,
                  (const bf16_t *)Hpre, (bf16_t *)out);
  else
    launch_kernel(gelu_bwd_kernel<float>,
                  dim3((unsigned)blocks), dim3(256), s, n, (const float *)dH, (const float *)Hpre,
                  (float *)out);
  return hipGetLastError();
}
#endif

}  // namespace pf
