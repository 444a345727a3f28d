// bf16 NT GEMM family for gfx950 with direct global -> LDS operand loads.
//
// Same products as the NT kernel of gemm_kernels.hip (forward and
// backward-data block-sparse products with the fused low-rank K-blocks, the
// dense comparator, the skinny rank-r products), restructured around the
// CDNA4 memory path:
//
//  * Operands move global -> LDS with buffer_load_dwordx4 ... lds: lane i of
//    a wave deposits its 16 bytes at LDS base + 16 i, so one wave instruction
//    fills a 1 KiB "window" and no VGPRs or ds_write instructions are spent
//    on staging.  The lane -> global address map places each 16-byte chunk
//    at an XOR-swizzled position so that the MFMA fragment reads below are
//    free of LDS bank conflicts.
//  * NS pipeline stages live in separate LDS arrays; the step loop is
//    unrolled by NS so every LDS access names its array at compile time.
//    The compiler tracks the LDS DMA of each array separately and therefore
//    only waits for the stage it is about to read.  The cross-wave handoff is
//    an explicit vmcnt wait (this wave's copies of the step have landed)
//    followed by s_barrier (every wave's have).
//  * Operands are swapped in the MFMA (D = W-tile . X-tile^T) so that each
//    lane ends up holding 4 consecutive output columns of one token row; the
//    epilogue transposes each wave's tile through LDS so that every store
//    covers whole 128-byte row segments.
//
// Tile: BM tokens x BN = G * BLK output columns, NW = 4 or 8 waves of 64
// output columns each by BM / (NW / (BN / 64)) tokens (the configurations
// are listed above ntd_cfg).  The virtual K range of a tile is its kept
// blocks, then the r / BLK low-rank blocks, then zero padding to a multiple
// of BK.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>
#include <type_traits>

#include "pf_dma.h"
#include "pf_launch.h"

// Token rows per group of the workgroup order (a group covers the token
// tiles of PF_GROUP_ROWS rows x a run of output tiles, so both operands are
// re-used from L2).
#ifndef PF_GROUP_ROWS
#define PF_GROUP_ROWS 512
#endif

namespace pf {
namespace {

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)lo) |
         ((uint32_t)__builtin_bit_cast(uint16_t, (__bf16)hi) << 16);
}
__device__ __forceinline__ float gelu(float x) {
  return 0.5f * x * (1.0f + erff(x * 0.70710678118654752f));
}
__device__ __forceinline__ float gelu_grad(float x) {
  const float Phi = 0.5f * (1.0f + erff(x * 0.70710678118654752f));
  return Phi + x * 0.39894228040143268f * __expf(-0.5f * x * x);
}

template <int BLK, int G, bool BKN, int BM, int BK, int NS, int NW, bool DENSE, int EPI, int OCC>
__global__ __launch_bounds__(64 * NW, OCC) void ntd_kernel(NTArgs a_arg) {
  const NTArgs a = a_arg;
  constexpr int BN = G * BLK;
  constexpr int KW = BK < BLK ? BK : BLK;  // K width of one sub-block
  constexpr int NH = BK / KW;              // sub-blocks per step
  // Waves: WGN = BN / 64 along N (64 output columns each), the rest along M.
  constexpr int WTN = 64, WGN = BN / WTN, WGM = NW / WGN, WTM = BM / WGM;
  constexpr int TM = WTM / 32, TN = WTN / 32;
  // A region: NH sub-blocks of [BM][KW]; B region: G x NH pieces of [BLK][KW]
  // (NT) or [KW][BLK] (B read as [k][n]).
  constexpr int RBA = KW * 2, RPWA = 1024 / RBA;
  constexpr int RBB = BKN ? BLK * 2 : KW * 2, RPWB = 1024 / RBB;
  constexpr int A_BYTES = BM * BK * 2, B_BYTES = BN * BK * 2;
  constexpr int PIECE = BLK * KW * 2;
  constexpr int AWW = A_BYTES / (1024 * NW), BWW = B_BYTES / (1024 * NW);  // windows per wave
  constexpr int WPH = BM / RPWA;                             // A windows per sub-block
  constexpr int WPP = PIECE / 1024;                          // B windows per piece
  constexpr int DPS = AWW + BWW;                             // copies per wave per step
  static_assert((NW == 4 || NW == 8) && WGN * WGM == NW && WGM * WTM == BM, "waves");
  static_assert(A_BYTES % (1024 * NW) == 0 && B_BYTES % (1024 * NW) == 0, "windows");
  static_assert(WPH % AWW == 0, "one sub-block per wave and step");
  static_assert(WPP % BWW == 0 || BWW % WPP == 0, "piece split");
  static_assert(TM >= 1 && TN >= 1 && WTM % 32 == 0 && WTN % 32 == 0, "wave tile");
  static_assert(NS >= 2 && NS <= 4 && DPS * (NS - 2) < 64, "stages");
  // The lane swizzle of 8-chunk rows alternates between even and odd
  // windows; every wave's first window of a sub-block or piece is even.
  static_assert(RBA != 128 || AWW % 2 == 0, "window parity (A)");
  static_assert(BKN || RBB != 128 || (BWW % 2 == 0 && WPP % 2 == 0), "window parity (B)");

  // Each stage holds its A and B operands in LDS arrays of their own: with
  // the transposed B reads addressed off a small array (frag_kn), the
  // compiler can tell them apart from the next stage's copies and keeps
  // those in flight instead of waiting for them before the reads.
  uint8_t *const sa0 = stage_buf<0, A_BYTES>(), *const sb0 = stage_buf<1, B_BYTES>();
  uint8_t *const sa1 = stage_buf<2, A_BYTES>(), *const sb1 = stage_buf<3, B_BYTES>();
  uint8_t *const sa2 = NS > 2 ? stage_buf<4, A_BYTES>() : sa0;
  uint8_t *const sb2 = NS > 2 ? stage_buf<5, B_BYTES>() : sb0;
  uint8_t *const sa3 = NS > 3 ? stage_buf<6, A_BYTES>() : sa1;
  uint8_t *const sb3 = NS > 3 ? stage_buf<7, B_BYTES>() : sb1;
  struct Stage {
    uint8_t *a, *b;
  };
  auto stage = [&](auto j) __attribute__((always_inline)) -> Stage {
    constexpr int J = decltype(j)::value;
    if constexpr (J == 0) return Stage{sa0, sb0};
    else if constexpr (J == 1) return Stage{sa1, sb1};
    else if constexpr (J == 2) return Stage{sa2, sb2};
    else return Stage{sa3, sb3};
  };

  const bf16_t *__restrict__ A = (const bf16_t *)a.A;
  const bf16_t *__restrict__ B = (const bf16_t *)a.B;
  const bf16_t *__restrict__ L = (const bf16_t *)a.L;
  const bf16_t *__restrict__ R = (const bf16_t *)a.R;

  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = w / WGN, wn = w % WGN;
  const int ntn = a.ntiles;
  const int mtiles = (int)((a.M + BM - 1) / BM);
  const int bid = xcd_remap(blockIdx.x, gridDim.x);
  constexpr int GM = PF_GROUP_ROWS / BM > 0 ? PF_GROUP_ROWS / BM : 1;  // token tiles per group
  const int split = bid / (mtiles * ntn);
  const int lin = bid % (mtiles * ntn);
  int mt, nt;
  if (!DENSE && !BKN && a.band > 0) {
    // Bands of output tiles, each walked by groups of GB token tiles: the
    // consecutive workgroups of one XCD keep one band's weight blocks in
    // its L2 while the token tiles stream past (16384 x 4096 forward at
    // b = 128: 559 -> 544 us, b = 64 389 -> 372 us, b = 32 354 -> 323 us).
    // Backward-data measured slower this way and keeps the groups below.
    constexpr int GB = 4;
    const int band = lin / (mtiles * a.band);
    const int bw = min(a.band, ntn - band * a.band);
    const int r = lin - band * mtiles * a.band;
    const int g = r / (GB * bw);
    const int gsz = min(GB, mtiles - g * GB);
    const int within = r - g * GB * bw;
    mt = g * GB + within % gsz;
    nt = band * a.band + within / gsz;
  } else {
    const int first_m = (lin / (GM * ntn)) * GM;
    const int gsz = min(GM, mtiles - first_m);
    const int within = lin - first_m * ntn;
    mt = first_m + within % gsz;
    nt = within / gsz;
  }
  const int64_t m0 = (int64_t)mt * BM;

  int g_valid, nsteps, kcol_off = 0, blk_off = 0;
  const NTTile *tile = DENSE ? nullptr : a.tiles + nt;
  if constexpr (DENSE) {
    g_valid = min(G, a.dense_nblk - nt * G);
    nsteps = a.dense_nsteps;
  } else {
    g_valid = ld_meta(&tile->g);
    nsteps = ld_meta(&tile->nsteps);
    kcol_off = ld_meta(&tile->kcol_off);
    blk_off = ld_meta(&tile->blk_off);
  }
  auto out_blk = [&](int g) __attribute__((always_inline)) -> int {
    if constexpr (DENSE) return nt * G + min(g, g_valid - 1);
    else return ld_meta(&tile->out_blk[g]);
  };
  const int vblocks = nsteps + a.nlr;
  const int total_all = (vblocks * BLK + BK - 1) / BK;
  const int per_split = (total_all + a.nsplit - 1) / a.nsplit;
  const int s_begin = split * per_split;
  const int total = max(0, min(total_all, s_begin + per_split) - s_begin);

  const bf16_t *const a_base = A + m0 * a.lda;
  const int64_t a_bytes = (a.M - m0) * a.lda * 2;
  const bf16_t *const l_base = DENSE ? A : L + m0 * a.ldl;
  const int64_t l_bytes = DENSE ? 0 : (a.M - m0) * a.ldl * 2;
  constexpr int64_t BIG = 0x7fffffff;

  // Sub-block h of step t: A base, byte range, row stride and column offset
  // (bytes).  Kept block, low-rank block or zero padding, chosen by selects.
  // Dense mode: token tile mt starts its K range mt steps in (mod total)
  // and wraps around.  In step with one another, every tile would read the
  // same columns of rows one operand stride apart (a power of two such as
  // 32 KiB), which concentrates the requests on few HBM channels; staggered
  // starts spread them (the S product at 16384 tokens, 16384 x 256: 219 ->
  // 194 us).  The order is fixed per tile, so results stay deterministic.
  const int rot = (DENSE && total > 0) ? mt % total : 0;
  auto rstep = [&](int t) __attribute__((always_inline)) -> int {
    if constexpr (DENSE) { const int u = t + rot; return u >= total ? u - total : u; }
    else return t;
  };
  auto a_src = [&](int t, int h, const bf16_t *&base, int64_t &bytes, uint32_t &ldb,
                   uint32_t &colb) __attribute__((always_inline)) {
    t = rstep(t);
    const int k0 = (s_begin + t) * BK + h * KW, c = k0 / BLK, kk = k0 % BLK;
    const bool sp = c < nsteps;
    const int kcol = DENSE ? c : ld_meta(&a.kcols[kcol_off + max(min(c, nsteps - 1), 0)]);
    base = sp ? a_base : l_base;
    bytes = sp ? a_bytes : (c < vblocks ? l_bytes : 0);
    ldb = (uint32_t)((sp ? a.lda : a.ldl) * 2);
    colb = (uint32_t)(((sp ? kcol : c - nsteps) * BLK + kk) * 2);
  };
  // Piece (g, h) of step t: B base at the piece, byte range, row stride.
  // ob: output block of piece g (the tile's out_blk[g]).
  auto b_src = [&](int t, int g, int h, int64_t ob, const bf16_t *&base,
                   int64_t &bytes, uint32_t &ldb) __attribute__((always_inline)) {
    t = rstep(t);
    const int k0 = (s_begin + t) * BK + h * KW, c = k0 / BLK, kk = k0 % BLK;
    if constexpr (DENSE) {
      ldb = (uint32_t)(a.ldb * 2);
      base = BKN ? B + ((int64_t)c * BLK + kk) * a.ldb + ob * BLK
                 : B + (ob * BLK) * a.ldb + (int64_t)c * BLK + kk;
      bytes = c < nsteps ? BIG : 0;
    } else {
      const bool sp = c < nsteps;
      const int64_t blk = ld_meta(&a.blks[blk_off + max(min(c, nsteps - 1), 0) * G + g]);
      const int cr = c - nsteps;
      const bf16_t *sp_base = B + blk * (BLK * BLK) + (BKN ? kk * BLK : kk);
      const bf16_t *lr_base = BKN ? R + ((int64_t)cr * BLK + kk) * a.ldr + ob * BLK
                                  : R + (ob * BLK) * a.ldr + (int64_t)cr * BLK + kk;
      base = sp ? sp_base : lr_base;
      bytes = (sp || c < vblocks) ? BIG : 0;
      ldb = (uint32_t)(sp ? BLK * 2 : a.ldr * 2);
    }
  };

  // Lane part of the copy addresses: row within the window and the
  // swizzled chunk (two variants for 8-chunk rows: even / odd window).
  constexpr int CPRA = RBA / 16, CPRB = RBB / 16;
  const uint32_t a_row = (uint32_t)(lane / CPRA);
  uint32_t a_c16[2];
  {
    const int pos = lane % CPRA;
    a_c16[0] = (uint32_t)((pos ^ ((lane >> 4) & 3)) << 4);
    a_c16[1] = (uint32_t)((pos ^ (((lane >> 4) & 3) | (CPRA == 8 ? 4 : 0))) << 4);
  }
  const uint32_t b_row = (uint32_t)(lane / CPRB);
  uint32_t b_c16[2];
  {
    const int pos = lane % CPRB;
    if constexpr (!BKN) {
      b_c16[0] = (uint32_t)((pos ^ ((lane >> 4) & 3)) << 4);
      b_c16[1] = (uint32_t)((pos ^ (((lane >> 4) & 3) | (CPRB == 8 ? 4 : 0))) << 4);
    } else {
      const int x = CPRB == 4 ? 0 : (CPRB == 8 ? (((lane >> 4) & 1) << 2) : ((lane >> 4) << 2));
      b_c16[0] = b_c16[1] = (uint32_t)((pos ^ x) << 4);
    }
  }

  constexpr int PPW = BWW > WPP ? BWW / WPP : 1;  // pieces per wave
  constexpr int WIN = BWW > WPP ? WPP : BWW;      // windows per piece and wave
  // Output block of each of this wave's B pieces (fixed for the tile).
  int64_t ob_w[PPW];
  sfor<PPW>([&](auto pi) __attribute__((always_inline)) {
    const int piece = __builtin_amdgcn_readfirstlane((w * BWW + pi * WIN) / WPP);
    ob_w[pi] = out_blk(piece / NH);
  });

  // Issue this wave's copies of step t into stage st.
  auto issue = [&](int t, Stage st) __attribute__((always_inline)) {
    {
      const int wa0 = w * AWW;
      const int h = __builtin_amdgcn_readfirstlane(wa0 / WPH), wr0 = wa0 % WPH;
      const bf16_t *base;
      int64_t bytes;
      uint32_t ldb, colb;
      a_src(t, h, base, bytes, ldb, colb);
      const rsrc_t r = make_rsrc(base, bytes);
      const uint32_t vrow = a_row * ldb;
      // Dense mode with B read [k][n] on 256-wide tiles is S = dY U of a
      // wide layer: it streams the whole of dY once, and non-temporal copies
      // keep those lines from displacing the rest of the cache (16384 x
      // 4096: S 144 -> 132 us; backward-data, which reads dY next, 2 us
      // slower).  Not on the 128-wide tiles of narrower products (the MLP
      // pair's S: its GELU backward-data then lost 6 us), nor for X in
      // T_lr = X V^T (the forward re-reads X right after).
      constexpr int AAUX = (DENSE && BKN && BN == 256) ? 2 : 0;
      sfor<AWW>([&](auto i) __attribute__((always_inline)) {
        const int wr = wr0 + i;
        dma16<AAUX>(r, st.a + (wa0 + i) * 1024, vrow + a_c16[i & 1],
                    (uint32_t)(wr * RPWA) * ldb + colb);
      });
    }
    sfor<PPW>([&](auto pi) __attribute__((always_inline)) {
      const int wb0 = w * BWW + pi * WIN;
      // Uniform; readfirstlane lets the block lookups stay scalar loads.
      const int piece = __builtin_amdgcn_readfirstlane(wb0 / WPP), wi0 = wb0 % WPP;
      const bf16_t *base;
      int64_t bytes;
      uint32_t ldb;
      b_src(t, piece / NH, piece % NH, ob_w[pi], base, bytes, ldb);
      const rsrc_t r = make_rsrc(base, bytes);
      const uint32_t vrow = b_row * ldb;
      sfor<WIN>([&](auto i) __attribute__((always_inline)) {
        dma16(r, st.b + (wb0 + i) * 1024, vrow + b_c16[i & 1],
              (uint32_t)((wi0 + i) * RPWB) * ldb);
      });
    });
  };

  f32x16 acc[TN][TM];
  sfor<TN>([&](auto i) __attribute__((always_inline)) {
    sfor<TM>([&](auto j) __attribute__((always_inline)) {
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;
    });
  });

  // Mixing weight: scale the kept-block sums once, at the first low-rank
  // K-block (virtual K index nsteps * BLK).
  const int kswitch = nsteps * BLK;
  // The switch check is a branch per K slice; launches without the mixing
  // weight run an instantiation without it (see the loop below).
  auto compute_m = [&](Stage st, int t, auto mix) __attribute__((always_inline)) {
    sfor<BK / 16>([&](auto ks) __attribute__((always_inline)) {
      constexpr int h = (ks * 16) / KW, kq = ks % (KW / 16);
      if (decltype(mix)::value && (s_begin + t) * BK + ks * 16 == kswitch) {
        sfor<TN>([&](auto tn) __attribute__((always_inline)) {
          sfor<TM>([&](auto tm) __attribute__((always_inline)) {
#pragma unroll
            for (int e = 0; e < 16; ++e) acc[tn][tm][e] *= a.mix_ratio;
          });
        });
      }
      bf16x8 xf[TM], wf[TN];
      sfor<TM>([&](auto tm) __attribute__((always_inline)) {
        xf[tm] = frag_rows<RBA>(st.a + h * (BM * RBA), wm * WTM + tm * 32, kq, lane);
      });
      sfor<TN>([&](auto tn) __attribute__((always_inline)) {
        const int n0 = wn * WTN + tn * 32;
        const int g = n0 / BLK, nl = n0 % BLK;
        const uint8_t *piece = st.b + (g * NH + h) * PIECE;
        if constexpr (BKN) wf[tn] = frag_kn<RBB>(piece, nl, kq, lane);
        else wf[tn] = frag_rows<RBB>(piece, nl, kq, lane);
      });
      sfor<TN>([&](auto tn) __attribute__((always_inline)) {
        sfor<TM>([&](auto tm) __attribute__((always_inline)) {
          acc[tn][tm] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wf[tn], xf[tm], acc[tn][tm], 0, 0, 0);
        });
      });
    });
  };

  // Pipeline: steps 0 .. NS-2 in flight before the loop; at step t the
  // copies of step t + NS - 1 go into the stage freed by step t - 1.
  sfor<NS - 1>([&](auto j) __attribute__((always_inline)) {
    if (j < total) issue(j, stage(j));
  });
  auto run = [&](auto mix) __attribute__((always_inline)) {
    auto compute = [&](Stage st, int t) __attribute__((always_inline)) {
      compute_m(st, t, mix);
    };
    for (int t0 = 0; t0 < total; t0 += NS) {
      bool done = false;
      sfor<NS>([&](auto j) __attribute__((always_inline)) {
        if (done) return;
        const int t = t0 + j;
        if (t >= total) {
          done = true;
          return;
        }
        // Copies of steps t+1 .. t+NS-2 that were issued may still be in
        // flight; step t's must have landed.
        const int ahead = min(NS - 2, total - 1 - t);
        if constexpr (NS == 2) {
          wait_vm<0>();
        } else if constexpr (NS == 3) {
          if (ahead >= 1) wait_vm<DPS>(); else wait_vm<0>();
        } else {
          if (ahead >= 2) wait_vm<2 * DPS>();
          else if (ahead == 1) wait_vm<DPS>();
          else wait_vm<0>();
        }
        barrier();
        if (t + NS - 1 < total) issue(t + NS - 1, stage(std::integral_constant<int, (j + NS - 1) % NS>{}));
        compute(stage(j), t);
      });
    }
  };
  if (a.mix) run(std::true_type{});
  else run(std::false_type{});

  // Epilogue.  Lane l of accumulator (tn, tm) holds token row tm*32 + l%32
  // and, for q = 0..3, output columns tn*32 + q*8 + (l/32)*4 + 0..3.  Full
  // 128-byte row segments store far faster than 8-byte pieces scattered
  // over 32 rows, so each wave transposes its tile through LDS, 32 rows at a
  // time (fp32 values in 16-byte chunks XOR-swizzled by row; plain bf16
  // outputs are rounded first and staged as bf16, see below), and every
  // lane then writes 8 consecutive columns of one row.  The staging area is the stage
  // buffer no wave reads in the last step; it needs no barrier because each
  // wave only touches its own slice and a wave's LDS accesses are ordered.
  constexpr int SROW = WTN * 4, SCH = SROW / 16;  // staged row bytes, chunks
  constexpr int SP = 32;                          // rows per pass
  constexpr int LPR = WTN / 8, RPI = 64 / LPR;    // lanes per row, rows per store step
  // Staging slices per stage (in its A array, then its B array); the stages
  // used are the ones after the stage read in the last step, so NW / WPS of
  // them must not wrap around to it.
  constexpr int SLICE = SP * SROW, SPA = A_BYTES / SLICE, SPB = B_BYTES / SLICE;
  constexpr int WPS = SPA + SPB < NW ? SPA + SPB : NW;
  static_assert(WPS >= 1 && (NW + WPS - 1) / WPS <= NS - 1, "staging room");
  static_assert((SCH & (SCH - 1)) == 0 && SP % RPI == 0, "staging");
  const int sidx = (total + w / WPS) % NS, slice = w % WPS;
  uint8_t *const sta = sidx == 0 ? sa0 : sidx == 1 ? sa1 : sidx == 2 ? sa2 : sa3;
  uint8_t *const stb = sidx == 0 ? sb0 : sidx == 1 ? sb1 : sidx == 2 ? sb2 : sb3;
  uint8_t *const stg = slice < SPA ? sta + slice * SLICE : stb + (slice - SPA) * SLICE;
  int ob[G];
  sfor<G>([&](auto g) __attribute__((always_inline)) { ob[g] = out_blk(g); });
  bf16_t *C = (bf16_t *)a.C;
  const int jl = lane % LPR, rl = lane / LPR;
  const int cn = wn * WTN + jl * 8;  // first of this lane's 8 columns in the tile
  const int gcol = cn / BLK;
  int obg = ob[0];
  sfor<G>([&](auto gg) __attribute__((always_inline)) { if (gcol == gg) obg = ob[gg]; });
  const int64_t col = (int64_t)obg * BLK + cn % BLK;
  const bool col_ok = gcol < g_valid;
  // Plain bf16 outputs of the block-sparse products (no GELU, no split
  // partials): round to bf16 first and stage half the bytes.  A staged row
  // is 64 columns = 16 units of 4 columns (8 bytes); lane l writes unit
  // u = tn*8 + q*2 + l/32 of row l%32 at unit position u ^ (row & 15), so
  // the 16 rows of a half-wave fill 16 different bank pairs.  A reader of
  // 8 columns (units 2j, 2j + 1) finds them in one 16-byte chunk, in order
  // when row & 1 is 0 and swapped when it is 1.  Same rounding as the fp32
  // path: each value is rounded once, after the mixing-weight scale.
  constexpr bool BF16_STAGE = !DENSE && EPI == 0;
  if constexpr (BF16_STAGE) {
    constexpr int SROW2 = WTN * 2;
    static_assert(SROW2 == 128 && 32 * SROW2 <= SLICE, "bf16 staging");
    sfor<TM>([&](auto tm) __attribute__((always_inline)) {
      const int r = lane & 31;
      sfor<TN>([&](auto tn) __attribute__((always_inline)) {
        sfor<4>([&](auto q) __attribute__((always_inline)) {
          float v0 = acc[tn][tm][q * 4 + 0], v1 = acc[tn][tm][q * 4 + 1];
          float v2 = acc[tn][tm][q * 4 + 2], v3 = acc[tn][tm][q * 4 + 3];
          if (a.mix) {
            v0 *= a.mix_out;
            v1 *= a.mix_out;
            v2 *= a.mix_out;
            v3 *= a.mix_out;
          }
          const int u = tn * 8 + q * 2 + (lane >> 5);
          *(u32x2 *)(stg + r * SROW2 + ((u ^ (r & 15)) << 3)) =
              u32x2{pack_bf16x2(v0, v1), pack_bf16x2(v2, v3)};
        });
      });
      sfor<32 / RPI>([&](auto it) __attribute__((always_inline)) {
        const int rr = it * RPI + rl, sw = rr & 15;
        u32x4 v = *(const u32x4 *)(stg + rr * SROW2 + ((((2 * jl) ^ sw) >> 1) << 4));
        if (sw & 1) v = u32x4{v[2], v[3], v[0], v[1]};
        const int64_t gm = m0 + wm * WTM + tm * 32 + rr;
        if (gm >= a.M || !col_ok) return;
        // Streaming store: the output is not read again by this launch, and
        // keeping it out of the caches leaves them to the operands (16384 x
        // 4096 step at b = 128: 1.754 -> 1.730 ms; S = dY U, which follows,
        // 158 -> 146 us).
        __builtin_nontemporal_store(v, (u32x4 *)(C + gm * a.ldc + col));
      });
    });
    return;
  }
  sfor<TM * (32 / SP)>([&](auto pass) __attribute__((always_inline)) {
    constexpr int tm = pass / (32 / SP), half = pass % (32 / SP);
    if ((lane & 31) / SP == half) {
      const int r = (lane & 31) % SP;
      sfor<TN>([&](auto tn) __attribute__((always_inline)) {
        sfor<4>([&](auto q) __attribute__((always_inline)) {
          const int c = tn * 8 + q * 2 + (lane >> 5);
          *(f32x4 *)(stg + r * SROW + ((c ^ (r & (SCH - 1))) << 4)) =
              f32x4{acc[tn][tm][q * 4 + 0], acc[tn][tm][q * 4 + 1], acc[tn][tm][q * 4 + 2],
                    acc[tn][tm][q * 4 + 3]};
        });
      });
    }
    sfor<SP / RPI>([&](auto it) __attribute__((always_inline)) {
      const int r = it * RPI + rl;
      const f32x4 lo = *(const f32x4 *)(stg + r * SROW + (((2 * jl) ^ (r & (SCH - 1))) << 4));
      const f32x4 hi = *(const f32x4 *)(stg + r * SROW + (((2 * jl + 1) ^ (r & (SCH - 1))) << 4));
      const int64_t gm = m0 + wm * WTM + tm * 32 + half * SP + r;
      if (gm >= a.M || !col_ok) return;
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
        *(u32x4 *)((bf16_t *)a.C2 + o) = u32x4{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]),
                                               pack_bf16x2(v[4], v[5]), pack_bf16x2(v[6], v[7])};
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = gelu(v[e]);
      } else if constexpr (EPI == 2) {  // backward GELU: scale by gelu'(pre-activation)
        const u32x4 x = *(const u32x4 *)((const bf16_t *)a.aux + o);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          v[2 * e] *= gelu_grad(__uint_as_float(x[e] << 16));
          v[2 * e + 1] *= gelu_grad(__uint_as_float(x[e] & 0xffff0000u));
        }
      }
      *(u32x4 *)(C + o) = u32x4{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]),
                                pack_bf16x2(v[4], v[5]), pack_bf16x2(v[6], v[7])};
    });
  });
}

template <int BLK, int G, bool BKN, int BM, int BK, int NS, int NW, bool DENSE, int OCC>
hipError_t ntd_go(const NTArgs &a, hipStream_t s) {
  const int64_t mtiles = (a.M + BM - 1) / BM;
  const int64_t grid = mtiles * a.ntiles * std::max(1, a.nsplit);
  if (grid <= 0 || grid > 0x7fffffff) return hipErrorInvalidValue;
  if (!DENSE && a.epi == 1) {
    if constexpr (!DENSE) {
      if constexpr (BKN)
        launch_kernel(ntd_kernel<BLK, G, BKN, BM, BK, NS, NW, DENSE, 2, OCC>,
                      dim3((unsigned)grid), dim3(64 * NW), s, a);
      else
        launch_kernel(ntd_kernel<BLK, G, BKN, BM, BK, NS, NW, DENSE, 1, OCC>,
                      dim3((unsigned)grid), dim3(64 * NW), s, a);
    }
  } else {
    launch_kernel(ntd_kernel<BLK, G, BKN, BM, BK, NS, NW, DENSE, 0, OCC>,
                  dim3((unsigned)grid), dim3(64 * NW), s, a);
  }
  return hipGetLastError();
}

// Tile configurations, chosen by the output tile width G * BLK:
//   128: 128 x 128 tiles, 4 waves, two workgroups per CU; or (tall) 512 x
//        128 tiles, 8 waves of 128 x 64, one workgroup per CU; or (short K
//        lists) 128 x 128 tiles with K-steps of 32 in three stages, three
//        workgroups per CU;
//   256: 256 x 256 tiles, 8 waves of 128 x 64, one workgroup per CU;
//    64: 256 x  64 tiles, 4 waves, two workgroups per CU.
// The others take K-steps of 64 in two stages.  The 8-wave tiles read half
// the operand bytes per flop of the 128 x 128 ones and keep two waves per
// SIMD; the short-K variant keeps more workgroups per CU in flight when each
// has only a few steps.
template <int BLK, int G, bool BKN, bool DENSE>
hipError_t ntd_cfg(int variant, const NTArgs &a, hipStream_t s) {
  constexpr int BN = G * BLK;
  if constexpr (BN == 128) {
    if (variant == NTD_TALL) return ntd_go<BLK, G, BKN, 512, 64, 2, 8, DENSE, 1>(a, s);
    if (variant == NTD_SHORT_K) return ntd_go<BLK, G, BKN, 128, 32, 3, 4, DENSE, 3>(a, s);
    return ntd_go<BLK, G, BKN, 128, 64, 2, 4, DENSE, 2>(a, s);
  } else if constexpr (BN == 256) {
    return ntd_go<BLK, G, BKN, 256, 64, 2, 8, DENSE, 1>(a, s);
  } else if constexpr (BN == 64) {
    return ntd_go<BLK, G, BKN, 256, 64, 2, 4, DENSE, 2>(a, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace

// The launcher of one (block size, B orientation) pair.  The build compiles
// this file once per pair (PF_PART_BLK, PF_PART_BKN) so that the
// instantiations compile in parallel; launch_ntd in the C ABI code picks the
// pair.
template <int BLK, bool BKN>
hipError_t launch_ntd_bb(int G, int variant, const NTArgs &a, hipStream_t s) {
  const bool dense = a.dense != 0;
  auto go = [&](auto g) {
    constexpr int GG = decltype(g)::value;
    return dense ? ntd_cfg<BLK, GG, BKN, true>(variant, a, s)
                 : ntd_cfg<BLK, GG, BKN, false>(variant, a, s);
  };
  if (G * BLK == 128) return go(std::integral_constant<int, 128 / BLK>{});
  if (G * BLK == 256) return go(std::integral_constant<int, 256 / BLK>{});
  if constexpr (BLK <= 64)
    if (G * BLK == 64) return go(std::integral_constant<int, 64 / BLK>{});
  return hipErrorInvalidValue;
}

#if defined(PF_PART_BLK) && defined(PF_PART_BKN)
template hipError_t launch_ntd_bb<PF_PART_BLK, (PF_PART_BKN != 0)>(int, int, const NTArgs &,
                                                                    hipStream_t);
#endif

}  // namespace pf
