// Internal declarations shared by the host library code and the HIP kernels.
// Not part of the public ABI (see include/pixelfly.h).
#pragma once

#include <hip/hip_runtime_api.h>
#include <stdint.h>

namespace pf {

// Events the next kernel launch of the calling thread records its start and
// end into (set by the C ABI's kernel timing hook; null when it is off).
// The timestamps come from the dispatch itself, so they bracket exactly the
// kernel's execution.
struct LaunchEvents {
  hipEvent_t start = nullptr, stop = nullptr;
};
LaunchEvents &next_launch_events();

// Maximum block rows one NT output tile covers, and blocks per side of a TN
// (weight-gradient) tile.
constexpr int kMaxG = 8;
constexpr int kTNMax = 4;
// Longest weight-gradient launch order carried in the kernel arguments.
constexpr int kTNOrderMax = 1280;

// One output column-tile of the block-sparse "NT" GEMM
//   C[:, out_blk[g]] = sum_c A[:, kcol(c)] . Bblk(g, c)^T  (+ low-rank)
// used by the forward (blocks of M o W) and by backward-data (blocks of the
// transposed layout).  All g rows of a tile share the same K-block list.
struct NTTile {
  int32_t g;         // valid block rows in this tile (<= the kernel's G)
  int32_t nsteps;    // kept K blocks
  int32_t kcol_off;  // offset into kcols: A column block of step c
  int32_t blk_off;   // offset into blks: [nsteps][G] packed block index
  int32_t out_blk[kMaxG];
};

// One weight-gradient tile: a (na*b) x (nb*b) slab of dY^T X of which the
// blocks with out_blk[ga*kTNMax + gb] >= 0 are kept (that CSR position).
struct TNItem {
  int32_t na, nb;
  int32_t a_col[kTNMax];  // dY column blocks (block rows of W)
  int32_t b_col[kTNMax];  // X column blocks (block columns of W)
  int32_t out_blk[kTNMax * kTNMax];
};

// Arguments of the NT kernel family.
struct NTArgs {
  const void *A;        // T x lda (X or dY)
  int64_t lda;
  const void *B;        // packed blocks (dense == 0) or a dense matrix
  int64_t ldb;          // dense B row stride
  int dense;            // 1: K-steps are 0..nsteps-1, B dense (comparator)
  int dense_nsteps;     // dense mode: K / b
  int dense_nblk;       // dense mode: output blocks (N / b)
  const void *L;        // low-rank left operand T x r (T_lr or S), or null
  int64_t ldl;
  const void *R;        // low-rank right operand: U (N x r) or V (r x K)
  int64_t ldr;
  int nlr;              // r / b low-rank K-blocks
  void *C;              // T x ldc output
  int64_t ldc;
  void *C2;             // GELU forward: pre-activation output
  const void *aux;      // GELU backward: pre-activation input
  int epi;
  int64_t M;            // tokens
  const NTTile *tiles;  // null in dense mode
  int ntiles;           // output column tiles (dense mode: ceil(nblk / G))
  const int32_t *kcols;
  const int32_t *blks;
  // Split of the K-steps across workgroups (dense mode only): each split
  // writes fp32 partial outputs P[split][M][ldp]; reduce_rows sums them.
  int nsplit;
  float *partials;
  int64_t ldp;
  // Mixing weight (block-sparse mode, nsplit 1): when mix is set the kept
  // blocks accumulate first, the accumulator is multiplied by mix_ratio at
  // the first low-rank K-block and the result by mix_out, giving
  // alpha * sparse + beta * low-rank with mix_ratio = alpha / beta and
  // mix_out = beta (or mix_out = alpha with no low-rank blocks).
  int mix;
  float mix_ratio, mix_out;
  // Workgroup order of a block-sparse launch with B read [n][k] (forward):
  // 0 walks groups of token tiles over all output tiles; band > 0 walks
  // bands of `band` output tiles, each over all token tiles in groups of
  // four, so that the workgroups of one XCD share one band's weight blocks.
  int band;
};

// A dense region of the TN kernel: out[a][b] = sum_t A[t][a] B[t][b] over
// na_blk x nb_blk blocks (e.g. dU = dY^T T_lr, dV = S^T X).
struct TNDense {
  const void *A;
  int64_t lda;
  const void *B;
  int64_t ldb;
  void *out;
  int64_t ldo;
  int na_blk, nb_blk;   // in blocks
};

struct TNArgs {
  const void *A;        // sparse region: dY (T x lda)
  int64_t lda;
  const void *B;        // sparse region: X (T x ldb)
  int64_t ldb;
  void *Wout;           // packed dW
  const TNItem *items;
  int n_items;
  TNDense dr[2];
  int n_dense;
  int64_t T;
  int nsplit;
  int64_t chunk;        // tokens per split (multiple of 64)
  float *partials;      // [items_total][nsplit][128*128] when nsplit > 1;
                        // the 256 x 256 kernel: two slots of 256*256 per workgroup
  // Mixing weight: stores scale the kept-block sums by scale_w and the dense
  // regions by scale_lr (1 and 1 otherwise).  With wdot set, every workgroup
  // that stores kept blocks also writes the sum over its stored elements of
  // (unscaled fp32 sum) x (the same element of the packed matrix wdot) to
  // wdot_out[item] (nsplit 1) or wdot_out[item * 16 + part] (the split
  // reduction), zero where it stores none.
  float scale_w, scale_lr;
  const void *wdot;
  float *wdot_out;
  // Launch order: launch position i (within a split) runs item order[i]
  // when n_order > 0, item i otherwise.
  int n_order;
  uint16_t order[kTNOrderMax];
};

// Rank-r product C[M x ncols] = A[M x K] . op(B) (bf16, skinny.hip):
// B is ncols x K ([n][k], V) or K x ncols ([k][n], U), row stride ldb.
struct SkinnyArgs {
  const void *A;
  int64_t lda;
  const void *B;
  int64_t ldb;
  void *C;
  int64_t ldc;
  int64_t M;
  int K, ncols;
};

struct AttnArgs {
  const void *Q, *K, *V, *O, *dO;
  void *Oout, *dQ, *dK, *dV;
  float *lse;
  const float *lse_in;
  float *delta;
  int BH, S, nbq;
  int nlong;            // leading block rows / columns kept whole (global stripes)
  int first;            // logical id of the launch's first workgroup (set by the launcher)
  float scale;
  const int32_t *row_ptr, *col_idx, *col_ptr, *row_idx;
};

// Kernel launchers (gemm_kernels.hip / attn_kernels.hip).  bm is the
// M-tile (tokens per workgroup): 128, or 64 for the skinny rank-r products.
hipError_t launch_nt(int dtype, int blk, int G, bool b_kn, int bm, const NTArgs &a,
                     hipStream_t s);
// b = 32 backward-data pairs: Wp[p] (64 x 64 bf16) from the blocks of W that
// src[4p .. 4p + 3] name (-1: zeros).
hipError_t launch_pair_gather(const void *W, const int32_t *src, int npair, void *Wp,
                              hipStream_t s);
// The weight gradient's way back: the blocks of pair blocks Wp[p] that
// src names (>= 0) copied to their places in W.
hipError_t launch_pair_scatter(const void *Wp, const int32_t *src, int npair, void *W,
                               hipStream_t s);
// bf16 NT family with direct global -> LDS operand copies (gemm_dma.hip).
// The output tile is G * blk = 64, 128 or 256 columns wide (the token tile
// follows: 256, 128, 256).  For 128-column tiles `variant` picks 512-token
// tiles (NTD_TALL) or short K-steps with more workgroups per CU
// (NTD_SHORT_K).
enum { NTD_DEFAULT = 0, NTD_TALL = 1, NTD_SHORT_K = 2 };
// Per-(block size, B orientation) parts (one object file each).
template <int BLK, bool BKN>
hipError_t launch_ntd_bb(int G, int variant, const NTArgs &a, hipStream_t s);
// Each part is instantiated in its own object only.
extern template hipError_t launch_ntd_bb<32, false>(int, int, const NTArgs &, hipStream_t);
extern template hipError_t launch_ntd_bb<32, true>(int, int, const NTArgs &, hipStream_t);
extern template hipError_t launch_ntd_bb<64, false>(int, int, const NTArgs &, hipStream_t);
extern template hipError_t launch_ntd_bb<64, true>(int, int, const NTArgs &, hipStream_t);
extern template hipError_t launch_ntd_bb<128, false>(int, int, const NTArgs &, hipStream_t);
extern template hipError_t launch_ntd_bb<128, true>(int, int, const NTArgs &, hipStream_t);
inline hipError_t launch_ntd(int blk, int G, bool b_kn, int variant, const NTArgs &a,
                             hipStream_t s) {
  switch (blk) {
    case 32: return b_kn ? launch_ntd_bb<32, true>(G, variant, a, s) : launch_ntd_bb<32, false>(G, variant, a, s);
    case 64: return b_kn ? launch_ntd_bb<64, true>(G, variant, a, s) : launch_ntd_bb<64, false>(G, variant, a, s);
    case 128: return b_kn ? launch_ntd_bb<128, true>(G, variant, a, s) : launch_ntd_bb<128, false>(G, variant, a, s);
  }
  return hipErrorInvalidValue;
}
// Sum split partials P[nsplit][M][ncols] (fp32) into C (dtype, row stride ldc).
hipError_t launch_reduce_rows(int dtype, int nsplit, const float *P, int64_t M, int64_t ncols,
                              void *C, int64_t ldc, hipStream_t s);
// The TN kernel, and (a.nsplit > 1) the pass that sums its split partials.
hipError_t launch_tn(int dtype, int blk, const TNArgs &a, hipStream_t s);
hipError_t launch_tn_reduce(int dtype, int blk, const TNArgs &a, hipStream_t s);
// bf16 weight gradient on 256 x 256 tiles (blk 64 or 128) on kTNWGrid
// workgroups, or one per item when fewer (gemm_tnw.hip), and the pass that
// sums its `shared` items.
constexpr int kTNWGrid = 256;
constexpr int kTNWMinItems = 192;  // fewest items the 256 x 256 kernel takes
constexpr int kTNWTile = 256;
hipError_t launch_tnw(int blk, int grid, const TNArgs &a, hipStream_t s);
hipError_t launch_tnw_reduce(int blk, int shared, const TNArgs &a, hipStream_t s);
// Per-element-type parts of the register-staged kernels (one object file
// each): T is uint16_t (bf16 storage) or float.
template <typename T, bool BKN>
hipError_t launch_nt_tb(int blk, int G, int bm, bool dense, const NTArgs &a, hipStream_t s);
template <typename T>
hipError_t launch_tn_t(int blk, const TNArgs &a, hipStream_t s);
template <typename T>
hipError_t launch_tn_reduce_t(int blk, const TNArgs &a, hipStream_t s);
extern template hipError_t launch_nt_tb<uint16_t, false>(int, int, int, bool, const NTArgs &, hipStream_t);
extern template hipError_t launch_nt_tb<uint16_t, true>(int, int, int, bool, const NTArgs &, hipStream_t);
extern template hipError_t launch_nt_tb<float, false>(int, int, int, bool, const NTArgs &, hipStream_t);
extern template hipError_t launch_nt_tb<float, true>(int, int, int, bool, const NTArgs &, hipStream_t);
extern template hipError_t launch_tn_t<uint16_t>(int, const TNArgs &, hipStream_t);
extern template hipError_t launch_tn_t<float>(int, const TNArgs &, hipStream_t);
extern template hipError_t launch_tn_reduce_t<uint16_t>(int, const TNArgs &, hipStream_t);
extern template hipError_t launch_tn_reduce_t<float>(int, const TNArgs &, hipStream_t);
// Work items of a TN launch on tile x tile tiles (128 or 256).
int tn_items_total(const TNArgs &a, int blk, int tile = 128);
hipError_t launch_skinny(bool b_kn, const SkinnyArgs &a, hipStream_t s);
// dgamma of the mixing weight: partial sums of <S, T_lr> (n elements,
// kMixDotParts workgroups), then one workgroup adds the kernel-stored partial
// dot products wparts[0 .. nw) and subtracts the S.T_lr partials, in a fixed
// order, into *dgamma.
constexpr int kMixDotParts = 256;
hipError_t launch_mix_dgamma(int dtype, const void *S, const void *T_lr, int64_t n,
                             const float *wparts, int nw, float *sparts, float *dgamma,
                             hipStream_t s);
hipError_t launch_gelu_bwd(int dtype, int64_t n, const void *dH,
                           const void *Hpre, void *out, hipStream_t s);
// Attention launches: part 0 covers every block row (column); with global
// stripes, part 1 runs their nlong long rows (columns) on the grouped
// kernels and part 2 the rest.
hipError_t launch_attn_fwd(const AttnArgs &a, int part, hipStream_t s);
hipError_t launch_attn_bwd_dq(const AttnArgs &a, int part, hipStream_t s);
hipError_t launch_attn_bwd_dkv(const AttnArgs &a, int part, hipStream_t s);
// Product form of the block butterfly (butterfly.hip): one launch applies
// every factor to TM-token x (k * 32)-feature tiles held in LDS.
constexpr int kBflyBlock = 32;
constexpr int kBflyMaxGroupCols = 1024;  // k * 32: the features of one group
struct BflyArgs {
  const void *in;  // X (forward) or dY (backward), T x n
  const void *F;   // factors, packed [nfac][nb][2][32][32] (block-CSR order)
  void *out;       // Y or dX, T x n
  void *save;      // [T][nfac][n]: factor inputs / output gradients, or null
  int64_t T, n;
  int nb, k, nfac;  // n / 32, 2^nfac (blocks per group), factors
};
hipError_t launch_bfly(bool bwd, const BflyArgs &a, hipStream_t s);

// The allocation-free attention backward keeps its row terms in a
// file-scope device array of kAttnScratchRows floats (16 MiB per GPU);
// attn_scratch gives this device's address of it (looked up on the first
// call on each device).
constexpr int64_t kAttnScratchRows = (int64_t)1 << 22;
hipError_t attn_scratch(float **ptr);

}  // namespace pf
