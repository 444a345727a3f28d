// Layout object: flat block butterfly block-CSR plus the kernel work lists.
#pragma once

#include <string>
#include <vector>

#include "pf_internal.h"
#include "pixelfly.h"

struct pf_layout {
  int64_t n_out = 0, n_in = 0;
  int32_t b = 0, max_stride = 0, eff_stride = 0, s = 0, nb_out = 0, nb_in = 0;
  int32_t global_blocks = 0;  // attention layouts: width of the global stripes (blocks)
  // Product-form butterfly layouts: the n x n matrix and its number of
  // factors (strides 2 .. 2^bfly_nfac); 0 for every other layout.
  int64_t bfly_n = 0;
  int32_t bfly_nfac = 0;
  int64_t nnzb = 0;
  std::vector<int32_t> row_ptr, col_idx, col_ptr, row_idx, tperm;

  // Work lists.  Forward NT tiles cover output block rows (tiles of G_fwd
  // rows with identical column sets); backward-data NT tiles cover block
  // columns (tiles of G_bwd columns with identical row sets); TN items cover
  // the kept blocks for the weight gradient.  The "_w" lists group up to
  // 256 / b rows (wide tiles of the bf16 kernels), the others up to 128 / b.
  int G_fwd = 1, G_bwd = 1, G_fwd_w = 1, G_bwd_w = 1;
  int kmax_fwd = 0, kmax_bwd = 0;  // most kept K-blocks of any forward / backward-data tile
  std::vector<pf::NTTile> fwd_tiles, bwd_tiles, fwd_tiles_w, bwd_tiles_w;
  std::vector<int32_t> kcols_fwd, blks_fwd, kcols_bwd, blks_bwd;
  std::vector<int32_t> kcols_fwd_w, blks_fwd_w, kcols_bwd_w, blks_bwd_w;
  std::vector<pf::TNItem> tn_items;
  // Weight-gradient items of the 256 x 256 bf16 kernel (b = 64 or 128):
  // bundles of 256 / b block rows x 256 / b block columns; empty otherwise.
  std::vector<pf::TNItem> tn_items_w;
  // Backward-data in 64-wide pairs (b = 32 with even block counts): block
  // rows and columns taken in aligned pairs (2i, 2i + 1), a 64 x 64 pair
  // block kept when any of its four b x b blocks is.  One tile per pair
  // column (kcols: its pair rows, blks: pair block indices); pair_src holds
  // for each pair block the CSR positions of its blocks (row half * 2 +
  // column half; -1 for a dropped block, read as zeros).  Empty otherwise.
  std::vector<pf::NTTile> bwd_tiles_p;
  std::vector<int32_t> kcols_bwd_p, blks_bwd_p, pair_src;
  int kmax_bwd_p = 0;
  // The pair blocks as a block-CSR of their own (pair rows x pair columns,
  // pair block ids in this order, pair_src indexed by them) and the
  // weight-gradient items of the 256 x 256 kernel over it (bundles of four
  // pair rows x runs of four pair columns).
  std::vector<int32_t> pr_ptr, pr_col;
  std::vector<pf::TNItem> tn_items_p;

  // Device copies (valid after pf_layout_upload).
  int device = -1;
  void *dev_mem = nullptr;
  const pf::NTTile *d_fwd_tiles = nullptr, *d_bwd_tiles = nullptr;
  const int32_t *d_kcols_fwd = nullptr, *d_blks_fwd = nullptr;
  const int32_t *d_kcols_bwd = nullptr, *d_blks_bwd = nullptr;
  const pf::NTTile *d_fwd_tiles_w = nullptr, *d_bwd_tiles_w = nullptr;
  const int32_t *d_kcols_fwd_w = nullptr, *d_blks_fwd_w = nullptr;
  const int32_t *d_kcols_bwd_w = nullptr, *d_blks_bwd_w = nullptr;
  const pf::TNItem *d_tn_items = nullptr, *d_tn_items_w = nullptr;
  const pf::NTTile *d_bwd_tiles_p = nullptr;
  const pf::TNItem *d_tn_items_p = nullptr;
  const int32_t *d_kcols_bwd_p = nullptr, *d_blks_bwd_p = nullptr, *d_pair_src = nullptr;
  const int32_t *d_row_ptr = nullptr, *d_col_idx = nullptr;
  const int32_t *d_col_ptr = nullptr, *d_row_idx = nullptr;
};

namespace pf {
// Build mask + block-CSR + work lists (host only).  Returns "" or an error.
std::string build_layout(pf_layout &L, int64_t n_out, int64_t n_in, int32_t b,
                         int32_t max_stride);
// Same from an explicit nb_out x nb_in block mask (row-major, nonzero =
// kept); every block row must keep at least one block.
std::string build_layout_from_mask(pf_layout &L, int32_t nb_out, int32_t nb_in, int32_t b,
                                   const uint8_t *mask);
// Attention layout: square flat block butterfly of side seq / b plus the
// first global_blocks block rows and columns.
std::string build_attention_layout(pf_layout &L, int64_t seq, int32_t b, int32_t max_stride,
                                   int32_t global_blocks);
// Layout of I + B_k (one factor of the butterfly product form), n x n.
std::string build_factor_layout(pf_layout &L, int64_t n, int32_t b, int32_t k);
// Layout of the (b, b)-block cover of an n_out x n_in element mask.
std::string build_cover_layout(pf_layout &L, int64_t n_out, int64_t n_in, int32_t b,
                               const uint8_t *elem_mask);
// Stacked factor supports of the product form of an n x n block butterfly
// with strides 2 .. max_stride: an (L nb) x (L nb) block-diagonal layout
// (L = log2 max_stride, nb = n / b) whose f-th diagonal block keeps (p, p)
// and (p, p XOR 2^f).  Its block-CSR order is the packing of the factors.
std::string build_butterfly_layout(pf_layout &L, int64_t n, int32_t b, int32_t max_stride);
std::string finish_layout(pf_layout &L);
// Re-verify the work lists against the block-CSR.  Returns "" or an error.
std::string check_layout(const pf_layout &L);
// Blocks per NT tile row-group the kernels are instantiated for (narrow and
// wide lists).
int max_group(int32_t b);
int max_group_wide(int32_t b);
}  // namespace pf
