// Flat block butterfly layout builder (host only).
//
// Mask: Section 3.1 (block butterfly factor B_k: [[D1 D2],[D3 D4]] with
// block-diagonal D_i; factor matrix: block-diagonal copies of one factor),
// Section 3.2 (flat butterfly of maximum stride k = I + B_2 + ... + B_k).
// In block units the support of B_k pairs p with p XOR k/2 (the two
// diagonal positions of one factor that share the in-quadrant offset), so the
// flat pattern keeps (p, q) iff p XOR q is 0 or a power of two below the
// maximum stride.  A square side s that is not a power of two is the
// power-of-two pattern cropped to s; rectangular weights repeat ("stretch")
// the s x s square along the longer dimension (appendix on method details,
// rectangular matrices).
#include "layout.h"

#include <algorithm>
#include <map>
#include <string>
#include <vector>

namespace pf {

// Widest NT output tile in columns (the tile is G blocks of b columns).
#ifndef PF_MAX_BN
#define PF_MAX_BN 128
#endif

int max_group(int32_t b) {
  if (b != 32 && b != 64 && b != 128) return 1;
  return std::max(1, std::min(4, PF_MAX_BN / b));
}

int max_group_wide(int32_t b) {
  if (b != 32 && b != 64 && b != 128) return 1;
  return std::max(1, std::min(kMaxG, 256 / b));
}

static int tn_group(int32_t b) {
  int g = b > 0 ? 128 / b : 1;
  return std::max(1, std::min(kTNMax, g));
}

static bool is_pow2(int64_t x) { return x > 0 && (x & (x - 1)) == 0; }

// Choose the largest G (power of two <= gmax) whose partial tiles waste at
// most a quarter of the tile rows.
static int choose_group(const std::vector<std::vector<int32_t>> &groups,
                        int gmax) {
  int64_t rows = 0;
  for (auto &g : groups) rows += (int64_t)g.size();
  for (int G = gmax; G > 1; G /= 2) {
    int64_t tiles = 0;
    for (auto &g : groups) tiles += ((int64_t)g.size() + G - 1) / G;
    if ((tiles * G - rows) * 4 <= rows) return G;
  }
  return 1;
}

// Group the block rows of a CSR-like structure by identical index lists.
static std::vector<std::vector<int32_t>> group_identical(
    const std::vector<int32_t> &ptr, const std::vector<int32_t> &idx) {
  std::map<std::vector<int32_t>, int> where;
  std::vector<std::vector<int32_t>> groups;
  int n = (int)ptr.size() - 1;
  for (int i = 0; i < n; ++i) {
    std::vector<int32_t> key(idx.begin() + ptr[i], idx.begin() + ptr[i + 1]);
    auto it = where.find(key);
    if (it == where.end()) {
      where.emplace(key, (int)groups.size());
      groups.push_back({i});
    } else {
      groups[it->second].push_back(i);
    }
  }
  return groups;
}

// NT tiles over the rows of (ptr, idx).  blk_of(row, slot) gives the packed
// block index of the slot-th kept block of that row.
template <class BlkOf>
static void build_nt_tiles(const std::vector<int32_t> &ptr,
                           const std::vector<int32_t> &idx, int gmax,
                           BlkOf blk_of, int &G, std::vector<NTTile> &tiles,
                           std::vector<int32_t> &kcols,
                           std::vector<int32_t> &blks) {
  auto groups = group_identical(ptr, idx);
  G = choose_group(groups, gmax);
  tiles.clear();
  kcols.clear();
  blks.clear();
  for (auto &grp : groups) {
    int r0 = grp[0];
    int nsteps = ptr[r0 + 1] - ptr[r0];
    int kcol_off = (int)kcols.size();
    for (int c = 0; c < nsteps; ++c) kcols.push_back(idx[ptr[r0] + c]);
    for (size_t t0 = 0; t0 < grp.size(); t0 += G) {
      NTTile t{};
      t.g = (int)std::min<size_t>(G, grp.size() - t0);
      t.nsteps = nsteps;
      t.kcol_off = kcol_off;
      t.blk_off = (int)blks.size();
      for (int g = 0; g < kMaxG; ++g)
        t.out_blk[g] = g < t.g ? grp[t0 + g] : grp[t0];
      for (int c = 0; c < nsteps; ++c)
        for (int g = 0; g < G; ++g)
          blks.push_back(blk_of(g < t.g ? grp[t0 + g] : grp[t0], c));
      tiles.push_back(t);
    }
  }
  // One step of padding: kernels read the tables at step max(min(c, nsteps
  // - 1), 0), so a tile without kept blocks (an empty block column on the
  // backward-data side) still reads inside them.
  kcols.push_back(0);
  for (int g = 0; g < G; ++g) blks.push_back(0);
}

static int32_t csr_pos(const pf_layout &L, int i, int j) {
  auto b = L.col_idx.begin() + L.row_ptr[i], e = L.col_idx.begin() + L.row_ptr[i + 1];
  auto it = std::lower_bound(b, e, j);
  return (it != e && *it == j) ? (int32_t)(it - L.col_idx.begin()) : -1;
}

// Weight-gradient items of GA x GA blocks: block rows with identical column
// lists bundled GA at a time (the rest bundled in row order), each bundle's
// column union cut into runs of GA columns.
static void build_tn_items(pf_layout &L, int GA, std::vector<TNItem> &out) {
  const int GB = GA;
  auto groups = group_identical(L.row_ptr, L.col_idx);
  std::vector<std::vector<int32_t>> bundles;
  std::vector<int32_t> leftover;
  for (auto &grp : groups) {
    size_t full = grp.size() / GA * GA;
    for (size_t t = 0; t < full; t += GA)
      bundles.emplace_back(grp.begin() + t, grp.begin() + t + GA);
    for (size_t t = full; t < grp.size(); ++t) leftover.push_back(grp[t]);
  }
  std::sort(leftover.begin(), leftover.end());
  for (size_t t = 0; t < leftover.size(); t += GA)
    bundles.emplace_back(leftover.begin() + t,
                         leftover.begin() + std::min(leftover.size(), t + GA));
  out.clear();
  for (auto &bun : bundles) {
    std::vector<int32_t> cols;
    for (int i : bun)
      cols.insert(cols.end(), L.col_idx.begin() + L.row_ptr[i],
                  L.col_idx.begin() + L.row_ptr[i + 1]);
    std::sort(cols.begin(), cols.end());
    cols.erase(std::unique(cols.begin(), cols.end()), cols.end());
    for (size_t c0 = 0; c0 < cols.size(); c0 += GB) {
      TNItem it{};
      it.na = (int)bun.size();
      it.nb = (int)std::min<size_t>(GB, cols.size() - c0);
      for (int a = 0; a < kTNMax; ++a) it.a_col[a] = a < it.na ? bun[a] : bun[0];
      for (int b = 0; b < kTNMax; ++b) it.b_col[b] = b < it.nb ? cols[c0 + b] : cols[c0];
      for (int a = 0; a < kTNMax; ++a)
        for (int b = 0; b < kTNMax; ++b)
          it.out_blk[a * kTNMax + b] =
              (a < it.na && b < it.nb) ? csr_pos(L, bun[a], cols[c0 + b]) : -1;
      out.push_back(it);
    }
  }
}

static void build_tn_items(pf_layout &L) {
  build_tn_items(L, tn_group(L.b), L.tn_items);
  L.tn_items_w.clear();
  if (L.b == 64 || L.b == 128) build_tn_items(L, 256 / L.b, L.tn_items_w);
}

std::string build_layout(pf_layout &L, int64_t n_out, int64_t n_in, int32_t b,
                         int32_t max_stride) {
  if (b < 1) return "block size b must be >= 1";
  if (n_out < 1 || n_in < 1) return "n_out and n_in must be >= 1";
  if (n_out % b || n_in % b) return "b must divide n_out and n_in";
  if (!is_pow2(max_stride)) return "max_stride must be a power of two >= 1";
  if (n_out / b > (1 << 30) || n_in / b > (1 << 30)) return "too many blocks";
  L.n_out = n_out;
  L.n_in = n_in;
  L.b = b;
  L.max_stride = max_stride;
  L.nb_out = (int32_t)(n_out / b);
  L.nb_in = (int32_t)(n_in / b);
  L.s = std::min(L.nb_out, L.nb_in);
  int64_t P = 1;
  while (P < L.s) P *= 2;
  L.eff_stride = (int32_t)std::min<int64_t>(max_stride, P);

  // Kept in-square columns of each square row.
  std::vector<std::vector<int32_t>> sq(L.s);
  for (int32_t ii = 0; ii < L.s; ++ii)
    for (int32_t jj = 0; jj < L.s; ++jj) {
      int32_t x = ii ^ jj;
      if (x == 0 || (is_pow2(x) && x < max_stride)) sq[ii].push_back(jj);
    }
  L.row_ptr.assign(1, 0);
  L.col_idx.clear();
  for (int32_t i = 0; i < L.nb_out; ++i) {
    for (int64_t base = 0; base < L.nb_in; base += L.s)
      for (int32_t jj : sq[i % L.s])
        if (base + jj < L.nb_in) L.col_idx.push_back((int32_t)(base + jj));
    L.row_ptr.push_back((int32_t)L.col_idx.size());
  }
  return finish_layout(L);
}

// Attention score layout: the square flat block butterfly of the sequence
// (block units nb = seq / b) plus the global component of the appendix on
// method details (low-rank in attention): the first global_blocks block rows
// (queries that attend to every key) and block columns (keys every query
// attends to), as a union of supports.
std::string build_attention_layout(pf_layout &L, int64_t seq, int32_t b, int32_t max_stride,
                                   int32_t global_blocks) {
  if (b < 1 || seq < 1 || seq % b) return "seq must be a positive multiple of b";
  if (seq / b > 16384) return "seq / b must be <= 16384";
  const int32_t nb = (int32_t)(seq / b);
  if (global_blocks < 0 || global_blocks > nb) return "global_blocks must be in [0, seq / b]";
  pf_layout sq;
  std::string e = build_layout(sq, seq, seq, b, max_stride);
  if (!e.empty()) return e;
  std::vector<uint8_t> m((size_t)nb * nb, 0);
  for (int32_t i = 0; i < nb; ++i) {
    for (int32_t p = sq.row_ptr[i]; p < sq.row_ptr[i + 1]; ++p) m[(size_t)i * nb + sq.col_idx[p]] = 1;
    for (int32_t j = 0; j < nb; ++j)
      if (i < global_blocks || j < global_blocks) m[(size_t)i * nb + j] = 1;
  }
  e = build_layout_from_mask(L, nb, nb, b, m.data());
  if (!e.empty()) return e;
  L.max_stride = sq.max_stride;
  L.eff_stride = sq.eff_stride;
  L.global_blocks = global_blocks;
  return "";
}

// One butterfly factor of the product form, I + B_k of the factor matrix
// B_k^{(n/b)} (Section 3.1: block-diagonal copies of a size-k factor whose
// quadrants are diagonal), in block units: (p, q) kept iff p == q or
// p XOR q == k / 2.
std::string build_factor_layout(pf_layout &L, int64_t n, int32_t b, int32_t k) {
  if (b < 1 || n < b || n % b) return "b must be >= 1 and divide n";
  const int64_t nb = n / b;
  if (nb > 16384) return "n / b must be <= 16384";
  if (k < 2 || (k & (k - 1)) || k > nb || nb % k)
    return "k must be a power of two >= 2 dividing n / b";
  std::vector<uint8_t> m((size_t)nb * nb, 0);
  for (int64_t p = 0; p < nb; ++p) {
    m[(size_t)p * nb + p] = 1;
    m[(size_t)p * nb + (p ^ (k / 2))] = 1;
  }
  std::string e = build_layout_from_mask(L, (int32_t)nb, (int32_t)nb, b, m.data());
  if (e.empty()) L.max_stride = L.eff_stride = k;
  return e;
}

// Product form of the block butterfly (Section 3.2, a product of factors
// each on the support of I + B_k, k = 2, 4, ..., max_stride): the layout
// holding every factor's kept blocks, factor f (stride 2^(f+1)) on the f-th
// diagonal block of an (L nb) x (L nb) grid.  Block row f nb + p keeps the
// columns f nb + p and f nb + (p XOR 2^f), ascending, which is also the
// order the factors are packed in.  The weight gradient of all factors is
// one masked product on this layout.
std::string build_butterfly_layout(pf_layout &L, int64_t n, int32_t b, int32_t max_stride) {
  if (b < 1 || n < b || n % b) return "b must be >= 1 and divide n";
  const int64_t nb = n / b;
  if (max_stride < 2 || !is_pow2(max_stride)) return "max_stride must be a power of two >= 2";
  if (nb % max_stride) return "max_stride must divide n / b";
  int nfac = 0;
  while ((1 << nfac) < max_stride) ++nfac;
  if ((int64_t)nfac * nb > (1 << 20)) return "too many blocks";
  const int32_t rows = (int32_t)(nfac * nb);
  L.n_out = L.n_in = (int64_t)rows * b;
  L.b = b;
  L.max_stride = L.eff_stride = max_stride;
  L.nb_out = L.nb_in = rows;
  L.s = rows;
  L.bfly_n = n;
  L.bfly_nfac = nfac;
  L.row_ptr.assign(1, 0);
  L.col_idx.clear();
  for (int f = 0; f < nfac; ++f) {
    const int64_t h = (int64_t)1 << f;
    for (int64_t p = 0; p < nb; ++p) {
      const int64_t q = p ^ h;
      L.col_idx.push_back((int32_t)(f * nb + std::min(p, q)));
      L.col_idx.push_back((int32_t)(f * nb + std::max(p, q)));
      L.row_ptr.push_back((int32_t)L.col_idx.size());
    }
  }
  return finish_layout(L);
}

// Layout of the (b, b)-block cover of an element mask (appendix on the cost
// model: the block-aligned mask with the fewest nonzeros containing it):
// block (i, j) is kept iff any element of it is nonzero.
std::string build_cover_layout(pf_layout &L, int64_t n_out, int64_t n_in, int32_t b,
                               const uint8_t *elem_mask) {
  if (!elem_mask) return "mask is NULL";
  if (b < 1 || n_out < b || n_in < b || n_out % b || n_in % b)
    return "b must be >= 1 and divide n_out and n_in";
  if (n_out / b > (1 << 20) || n_in / b > (1 << 20) || (n_out / b) * (n_in / b) > (1 << 26))
    return "too many blocks";
  const int32_t nbo = (int32_t)(n_out / b), nbi = (int32_t)(n_in / b);
  std::vector<uint8_t> m((size_t)nbo * nbi, 0);
  for (int64_t i = 0; i < n_out; ++i) {
    const uint8_t *row = elem_mask + i * n_in;
    uint8_t *mb = m.data() + (size_t)(i / b) * nbi;
    for (int64_t j = 0; j < n_in; ++j)
      if (row[j]) mb[j / b] = 1;
  }
  return build_layout_from_mask(L, nbo, nbi, b, m.data());
}

std::string build_layout_from_mask(pf_layout &L, int32_t nb_out, int32_t nb_in, int32_t b,
                                   const uint8_t *mask) {
  if (b < 1) return "block size b must be >= 1";
  if (nb_out < 1 || nb_in < 1) return "nb_out and nb_in must be >= 1";
  if (!mask) return "mask is NULL";
  if ((int64_t)nb_out * b > ((int64_t)1 << 40) || (int64_t)nb_in * b > ((int64_t)1 << 40))
    return "too large";
  L.n_out = (int64_t)nb_out * b;
  L.n_in = (int64_t)nb_in * b;
  L.b = b;
  L.max_stride = 0;
  L.eff_stride = 0;
  L.nb_out = nb_out;
  L.nb_in = nb_in;
  L.s = std::min(nb_out, nb_in);
  L.row_ptr.assign(1, 0);
  L.col_idx.clear();
  for (int32_t i = 0; i < nb_out; ++i) {
    for (int32_t j = 0; j < nb_in; ++j)
      if (mask[(int64_t)i * nb_in + j]) L.col_idx.push_back(j);
    if (L.col_idx.size() == (size_t)L.row_ptr.back())
      return "every block row needs at least one kept block";
    L.row_ptr.push_back((int32_t)L.col_idx.size());
  }
  return finish_layout(L);
}

// Pair lists of b = 32 layouts with even block counts (see pf_layout): the
// pair block-CSR, each pair block's sources, one backward-data tile per pair
// column (pair rows ascending) and the weight-gradient items.
static void build_pairs(pf_layout &L) {
  L.bwd_tiles_p.clear();
  L.kcols_bwd_p.clear();
  L.blks_bwd_p.clear();
  L.pair_src.clear();
  L.pr_ptr.clear();
  L.pr_col.clear();
  L.tn_items_p.clear();
  L.kmax_bwd_p = 0;
  if (L.b != 32 || L.nb_out % 2 || L.nb_in % 2) return;
  const int32_t npr = L.nb_out / 2, npc = L.nb_in / 2;
  L.pr_ptr.assign(1, 0);
  std::vector<int32_t> cols;
  for (int32_t R = 0; R < npr; ++R) {
    cols.clear();
    for (int32_t i = 2 * R; i < 2 * R + 2; ++i)
      for (int32_t p = L.row_ptr[i]; p < L.row_ptr[i + 1]; ++p) cols.push_back(L.col_idx[p] / 2);
    std::sort(cols.begin(), cols.end());
    cols.erase(std::unique(cols.begin(), cols.end()), cols.end());
    for (int32_t Q : cols) {
      L.pr_col.push_back(Q);
      for (int a = 0; a < 2; ++a)
        for (int c = 0; c < 2; ++c) L.pair_src.push_back(csr_pos(L, 2 * R + a, 2 * Q + c));
    }
    L.pr_ptr.push_back((int32_t)L.pr_col.size());
  }
  // Backward-data: per pair column, its pair rows (ascending) and their ids.
  std::vector<std::vector<int32_t>> rows_of(npc), ids_of(npc);
  for (int32_t R = 0; R < npr; ++R)
    for (int32_t id = L.pr_ptr[R]; id < L.pr_ptr[R + 1]; ++id) {
      rows_of[L.pr_col[id]].push_back(R);
      ids_of[L.pr_col[id]].push_back(id);
    }
  for (int32_t q = 0; q < npc; ++q) {
    NTTile t{};
    t.g = 1;
    t.nsteps = (int32_t)rows_of[q].size();
    t.kcol_off = (int32_t)L.kcols_bwd_p.size();
    t.blk_off = (int32_t)L.blks_bwd_p.size();
    for (int g = 0; g < kMaxG; ++g) t.out_blk[g] = g == 0 ? q : -1;
    L.kcols_bwd_p.insert(L.kcols_bwd_p.end(), rows_of[q].begin(), rows_of[q].end());
    L.blks_bwd_p.insert(L.blks_bwd_p.end(), ids_of[q].begin(), ids_of[q].end());
    L.kmax_bwd_p = std::max(L.kmax_bwd_p, t.nsteps);
    L.bwd_tiles_p.push_back(t);
  }
  // Weight-gradient items over the pair block-CSR, as for b = 64.
  pf_layout P;
  P.b = 64;
  P.nb_out = npr;
  P.nb_in = npc;
  P.row_ptr = L.pr_ptr;
  P.col_idx = L.pr_col;
  build_tn_items(P, 4, L.tn_items_p);
}

// CSC, work lists and their self-check, from row_ptr / col_idx.
std::string finish_layout(pf_layout &L) {
  L.nnzb = (int64_t)L.col_idx.size();
  if (L.nnzb > (int64_t)1 << 30) return "too many kept blocks";

  // Transpose (CSC); rows ascending within a column.
  L.col_ptr.assign(L.nb_in + 1, 0);
  for (int32_t j : L.col_idx) L.col_ptr[j + 1]++;
  for (int32_t j = 0; j < L.nb_in; ++j) L.col_ptr[j + 1] += L.col_ptr[j];
  L.row_idx.assign(L.nnzb, 0);
  L.tperm.assign(L.nnzb, 0);
  std::vector<int32_t> fill(L.col_ptr.begin(), L.col_ptr.end() - 1);
  for (int32_t i = 0; i < L.nb_out; ++i)
    for (int32_t p = L.row_ptr[i]; p < L.row_ptr[i + 1]; ++p) {
      int32_t q = fill[L.col_idx[p]]++;
      L.row_idx[q] = i;
      L.tperm[q] = p;
    }

  const int gmax = max_group(L.b);
  build_nt_tiles(
      L.row_ptr, L.col_idx, gmax,
      [&](int row, int c) { return L.row_ptr[row] + c; }, L.G_fwd,
      L.fwd_tiles, L.kcols_fwd, L.blks_fwd);
  build_nt_tiles(
      L.col_ptr, L.row_idx, gmax,
      [&](int col, int c) { return L.tperm[L.col_ptr[col] + c]; }, L.G_bwd,
      L.bwd_tiles, L.kcols_bwd, L.blks_bwd);
  build_nt_tiles(
      L.row_ptr, L.col_idx, max_group_wide(L.b),
      [&](int row, int c) { return L.row_ptr[row] + c; }, L.G_fwd_w,
      L.fwd_tiles_w, L.kcols_fwd_w, L.blks_fwd_w);
  build_nt_tiles(
      L.col_ptr, L.row_idx, max_group_wide(L.b),
      [&](int col, int c) { return L.tperm[L.col_ptr[col] + c]; }, L.G_bwd_w,
      L.bwd_tiles_w, L.kcols_bwd_w, L.blks_bwd_w);
  build_tn_items(L);
  build_pairs(L);
  L.kmax_fwd = L.kmax_bwd = 0;
  for (auto &t : L.fwd_tiles) L.kmax_fwd = std::max(L.kmax_fwd, (int)t.nsteps);
  for (auto &t : L.bwd_tiles) L.kmax_bwd = std::max(L.kmax_bwd, (int)t.nsteps);
  return check_layout(L);
}

std::string check_layout(const pf_layout &L) {
  std::vector<int> seen(L.nnzb, 0);
  auto sweep = [&](const std::vector<NTTile> &tiles,
                   const std::vector<int32_t> &kcols,
                   const std::vector<int32_t> &blks, int G,
                   bool transposed) -> std::string {
    std::fill(seen.begin(), seen.end(), 0);
    for (auto &t : tiles) {
      if (t.g < 1 || t.g > G) return "tile row count out of range";
      for (int c = 0; c < t.nsteps; ++c)
        for (int g = 0; g < t.g; ++g) {
          int k = kcols[t.kcol_off + c], o = t.out_blk[g];
          int32_t want = transposed ? csr_pos(L, k, o) : csr_pos(L, o, k);
          int32_t got = blks[t.blk_off + c * G + g];
          if (want < 0 || got != want) return "tile block index mismatch";
          seen[got]++;
        }
    }
    for (int v : seen)
      if (v != 1) return "tiles do not cover each kept block exactly once";
    return "";
  };
  std::string e = sweep(L.fwd_tiles, L.kcols_fwd, L.blks_fwd, L.G_fwd, false);
  if (!e.empty()) return "forward: " + e;
  e = sweep(L.fwd_tiles_w, L.kcols_fwd_w, L.blks_fwd_w, L.G_fwd_w, false);
  if (!e.empty()) return "forward (wide): " + e;
  e = sweep(L.bwd_tiles, L.kcols_bwd, L.blks_bwd, L.G_bwd, true);
  if (!e.empty()) return "backward-data: " + e;
  e = sweep(L.bwd_tiles_w, L.kcols_bwd_w, L.blks_bwd_w, L.G_bwd_w, true);
  if (!e.empty()) return "backward-data (wide): " + e;
  if (!L.bwd_tiles_p.empty()) {
    // Pair lists: each pair block's sources are the CSR positions of its
    // four blocks, and every kept block is one pair block's source once.
    std::fill(seen.begin(), seen.end(), 0);
    if (L.bwd_tiles_p.size() != (size_t)(L.nb_in / 2)) return "backward-data pairs: tile count";
    for (size_t q = 0; q < L.bwd_tiles_p.size(); ++q) {
      const NTTile &t = L.bwd_tiles_p[q];
      if (t.g != 1 || t.out_blk[0] != (int32_t)q) return "backward-data pairs: tile column";
      for (int c = 0; c < t.nsteps; ++c) {
        const int32_t r = L.kcols_bwd_p[t.kcol_off + c], pb = L.blks_bwd_p[t.blk_off + c];
        if (r < 0 || 2 * r + 1 >= L.nb_out || pb < 0 || 4 * (size_t)pb + 3 >= L.pair_src.size())
          return "backward-data pairs: index out of range";
        int any = 0;
        for (int a = 0; a < 2; ++a)
          for (int h = 0; h < 2; ++h) {
            const int32_t src = L.pair_src[4 * pb + 2 * a + h];
            if (src != csr_pos(L, 2 * r + a, 2 * (int32_t)q + h))
              return "backward-data pairs: block source mismatch";
            if (src >= 0) {
              seen[src]++;
              any = 1;
            }
          }
        if (!any) return "backward-data pairs: empty pair block";
      }
    }
    for (int v : seen)
      if (v != 1) return "backward-data pairs do not cover each kept block exactly once";
    // Weight-gradient items over the pair blocks: each pair block once, at
    // its pair block-CSR position.
    const size_t npair = L.pair_src.size() / 4;
    std::vector<int> pseen(npair, 0);
    auto pair_pos = [&](int R, int Q) -> int32_t {
      auto b = L.pr_col.begin() + L.pr_ptr[R], e = L.pr_col.begin() + L.pr_ptr[R + 1];
      auto it = std::lower_bound(b, e, Q);
      return (it != e && *it == Q) ? (int32_t)(it - L.pr_col.begin()) : -1;
    };
    for (auto &it : L.tn_items_p)
      for (int a = 0; a < kTNMax; ++a)
        for (int b = 0; b < kTNMax; ++b) {
          const int32_t p = it.out_blk[a * kTNMax + b];
          if (a < it.na && b < it.nb) {
            if (it.a_col[a] < 0 || it.a_col[a] >= L.nb_out / 2 || p != pair_pos(it.a_col[a], it.b_col[b]))
              return "weight-gradient pair item block index mismatch";
            if (p >= 0) pseen[p]++;
          } else if (p != -1) {
            return "weight-gradient pair item padding not empty";
          }
        }
    for (int v : pseen)
      if (v != 1) return "weight-gradient pair items do not cover each pair block exactly once";
  }
  auto items = [&](const std::vector<TNItem> &list, const char *what) -> std::string {
    std::fill(seen.begin(), seen.end(), 0);
    for (auto &it : list) {
      for (int a = 0; a < kTNMax; ++a)
        for (int b = 0; b < kTNMax; ++b) {
          const int32_t p = it.out_blk[a * kTNMax + b];
          if (a < it.na && b < it.nb) {
            if (p != csr_pos(L, it.a_col[a], it.b_col[b]))
              return std::string(what) + " item block index mismatch";
            if (p >= 0) seen[p]++;
          } else if (p >= 0) {
            return std::string(what) + " item keeps a block outside its extent";
          }
        }
    }
    for (int v : seen)
      if (v != 1) return std::string(what) + " items do not cover each kept block once";
    return "";
  };
  e = items(L.tn_items, "weight-gradient");
  if (!e.empty()) return e;
  if (!L.tn_items_w.empty()) return items(L.tn_items_w, "weight-gradient (wide)");
  return "";
}

}  // namespace pf
