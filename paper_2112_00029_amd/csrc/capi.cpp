// C ABI of libpixelfly.so: argument validation (all before any enqueue) and
// dispatch to the HIP kernels.  See include/pixelfly.h for the contract.
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <cmath>
#include <atomic>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "layout.h"
#include "pf_internal.h"
#include "pixelfly.h"

namespace pf {
LaunchEvents &next_launch_events() {
  thread_local LaunchEvents e;
  return e;
}

int tn_items_total(const TNArgs &a, int blk, int tile) {
  const int GT = tile / blk;
  int n = a.n_items;
  for (int r = 0; r < a.n_dense; ++r)
    n += ((a.dr[r].na_blk + GT - 1) / GT) * ((a.dr[r].nb_blk + GT - 1) / GT);
  return n;
}
}  // namespace pf

namespace {

thread_local std::string g_err;

pf_status fail(pf_status s, const std::string &msg) {
  g_err = msg;
  return s;
}

bool aligned16(const void *p) { return ((uintptr_t)p & 15) == 0; }

// Kernel timing hook (pf_timing_begin / pf_timing_end): per kernel class,
// event pairs recorded around the next `cap` launches.
struct KernelTimer {
  std::mutex mu;
  std::atomic<int> armed{0};
  int cap = 0;
  std::vector<hipEvent_t> ev[PF_KERNEL_COUNT];  // 2 * cap each: start, end
  int n[PF_KERNEL_COUNT] = {};

  void release() {
    for (auto &v : ev) {
      for (hipEvent_t e : v)
        if (e) (void)hipEventDestroy(e);
      v.clear();
    }
    std::fill(n, n + PF_KERNEL_COUNT, 0);
    cap = 0;
  }
};
KernelTimer g_kt;

// Scope around one kernel launch: when the hook is armed and the class has
// room, hands the next launch a pair of events (recorded by the dispatch at
// the kernel's start and end) and counts it if the launch took them.
class Timed {
 public:
  Timed(pf_kernel_class k, hipStream_t) : k_(k) {
    if (!g_kt.armed.load(std::memory_order_acquire) || g_kt.n[k] >= g_kt.cap) return;
    pf::next_launch_events() = {g_kt.ev[k][2 * g_kt.n[k]], g_kt.ev[k][2 * g_kt.n[k] + 1]};
    on_ = true;
  }
  ~Timed() {
    if (!on_) return;
    pf::LaunchEvents &e = pf::next_launch_events();
    if (!e.start) g_kt.n[k_]++;  // consumed by a launch
    e.start = e.stop = nullptr;
  }
  Timed(const Timed &) = delete;
  Timed &operator=(const Timed &) = delete;

 private:
  pf_kernel_class k_;
  bool on_ = false;
};

pf_status need_ptr(const void *p, const char *name) {
  if (!p) return fail(PF_ERR_INVALID_ARG, std::string(name) + " is NULL");
  if (!aligned16(p))
    return fail(PF_ERR_INVALID_ARG, std::string(name) + " is not 16-byte aligned");
  return PF_OK;
}

bool kernel_block(int32_t b) { return b == 32 || b == 64 || b == 128; }

pf_status check_layout_arg(const pf_layout *L) {
  if (!L) return fail(PF_ERR_INVALID_ARG, "layout is NULL");
  if (!kernel_block(L->b))
    return fail(PF_ERR_UNSUPPORTED, "kernels support b in {32, 64, 128}");
  return PF_OK;
}

// Called after all argument checks: the layout must live on this device.
pf_status check_state(const pf_layout *L) {
  if (L->device < 0 || !L->dev_mem)
    return fail(PF_ERR_STATE, "layout not uploaded (call pf_layout_upload)");
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev != L->device)
    return fail(PF_ERR_STATE, "layout was uploaded to another device");
  return PF_OK;
}

// Kernels address a tile of up to 512 token rows of any operand with 32-bit
// buffer offsets: 512 rows of the widest operand must stay below 2^31 bytes.
constexpr int64_t kMaxRowBytes = 0x7fffffffLL / 512;

pf_status check_dtype_r(pf_dtype dt, int64_t T, int32_t r, int32_t b) {
  if (dt != PF_BF16 && dt != PF_FP32) return fail(PF_ERR_INVALID_ARG, "bad dtype");
  if (T < 1) return fail(PF_ERR_INVALID_ARG, "T must be >= 1");
  if (T > ((int64_t)1 << 31) / 2) return fail(PF_ERR_INVALID_ARG, "T too large");
  if (r < 0 || r % b) return fail(PF_ERR_INVALID_ARG, "r must be a non-negative multiple of b");
  return PF_OK;
}

pf_status check_extent(const pf_layout *L, pf_dtype dt, int32_t r) {
  const int64_t es = dt == PF_BF16 ? 2 : 4;
  if (std::max<int64_t>({L->n_out, L->n_in, r}) * es > kMaxRowBytes)
    return fail(PF_ERR_UNSUPPORTED, "rows wider than " + std::to_string(kMaxRowBytes) +
                                        " bytes are not supported");
  return PF_OK;
}

pf_status hip_status(hipError_t e, const char *what) {
  if (e == hipSuccess) return PF_OK;
  return fail(PF_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

// Largest power of two <= min(gmax, n).
int pow2_group(int gmax, int n) {
  int g = 1;
  while (g * 2 <= gmax && g * 2 <= n) g *= 2;
  return g;
}

// NT launch: bf16 tiles 64 (b <= 64), 128 or 256 columns wide go to the
// direct-to-LDS kernel family; fp32 and 32-column bf16 tiles go to the
// register-staged one (faster for single 32-wide block columns).
#ifndef PF_NTD
#define PF_NTD 1
#endif

bool ntd_width(int dtype, int blk, int G) {
  const int w = G * blk;
  return PF_NTD && dtype == 0 && (w == 128 || w == 256 || (w == 64 && blk <= 64));
}

// The NT kernel one launch runs: the family (direct-to-LDS or
// register-staged), its variant, and the token x column output tile.
struct NTChoice {
  bool dma;
  int variant;
  int bm, bn;
};

// kmax: the most K-blocks (kept + low-rank) of any tile of the launch; bm:
// token tile of the register-staged family.
NTChoice nt_choose(int dtype, int blk, int G, int bm, int kmax, int64_t M, int ntiles, int nsplit,
                   bool dense) {
  if (!ntd_width(dtype, blk, G)) return NTChoice{false, 0, bm, G * blk};
  // 128-column outputs: 512-token tiles once they still make 512+
  // workgroups; for block-sparse tiles, short K-steps with three workgroups
  // per CU when every tile has at most 8 steps of 64 and one round of
  // workgroups covers them.
  const int w = G * blk;
  if (w == 128) {
    const int64_t ns = std::max(1, nsplit);
    const int64_t wg = ((M + 127) / 128) * ntiles * ns;
    const int64_t steps = ((int64_t)kmax * blk + 63) / 64;
    if (((M + 511) / 512) * ntiles * ns >= 512) return NTChoice{true, pf::NTD_TALL, 512, 128};
    if (!dense && steps <= 8 && wg <= 768) return NTChoice{true, pf::NTD_SHORT_K, 128, 128};
    return NTChoice{true, pf::NTD_DEFAULT, 128, 128};
  }
  return NTChoice{true, pf::NTD_DEFAULT, 256, w};  // 256 x 256 and 256 x 64 tiles
}

// Output tiles per band of the forward's workgroup order: one band per XCD
// once there are 64 or more output tiles (fewer: the token-tile groups).
int nt_band(bool dense, bool b_kn, int ntiles) {
  return !dense && !b_kn && ntiles >= 64 ? (ntiles + 7) / 8 : 0;
}

hipError_t nt_launch(pf_kernel_class kc, int dtype, int blk, int G, bool b_kn, int bm, int kmax,
                     const pf::NTArgs &a_in, hipStream_t s) {
  Timed t(kc, s);
  pf::NTArgs a = a_in;
  a.band = nt_band(a.dense != 0, b_kn, a.ntiles);
  const NTChoice c = nt_choose(dtype, blk, G, bm, kmax, a.M, a.ntiles, a.nsplit, a.dense != 0);
  if (c.dma) return pf::launch_ntd(blk, G, b_kn, c.variant, a, s);
  return pf::launch_nt(dtype, blk, G, b_kn, bm, a, s);
}

// Wide (256-column, 256-token) bf16 tiles pay off once there are enough
// token rows to fill them.
#ifndef PF_WIDE_MIN_T
#define PF_WIDE_MIN_T 2048
#endif

// Dense-mode NT launch: C[M x nblk*b] = A[M x nsteps*b] . B^T (B [n][k]) or
// A . B (B [k][n]), with M-tile bm; split over K when ws gives room.
pf_status dense_nt(pf_kernel_class kc, int dtype, int blk, int G, bool b_kn, int bm, int64_t M,
                   const void *A, int64_t lda, const void *B, int64_t ldb, int nsteps, int nblk,
                   void *C, int64_t ldc, int nsplit, float *ws, hipStream_t s, const char *what) {
  pf::NTArgs a{};
  a.A = A; a.lda = lda; a.B = B; a.ldb = ldb;
  a.dense = 1; a.dense_nsteps = nsteps; a.dense_nblk = nblk;
  a.C = C; a.ldc = ldc; a.M = M;
  a.ntiles = (nblk + G - 1) / G;
  a.nsplit = nsplit;
  a.partials = ws;
  a.ldp = (int64_t)nblk * blk;
  const int per_split = (nsteps + std::max(1, nsplit) - 1) / std::max(1, nsplit);
  pf_status st = hip_status(nt_launch(kc, dtype, blk, G, b_kn, bm, per_split, a, s), what);
  if (st != PF_OK || nsplit <= 1) return st;
  Timed t(PF_KERNEL_REDUCE, s);
  return hip_status(pf::launch_reduce_rows(dtype, nsplit, ws, M, (int64_t)nblk * blk, C, ldc, s), what);
}

// The bf16 rank-r kernel (32-token x 64-column workgroups, no split) runs a
// product when 128 x 128 tiles would cover less than a quarter of the CUs
// (those then need a deep K split, fp32 partials and a reduction pass).
// With more tiles the tile kernel re-reads the small operand far less and
// measured faster (4096 tokens, r = 96: rank-r kernel; 8192 tokens,
// r = 128: tiles).
// Rank-r products go to the rank-r kernel while 128 x 128 tiles would cover
// fewer than PF_SKINNY_MAX_TILES of them (a quarter of the CUs).
#ifndef PF_SKINNY_MAX_TILES
#define PF_SKINNY_MAX_TILES 64
#endif
// The rank-r kernel addresses its operands through 32-bit buffer ranges and
// points steps past the end at the offset 0x7ffffff0, which must lie outside
// every range: A's 32-row tile (32 K-long rows) and the whole r x K (or
// K x r) second operand.  Larger shapes take the tile kernel.
bool skinny_fits(int64_t K, int r) {
  const int64_t lim = 0x7ffffff0LL;
  return 32 * K * 2 < lim && (int64_t)r * K * 2 < lim;
}
bool use_skinny(int dtype, int64_t T, int r, int64_t K) {
  return dtype == 0 && r > 0 && ((T + 127) / 128) * ((r + 127) / 128) < PF_SKINNY_MAX_TILES &&
         skinny_fits(K, r);
}

// bf16 rank-r product C[M x r] = A[M x K] . op(B) on the rank-r kernel
// (B [n][k] for V, [k][n] for U); one launch, no workspace.
pf_status skinny_bf16(pf_kernel_class kc, bool b_kn, int64_t M, const void *A, int64_t lda,
                      const void *B, int64_t ldb, int K, int r, void *C, hipStream_t s,
                      const char *what) {
  pf::SkinnyArgs a{};
  a.A = A; a.lda = lda; a.B = B; a.ldb = ldb; a.C = C; a.ldc = r;
  a.M = M; a.K = K; a.ncols = r;
  Timed t(kc, s);
  return hip_status(pf::launch_skinny(b_kn, a, s), what);
}

// Workgroups a launch aims for (2 per CU on 256 CUs) before splitting K.
#ifndef PF_WG_TARGET
#define PF_WG_TARGET 512
#endif
#ifndef PF_MAX_SPLIT
#define PF_MAX_SPLIT 4
#endif

// Plan of a skinny rank-r product (M = T tokens, K = kblocks * b, r / b
// output blocks): token tile bm and the split of the K range over
// workgroups.  bf16 runs on the direct-to-LDS kernel with 128 x 128 tiles
// and K-steps of 64; it splits until about 512 workgroups are in flight but
// keeps at least 6 steps per split (the fp32 partials and their reduction
// cost more than they save below that).  fp32 uses 64-token tiles, K-steps
// of 32 and at most PF_MAX_SPLIT splits.
struct SkinnyPlan {
  int bm;
  int nsplit;
  size_t ws;
  int G;  // output blocks per tile (128 or 256 columns)
  int blk = 0;  // block width of the product's K-steps and output blocks
};
SkinnyPlan skinny_plan(int dtype, int blk, int64_t T, int kblocks, int r) {
  SkinnyPlan p{dtype == 0 ? 128 : 64, 1, 0, 128 / blk};
  if (dtype != 0 && r > 0 && r < 128) {
    // fp32, r below one 128-column tile: one block per tile (no dead columns).
    p.G = 1;
    p.bm = blk == 32 ? 128 : 64;
  }
  if (r <= 0 || use_skinny(dtype, T, r, (int64_t)kblocks * blk)) return p;  // no split
  if (dtype == 0 && r % 256 == 0 && T >= 2048 && (int64_t)kblocks * blk >= 8192) {
    // Deep products (S = dY U of a wide layer): 256 x 256 tiles, eight
    // waves, one workgroup per CU, split until about 256 workgroups run, at
    // least 8 steps of 64 per split.  They read half the operand bytes per
    // flop of the 128 x 128 tiles (16384 x 16384 by 256: 181 -> 158 us
    // with four splits, the reduction 5 us longer).
    p.G = 256 / blk;
    p.bm = 256;
    const int64_t tiles = ((T + 255) / 256) * (r / 256);
    const int64_t steps = ((int64_t)kblocks * blk) / 64;
    const int64_t want = std::max<int64_t>(1, 256 / tiles);
    const int64_t cap = std::max<int64_t>(1, steps / 8);
    int64_t ns = 1;
    while (ns * 2 <= std::min(want, cap)) ns *= 2;
    if (ns > 1) {
      p.nsplit = (int)ns;
      p.ws = (size_t)ns * T * r * sizeof(float);
    }
    return p;
  }
  const int64_t mtiles = (T + p.bm - 1) / p.bm, ntiles = (r + p.G * blk - 1) / (p.G * blk);
  const int64_t steps = ((int64_t)kblocks * blk) / (dtype == 0 ? 64 : 32);
  int64_t ns;
  if (dtype == 0) {
    const int64_t want = std::max<int64_t>(1, 512 / (mtiles * ntiles));
    const int64_t cap = std::max<int64_t>(1, steps / 6);
    ns = 1;
    while (ns * 2 <= std::min(want, cap)) ns *= 2;
    if (ns == 2 && steps < 16) ns = 1;
  } else {
    const int64_t want = (PF_WG_TARGET + mtiles * ntiles - 1) / (mtiles * ntiles);
    ns = std::min<int64_t>({want, p.G == 1 ? 2 * PF_MAX_SPLIT : PF_MAX_SPLIT,
                            std::max<int64_t>(1, steps / 4)});
  }
  if (ns > 1) {
    p.nsplit = (int)ns;
    p.ws = (size_t)ns * T * r * sizeof(float);
  }
  return p;
}

// Block width of a rank-r product: the products are dense, so bf16 takes
// 128 (else 64) when r and K allow it, whatever the layout's b: b = 32
// blocks would give K-steps of 32-column (64-byte) row halves (S = dY U at
// 16384 x 4096 b = 32: 157 -> 132 us).  fp32 keeps b.
int rank_blk(const pf_layout *L, int dtype, int32_t r, int64_t K) {
  if (dtype == PF_BF16)
    for (int cb : {128, 64})
      if (r % cb == 0 && K % cb == 0) return cb;
  return L->b;
}
// Plan of T_lr = X V^T (s_side false, K = n_in) or S = dY U (K = n_out).
SkinnyPlan rank_plan(const pf_layout *L, int dtype, int64_t T, int32_t r, bool s_side) {
  const int64_t K = s_side ? L->n_out : L->n_in;
  const int rb = rank_blk(L, dtype, r, K);
  SkinnyPlan p = skinny_plan(dtype, rb, T, (int)(K / rb), r);
  p.blk = rb;
  return p;
}

// Split-token plan of the TN kernel.  Few work items (under one round of
// kTNSlots resident workgroups): the split of at most PF_TN_MAX_SPLIT parts of
// at least min_tokens tokens that minimises rounds x steps per workgroup.  Many
// items: aim for about 4096 workgroups (token splits also shorten each
// workgroup's serial chain and its L2 footprint) with power-of-two splits of
// at least 512 tokens, at most PF_TN_MAX_SPLIT, keeping the fp32 partial
// traffic in check.  Always enough splits that one split's rows stay below
// 2^31 bytes (32-bit buffer offsets).
constexpr int64_t kTNSlots = 512;  // two TN workgroups per CU on 256 CUs
#ifndef PF_TN_ROUND_ITEMS
#define PF_TN_ROUND_ITEMS kTNSlots
#endif
#ifndef PF_TN_MAX_SPLIT
#define PF_TN_MAX_SPLIT 8
#endif
struct TNPlan {
  int nsplit;
  int64_t chunk;
  size_t ws;
  // 256 x 256 kernel: items shared by several workgroups (summed from the
  // partial slots by a second pass).
  bool wide = false;
  int shared = 0;
  int grid = 0;  // 256 x 256 kernel: workgroups
  // b = 32 on pair blocks (256 x 256 kernel as b = 64): the pair-block
  // gradients go to the workspace at pair_off, then scatter into dW.
  bool pairs = false;
  size_t pair_off = 0;
};

// row_bytes: the largest operand row stride in bytes.
int64_t tn_min_tokens(int dtype) { return dtype == 0 ? 512 : 64; }

// min_tokens: fewest tokens per split (512 for bf16, whose weight gradient
// is bound by operand traffic; 64 for fp32, bound by its long MFMAs).
TNPlan tn_plan(int items, int64_t T, int64_t row_bytes, int64_t min_tokens = 512) {
  TNPlan p{1, ((T + 63) / 64) * 64, 0};
  const int64_t min_split = (T * row_bytes + 0x7fffffffLL - 1) / 0x7fffffffLL;
  int64_t ns = 1;
  const int64_t cap = std::max<int64_t>(1, std::min<int64_t>(PF_TN_MAX_SPLIT, T / min_tokens));
  if (items < PF_TN_ROUND_ITEMS) {
    // Few items: the split that finishes soonest when kTNSlots workgroups
    // run at a time, i.e. fewest (rounds x 64-token steps per workgroup);
    // the smaller split on ties (fewer partials).
    int64_t best = -1;
    for (int64_t c = 1; c <= cap; ++c) {
      const int64_t chunk = ((T + c - 1) / c + 63) / 64 * 64, nsr = (T + chunk - 1) / chunk;
      const int64_t cost = ((items * nsr + kTNSlots - 1) / kTNSlots) * (chunk / 64);
      if (best < 0 || cost < best) {
        best = cost;
        ns = nsr;
      }
    }
  } else {
    const int64_t want = std::max<int64_t>(1, 4096 / std::max(1, items));
    while (ns * 2 <= std::min(want, cap)) ns *= 2;
  }
  ns = std::max(ns, min_split);
  if (ns > 1) {
    int64_t chunk = ((T + ns - 1) / ns + 63) / 64 * 64;
    // Rounding the chunk up to whole 64-token steps can push a split's rows
    // past the 32-bit buffer range again: take more splits until it fits.
    while (chunk * row_bytes > 0x7fffffffLL && chunk > 64) {
      ++ns;
      chunk = ((T + ns - 1) / ns + 63) / 64 * 64;
    }
    ns = (T + chunk - 1) / chunk;
    if (ns > 1) {
      p.nsplit = (int)ns;
      p.chunk = chunk;
      p.ws = (size_t)items * ns * 128 * 128 * sizeof(float);
    }
  }
  return p;
}

// The 256 x 256 weight-gradient kernel runs a call when: bf16, b of 64 or
// 128, no mixing weight, at least PF_WIDE_MIN_T tokens, at least one full
// round of work items (kTNWGrid), every operand's rows over the whole token
// range addressable with 32-bit offsets, and the wide items waste at most a
// fifth of their block slots (kept blocks over rows x kept columns of every
// item; a wave whose columns keep nothing skips its MFMAs).  With fewer
// items than workgroups every item is shared: workgroups then read
// different token rows of the same columns at a time, L2 stops serving the
// neighbours, and the 128 x 128 kernel measured faster (the 16384 x 4096
// layer at b = 64: 208 items, 540 against 466 us).
void fill_tn_regions(pf::TNArgs &a, const pf_layout *L, int32_t r, const void *dY,
                     const void *X, const void *T_lr, const void *S, void *dU, void *dV,
                     int blk = 0);
bool tn_wide(const pf_layout *L, int dtype, int64_t T, int32_t r, bool mixed) {
  if (dtype != 0 || mixed || (L->b != 64 && L->b != 128) || L->tn_items_w.empty()) return false;
  if (T < PF_WIDE_MIN_T) return false;
  pf::TNArgs w{};
  w.n_items = (int)L->tn_items_w.size();
  fill_tn_regions(w, L, r, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr);
  // Fewer items than workgroups run one workgroup per item (no shared
  // items, no second pass) while they still fill three quarters of the CUs:
  // at 16384 x 4096, b = 64 (208 items) that took the weight gradient from
  // 475 us on the 128 x 128 kernel (4 token splits + reduction) to 402 us.
  if (pf::tn_items_total(w, L->b, pf::kTNWTile) < pf::kTNWMinItems) return false;
  const int64_t row_bytes = std::max<int64_t>({L->n_out, L->n_in, (int64_t)r}) * 2;
  // Copies run up to seven 32-token steps past a segment (read as zeros).
  if ((T + 512) * row_bytes > 0x7fffffffLL) return false;
  const int GT = 256 / L->b;
  int64_t slots = 0;
  for (auto &it : L->tn_items_w) slots += (int64_t)GT * it.nb;
  return L->nnzb * 5 >= slots * 4;
}

// b = 32 weight gradient on the pair blocks (T x K of 4M or more, rank a
// multiple of 64, the 256 x 256 item count of b = 64): the 32-token steps of
// the 128 x 128 kernel read 64-byte row halves of both operands; the pair
// items read whole 128-byte segments and compute the dropped quarters too.
bool tn_pairs(const pf_layout *L, int dtype, int64_t T, int32_t r, bool mixed) {
  if (dtype != 0 || mixed || L->b != 32 || L->tn_items_p.empty() || r % 64) return false;
  if (T < PF_WIDE_MIN_T || T * L->n_in < ((int64_t)1 << 22)) return false;
  pf::TNArgs w{};
  w.n_items = (int)L->tn_items_p.size();
  fill_tn_regions(w, L, r, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, 64);
  if (pf::tn_items_total(w, 64, pf::kTNWTile) < pf::kTNWMinItems) return false;
  const int64_t row_bytes = std::max<int64_t>({L->n_out, L->n_in, (int64_t)r}) * 2;
  return (T + 512) * row_bytes <= 0x7fffffffLL;
}

// Plan of the 256 x 256 kernel over `items` work items: kTNWGrid
// workgroups (one per item when there are fewer items); the items past the
// last full round are shared.  Workspace: two fp32 partial slots of
// 256 x 256 per workgroup.
TNPlan tn_plan_wide(int items, int64_t T) {
  TNPlan p{1, ((T + 63) / 64) * 64, 0};
  p.wide = true;
  p.grid = std::min(items, pf::kTNWGrid);
  p.shared = items % p.grid;
  if (p.shared > 0)
    p.ws = (size_t)2 * pf::kTNWGrid * pf::kTNWTile * pf::kTNWTile * sizeof(float);
  return p;
}

pf::TNArgs tn_args(const pf_layout *L, pf_dtype dtype, int64_t T, int32_t r, const void *dY,
                   const void *X, const void *T_lr, const void *S, void *dWblk, void *dU,
                   void *dV, TNPlan *plan, bool mixed = false);

// Workspace the mixed weight-gradient call adds after the split partials:
// the kept-block dot partials (one per item, or 16 per item after a split)
// and the S.T_lr partials, 256-byte aligned.
size_t mix_dgamma_bytes(int items) {
  return ((size_t)items * 16 + pf::kMixDotParts) * sizeof(float) + 256;
}
size_t align256(size_t x) { return (x + 255) / 256 * 256; }

// Tile list of a block-sparse NT launch: the wide list (256-column bf16
// tiles) once the token count fills them, else the narrow one.
struct NTList {
  bool wide;
  int G, ntiles, kmax;
  const pf::NTTile *tiles;
  const int32_t *kcols, *blks;
};
NTList fwd_list(const pf_layout *L, int dt, int64_t T) {
  const bool wide = ntd_width(dt, L->b, L->G_fwd_w) && L->G_fwd_w * L->b == 256 && T >= PF_WIDE_MIN_T;
  if (wide)
    return NTList{true, L->G_fwd_w, (int)L->fwd_tiles_w.size(), L->kmax_fwd, L->d_fwd_tiles_w,
                  L->d_kcols_fwd_w, L->d_blks_fwd_w};
  return NTList{false, L->G_fwd, (int)L->fwd_tiles.size(), L->kmax_fwd, L->d_fwd_tiles,
                L->d_kcols_fwd, L->d_blks_fwd};
}
NTList bwd_list(const pf_layout *L, int dt, int64_t T) {
  const bool wide = ntd_width(dt, L->b, L->G_bwd_w) && L->G_bwd_w * L->b == 256 && T >= PF_WIDE_MIN_T;
  if (wide)
    return NTList{true, L->G_bwd_w, (int)L->bwd_tiles_w.size(), L->kmax_bwd, L->d_bwd_tiles_w,
                  L->d_kcols_bwd_w, L->d_blks_bwd_w};
  return NTList{false, L->G_bwd, (int)L->bwd_tiles.size(), L->kmax_bwd, L->d_bwd_tiles,
                L->d_kcols_bwd, L->d_blks_bwd};
}

// b = 32 backward-data on 64-wide pair tiles (bf16, no two block columns
// sharing their kept rows, rank a multiple of 64, T x K of 4M or more): the
// 32-wide tiles read dY in half 128-byte row segments; the pair tiles read
// whole ones and multiply the dropped blocks of each pair block as zeros
// (16384 x 4096: 468 -> 276 us plus a 5 us gather).  Small products do not
// repay the gather launch (2048 tokens x 1024: 7.0 -> 8.7 + 4.4 us).
bool use_bwd_pairs(const pf_layout *L, int dt, int64_t T, int32_t r) {
  return dt == PF_BF16 && !L->bwd_tiles_p.empty() && L->G_bwd == 1 && L->G_bwd_w == 1 &&
         r % 64 == 0 && T * L->n_in >= ((int64_t)1 << 22);
}
size_t pair_ws_bytes(const pf_layout *L, int dt, int64_t T, int32_t r) {
  return use_bwd_pairs(L, dt, T, r) ? (L->pair_src.size() / 4) * 64 * 64 * 2 : 0;
}

// blk: block size of the regions' tiling (0: the layout's).
void fill_tn_regions(pf::TNArgs &a, const pf_layout *L, int32_t r, const void *dY,
                     const void *X, const void *T_lr, const void *S, void *dU, void *dV,
                     int blk) {
  const int b = blk ? blk : L->b;
  a.n_dense = 0;
  if (r > 0) {
    a.dr[0] = pf::TNDense{dY, L->n_out, T_lr, r, dU, r, (int)(L->n_out / b), r / b};
    a.dr[1] = pf::TNDense{S, r, X, L->n_in, dV, L->n_in, r / b, (int)(L->n_in / b)};
    a.n_dense = 2;
  }
}

}  // namespace

extern "C" {

const char *pf_status_string(pf_status s) {
  switch (s) {
    case PF_OK: return "ok";
    case PF_ERR_INVALID_ARG: return "invalid argument";
    case PF_ERR_UNSUPPORTED: return "unsupported";
    case PF_ERR_WORKSPACE: return "workspace too small";
    case PF_ERR_HIP: return "HIP error";
    case PF_ERR_NOMEM: return "out of memory";
    case PF_ERR_STATE: return "layout not ready";
  }
  return "unknown status";
}

const char *pf_last_error(void) { return g_err.c_str(); }

pf_status pf_timing_begin(int32_t max_launches_per_class) {
  if (max_launches_per_class < 1 || max_launches_per_class > (1 << 20))
    return fail(PF_ERR_INVALID_ARG, "max_launches_per_class must be in [1, 2^20]");
  std::lock_guard<std::mutex> lk(g_kt.mu);
  g_kt.armed.store(0, std::memory_order_release);
  g_kt.release();
  try {
    for (auto &v : g_kt.ev) v.assign(2 * (size_t)max_launches_per_class, nullptr);
  } catch (const std::bad_alloc &) {
    g_kt.release();
    return fail(PF_ERR_NOMEM, "host allocation failed");
  }
  for (auto &v : g_kt.ev)
    for (hipEvent_t &e : v)
      if (hipEventCreate(&e) != hipSuccess) {
        e = nullptr;
        g_kt.release();
        return fail(PF_ERR_HIP, "hipEventCreate failed");
      }
  g_kt.cap = max_launches_per_class;
  g_kt.armed.store(1, std::memory_order_release);
  return PF_OK;
}

pf_status pf_timing_end(int32_t *counts, double *avg_ms) {
  std::lock_guard<std::mutex> lk(g_kt.mu);
  if (!g_kt.armed.load(std::memory_order_acquire)) return fail(PF_ERR_STATE, "timing not begun");
  g_kt.armed.store(0, std::memory_order_release);
  pf_status st = PF_OK;
  for (int k = 0; k < PF_KERNEL_COUNT; ++k) {
    double sum = 0;
    for (int i = 0; i < g_kt.n[k]; ++i) {
      float ms = 0;
      if (hipEventSynchronize(g_kt.ev[k][2 * i + 1]) != hipSuccess ||
          hipEventElapsedTime(&ms, g_kt.ev[k][2 * i], g_kt.ev[k][2 * i + 1]) != hipSuccess) {
        st = fail(PF_ERR_HIP, "reading timing events failed");
        break;
      }
      sum += ms;
    }
    if (counts) counts[k] = g_kt.n[k];
    if (avg_ms) avg_ms[k] = g_kt.n[k] ? sum / g_kt.n[k] : 0.0;
  }
  g_kt.release();
  return st;
}

pf_status pf_layout_create(int64_t n_out, int64_t n_in, int32_t b, int32_t max_stride,
                           pf_layout **out) {
  if (!out) return fail(PF_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  pf_layout *L = new (std::nothrow) pf_layout();
  if (!L) return fail(PF_ERR_NOMEM, "host allocation failed");
  std::string e;
  try {
    e = pf::build_layout(*L, n_out, n_in, b, max_stride);
  } catch (const std::bad_alloc &) {
    delete L;
    return fail(PF_ERR_NOMEM, "host allocation failed");
  } catch (...) {
    delete L;
    return fail(PF_ERR_INVALID_ARG, "layout build failed");
  }
  if (!e.empty()) {
    delete L;
    return fail(PF_ERR_INVALID_ARG, e);
  }
  *out = L;
  return PF_OK;
}

pf_status pf_layout_create_from_mask(int32_t nb_out, int32_t nb_in, int32_t b,
                                     const uint8_t *block_mask, pf_layout **out) {
  if (!out) return fail(PF_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  pf_layout *L = new (std::nothrow) pf_layout();
  if (!L) return fail(PF_ERR_NOMEM, "host allocation failed");
  std::string e;
  try {
    e = pf::build_layout_from_mask(*L, nb_out, nb_in, b, block_mask);
  } catch (const std::bad_alloc &) {
    delete L;
    return fail(PF_ERR_NOMEM, "host allocation failed");
  } catch (...) {
    delete L;
    return fail(PF_ERR_INVALID_ARG, "layout build failed");
  }
  if (!e.empty()) {
    delete L;
    return fail(PF_ERR_INVALID_ARG, e);
  }
  *out = L;
  return PF_OK;
}

pf_status pf_layout_create_attention(int64_t seq, int32_t b, int32_t max_stride,
                                     int32_t global_blocks, pf_layout **out) {
  if (!out) return fail(PF_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  pf_layout *L = new (std::nothrow) pf_layout();
  if (!L) return fail(PF_ERR_NOMEM, "host allocation failed");
  std::string e;
  try {
    e = pf::build_attention_layout(*L, seq, b, max_stride, global_blocks);
  } catch (const std::bad_alloc &) {
    delete L;
    return fail(PF_ERR_NOMEM, "host allocation failed");
  } catch (...) {
    delete L;
    return fail(PF_ERR_INVALID_ARG, "layout build failed");
  }
  if (!e.empty()) {
    delete L;
    return fail(PF_ERR_INVALID_ARG, e);
  }
  *out = L;
  return PF_OK;
}

pf_status pf_layout_create_from_element_mask(int64_t n_out, int64_t n_in, int32_t b,
                                             const uint8_t *elem_mask, pf_layout **out) {
  if (!out) return fail(PF_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  pf_layout *L = new (std::nothrow) pf_layout();
  if (!L) return fail(PF_ERR_NOMEM, "host allocation failed");
  std::string e;
  try {
    e = pf::build_cover_layout(*L, n_out, n_in, b, elem_mask);
  } catch (const std::bad_alloc &) {
    delete L;
    return fail(PF_ERR_NOMEM, "host allocation failed");
  } catch (...) {
    delete L;
    return fail(PF_ERR_INVALID_ARG, "layout build failed");
  }
  if (!e.empty()) {
    delete L;
    return fail(PF_ERR_INVALID_ARG, e);
  }
  *out = L;
  return PF_OK;
}

pf_status pf_layout_create_factor(int64_t n, int32_t b, int32_t k, pf_layout **out) {
  if (!out) return fail(PF_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  pf_layout *L = new (std::nothrow) pf_layout();
  if (!L) return fail(PF_ERR_NOMEM, "host allocation failed");
  std::string e;
  try {
    e = pf::build_factor_layout(*L, n, b, k);
  } catch (const std::bad_alloc &) {
    delete L;
    return fail(PF_ERR_NOMEM, "host allocation failed");
  } catch (...) {
    delete L;
    return fail(PF_ERR_INVALID_ARG, "layout build failed");
  }
  if (!e.empty()) {
    delete L;
    return fail(PF_ERR_INVALID_ARG, e);
  }
  *out = L;
  return PF_OK;
}

pf_status pf_layout_create_butterfly(int64_t n, int32_t b, int32_t max_stride, pf_layout **out) {
  if (!out) return fail(PF_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  pf_layout *L = new (std::nothrow) pf_layout();
  if (!L) return fail(PF_ERR_NOMEM, "host allocation failed");
  std::string e;
  try {
    e = pf::build_butterfly_layout(*L, n, b, max_stride);
  } catch (const std::bad_alloc &) {
    delete L;
    return fail(PF_ERR_NOMEM, "host allocation failed");
  } catch (...) {
    delete L;
    return fail(PF_ERR_INVALID_ARG, "layout build failed");
  }
  if (!e.empty()) {
    delete L;
    return fail(PF_ERR_INVALID_ARG, e);
  }
  *out = L;
  return PF_OK;
}

pf_status pf_select_mask(int64_t n_out, int64_t n_in, int32_t b, double budget,
                         double lowrank_share, int32_t *r_out, int32_t *max_stride_out,
                         int64_t *params_out) {
  if (!r_out || !max_stride_out) return fail(PF_ERR_INVALID_ARG, "NULL output");
  if (b < 1 || n_out < b || n_in < b || n_out % b || n_in % b)
    return fail(PF_ERR_INVALID_ARG, "b must be >= 1 and divide n_out and n_in");
  if (!(budget > 0.0 && budget <= 1.0)) return fail(PF_ERR_INVALID_ARG, "budget must be in (0, 1]");
  if (!(lowrank_share >= 0.0 && lowrank_share <= 1.0))
    return fail(PF_ERR_INVALID_ARG, "lowrank_share must be in [0, 1]");
  // Cost of a configuration: kept weight entries plus low-rank entries (the
  // per-token FLOPs are twice this), against budget * n_out * n_in.
  const double dense = (double)n_out * (double)n_in, total = budget * dense;
  const int64_t per_rank = n_out + n_in;
  const int64_t rmax = std::min(n_out, n_in) / b * b;
  int64_t r = (int64_t)std::floor(lowrank_share * total / (double)per_rank);
  r = std::max<int64_t>(0, std::min(rmax, r / b * b));
  const int64_t s = std::min(n_out, n_in) / b;
  int64_t top = 1;
  while (top < s) top *= 2;  // strides past the next power of two of s change nothing
  int32_t best = 1;
  int64_t best_params = -1;
  try {
    for (int64_t ms = 1; ms <= top; ms *= 2) {
      pf_layout L;
      std::string e = pf::build_layout(L, n_out, n_in, b, (int32_t)ms);
      if (!e.empty()) return fail(PF_ERR_INVALID_ARG, e);
      const int64_t params = L.nnzb * (int64_t)b * b + r * per_rank;
      if (ms == 1 || (double)params <= total) {
        best = (int32_t)ms;
        best_params = params;
      }
      if ((double)params > total) break;
    }
  } catch (const std::bad_alloc &) {
    return fail(PF_ERR_NOMEM, "host allocation failed");
  }
  *r_out = (int32_t)r;
  *max_stride_out = best;
  if (params_out) *params_out = best_params;
  return PF_OK;
}

pf_status pf_layout_info_get(const pf_layout *L, pf_layout_info *o) {
  if (!L || !o) return fail(PF_ERR_INVALID_ARG, "NULL argument");
  o->n_out = L->n_out;
  o->n_in = L->n_in;
  o->b = L->b;
  o->max_stride = L->max_stride;
  o->eff_stride = L->eff_stride;
  o->s = L->s;
  o->nb_out = L->nb_out;
  o->nb_in = L->nb_in;
  o->nnzb = L->nnzb;
  o->row_ptr = L->row_ptr.data();
  o->col_idx = L->col_idx.data();
  o->col_ptr = L->col_ptr.data();
  o->row_idx = L->row_idx.data();
  o->tperm = L->tperm.data();
  return PF_OK;
}

pf_status pf_layout_check(const pf_layout *L) {
  if (!L) return fail(PF_ERR_INVALID_ARG, "layout is NULL");
  std::string e = pf::check_layout(*L);
  if (!e.empty()) return fail(PF_ERR_INVALID_ARG, e);
  return PF_OK;
}

pf_status pf_layout_plan_get(const pf_layout *L, int32_t *stats, int32_t n) {
  if (!L || !stats || n < 6) return fail(PF_ERR_INVALID_ARG, "bad arguments");
  if (n >= 10) {
    stats[6] = L->G_fwd_w;
    stats[7] = (int32_t)L->fwd_tiles_w.size();
    stats[8] = L->G_bwd_w;
    stats[9] = (int32_t)L->bwd_tiles_w.size();
  }
  stats[0] = L->G_fwd;
  stats[1] = (int32_t)L->fwd_tiles.size();
  stats[2] = L->G_bwd;
  stats[3] = (int32_t)L->bwd_tiles.size();
  stats[4] = (int32_t)L->tn_items.size();
  int kept = 0;
  for (auto &it : L->tn_items)
    for (int q = 0; q < pf::kTNMax * pf::kTNMax; ++q) kept += it.out_blk[q] >= 0;
  stats[5] = kept;
  return PF_OK;
}

pf_status pf_layout_upload(pf_layout *L, void *stream) {
  if (!L) return fail(PF_ERR_INVALID_ARG, "layout is NULL");
  if (!kernel_block(L->b))
    return fail(PF_ERR_UNSUPPORTED, "kernels support b in {32, 64, 128}");
  if (L->dev_mem) return PF_OK;
  int dev = -1;
  pf_status st = hip_status(hipGetDevice(&dev), "hipGetDevice");
  if (st != PF_OK) return st;
  // Every host array goes into one device allocation, 256-byte aligned
  // pieces; `dst` receives each piece's device address.
  struct Piece {
    const void *src;
    size_t bytes;
    const void **dst;
  };
  auto vec = [](auto &v, auto &d) {
    return Piece{v.data(), v.size() * sizeof(v[0]), (const void **)&d};
  };
  const Piece pieces[] = {
      vec(L->fwd_tiles, L->d_fwd_tiles),     vec(L->bwd_tiles, L->d_bwd_tiles),
      vec(L->kcols_fwd, L->d_kcols_fwd),     vec(L->blks_fwd, L->d_blks_fwd),
      vec(L->kcols_bwd, L->d_kcols_bwd),     vec(L->blks_bwd, L->d_blks_bwd),
      vec(L->fwd_tiles_w, L->d_fwd_tiles_w), vec(L->bwd_tiles_w, L->d_bwd_tiles_w),
      vec(L->kcols_fwd_w, L->d_kcols_fwd_w), vec(L->blks_fwd_w, L->d_blks_fwd_w),
      vec(L->kcols_bwd_w, L->d_kcols_bwd_w), vec(L->blks_bwd_w, L->d_blks_bwd_w),
      vec(L->tn_items, L->d_tn_items),       vec(L->tn_items_w, L->d_tn_items_w),
      vec(L->bwd_tiles_p, L->d_bwd_tiles_p), vec(L->kcols_bwd_p, L->d_kcols_bwd_p),
      vec(L->blks_bwd_p, L->d_blks_bwd_p),   vec(L->pair_src, L->d_pair_src),
      vec(L->tn_items_p, L->d_tn_items_p),
      vec(L->row_ptr, L->d_row_ptr),
      vec(L->col_idx, L->d_col_idx),         vec(L->col_ptr, L->d_col_ptr),
      vec(L->row_idx, L->d_row_idx)};
  constexpr int NP = (int)(sizeof(pieces) / sizeof(pieces[0]));
  size_t off[NP], total = 0;
  for (int i = 0; i < NP; ++i) {
    off[i] = total;
    total += (pieces[i].bytes + 255) / 256 * 256;
  }
  void *mem = nullptr;
  if (hipMalloc(&mem, std::max<size_t>(total, 256)) != hipSuccess)
    return fail(PF_ERR_NOMEM, "hipMalloc for layout failed");
  hipStream_t s = (hipStream_t)stream;
  for (int i = 0; i < NP; ++i)
    if (pieces[i].bytes) {
      hipError_t e = hipMemcpyAsync((char *)mem + off[i], pieces[i].src, pieces[i].bytes,
                                    hipMemcpyHostToDevice, s);
      if (e != hipSuccess) {
        (void)hipFree(mem);
        return hip_status(e, "layout upload");
      }
    }
  hipError_t e = hipStreamSynchronize(s);
  if (e != hipSuccess) {
    (void)hipFree(mem);
    return hip_status(e, "layout upload sync");
  }
  for (int i = 0; i < NP; ++i) *pieces[i].dst = (const char *)mem + off[i];
  L->dev_mem = mem;
  L->device = dev;
  return PF_OK;
}

void pf_layout_destroy(pf_layout *L) {
  if (!L) return;
  if (L->dev_mem) {
    int cur = -1;
    (void)hipGetDevice(&cur);
    if (cur != L->device) (void)hipSetDevice(L->device);
    (void)hipFree(L->dev_mem);
    if (cur >= 0 && cur != L->device) (void)hipSetDevice(cur);
  }
  delete L;
}

size_t pf_workspace_bytes(const pf_layout *L, int64_t T, int32_t r, pf_dtype dtype) {
  if (!L || T < 1 || r < 0 || !kernel_block(L->b) || r % L->b) return 0;
  if (dtype != PF_BF16 && dtype != PF_FP32) return 0;
  pf::TNArgs a{};
  a.n_items = (int)L->tn_items.size();
  fill_tn_regions(a, L, r, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr);
  const int64_t es = dtype == PF_BF16 ? 2 : 4;
  const int items = pf::tn_items_total(a, L->b);
  // The 128 x 128 plan (mixed calls, and the rest when the wide kernel does
  // not apply) and, where it applies, the 256 x 256 one.
  const size_t tn = tn_plan(items, T, std::max(L->n_out, L->n_in) * es, tn_min_tokens(dtype)).ws;
  size_t tnw = 0;
  if (tn_wide(L, (int)dtype, T, r, false) || tn_pairs(L, (int)dtype, T, r, false)) {
    TNPlan wp;
    (void)tn_args(L, dtype, T, r, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr,
                  &wp);
    tnw = wp.ws;
  }
  const size_t fwd = rank_plan(L, (int)dtype, T, r, false).ws;
  const size_t sws = rank_plan(L, (int)dtype, T, r, true).ws;
  const size_t pws = pair_ws_bytes(L, (int)dtype, T, r);
  const size_t bwd = pws ? align256(sws) + pws : sws;
  return std::max({tn, tnw, fwd, bwd}) + mix_dgamma_bytes(items);
}

pf_status pf_linear_plan_get(const pf_layout *L, pf_dtype dtype, int64_t T, int32_t r,
                             pf_linear_plan *o) {
  if (!o) return fail(PF_ERR_INVALID_ARG, "out is NULL");
  pf_status st = check_layout_arg(L);
  if (st != PF_OK) return st;
  if ((st = check_dtype_r(dtype, T, r, L->b)) != PF_OK) return st;
  if ((st = check_extent(L, dtype, r)) != PF_OK) return st;
  const int dt = (int)dtype, b = L->b;
  pf_linear_plan p{};
  // Rank-r products: the same decisions as enqueue of T_lr and S.
  auto rank = [&](int64_t K, int kblocks, bool b_kn, int32_t *v) {
    (void)kblocks;
    if (r <= 0) return;
    if (use_skinny(dt, T, r, K)) {
      v[0] = 1;
      v[1] = 1;
      v[2] = 32;
      v[3] = 64;
      return;
    }
    const SkinnyPlan sp = rank_plan(L, dt, T, r, b_kn);
    const int G = sp.G, rb = sp.blk;
    const int ksteps = (int)(K / rb);
    const NTChoice c = nt_choose(dt, rb, G, sp.bm, (ksteps + sp.nsplit - 1) / sp.nsplit, T,
                                 (r / rb + G - 1) / G, sp.nsplit, true);
    v[0] = 2;
    v[1] = sp.nsplit;
    v[2] = c.bm;
    v[3] = c.bn;
  };
  int32_t t[4] = {0, 0, 0, 0}, sv[4] = {0, 0, 0, 0};
  rank(L->n_in, L->nb_in, false, t);
  rank(L->n_out, L->nb_out, true, sv);
  p.lowrank_t_kernel = t[0];
  p.lowrank_t_split = t[1];
  p.lowrank_t_tile_m = t[2];
  p.lowrank_t_tile_n = t[3];
  p.lowrank_s_kernel = sv[0];
  p.lowrank_s_split = sv[1];
  p.lowrank_s_tile_m = sv[2];
  p.lowrank_s_tile_n = sv[3];
  const NTList f = fwd_list(L, dt, T), g = bwd_list(L, dt, T);
  const NTChoice cf = nt_choose(dt, b, f.G, 128, f.kmax + r / b, T, f.ntiles, 1, false);
  const NTChoice cg =
      use_bwd_pairs(L, dt, T, r)
          ? nt_choose(dt, 64, 1, 128, L->kmax_bwd_p + r / 64, T, (int)L->bwd_tiles_p.size(), 1, false)
          : nt_choose(dt, b, g.G, 128, g.kmax + r / b, T, g.ntiles, 1, false);
  p.fwd_tile_m = cf.bm;
  p.fwd_tile_n = cf.bn;
  p.fwd_direct_lds = cf.dma;
  p.bwd_tile_m = cg.bm;
  p.bwd_tile_n = cg.bn;
  p.bwd_direct_lds = cg.dma;
  TNPlan tp;
  const pf::TNArgs a =
      tn_args(L, dtype, T, r, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, &tp);
  p.tn_items = pf::tn_items_total(a, tp.pairs ? 64 : b, tp.wide ? pf::kTNWTile : 128);
  p.tn_split = tp.nsplit;
  p.tn_chunk = tp.chunk;
  p.tn_tile = tp.wide ? pf::kTNWTile : 128;
  p.tn_shared = tp.shared;
  p.workspace_bytes = pf_workspace_bytes(L, T, r, dtype);
  *o = p;
  return PF_OK;
}

// Checks a caller workspace against a need of `need` bytes.
static pf_status need_ws(size_t need, const void *ws, size_t ws_bytes) {
  if (need == 0) return PF_OK;
  if (ws_bytes < need)
    return fail(PF_ERR_WORKSPACE, "workspace needs " + std::to_string(need) + " bytes");
  return need_ptr(ws, "workspace");
}

}  // extern "C"

namespace {

// Mixing weight of the mixed calls: alpha on the block-sparse part, beta on
// the low-rank part (alpha = gamma, beta = 1 - gamma).
struct Mix {
  bool on;
  float alpha, beta;
};
constexpr Mix kNoMix{false, 1.f, 1.f};

pf_status check_gamma(float gamma) {
  if (!std::isfinite(gamma)) return fail(PF_ERR_INVALID_ARG, "gamma must be finite");
  return PF_OK;
}

// The NT arguments' mixing fields for low-rank blocks nlr (0: none, or
// skipped because beta is 0).
void set_mix(pf::NTArgs &a, const Mix &m) {
  if (!m.on) return;
  a.mix = 1;
  if (a.nlr > 0 && m.beta != 0.f) {
    a.mix_ratio = m.alpha / m.beta;
    a.mix_out = m.beta;
  } else {
    a.nlr = 0;
    a.mix_ratio = 1.f;
    a.mix_out = m.alpha;
  }
}

pf_status linear_fwd(const pf_layout *L, pf_dtype dtype, int64_t T, int32_t r, const Mix &mix,
                     const void *X, const void *Wblk, const void *U, const void *V, void *Y,
                     void *T_lr, pf_epilogue epi, void *Y_pre, void *workspace, size_t ws_bytes,
                     void *stream) {
  pf_status st = check_layout_arg(L);
  if (st != PF_OK) return st;
  if ((st = check_dtype_r(dtype, T, r, L->b)) != PF_OK) return st;
  if ((st = check_extent(L, dtype, r)) != PF_OK) return st;
  if ((st = need_ptr(X, "X")) != PF_OK || (st = need_ptr(Wblk, "Wblk")) != PF_OK ||
      (st = need_ptr(Y, "Y")) != PF_OK)
    return st;
  if (r > 0 && ((st = need_ptr(U, "U")) != PF_OK || (st = need_ptr(V, "V")) != PF_OK ||
                (st = need_ptr(T_lr, "T_lr")) != PF_OK))
    return st;
  if (epi != PF_EPI_NONE && epi != PF_EPI_GELU) return fail(PF_ERR_INVALID_ARG, "bad epilogue");
  if (epi == PF_EPI_GELU && (st = need_ptr(Y_pre, "Y_pre")) != PF_OK) return st;
  if (epi == PF_EPI_NONE && Y_pre) return fail(PF_ERR_INVALID_ARG, "Y_pre given without GELU epilogue");
  const SkinnyPlan sp = rank_plan(L, (int)dtype, T, r, false);
  if ((st = need_ws(sp.ws, workspace, ws_bytes)) != PF_OK) return st;
  if ((st = check_state(L)) != PF_OK) return st;
  hipStream_t s = (hipStream_t)stream;
  const int dt = (int)dtype, b = L->b;
  if (use_skinny(dt, T, r, L->n_in)) {
    st = skinny_bf16(PF_KERNEL_LOWRANK_T, false, T, X, L->n_in, V, L->n_in, (int)L->n_in, r, T_lr,
                     s, "T_lr kernel");
    if (st != PF_OK) return st;
  } else if (r > 0) {
    // T_lr = X V^T: dense NT over K, r / blk output blocks.
    const int rb = sp.blk;
    st = dense_nt(PF_KERNEL_LOWRANK_T, dt, rb, sp.G, false, sp.bm, T, X, L->n_in, V, L->n_in,
                  (int)(L->n_in / rb), r / rb, T_lr, r, sp.nsplit, (float *)workspace, s,
                  "T_lr kernel");
    if (st != PF_OK) return st;
  }
  pf::NTArgs a{};
  a.A = X; a.lda = L->n_in;
  a.B = Wblk;
  a.L = T_lr; a.ldl = r; a.R = U; a.ldr = r; a.nlr = r / b;
  a.C = Y; a.ldc = L->n_out;
  a.C2 = epi == PF_EPI_GELU ? Y_pre : nullptr;
  a.epi = (int)epi;
  a.M = T;
  const NTList tl = fwd_list(L, dt, T);
  a.tiles = tl.tiles;
  a.ntiles = tl.ntiles;
  a.kcols = tl.kcols;
  a.blks = tl.blks;
  a.nsplit = 1;
  set_mix(a, mix);
  return hip_status(nt_launch(PF_KERNEL_SPMM_FWD, dt, b, tl.G, false, 128, tl.kmax + a.nlr, a, s),
                    "forward kernel");
}

}  // namespace

extern "C" {

pf_status pf_linear_fwd(const pf_layout *L, pf_dtype dtype, int64_t T, int32_t r, const void *X,
                        const void *Wblk, const void *U, const void *V, void *Y, void *T_lr,
                        pf_epilogue epi, void *Y_pre, void *workspace, size_t ws_bytes,
                        void *stream) {
  return linear_fwd(L, dtype, T, r, kNoMix, X, Wblk, U, V, Y, T_lr, epi, Y_pre, workspace,
                    ws_bytes, stream);
}

pf_status pf_linear_fwd_mixed(const pf_layout *L, pf_dtype dtype, int64_t T, int32_t r,
                              float gamma, const void *X, const void *Wblk, const void *U,
                              const void *V, void *Y, void *T_lr, pf_epilogue epi, void *Y_pre,
                              void *workspace, size_t ws_bytes, void *stream) {
  pf_status st = check_gamma(gamma);
  if (st != PF_OK) return st;
  return linear_fwd(L, dtype, T, r, Mix{true, gamma, 1.f - gamma}, X, Wblk, U, V, Y, T_lr, epi,
                    Y_pre, workspace, ws_bytes, stream);
}

}  // extern "C"

namespace {

// Argument checks of the backward calls (everything before any enqueue).
pf_status check_bwd_data_args(const pf_layout *L, pf_dtype dtype, int64_t T, int32_t r,
                              const void *dY, const void *Wblk, const void *U, const void *V,
                              const void *S, const void *dX, pf_epilogue epi, const void *aux) {
  pf_status st = check_layout_arg(L);
  if (st != PF_OK) return st;
  if ((st = check_dtype_r(dtype, T, r, L->b)) != PF_OK) return st;
  if ((st = check_extent(L, dtype, r)) != PF_OK) return st;
  if ((st = need_ptr(dY, "dY")) != PF_OK || (st = need_ptr(Wblk, "Wblk")) != PF_OK ||
      (st = need_ptr(dX, "dX")) != PF_OK)
    return st;
  if (r > 0 && ((st = need_ptr(U, "U")) != PF_OK || (st = need_ptr(V, "V")) != PF_OK ||
                (st = need_ptr(S, "S")) != PF_OK))
    return st;
  if (epi != PF_EPI_NONE && epi != PF_EPI_GELU) return fail(PF_ERR_INVALID_ARG, "bad epilogue");
  if (epi == PF_EPI_GELU && (st = need_ptr(aux, "aux")) != PF_OK) return st;
  return PF_OK;
}

pf_status check_bwd_weight_args(const pf_layout *L, pf_dtype dtype, int64_t T, int32_t r,
                                const void *dY, const void *X, const void *T_lr, const void *S,
                                const void *dWblk, const void *dU, const void *dV) {
  pf_status st = check_layout_arg(L);
  if (st != PF_OK) return st;
  if ((st = check_dtype_r(dtype, T, r, L->b)) != PF_OK) return st;
  if ((st = check_extent(L, dtype, r)) != PF_OK) return st;
  if ((st = need_ptr(dY, "dY")) != PF_OK || (st = need_ptr(X, "X")) != PF_OK ||
      (st = need_ptr(dWblk, "dWblk")) != PF_OK)
    return st;
  if (r > 0 && ((st = need_ptr(T_lr, "T_lr")) != PF_OK || (st = need_ptr(S, "S")) != PF_OK ||
                (st = need_ptr(dU, "dU")) != PF_OK || (st = need_ptr(dV, "dV")) != PF_OK))
    return st;
  return PF_OK;
}

// S = dY U (rank-r product, dense over N with U read as [k][n]).
pf_status enqueue_s(const pf_layout *L, int dt, int64_t T, int32_t r, const void *dY,
                    const void *U, void *S, const SkinnyPlan &sp, float *ws, hipStream_t s) {
  if (r <= 0) return PF_OK;
  if (use_skinny(dt, T, r, L->n_out))
    return skinny_bf16(PF_KERNEL_LOWRANK_S, true, T, dY, L->n_out, U, r, (int)L->n_out, r, S, s,
                       "S kernel");
  const int rb = sp.blk;
  return dense_nt(PF_KERNEL_LOWRANK_S, dt, rb, sp.G, true, sp.bm, T, dY, L->n_out, U, r,
                  (int)(L->n_out / rb), r / rb, S, r, sp.nsplit, ws, s, "S kernel");
}

// dX = dY (M o W) + S V (optionally times gelu'(aux)).  pair_ws: room for
// the pair blocks when use_bwd_pairs holds (pair_ws_bytes).
pf_status enqueue_dx(const pf_layout *L, int dt, int64_t T, int32_t r, const void *dY,
                     const void *Wblk, const void *S, const void *V, void *dX, pf_epilogue epi,
                     const void *aux, void *pair_ws, hipStream_t s, const Mix &mix = kNoMix) {
  const int b = L->b;
  pf::NTArgs a{};
  a.A = dY; a.lda = L->n_out;
  a.B = Wblk;
  a.L = S; a.ldl = r; a.R = V; a.ldr = L->n_in; a.nlr = r / b;
  a.C = dX; a.ldc = L->n_in;
  a.aux = aux;
  a.epi = (int)epi;
  a.M = T;
  if (use_bwd_pairs(L, dt, T, r)) {
    const int npair = (int)(L->pair_src.size() / 4);
    {
      Timed t(PF_KERNEL_REDUCE, s);
      pf_status st = hip_status(pf::launch_pair_gather(Wblk, L->d_pair_src, npair, pair_ws, s),
                                "pair gather kernel");
      if (st != PF_OK) return st;
    }
    a.B = pair_ws;
    a.nlr = r / 64;
    a.tiles = L->d_bwd_tiles_p;
    a.ntiles = (int)L->bwd_tiles_p.size();
    a.kcols = L->d_kcols_bwd_p;
    a.blks = L->d_blks_bwd_p;
    a.nsplit = 1;
    set_mix(a, mix);
    return hip_status(nt_launch(PF_KERNEL_SPMM_BWD_DATA, dt, 64, 1, true, 128,
                                L->kmax_bwd_p + a.nlr, a, s),
                      "backward-data kernel");
  }
  const NTList tl = bwd_list(L, dt, T);
  a.tiles = tl.tiles;
  a.ntiles = tl.ntiles;
  a.kcols = tl.kcols;
  a.blks = tl.blks;
  a.nsplit = 1;
  set_mix(a, mix);
  return hip_status(nt_launch(PF_KERNEL_SPMM_BWD_DATA, dt, b, tl.G, true, 128, tl.kmax + a.nlr, a, s),
                    "backward-data kernel");
}

// Launch order of the weight-gradient items.  Workgroups reach the eight
// XCDs in contiguous runs of launch positions, each XCD with its own L2, and
// the dU items read whole dY column blocks that kept-block items read too:
// placed apart, the same dY rows are fetched into two L2s.  So the dV items
// (S and X only) go first, then, for each group of dY block columns linked
// by a shared item (union-find over block rows of W), the group's kept-block
// items followed by its dU items.  Without the low-rank regions, or with
// more items than the order holds, the natural order stays.  `items` is the
// kept-block list of the launch, tiles of GT x GT blocks.
void set_tn_order(pf::TNArgs &a, const pf_layout *L, const std::vector<pf::TNItem> &items,
                  int GT) {
  a.n_order = 0;
  if (a.n_dense < 2) return;
  const pf::TNDense &d0 = a.dr[0], &d1 = a.dr[1];
  const int nsp = a.n_items;
  const int nbg0 = (d0.nb_blk + GT - 1) / GT, n0 = ((d0.na_blk + GT - 1) / GT) * nbg0;
  const int n1 = ((d1.na_blk + GT - 1) / GT) * ((d1.nb_blk + GT - 1) / GT);
  const int total = nsp + n0 + n1;
  if (total > pf::kTNOrderMax || total <= 0) return;
  std::vector<int> parent(L->nb_out);
  for (int i = 0; i < L->nb_out; ++i) parent[i] = i;
  auto find = [&](int x) {
    while (parent[x] != x) x = parent[x] = parent[parent[x]];
    return x;
  };
  auto unite = [&](int x, int y) { parent[find(x)] = find(y); };
  auto du_rows = [&](int q, int &r0, int &r1) {
    r0 = (q / nbg0) * GT;
    r1 = std::min(r0 + GT, d0.na_blk);
  };
  for (int i = 0; i < nsp; ++i) {
    const pf::TNItem &it = items[i];
    for (int g = 1; g < it.na; ++g) unite(it.a_col[g], it.a_col[0]);
  }
  for (int q = 0; q < n0; ++q) {
    int r0, r1;
    du_rows(q, r0, r1);
    for (int rr = r0 + 1; rr < r1; ++rr) unite(rr, r0);
  }
  // Buckets per group root, in order of first appearance.
  std::vector<std::vector<int>> sp_of(L->nb_out), du_of(L->nb_out);
  std::vector<int> roots;
  auto note = [&](int root) {
    if (sp_of[root].empty() && du_of[root].empty()) roots.push_back(root);
  };
  for (int i = 0; i < nsp; ++i) {
    const int root = find(items[i].a_col[0]);
    note(root);
    sp_of[root].push_back(i);
  }
  for (int q = 0; q < n0; ++q) {
    int r0, r1;
    du_rows(q, r0, r1);
    const int root = find(r0);
    note(root);
    du_of[root].push_back(nsp + q);
  }
  int k = 0;
  for (int q = 0; q < n1; ++q) a.order[k++] = (uint16_t)(nsp + n0 + q);
  for (int root : roots) {
    for (int i : sp_of[root]) a.order[k++] = (uint16_t)i;
    for (int i : du_of[root]) a.order[k++] = (uint16_t)i;
  }
  if (k == total) a.n_order = total;
}

// Weight-gradient work list and its token split (the 256 x 256 kernel when
// tn_wide allows; mixed calls always take the 128 x 128 one).
pf::TNArgs tn_args(const pf_layout *L, pf_dtype dtype, int64_t T, int32_t r, const void *dY,
                   const void *X, const void *T_lr, const void *S, void *dWblk, void *dU,
                   void *dV, TNPlan *plan, bool mixed) {
  pf::TNArgs a{};
  a.A = dY; a.lda = L->n_out;
  a.B = X; a.ldb = L->n_in;
  a.Wout = dWblk;
  a.T = T;
  a.scale_w = a.scale_lr = 1.f;
  if (tn_pairs(L, (int)dtype, T, r, mixed)) {
    fill_tn_regions(a, L, r, dY, X, T_lr, S, dU, dV, 64);
    a.items = L->d_tn_items_p; a.n_items = (int)L->tn_items_p.size();
    a.n_order = 0;
    *plan = tn_plan_wide(pf::tn_items_total(a, 64, pf::kTNWTile), T);
    plan->pairs = true;
    plan->pair_off = align256(plan->ws);
    plan->ws = plan->pair_off + (L->pair_src.size() / 4) * 64 * 64 * 2;
    a.nsplit = plan->nsplit;
    a.chunk = plan->chunk;
    return a;
  }
  fill_tn_regions(a, L, r, dY, X, T_lr, S, dU, dV);
  if (tn_wide(L, (int)dtype, T, r, mixed)) {
    a.items = L->d_tn_items_w; a.n_items = (int)L->tn_items_w.size();
    set_tn_order(a, L, L->tn_items_w, pf::kTNWTile / L->b);
    *plan = tn_plan_wide(pf::tn_items_total(a, L->b, pf::kTNWTile), T);
  } else {
    a.items = L->d_tn_items; a.n_items = (int)L->tn_items.size();
    set_tn_order(a, L, L->tn_items, 128 / L->b);
    *plan = tn_plan(pf::tn_items_total(a, L->b), T,
                    std::max(L->n_out, L->n_in) * (dtype == PF_BF16 ? 2 : 4), tn_min_tokens(dtype));
  }
  a.nsplit = plan->nsplit;
  a.chunk = plan->chunk;
  return a;
}

// dW on the mask, dU, dV (and the pass over split partials).
pf_status enqueue_tn(const pf_layout *L, int dt, pf::TNArgs a, const TNPlan &p, float *ws,
                     hipStream_t s) {
  a.partials = ws;
  if (p.wide) {
    const int blk = p.pairs ? 64 : L->b;
    void *const dW = a.Wout;
    if (p.pairs) a.Wout = (char *)ws + p.pair_off;
    {
      Timed t(PF_KERNEL_SDDMM, s);
      pf_status st = hip_status(pf::launch_tnw(blk, p.grid, a, s), "weight-gradient kernel");
      if (st != PF_OK) return st;
    }
    if (p.shared > 0) {
      Timed t(PF_KERNEL_REDUCE, s);
      pf_status st =
          hip_status(pf::launch_tnw_reduce(blk, p.shared, a, s), "weight-gradient reduction");
      if (st != PF_OK) return st;
    }
    if (!p.pairs) return PF_OK;
    Timed t(PF_KERNEL_REDUCE, s);
    return hip_status(pf::launch_pair_scatter(a.Wout, L->d_pair_src, (int)(L->pair_src.size() / 4),
                                              dW, s),
                      "pair scatter kernel");
  }
  {
    Timed t(PF_KERNEL_SDDMM, s);
    pf_status st = hip_status(pf::launch_tn(dt, L->b, a, s), "weight-gradient kernel");
    if (st != PF_OK) return st;
  }
  if (a.nsplit <= 1) return PF_OK;
  Timed t(PF_KERNEL_REDUCE, s);
  return hip_status(pf::launch_tn_reduce(dt, L->b, a, s), "weight-gradient reduction");
}

}  // namespace

extern "C" {

pf_status pf_linear_bwd_data(const pf_layout *L, pf_dtype dtype, int64_t T, int32_t r,
                             const void *dY, const void *Wblk, const void *U, const void *V,
                             void *S, void *dX, pf_epilogue epi, const void *aux,
                             void *workspace, size_t ws_bytes, void *stream) {
  pf_status st = check_bwd_data_args(L, dtype, T, r, dY, Wblk, U, V, S, dX, epi, aux);
  if (st != PF_OK) return st;
  const SkinnyPlan sp = rank_plan(L, (int)dtype, T, r, true);
  const size_t pws = pair_ws_bytes(L, (int)dtype, T, r);
  if ((st = need_ws(pws ? align256(sp.ws) + pws : sp.ws, workspace, ws_bytes)) != PF_OK) return st;
  if ((st = check_state(L)) != PF_OK) return st;
  hipStream_t s = (hipStream_t)stream;
  if ((st = enqueue_s(L, (int)dtype, T, r, dY, U, S, sp, (float *)workspace, s)) != PF_OK) return st;
  return enqueue_dx(L, (int)dtype, T, r, dY, Wblk, S, V, dX, epi, aux,
                    (char *)workspace + align256(sp.ws), s);
}

pf_status pf_linear_bwd_weight(const pf_layout *L, pf_dtype dtype, int64_t T, int32_t r,
                               const void *dY, const void *X, const void *T_lr, const void *S,
                               void *dWblk, void *dU, void *dV, void *workspace, size_t ws_bytes,
                               void *stream) {
  pf_status st = check_bwd_weight_args(L, dtype, T, r, dY, X, T_lr, S, dWblk, dU, dV);
  if (st != PF_OK) return st;
  if ((st = check_state(L)) != PF_OK) return st;
  TNPlan p;
  const pf::TNArgs a = tn_args(L, dtype, T, r, dY, X, T_lr, S, dWblk, dU, dV, &p);
  if ((st = need_ws(p.ws, workspace, ws_bytes)) != PF_OK) return st;
  return enqueue_tn(L, (int)dtype, a, p, (float *)workspace, (hipStream_t)stream);
}

pf_status pf_linear_bwd_data_mixed(const pf_layout *L, pf_dtype dtype, int64_t T, int32_t r,
                                   float gamma, const void *dY, const void *Wblk, const void *U,
                                   const void *V, void *S, void *dX, pf_epilogue epi,
                                   const void *aux, void *workspace, size_t ws_bytes,
                                   void *stream) {
  pf_status st = check_gamma(gamma);
  if (st != PF_OK) return st;
  if ((st = check_bwd_data_args(L, dtype, T, r, dY, Wblk, U, V, S, dX, epi, aux)) != PF_OK) return st;
  const SkinnyPlan sp = rank_plan(L, (int)dtype, T, r, true);
  const size_t pws = pair_ws_bytes(L, (int)dtype, T, r);
  if ((st = need_ws(pws ? align256(sp.ws) + pws : sp.ws, workspace, ws_bytes)) != PF_OK) return st;
  if ((st = check_state(L)) != PF_OK) return st;
  hipStream_t s = (hipStream_t)stream;
  if ((st = enqueue_s(L, (int)dtype, T, r, dY, U, S, sp, (float *)workspace, s)) != PF_OK) return st;
  return enqueue_dx(L, (int)dtype, T, r, dY, Wblk, S, V, dX, epi, aux,
                    (char *)workspace + align256(sp.ws), s, Mix{true, gamma, 1.f - gamma});
}

pf_status pf_linear_bwd_weight_mixed(const pf_layout *L, pf_dtype dtype, int64_t T, int32_t r,
                                     float gamma, const void *dY, const void *X,
                                     const void *Wblk, const void *T_lr, const void *S,
                                     void *dWblk, void *dU, void *dV, float *dgamma,
                                     void *workspace, size_t ws_bytes, void *stream) {
  pf_status st = check_gamma(gamma);
  if (st != PF_OK) return st;
  if ((st = check_bwd_weight_args(L, dtype, T, r, dY, X, T_lr, S, dWblk, dU, dV)) != PF_OK) return st;
  if ((st = need_ptr(Wblk, "Wblk")) != PF_OK) return st;
  if (!dgamma || ((uintptr_t)dgamma & 3)) return fail(PF_ERR_INVALID_ARG, "dgamma NULL or misaligned");
  if ((st = check_state(L)) != PF_OK) return st;
  TNPlan p;
  pf::TNArgs a = tn_args(L, dtype, T, r, dY, X, T_lr, S, dWblk, dU, dV, &p, true);
  const int items = pf::tn_items_total(a, L->b);
  const size_t off = align256(p.ws);
  const size_t need = off + mix_dgamma_bytes(items);
  if ((st = need_ws(need, workspace, ws_bytes)) != PF_OK) return st;
  a.scale_w = gamma;
  a.scale_lr = 1.f - gamma;
  a.wdot = Wblk;
  float *wparts = (float *)((char *)workspace + off);
  float *sparts = wparts + (size_t)items * 16;
  a.wdot_out = wparts;
  hipStream_t s = (hipStream_t)stream;
  if ((st = enqueue_tn(L, (int)dtype, a, p, (float *)workspace, s)) != PF_OK) return st;
  Timed t(PF_KERNEL_REDUCE, s);
  return hip_status(pf::launch_mix_dgamma((int)dtype, S, T_lr, r > 0 ? T * r : 0, wparts,
                                          a.nsplit > 1 ? items * 16 : items, sparts, dgamma, s),
                    "dgamma kernels");
}

pf_status pf_gelu_bwd(pf_dtype dtype, int64_t n, const void *dH, const void *H_pre, void *dH_pre,
                      void *stream) {
  if (dtype != PF_BF16 && dtype != PF_FP32) return fail(PF_ERR_INVALID_ARG, "bad dtype");
  if (n < 0) return fail(PF_ERR_INVALID_ARG, "n must be >= 0");
  if (n == 0) return PF_OK;
  pf_status st;
  if ((st = need_ptr(dH, "dH")) != PF_OK || (st = need_ptr(H_pre, "H_pre")) != PF_OK ||
      (st = need_ptr(dH_pre, "dH_pre")) != PF_OK)
    return st;
  Timed t(PF_KERNEL_GELU_BWD, (hipStream_t)stream);
  return hip_status(pf::launch_gelu_bwd((int)dtype, n, dH, H_pre, dH_pre, (hipStream_t)stream),
                    "gelu backward kernel");
}

static pf_status attn_check(const pf_layout *L, int32_t B, int32_t H, int32_t Sq, int32_t d) {
  pf_status st = check_layout_arg(L);
  if (st != PF_OK) return st;
  if (B < 1 || H < 1 || Sq < 1) return fail(PF_ERR_INVALID_ARG, "B, H, Sq must be >= 1");
  if (L->n_out != L->n_in || L->n_out != Sq)
    return fail(PF_ERR_INVALID_ARG, "attention layout must be square with side Sq");
  if (L->b != 64 || d != 64) return fail(PF_ERR_UNSUPPORTED, "attention supports b = 64, d = 64");
  if ((int64_t)B * H > 0x7fffffff / (Sq / 64)) return fail(PF_ERR_INVALID_ARG, "too many blocks");
  return PF_OK;
}

pf_status pf_attn_fwd(const pf_layout *L, int32_t B, int32_t H, int32_t Sq, int32_t d, float scale,
                      const void *Q, const void *K, const void *V, void *O, float *lse, void *stream) {
  pf_status st = attn_check(L, B, H, Sq, d);
  if (st != PF_OK) return st;
  if ((st = need_ptr(Q, "Q")) != PF_OK || (st = need_ptr(K, "K")) != PF_OK ||
      (st = need_ptr(V, "V")) != PF_OK || (st = need_ptr(O, "O")) != PF_OK ||
      (st = need_ptr(lse, "lse")) != PF_OK)
    return st;
  if ((st = check_state(L)) != PF_OK) return st;
  pf::AttnArgs a{};
  a.Q = Q; a.K = K; a.V = V; a.Oout = O; a.lse = lse;
  a.BH = B * H; a.S = Sq; a.nbq = Sq / 64; a.scale = scale;
  a.nlong = L->global_blocks;
  a.row_ptr = L->d_row_ptr; a.col_idx = L->d_col_idx;
  a.col_ptr = L->d_col_ptr; a.row_idx = L->d_row_idx;
  hipStream_t s = (hipStream_t)stream;
  if (a.nlong > 0) {
    {
      Timed t(PF_KERNEL_ATTN_FWD, s);
      if ((st = hip_status(pf::launch_attn_fwd(a, 1, s), "attention forward kernel")) != PF_OK) return st;
    }
    if (a.nlong == a.nbq) return PF_OK;
    Timed t(PF_KERNEL_ATTN_FWD, s);
    return hip_status(pf::launch_attn_fwd(a, 2, s), "attention forward kernel");
  }
  Timed t(PF_KERNEL_ATTN_FWD, s);
  return hip_status(pf::launch_attn_fwd(a, 0, s), "attention forward kernel");
}

size_t pf_attn_workspace_bytes(int32_t B, int32_t H, int32_t Sq) {
  if (B < 1 || H < 1 || Sq < 1) return 0;
  return ((size_t)B * H * Sq * sizeof(float) + 255) / 256 * 256;
}

}  // extern "C"

namespace {

// Argument checks of both attention backward calls (before any enqueue).
pf_status attn_bwd_check(const pf_layout *L, int32_t B, int32_t H, int32_t Sq, int32_t d,
                         const void *Q, const void *K, const void *V, const void *O,
                         const float *lse, const void *dO, void *dQ, void *dK, void *dV) {
  pf_status st = attn_check(L, B, H, Sq, d);
  if (st != PF_OK) return st;
  if ((st = need_ptr(Q, "Q")) != PF_OK || (st = need_ptr(K, "K")) != PF_OK ||
      (st = need_ptr(V, "V")) != PF_OK || (st = need_ptr(O, "O")) != PF_OK ||
      (st = need_ptr(lse, "lse")) != PF_OK || (st = need_ptr(dO, "dO")) != PF_OK ||
      (st = need_ptr(dQ, "dQ")) != PF_OK || (st = need_ptr(dK, "dK")) != PF_OK ||
      (st = need_ptr(dV, "dV")) != PF_OK)
    return st;
  return PF_OK;
}

// dQ (with delta = rowsum(dO o O) into `delta`, B*H*Sq floats), then dK, dV.
pf_status attn_bwd_enqueue(const pf_layout *L, int32_t B, int32_t H, int32_t Sq, float scale,
                           const void *Q, const void *K, const void *V, const void *O,
                           const float *lse, const void *dO, void *dQ, void *dK, void *dV,
                           float *delta, hipStream_t s) {
  pf::AttnArgs a{};
  a.Q = Q; a.K = K; a.V = V; a.O = O; a.dO = dO;
  a.dQ = dQ; a.dK = dK; a.dV = dV;
  a.lse_in = lse; a.delta = delta;
  a.BH = B * H; a.S = Sq; a.nbq = Sq / 64; a.scale = scale;
  a.nlong = L->global_blocks;
  a.row_ptr = L->d_row_ptr; a.col_idx = L->d_col_idx;
  a.col_ptr = L->d_col_ptr; a.row_idx = L->d_row_idx;
  // Parts: 0 (all rows) without global stripes, else 1 (the stripes'
  // long rows / columns, grouped kernels) then 2 (the rest).
  const int parts[2] = {a.nlong > 0 ? 1 : 0, 2};
  const int nparts = a.nlong > 0 && a.nlong < a.nbq ? 2 : 1;
  pf_status st;
  for (int i = 0; i < nparts; ++i) {
    Timed t(PF_KERNEL_ATTN_BWD_DQ, s);
    if ((st = hip_status(pf::launch_attn_bwd_dq(a, parts[i], s), "attention dQ kernel")) != PF_OK)
      return st;
  }
  for (int i = 0; i < nparts; ++i) {
    Timed t(PF_KERNEL_ATTN_BWD_DKV, s);
    if ((st = hip_status(pf::launch_attn_bwd_dkv(a, parts[i], s), "attention dK/dV kernel")) != PF_OK)
      return st;
  }
  return PF_OK;
}

}  // namespace

extern "C" {

pf_status pf_attn_bwd(const pf_layout *L, int32_t B, int32_t H, int32_t Sq, int32_t d, float scale,
                      const void *Q, const void *K, const void *V, const void *O, const float *lse,
                      const void *dO, void *dQ, void *dK, void *dV, void *workspace, size_t ws_bytes,
                      void *stream) {
  pf_status st = attn_bwd_check(L, B, H, Sq, d, Q, K, V, O, lse, dO, dQ, dK, dV);
  if (st != PF_OK) return st;
  if (ws_bytes < pf_attn_workspace_bytes(B, H, Sq))
    return fail(PF_ERR_WORKSPACE, "workspace too small");
  if ((st = need_ptr(workspace, "workspace")) != PF_OK) return st;
  if ((st = check_state(L)) != PF_OK) return st;
  return attn_bwd_enqueue(L, B, H, Sq, scale, Q, K, V, O, lse, dO, dQ, dK, dV,
                          (float *)workspace, (hipStream_t)stream);
}

pf_status pf_attn_bwd_noalloc(const pf_layout *L, int32_t B, int32_t H, int32_t Sq, int32_t d,
                              float scale, const void *Q, const void *K, const void *V,
                              const void *O, const float *lse, const void *dO, void *dQ, void *dK,
                              void *dV, void *stream) {
  pf_status st = attn_bwd_check(L, B, H, Sq, d, Q, K, V, O, lse, dO, dQ, dK, dV);
  if (st != PF_OK) return st;
  const int64_t rows = (int64_t)B * H * Sq;
  if (rows > pf::kAttnScratchRows)
    return fail(PF_ERR_UNSUPPORTED, "B * H * Sq = " + std::to_string(rows) +
                                        " query rows exceed the allocation-free scratch of " +
                                        std::to_string(pf::kAttnScratchRows) +
                                        " rows; use pf_attn_bwd with a workspace");
  if ((st = check_state(L)) != PF_OK) return st;
  float *delta = nullptr;
  if ((st = hip_status(pf::attn_scratch(&delta), "attention scratch lookup")) != PF_OK) return st;
  return attn_bwd_enqueue(L, B, H, Sq, scale, Q, K, V, O, lse, dO, dQ, dK, dV, delta,
                          (hipStream_t)stream);
}

}  // extern "C"

namespace {

// The product-form butterfly calls: validation (before any enqueue) and
// the one launch.
pf_status butterfly_call(bool bwd, const pf_layout *L, int64_t T, const void *in, const void *F,
                         void *out, void *save, void *stream) {
  if (!L) return fail(PF_ERR_INVALID_ARG, "layout is NULL");
  if (L->bfly_nfac < 1) return fail(PF_ERR_INVALID_ARG, "not a product-form butterfly layout");
  const int64_t k = (int64_t)1 << L->bfly_nfac;
  if (L->b != pf::kBflyBlock || k * L->b > pf::kBflyMaxGroupCols)
    return fail(PF_ERR_UNSUPPORTED, "the product kernel supports b = 32, max_stride <= 32");
  if (T < 1 || T > ((int64_t)1 << 30)) return fail(PF_ERR_INVALID_ARG, "T must be in [1, 2^30]");
  if (L->bfly_n * L->bfly_nfac * 2 > kMaxRowBytes)
    return fail(PF_ERR_UNSUPPORTED, "rows of the saved activations too wide");
  pf_status st;
  if ((st = need_ptr(in, bwd ? "dY" : "X")) != PF_OK || (st = need_ptr(F, "F")) != PF_OK ||
      (st = need_ptr(out, bwd ? "dX" : "Y")) != PF_OK)
    return st;
  if (save && (st = need_ptr(save, bwd ? "grads" : "acts")) != PF_OK) return st;
  pf::BflyArgs a{};
  a.in = in;
  a.F = F;
  a.out = out;
  a.save = save;
  a.T = T;
  a.n = L->bfly_n;
  a.nb = (int)(L->bfly_n / L->b);
  a.k = (int)k;
  a.nfac = L->bfly_nfac;
  hipStream_t s = (hipStream_t)stream;
  Timed t(PF_KERNEL_BUTTERFLY, s);
  return hip_status(pf::launch_bfly(bwd, a, s), "butterfly product kernel");
}

}  // namespace

extern "C" {

pf_status pf_butterfly_fwd(const pf_layout *L, int64_t T, const void *X, const void *F, void *Y,
                           void *acts, void *stream) {
  return butterfly_call(false, L, T, X, F, Y, acts, stream);
}

pf_status pf_butterfly_bwd_data(const pf_layout *L, int64_t T, const void *dY, const void *F,
                                void *dX, void *grads, void *stream) {
  return butterfly_call(true, L, T, dY, F, dX, grads, stream);
}

size_t pf_dense_workspace_bytes(pf_dtype dtype, pf_gemm_op op, int64_t M, int64_t N, int64_t K) {
  if (dtype != PF_BF16 && dtype != PF_FP32) return 0;
  if (op != PF_OP_TN || M < 64 || N < 64 || K < 1 || M % 64 || N % 64) return 0;
  int items = (int)(((M / 64 + 1) / 2) * ((N / 64 + 1) / 2));
  return tn_plan(items, K, std::max(M, N) * (dtype == PF_BF16 ? 2 : 4), tn_min_tokens(dtype)).ws;
}

// Blocks of 64 columns per dense comparator tile: 256-wide bf16 tiles when
// the shape fills them, else 128.
static int dense_g(int dt, int64_t M, int64_t N) {
  return (ntd_width(dt, 64, 4) && N % 256 == 0 && M >= PF_WIDE_MIN_T) ? 4 : 2;
}

pf_status pf_dense_gemm(pf_dtype dtype, pf_gemm_op op, int64_t M, int64_t N, int64_t K,
                        const void *A, const void *B, void *C, void *workspace, size_t ws_bytes,
                        void *stream) {
  if (dtype != PF_BF16 && dtype != PF_FP32) return fail(PF_ERR_INVALID_ARG, "bad dtype");
  if (M < 1 || N < 1 || K < 1) return fail(PF_ERR_INVALID_ARG, "M, N, K must be >= 1");
  if (M % 64 || N % 64) return fail(PF_ERR_UNSUPPORTED, "M and N must be multiples of 64");
  if (op != PF_OP_TN && K % 64) return fail(PF_ERR_UNSUPPORTED, "K must be a multiple of 64");
  if (M / 64 > (1 << 24) || N / 64 > (1 << 24) || K / 64 > (1 << 24))
    return fail(PF_ERR_INVALID_ARG, "dimensions too large");
  pf_status st;
  if ((st = need_ptr(A, "A")) != PF_OK || (st = need_ptr(B, "B")) != PF_OK ||
      (st = need_ptr(C, "C")) != PF_OK)
    return st;
  hipStream_t s = (hipStream_t)stream;
  const int dt = (int)dtype;
  switch (op) {
    case PF_OP_NT:
      return dense_nt(PF_KERNEL_DENSE, dt, 64, dense_g(dt, M, N), false, 128, M, A, K, B, K,
                      (int)(K / 64), (int)(N / 64), C, N, 1, nullptr, s, "dense NT");
    case PF_OP_NN:
      return dense_nt(PF_KERNEL_DENSE, dt, 64, dense_g(dt, M, N), true, 128, M, A, K, B, N,
                      (int)(K / 64), (int)(N / 64), C, N, 1, nullptr, s, "dense NN");
    case PF_OP_TN: {
      pf::TNArgs a{};
      a.n_items = 0;
      a.scale_w = a.scale_lr = 1.f;
      a.dr[0] = pf::TNDense{A, M, B, N, C, N, (int)(M / 64), (int)(N / 64)};
      a.n_dense = 1;
      a.T = K;
      TNPlan p = tn_plan(pf::tn_items_total(a, 64), K, std::max(M, N) * (dtype == PF_BF16 ? 2 : 4),
                         tn_min_tokens(dtype));
      if ((st = need_ws(p.ws, workspace, ws_bytes)) != PF_OK) return st;
      a.nsplit = p.nsplit;
      a.chunk = p.chunk;
      a.partials = (float *)workspace;
      {
        Timed t(PF_KERNEL_DENSE, s);
        st = hip_status(pf::launch_tn(dt, 64, a, s), "dense TN");
        if (st != PF_OK) return st;
      }
      if (a.nsplit <= 1) return PF_OK;
      Timed t(PF_KERNEL_REDUCE, s);
      return hip_status(pf::launch_tn_reduce(dt, 64, a, s), "dense TN reduction");
    }
  }
  return fail(PF_ERR_INVALID_ARG, "bad op");
}

}  // extern "C"
