// Host-only driver of the C ABI for the sanitizer build: builds every kind
// of layout over the workload shapes and a sweep of sizes, checks each with
// the library's own verifier, queries launch plans and workspace sizes over
// token counts and ranks, and calls every entry point with bad arguments.
// No device is used.  Exits 0 when every expectation holds.
#include <cstdint>
#include <cstdio>
#include <random>
#include <vector>

#include "pixelfly.h"

static int g_fail = 0;
#define EXPECT(cond)                                                            \
  do {                                                                          \
    if (!(cond)) {                                                              \
      ++g_fail;                                                                 \
      std::fprintf(stderr, "%s:%d: expectation failed: %s (%s)\n", __FILE__,    \
                   __LINE__, #cond, pf_last_error());                           \
    }                                                                           \
  } while (0)

// Plan and workspace queries over token counts and ranks; the weight
// gradient's token split keeps each split's rows below 2^31 bytes.
static void exercise_plans(const pf_layout *L, const pf_layout_info &info) {
  const int64_t Ts[] = {1, 63, 64, 65, 200, 1000, 4096, 8191, 16384, 32767};
  for (pf_dtype dt : {PF_BF16, PF_FP32}) {
    const int64_t es = dt == PF_BF16 ? 2 : 4;
    for (int64_t T : Ts)
      for (int32_t r : {0, info.b, 4 * info.b}) {
        pf_linear_plan p;
        pf_status st = pf_linear_plan_get(L, dt, T, r, &p);
        if (st != PF_OK) {
          EXPECT(st == PF_ERR_UNSUPPORTED || st == PF_ERR_INVALID_ARG);
          continue;
        }
        EXPECT(p.tn_split >= 1 && p.tn_chunk >= 1 && p.tn_chunk % 64 == 0);
        EXPECT((int64_t)p.tn_split * p.tn_chunk >= T);
        const int64_t row = (info.n_out > info.n_in ? info.n_out : info.n_in) * es;
        EXPECT(p.tn_split == 1 || p.tn_chunk * row <= 0x7fffffffLL);
        EXPECT(p.workspace_bytes == pf_workspace_bytes(L, T, r, dt));
        EXPECT(r > 0 || (p.lowrank_t_kernel == 0 && p.lowrank_s_kernel == 0));
      }
  }
}

static void exercise_layout(pf_layout *L) {
  EXPECT(pf_layout_check(L) == PF_OK);
  pf_layout_info info;
  EXPECT(pf_layout_info_get(L, &info) == PF_OK);
  EXPECT(info.row_ptr[0] == 0 && info.row_ptr[info.nb_out] == info.nnzb);
  EXPECT(info.col_ptr[0] == 0 && info.col_ptr[info.nb_in] == info.nnzb);
  for (int64_t q = 0; q < info.nnzb; ++q) {
    EXPECT(info.tperm[q] >= 0 && info.tperm[q] < info.nnzb);
    EXPECT(info.col_idx[info.tperm[q]] >= 0 && info.col_idx[info.tperm[q]] < info.nb_in);
  }
  int32_t stats[10];
  EXPECT(pf_layout_plan_get(L, stats, 10) == PF_OK);
  if (info.b == 32 || info.b == 64 || info.b == 128) {
    EXPECT(stats[5] == info.nnzb);
    exercise_plans(L, info);
  }
}

// Every compute call with NULL or misaligned pointers, and with plausible
// pointers on a layout that was never uploaded: each must fail on the host.
static void exercise_compute_errors(pf_layout *L, int32_t b) {
  void *const fake = reinterpret_cast<void *>(uintptr_t(1) << 40);  // aligned, never read
  void *const odd = reinterpret_cast<void *>((uintptr_t(1) << 40) + 2);
  const int32_t r = b;
  EXPECT(pf_linear_fwd(L, PF_BF16, 64, r, nullptr, fake, fake, fake, fake, fake, PF_EPI_NONE,
                       nullptr, fake, 1 << 30, nullptr) == PF_ERR_INVALID_ARG);
  EXPECT(pf_linear_fwd(L, PF_BF16, 64, r, odd, fake, fake, fake, fake, fake, PF_EPI_NONE, nullptr,
                       fake, 1 << 30, nullptr) == PF_ERR_INVALID_ARG);
  EXPECT(pf_linear_fwd(L, PF_BF16, 0, r, fake, fake, fake, fake, fake, fake, PF_EPI_NONE, nullptr,
                       fake, 1 << 30, nullptr) == PF_ERR_INVALID_ARG);
  EXPECT(pf_linear_fwd(L, PF_BF16, 64, r + 1, fake, fake, fake, fake, fake, fake, PF_EPI_NONE,
                       nullptr, fake, 1 << 30, nullptr) == PF_ERR_INVALID_ARG);
  EXPECT(pf_linear_fwd(L, PF_BF16, 64, r, fake, fake, fake, fake, fake, fake, PF_EPI_NONE,
                       nullptr, fake, 1 << 30, nullptr) == PF_ERR_STATE);
  EXPECT(pf_linear_fwd(L, PF_BF16, 64, r, fake, fake, fake, fake, fake, fake, PF_EPI_GELU,
                       nullptr, fake, 1 << 30, nullptr) == PF_ERR_INVALID_ARG);
  EXPECT(pf_linear_bwd_data(L, PF_FP32, 64, r, fake, fake, fake, fake, nullptr, fake,
                            PF_EPI_NONE, nullptr, fake, 1 << 30, nullptr) == PF_ERR_INVALID_ARG);
  EXPECT(pf_linear_bwd_data(L, PF_FP32, 64, r, fake, fake, fake, fake, fake, fake, PF_EPI_NONE,
                            nullptr, fake, 1 << 30, nullptr) == PF_ERR_STATE);
  EXPECT(pf_linear_bwd_weight(L, PF_BF16, 64, r, fake, fake, fake, fake, fake, nullptr, fake,
                              fake, 1 << 30, nullptr) == PF_ERR_INVALID_ARG);
  EXPECT(pf_linear_bwd_weight(L, PF_BF16, 64, r, fake, fake, fake, fake, fake, fake, fake, fake,
                              1 << 30, nullptr) == PF_ERR_STATE);
  EXPECT(pf_linear_fwd_mixed(L, PF_BF16, 64, r, 1.0f / 0.0f, fake, fake, fake, fake, fake, fake,
                             PF_EPI_NONE, nullptr, fake, 1 << 30, nullptr) == PF_ERR_INVALID_ARG);
  EXPECT(pf_linear_bwd_weight_mixed(L, PF_BF16, 64, r, 0.5f, fake, fake, fake, fake, fake, fake,
                                    fake, fake, nullptr, fake, 1 << 30,
                                    nullptr) == PF_ERR_INVALID_ARG);
  EXPECT(pf_workspace_bytes(nullptr, 64, r, PF_BF16) == 0);
  EXPECT(pf_workspace_bytes(L, 0, r, PF_BF16) == 0);
}

int main() {
  std::mt19937 rng(2112);
  std::vector<pf_layout *> all;
  // keep(status, layout): call with the layout after the create call has
  // returned (a separate statement: argument evaluation order is unspecified).
  auto keep = [&](pf_status st, pf_layout *L) {
    EXPECT(st == PF_OK && L != nullptr);
    if (st == PF_OK && L) {
      exercise_layout(L);
      all.push_back(L);
    }
  };

  // The workload shapes.
  const int64_t shapes[][4] = {{1024, 1024, 32, 32},  {3072, 768, 32, 16},   {4096, 1024, 64, 16},
                               {1024, 4096, 64, 16},  {16384, 4096, 128, 32}, {16384, 4096, 64, 32},
                               {16384, 4096, 32, 32}, {4096, 4096, 32, 128}, {1024, 1024, 32, 2}};
  for (auto &s : shapes) {
    pf_layout *L = nullptr;
    {
      const pf_status st_ = pf_layout_create(s[0], s[1], (int32_t)s[2], (int32_t)s[3], &L);
      keep(st_, L);
    }
    if (L) exercise_compute_errors(L, (int32_t)s[2]);
  }
  // A sweep of sides, block sizes (including ones the kernels refuse) and
  // strides, square and rectangular both ways.
  for (int it = 0; it < 120; ++it) {
    const int32_t bs[] = {1, 2, 16, 32, 64, 128};
    const int32_t b = bs[rng() % 6];
    const int64_t nbo = 1 + rng() % 40, nbi = 1 + rng() % 40;
    const int32_t ms = 1 << (rng() % 8);
    pf_layout *L = nullptr;
    {
      const pf_status st_ = pf_layout_create(nbo * b, nbi * b, b, ms, &L);
      keep(st_, L);
    }
  }
  // Explicit block masks, attention masks with global stripes, factor
  // layouts, block covers of element masks.
  for (int it = 0; it < 40; ++it) {
    const int32_t nbo = 1 + rng() % 24, nbi = 1 + rng() % 24, b = 32 << (rng() % 3);
    std::vector<uint8_t> m((size_t)nbo * nbi, 0);
    for (auto &x : m) x = (rng() % 5) == 0;
    for (int32_t i = 0; i < nbo; ++i) m[(size_t)i * nbi + rng() % nbi] = 1;
    pf_layout *L = nullptr;
    {
      const pf_status st_ = pf_layout_create_from_mask(nbo, nbi, b, m.data(), &L);
      keep(st_, L);
    }
  }
  for (int32_t g : {0, 1, 3}) {
    pf_layout *L = nullptr;
    {
      const pf_status st_ = pf_layout_create_attention(4096, 64, 64, g, &L);
      keep(st_, L);
    }
  }
  for (int32_t k : {2, 4, 8, 16, 32}) {
    pf_layout *L = nullptr;
    {
      const pf_status st_ = pf_layout_create_factor(1024, 32, k, &L);
      keep(st_, L);
    }
  }
  {
    const int64_t n = 256;
    std::vector<uint8_t> e((size_t)n * n);
    for (auto &x : e) x = (rng() % 10) == 0;
    pf_layout *L = nullptr;
    {
      const pf_status st_ = pf_layout_create_from_element_mask(n, n, 32, e.data(), &L);
      keep(st_, L);
    }
  }
  // A token split whose rounding to whole steps would pass 2^31 bytes per
  // split, and a rank-r product whose second operand exceeds the rank-r
  // kernel's 32-bit range (tile kernel instead).
  {
    pf_layout *L = nullptr;
    {
      const pf_status st_ = pf_layout_create(65536, 65536, 128, 2, &L);
      keep(st_, L);
    }
    pf_linear_plan p;
    EXPECT(pf_linear_plan_get(L, PF_BF16, 32767, 0, &p) == PF_OK);
    EXPECT(p.tn_split >= 3 && p.tn_chunk * 65536 * 2 <= 0x7fffffffLL);
    pf_layout *W = nullptr;
    {
      const pf_status st_ = pf_layout_create(1024, 1 << 20, 128, 8, &W);
      keep(st_, W);
    }
    EXPECT(pf_linear_plan_get(W, PF_BF16, 64, 1024, &p) == PF_OK);
    EXPECT(p.lowrank_t_kernel == 2);
    EXPECT(pf_linear_plan_get(W, PF_BF16, 64, 128, &p) == PF_OK);
    EXPECT(p.lowrank_t_kernel == 1);
    pf_layout *X = nullptr;
    {
      const pf_status st_ = pf_layout_create(1024, 1 << 22, 128, 8, &X);
      keep(st_, X);
    }
    EXPECT(pf_linear_plan_get(X, PF_BF16, 64, 128, &p) == PF_ERR_UNSUPPORTED);
  }

  // Creation errors.
  pf_layout *L = nullptr;
  EXPECT(pf_layout_create(1024, 1024, 32, 3, &L) == PF_ERR_INVALID_ARG && L == nullptr);
  EXPECT(pf_layout_create(1000, 1024, 32, 4, &L) == PF_ERR_INVALID_ARG);
  EXPECT(pf_layout_create(1024, 1024, 0, 4, &L) == PF_ERR_INVALID_ARG);
  EXPECT(pf_layout_create(1024, 1024, 32, 4, nullptr) == PF_ERR_INVALID_ARG);
  EXPECT(pf_layout_create_from_mask(4, 4, 32, nullptr, &L) == PF_ERR_INVALID_ARG);
  {
    std::vector<uint8_t> m(16, 0);
    m[0] = 1;
    EXPECT(pf_layout_create_from_mask(4, 4, 32, m.data(), &L) == PF_ERR_INVALID_ARG);
  }
  EXPECT(pf_layout_create_attention(4096, 64, 64, 65, &L) == PF_ERR_INVALID_ARG);
  EXPECT(pf_layout_create_factor(1024, 32, 3, &L) == PF_ERR_INVALID_ARG);
  EXPECT(pf_layout_create_factor(1024, 32, 64, &L) == PF_ERR_INVALID_ARG);
  int32_t r = 0, ms = 0;
  int64_t params = 0;
  EXPECT(pf_select_mask(1024, 1024, 32, 0.25, 0.25, &r, &ms, &params) == PF_OK);
  EXPECT(r == 32 && ms == 32 && params == 262144);
  EXPECT(pf_select_mask(1024, 1024, 32, 0.0, 0.25, &r, &ms, &params) == PF_ERR_INVALID_ARG);
  EXPECT(pf_layout_upload(nullptr, nullptr) == PF_ERR_INVALID_ARG);
  EXPECT(pf_layout_check(nullptr) == PF_ERR_INVALID_ARG);
  EXPECT(pf_timing_end(nullptr, nullptr) == PF_ERR_STATE);
  EXPECT(pf_timing_begin(0) == PF_ERR_INVALID_ARG);
  EXPECT(pf_gelu_bwd(PF_BF16, -1, nullptr, nullptr, nullptr, nullptr) == PF_ERR_INVALID_ARG);
  EXPECT(pf_gelu_bwd(PF_BF16, 0, nullptr, nullptr, nullptr, nullptr) == PF_OK);
  EXPECT(pf_dense_gemm(PF_BF16, PF_OP_NT, 256, 128, 200, nullptr, nullptr, nullptr, nullptr, 0,
                       nullptr) == PF_ERR_UNSUPPORTED);
  EXPECT(!all.empty());
  if (!all.empty())
    EXPECT(pf_attn_fwd(all[0], 1, 1, 1024, 64, 0.125f, nullptr, nullptr, nullptr, nullptr, nullptr,
                     nullptr) == PF_ERR_UNSUPPORTED);  // b = 32 layout: attention needs b = 64
  EXPECT(pf_status_string(PF_ERR_STATE) != nullptr);

  for (pf_layout *x : all) pf_layout_destroy(x);
  pf_layout_destroy(nullptr);
  std::printf("host ABI check: %zu layouts, %d failed expectations\n", all.size(), g_fail);
  return g_fail == 0 ? 0 : 1;
}
