// Weight-gradient product on 256 x 256 tiles (bf16, b = 64 or 128):
//   dW = dY^T X on the kept blocks, dU = dY^T T_lr, dV = S^T X
// reduced over all tokens (Appendix on gradient computation: the gradient of
// a block-sparse weight is the dense gradient restricted to its mask).
//
// Compared with the 128 x 128 TN kernel of gemm_kernels.hip this one
//  * copies operands global -> LDS directly (buffer_load ... lds, 16 bytes a
//    lane, chunks XOR-swizzled so the transpose fragment reads are free of
//    bank conflicts), four stages of 32 tokens, three steps in flight;
//  * runs 8 waves of 128 x 64 on a 256 x 256 tile: 128 flop per operand
//    byte staged through LDS (the 128 x 128 tile has 64);
//  * covers the token range without a split into fp32 partials for every
//    item: the grid is one workgroup per CU, and each workgroup first runs
//    whole items (item g, g + G, ... while full rounds of G remain; the
//    workgroups of a round move through the tokens in step, so items that
//    share operand columns find them in L2), then a contiguous share of the
//    (item, step) space of the remaining items, so every workgroup gets the
//    same number of steps.  A segment of a shared item goes to the
//    workgroup's own fp32 slot (slot 0: the first segment of its share,
//    slot 1: the last), and tnw_reduce_kernel adds an item's segments in
//    token order (deterministic) and stores it.
//
// Output tile orientation: the MFMA takes the X-side fragment as its first
// operand, so each lane holds 4 consecutive columns of one row of dW (or of
// dU / dV) and stores them as 8 bytes.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

#include "pf_dma.h"
#include "pf_launch.h"

namespace pf {
namespace {

constexpr int kWT = 256;      // tile side
constexpr int kWK = 32;          // tokens per step
constexpr int kWNS = 4;          // pipeline stages (three steps in flight)
constexpr int kWOp = kWK * 512;  // bytes of one operand in a stage
constexpr int kWDma = 2 * (kWOp / 1024) / 8;  // copies per wave and step
constexpr int kWSlot = kWT * kWT;  // floats of one partial slot

// A work item on 256 x 256 tiles: a kept-block item of the wide list or a
// tile of a dense region (dU, dV).
template <int BLK>
struct WItem {
  static constexpr int GT = kWT / BLK;
  bool sparse;
  const TNItem *it;
  int na, nb, ag, bg;
  const bf16_t *Ab, *Bb;
  int64_t lda, ldb, ldo;
  bf16_t *dout;

  __device__ __forceinline__ void decode(const TNArgs &a, int item) {
    const int n0 = a.n_dense > 0 ? ((a.dr[0].na_blk + GT - 1) / GT) * ((a.dr[0].nb_blk + GT - 1) / GT) : 0;
    sparse = item < a.n_items;
    it = sparse ? a.items + item : nullptr;
    ag = bg = 0;
    dout = nullptr;
    ldo = 0;
    if (sparse) {
      Ab = (const bf16_t *)a.A; lda = a.lda;
      Bb = (const bf16_t *)a.B; ldb = a.ldb;
      na = ld_meta(&it->na); nb = ld_meta(&it->nb);
    } else {
      int q = item - a.n_items, r = 0;
      if (q >= n0) { q -= n0; r = 1; }
      const TNDense &d = a.dr[r];
      const int nbg = (d.nb_blk + GT - 1) / GT;
      ag = q / nbg; bg = q % nbg;
      Ab = (const bf16_t *)d.A; lda = d.lda;
      Bb = (const bf16_t *)d.B; ldb = d.ldb;
      na = min(GT, d.na_blk - ag * GT);
      nb = min(GT, d.nb_blk - bg * GT);
      dout = (bf16_t *)d.out;
      ldo = d.ldo;
    }
  }
  __device__ __forceinline__ int acol(int g) const {
    return sparse ? ld_meta(&it->a_col[g]) : ag * GT + min(g, na - 1);
  }
  __device__ __forceinline__ int bcol(int g) const {
    return sparse ? ld_meta(&it->b_col[g]) : bg * GT + min(g, nb - 1);
  }
  __device__ __forceinline__ int oblk(int ga, int gb) const {
    return sparse ? ld_meta(&it->out_blk[ga * kTNMax + gb]) : ((ga < na && gb < nb) ? 0 : -1);
  }
};

__device__ __forceinline__ int wide_items_total(const TNArgs &a, int GT) {
  int n = a.n_items;
  for (int r = 0; r < a.n_dense; ++r)
    n += ((a.dr[r].na_blk + GT - 1) / GT) * ((a.dr[r].nb_blk + GT - 1) / GT);
  return n;
}

// Workgroup whose share of the remaining (item, step) space [0, Lw) holds
// position x: the largest q with floor(Lw q / G) <= x.
__device__ __forceinline__ int share_of(int64_t x, int64_t Lw, int G) {
  int q = (int)((x * G) / Lw);
  while (q + 1 < G && (Lw * (q + 1)) / G <= x) ++q;
  while (q > 0 && (Lw * q) / G > x) --q;
  return q;
}

// Store 4 consecutive values of a tile (row R, columns C .. C+3, both
// within the 256 x 256 tile) as bf16: into the packed dW block, or into a
// dense region's rows; nothing where the tile keeps no block.
template <int BLK>
__device__ __forceinline__ void store4(const TNArgs &a, const WItem<BLK> &v, int R, int C, f32x4 f) {
  const int ga = R / BLK, gb = C / BLK;
  const int blk = v.oblk(ga, gb);
  if (blk < 0) return;
  const int rl = R % BLK, cl = C % BLK;
  bf16_t *dst = v.sparse ? (bf16_t *)a.Wout + (int64_t)blk * (BLK * BLK) + rl * BLK + cl
                         : v.dout + ((int64_t)v.acol(ga) * BLK + rl) * v.ldo + (int64_t)v.bcol(gb) * BLK + cl;
  *(u32x2 *)dst = u32x2{(uint32_t)__builtin_bit_cast(uint16_t, (__bf16)f[0]) |
                            ((uint32_t)__builtin_bit_cast(uint16_t, (__bf16)f[1]) << 16),
                        (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)f[2]) |
                            ((uint32_t)__builtin_bit_cast(uint16_t, (__bf16)f[3]) << 16)};
}

// Offset in a partial slot of the 4 values (tn, tm, q) of thread tid:
// lane-contiguous, so each wave's store or load covers 1 KiB.
__device__ __forceinline__ int slot_idx(int tn, int tm, int q, int tid) {
  return (((tn * 4 + tm) * 4 + q) * 512 + tid) * 4;
}

template <int BLK>
__global__ __launch_bounds__(512, 1) void tnw_kernel(TNArgs a_arg) {
  const TNArgs a = a_arg;
  constexpr int GT = kWT / BLK;
  constexpr int TM = 4, TN = 2;  // wave tile: 128 dW rows x 64 dW columns
  constexpr int CPB = BLK / 8;   // 16-byte chunks per block row
  static_assert(GT <= kTNMax, "item width");
  // One LDS object per stage (A at 0, B at kWOp), each read at one integer
  // offset from its object (see frag_kn), so the copies into the next stages
  // stay in flight while this one is read.
  uint8_t *const lds0 = stage_buf<0, 2 * kWOp>(), *const lds1 = stage_buf<1, 2 * kWOp>();
  uint8_t *const lds2 = stage_buf<2, 2 * kWOp>(), *const lds3 = stage_buf<3, 2 * kWOp>();
  struct Stage {
    uint8_t *a, *b;
  };
  auto stage = [&](auto j) __attribute__((always_inline)) -> Stage {
    constexpr int J = decltype(j)::value % kWNS;
    if constexpr (J == 0) return Stage{lds0, lds0 + kWOp};
    else if constexpr (J == 1) return Stage{lds1, lds1 + kWOp};
    else if constexpr (J == 2) return Stage{lds2, lds2 + kWOp};
    else return Stage{lds3, lds3 + kWOp};
  };

  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  // dW rows (dY columns) in two halves, dW columns (X columns) in quarters;
  // waves w and w + 4 (which share a SIMD) take different column quarters,
  // so a tile whose right half holds no kept block keeps every SIMD busy.
  const int wm = w & 1, wn = w >> 1;
  const int G = gridDim.x;
  const int g = xcd_remap(blockIdx.x, G);
  const int I = wide_items_total(a, GT);
  const int S = (int)((a.T + kWK - 1) / kWK);
  const int full = I / G, left = I - full * G;
  const int64_t Lw = (int64_t)left * S;
  const int64_t r0 = Lw * g / G, r1 = Lw * (g + 1) / G;

  // Lane part of the copies: row 2 win + rr of a window, LDS chunk position
  // p, and the global chunk it holds for even / odd windows.
  const int rr = lane >> 5, p = lane & 31;
  int cg[2];
#pragma unroll
  for (int par = 0; par < 2; ++par) cg[par] = p ^ ((((par << 1) | rr)) << 2);

  f32x16 acc[TN][TM];
  int rd = 0;
  int64_t x = r0;
  for (;;) {
    int pos, s0, s1, which = 0;
    bool whole;
    if (rd < full) {
      pos = rd * G + g;
      s0 = 0;
      s1 = S;
      whole = true;
      ++rd;
    } else if (x < r1) {
      const int li = (int)(x / S);
      s0 = (int)(x % S);
      s1 = (int)std::min<int64_t>(S, s0 + (r1 - x));
      pos = full * G + li;
      whole = s0 == 0 && s1 == S;
      which = x == r0 ? 0 : 1;
      x += s1 - s0;
    } else {
      break;
    }
    const int item = a.n_order > 0 ? (int)a_arg.order[pos] : pos;
    WItem<BLK> v;
    v.decode(a, item);

    // This wave's 128 x 64 piece of the tile holds a kept block?
    bool live_w = false;
#pragma unroll
    for (int tm = 0; tm < TM; ++tm)
      live_w |= v.oblk((wm * 128 + tm * 32) / BLK, (wn * 64) / BLK) >= 0;

    const int64_t t0 = (int64_t)s0 * kWK, t1 = std::min<int64_t>(a.T, (int64_t)s1 * kWK);
    const uint32_t lda_b = (uint32_t)(v.lda * 2), ldb_b = (uint32_t)(v.ldb * 2);
    const rsrc_t rA = make_rsrc(v.Ab + t0 * v.lda, (t1 - t0) * (int64_t)lda_b);
    const rsrc_t rB = make_rsrc(v.Bb + t0 * v.ldb, (t1 - t0) * (int64_t)ldb_b);
    uint32_t voA[2], voB[2];
#pragma unroll
    for (int par = 0; par < 2; ++par) {
      const int grp = cg[par] / CPB, inb = (cg[par] % CPB) * 16;
      voA[par] = rr * lda_b + (uint32_t)(v.acol(grp) * BLK * 2 + inb);
      voB[par] = rr * ldb_b + (uint32_t)(v.bcol(grp) * BLK * 2 + inb);
    }
    // Windows 2w, 2w+1 of each operand: token rows 4w .. 4w+3 of the step.
    constexpr int WPW = kWDma / 2;
    auto issue = [&](int t, Stage st) __attribute__((always_inline)) {
      sfor<WPW>([&](auto i) __attribute__((always_inline)) {
        const int win = w * WPW + i;
        const uint32_t row = (uint32_t)(t * kWK + 2 * win);
        dma16(rA, st.a + win * 1024, voA[i & 1], row * lda_b);
        dma16(rB, st.b + win * 1024, voB[i & 1], row * ldb_b);
      });
    };
    auto compute = [&](Stage st) __attribute__((always_inline)) {
      if (!live_w) return;
      sfor<kWK / 16>([&](auto kq) __attribute__((always_inline)) {
        bf16x8 af[TM], bfr[TN];
        sfor<TM>([&](auto tm) __attribute__((always_inline)) {
          af[tm] = frag_kn<512>(st.a, wm * 128 + tm * 32, kq, lane);
        });
        sfor<TN>([&](auto tn) __attribute__((always_inline)) {
          bfr[tn] = frag_kn<512>(st.b, wn * 64 + tn * 32, kq, lane);
        });
        sfor<TN>([&](auto tn) __attribute__((always_inline)) {
          sfor<TM>([&](auto tm) __attribute__((always_inline)) {
            acc[tn][tm] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bfr[tn], af[tm], acc[tn][tm], 0, 0, 0);
          });
        });
      });
    };

    sfor<TN>([&](auto tn) __attribute__((always_inline)) {
      sfor<TM>([&](auto tm) __attribute__((always_inline)) {
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[tn][tm][e] = 0.f;
      });
    });
    // Every wave is past the previous segment's reads of both stages.
    barrier();
    const int n = s1 - s0;
    // Steps 0 .. 2 in flight before the loop; at step t the copies of step
    // t + 3 go into the stage step t - 1 read (every wave is past it after
    // the barrier), and the wait leaves the two younger steps' copies in
    // flight.  The loop runs whole groups of four steps with no branch
    // around a copy (copies and waits under a branch make the compiler wait
    // for every copy before the reads): steps past the segment read rows
    // outside the buffer range, i.e. zeros, and add nothing.
    sfor<kWNS - 1>([&](auto j) __attribute__((always_inline)) { issue(j, stage(j)); });
    for (int t0 = 0; t0 < n; t0 += kWNS) {
      sfor<kWNS>([&](auto j) __attribute__((always_inline)) {
        wait_vm<2 * kWDma>();
        barrier();
        issue(t0 + j + kWNS - 1, stage(std::integral_constant<int, j + kWNS - 1>{}));
        compute(stage(j));
      });
    }
    // The copies still in flight land in LDS; none may outlive the segment.
    wait_vm<0>();

    auto own4 = [&](auto tn, auto tm, auto q) __attribute__((always_inline)) -> f32x4 {
      return f32x4{acc[tn][tm][q * 4 + 0], acc[tn][tm][q * 4 + 1], acc[tn][tm][q * 4 + 2],
                   acc[tn][tm][q * 4 + 3]};
    };
    if (whole) {
      sfor<TN>([&](auto tn) __attribute__((always_inline)) {
        sfor<TM>([&](auto tm) __attribute__((always_inline)) {
          sfor<4>([&](auto q) __attribute__((always_inline)) {
            store4(a, v, wm * 128 + tm * 32 + (lane & 31), wn * 64 + tn * 32 + q * 8 + (lane >> 5) * 4,
                   own4(tn, tm, q));
          });
        });
      });
    } else {
      float *slot = a.partials + ((int64_t)g * 2 + which) * kWSlot;
      sfor<TN>([&](auto tn) __attribute__((always_inline)) {
        sfor<TM>([&](auto tm) __attribute__((always_inline)) {
          sfor<4>([&](auto q) __attribute__((always_inline)) {
            *(f32x4 *)(slot + slot_idx(tn, tm, q, tid)) = own4(tn, tm, q);
          });
        });
      });
    }
  }
}

// Second pass over the shared items: workgroup (li, part) sums 1024 values
// of shared item li (4 per thread, the lane-contiguous slot order) over the
// segments of the workgroups whose shares hold it, in token order, and
// stores the kept ones.  Workgroups whose share is empty (fewer remaining
// steps than workgroups) hold no segment.
template <int BLK>
__global__ __launch_bounds__(256) void tnw_reduce_kernel(TNArgs a_arg) {
  const TNArgs a = a_arg;
  constexpr int GT = kWT / BLK;
  constexpr int G = kTNWGrid;
  const int I = wide_items_total(a, GT);
  const int S = (int)((a.T + kWK - 1) / kWK);
  const int full = I / G, left = I - full * G;
  const int64_t Lw = (int64_t)left * S;
  const int li = blockIdx.x / 64, part = blockIdx.x % 64;
  if (li >= left) return;
  const int pos = full * G + li;
  const int item = a.n_order > 0 ? (int)a_arg.order[pos] : pos;
  WItem<BLK> v;
  v.decode(a, item);
  // Slot position -> (tn, tm, q, thread) -> tile row and first of 4 columns.
  const int e = (part * 256 + threadIdx.x) * 4;
  const int chunk = e / 2048, th = (e % 2048) / 4;
  const int q = chunk % 4, tm = (chunk / 4) % 4, tn = chunk / 16;
  const int w = th / 64, lane = th % 64, wm = w & 1, wn = w >> 1;
  const int g_first = share_of((int64_t)li * S, Lw, G);
  const int g_last = share_of((int64_t)(li + 1) * S - 1, Lw, G);
  // Segments in batches of 8: the batch's loads are issued together, then
  // added in token order.
  f32x4 tot = {0.f, 0.f, 0.f, 0.f};
  bool first = true;
  for (int g0 = g_first; g0 <= g_last; g0 += 8) {
    f32x4 term[8];
    bool have[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int gk = g0 + u;
      // Empty shares (and positions past g_last) hold no segment; the item
      // is gk's first segment when gk's share starts in it.
      have[u] = gk <= g_last && (Lw * (gk + 1)) / G > (Lw * gk) / G;
      const int wk = (Lw * gk) / G >= (int64_t)li * S ? 0 : 1;
      if (have[u]) term[u] = *(const f32x4 *)(a.partials + ((int64_t)gk * 2 + wk) * kWSlot + e);
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      if (!have[u]) continue;
      tot = first ? term[u] : tot + term[u];
      first = false;
    }
  }
  store4(a, v, wm * 128 + tm * 32 + (lane & 31), wn * 64 + tn * 32 + q * 8 + (lane >> 5) * 4, tot);
}

}  // namespace

hipError_t launch_tnw(int blk, int grid, const TNArgs &a, hipStream_t s) {
  if (grid <= 0) return hipErrorInvalidValue;
  if (blk == 128) launch_kernel(tnw_kernel<128>, dim3((unsigned)grid), dim3(512), s, a);
  else if (blk == 64) launch_kernel(tnw_kernel<64>, dim3((unsigned)grid), dim3(512), s, a);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_tnw_reduce(int blk, int shared, const TNArgs &a, hipStream_t s) {
  if (shared <= 0) return hipSuccess;
  const dim3 grid((unsigned)shared * 64);
  if (blk == 128) launch_kernel(tnw_reduce_kernel<128>, grid, dim3(256), s, a);
  else if (blk == 64) launch_kernel(tnw_reduce_kernel<64>, grid, dim3(256), s, a);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}


}  // namespace pf
