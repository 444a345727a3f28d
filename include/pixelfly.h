/*
 * pixelfly.h -- C ABI of libpixelfly.so, the MI355X (gfx950) hot path of
 * Pixelated Butterfly: the flat block butterfly + low-rank linear layer
 *
 *     Y = X (M o W)^T + (X V^T) U^T                      (Section 3.3)
 *
 * run forward and backward, and block-sparse softmax attention on the same
 * mask family (appendix on method details, attention).
 *
 * Conventions shared by every call
 *   - Matrices are row-major.  X: T x K (tokens x in-features), Y: T x N,
 *     U: N x r, V: r x K.  W is stored packed: the kept b x b blocks in
 *     block-CSR order (block row ascending, then block column ascending),
 *     element (q, c) of packed block p being W[i*b + q][j*b + c] for the
 *     block (i, j) at CSR position p.
 *   - Device pointers are plain device addresses (e.g. torch
 *     tensor.data_ptr()); `stream` is a hipStream_t passed as void* (NULL is
 *     the null stream).  The caller owns every device buffer it passes.
 *   - dtype is uniform per call: PF_BF16 (bfloat16 storage, fp32
 *     accumulation, round-to-nearest-even stores) or PF_FP32.
 *   - Compute calls validate every argument on the host before enqueuing
 *     anything; on error they return a negative pf_status, enqueue nothing
 *     and leave outputs untouched (pf_last_error() gives the detail).  They
 *     never allocate, never synchronise and return as soon as the kernels
 *     are enqueued on `stream`.
 *   - Calls that take a workspace need at least pf_workspace_bytes(...)
 *     bytes of device memory (16-byte aligned) whose contents on entry do
 *     not matter; the library uses it for fp32 partial sums when it splits a
 *     reduction over several workgroups.  Partials are summed in a fixed
 *     order, so results are deterministic.  A workspace must not be shared
 *     by calls that may run concurrently.  With a size of 0 the pointer may
 *     be NULL.
 *   - No C++ exception crosses this ABI.  Kernel launch failures map to
 *     PF_ERR_HIP.
 */
#ifndef PIXELFLY_H
#define PIXELFLY_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  PF_OK = 0,
  PF_ERR_INVALID_ARG = -1, /* bad dimension, null or misaligned pointer ... */
  PF_ERR_UNSUPPORTED = -2, /* valid but not implemented (e.g. b = 16)       */
  PF_ERR_WORKSPACE = -3,   /* workspace smaller than pf_workspace_bytes     */
  PF_ERR_HIP = -4,         /* a HIP runtime call or launch failed           */
  PF_ERR_NOMEM = -5,       /* host or device allocation failed (setup only) */
  PF_ERR_STATE = -6        /* layout not uploaded before a compute call     */
} pf_status;

typedef enum { PF_BF16 = 0, PF_FP32 = 1 } pf_dtype;

typedef enum {
  PF_EPI_NONE = 0,
  /* forward: Y_pre = acc, Y = gelu(acc) (exact erf GELU);
     backward-data: dX = acc * gelu'(aux) with aux = the forward's Y_pre. */
  PF_EPI_GELU = 1
} pf_epilogue;

typedef enum { PF_OP_NT = 0, PF_OP_NN = 1, PF_OP_TN = 2 } pf_gemm_op;

typedef struct pf_layout pf_layout; /* opaque; immutable after create */

/* Host views of a layout's block-CSR (valid until pf_layout_destroy). */
typedef struct {
  int64_t n_out, n_in;     /* N, K in elements                          */
  int32_t b;               /* block size                                */
  int32_t max_stride;      /* as requested, in blocks                   */
  int32_t eff_stride;      /* clamped to the next power of two >= s      */
  int32_t s;               /* square side min(nb_out, nb_in) in blocks   */
  int32_t nb_out, nb_in;   /* N / b, K / b                               */
  int64_t nnzb;            /* kept blocks                                */
  const int32_t *row_ptr;  /* [nb_out + 1]                               */
  const int32_t *col_idx;  /* [nnzb], CSR order                          */
  const int32_t *col_ptr;  /* [nb_in + 1]                                */
  const int32_t *row_idx;  /* [nnzb], CSC order                          */
  const int32_t *tperm;    /* [nnzb]: CSR position of the p-th CSC block */
} pf_layout_info;

/*
 * Build the flat block butterfly mask of an n_out x n_in weight with block
 * size b and maximum stride max_stride (in blocks) and its block-CSR.
 * Definitions: block butterfly factor and factor matrix (Section 3.1), flat
 * butterfly of maximum stride k = I + sum of factors B_2..B_k (Section 3.2),
 * mask selection by block size and maximum stride (Section 3.3, step 2),
 * rectangular "stretch" (appendix on method details).  In block units,
 * with s = min(n_out/b, n_in/b): block (i, j) is kept iff
 * x = (i mod s) XOR (j mod s) is 0 or a power of two below max_stride; the
 * s x s square is the power-of-two pattern cropped to s (partners >= s are
 * dropped) and is tiled along the longer dimension.
 * Requires b >= 1 dividing n_out and n_in, max_stride a power of two >= 1.
 * Host only (no device work).  *out receives a new layout (free with
 * pf_layout_destroy).  Errors: INVALID_ARG, NOMEM.
 */
pf_status pf_layout_create(int64_t n_out, int64_t n_in, int32_t b,
                           int32_t max_stride, pf_layout **out);

/*
 * Layout from an explicit block mask instead of the butterfly rule: block
 * (i, j) of the nb_out x nb_in grid is kept iff block_mask[i*nb_in + j] != 0
 * (row-major, host memory, read during the call only).  Serves the dense
 * comparator (all blocks kept) and other block patterns, e.g. the random
 * block patterns of the paper's microbenchmark (appendix on
 * microbenchmarking).  Every block row must keep at least one block.
 * max_stride and eff_stride of the layout read 0.  Host only.
 * Errors: INVALID_ARG, NOMEM.
 */
pf_status pf_layout_create_from_mask(int32_t nb_out, int32_t nb_in, int32_t b,
                                     const uint8_t *block_mask, pf_layout **out);

/*
 * Attention score layout for a sequence of seq tokens, block size b: the
 * square flat block butterfly of side seq / b (as pf_layout_create with
 * n_out = n_in = seq) plus the "global" component of the appendix on method
 * details (low-rank in attention): block rows and block columns
 * 0 .. global_blocks-1 are kept whole, i.e. the first global_blocks * b
 * queries attend to every key and every query attends to the first
 * global_blocks * b keys (stripes of width w = global_blocks * b, a term of
 * rank at most 2w).  global_blocks = 0 gives the plain butterfly mask.  The
 * layout serves pf_attn_fwd / pf_attn_bwd (which need b = 64).
 * Requires b >= 1 dividing seq, seq / b <= 16384, max_stride a power of two
 * >= 1, 0 <= global_blocks <= seq / b.  Host only; *out receives a new
 * layout (free with pf_layout_destroy).  Errors: INVALID_ARG, NOMEM.
 */
pf_status pf_layout_create_attention(int64_t seq, int32_t b, int32_t max_stride,
                                     int32_t global_blocks, pf_layout **out);

/*
 * Layout of the (b, b)-block cover of an arbitrary element mask (appendix on
 * the cost model: the block cover is the block-aligned mask with the fewest
 * nonzeros containing the mask; the kernels touch exactly its blocks, so
 * its density is the "actual density" of the appendix on
 * microbenchmarking).  elem_mask: n_out x n_in bytes, row-major host
 * memory, nonzero = kept element, read during the call only.  Block (i, j)
 * is kept iff any element of it is.  Values of W inside a kept block but
 * outside the element mask are the caller's (zeros reproduce the finer
 * mask).  Requires b >= 1 dividing n_out and n_in, at most 2^26 blocks, and
 * every block row keeping at least one block.  max_stride and eff_stride
 * read 0.  Host only.  Errors: INVALID_ARG, NOMEM.
 */
pf_status pf_layout_create_from_element_mask(int64_t n_out, int64_t n_in, int32_t b,
                                             const uint8_t *elem_mask, pf_layout **out);

/*
 * Layout of one factor of the butterfly product form, I + B_k, for an n x n
 * matrix with block size b: the butterfly factor matrix B_k^{(n/b)}
 * (Section 3.1: n/(b k) block-diagonal copies of a size-k factor
 * [[D1 D2],[D3 D4]] with diagonal D_i, in b x b block units) plus the
 * identity, i.e. block (p, q) kept iff p == q or p XOR q == k / 2: two
 * blocks per block row.  The residual butterfly (I + lam B_n) ... (I +
 * lam B_2) (Section 3.2) runs as a chain of layers on these layouts, its
 * flat first-order term as one layer on pf_layout_create(n, n, b, k_max);
 * the appendix on benchmarking the butterfly multiply compares the two.
 * Requires b >= 1 dividing n, n / b <= 16384, k a power of two >= 2
 * dividing n / b.  max_stride and eff_stride read k.  Host only.
 * Errors: INVALID_ARG, NOMEM.
 */
pf_status pf_layout_create_factor(int64_t n, int32_t b, int32_t k, pf_layout **out);

/*
 * Product form of an n x n block butterfly (Section 3.2: the product of
 * factors F_L ... F_1, each a general matrix on the support of I + B_k,
 * k = 2, 4, ..., max_stride; appendix on benchmarking the butterfly
 * multiply), as a layer on token rows: Y = X (F_L ... F_1)^T, smallest
 * stride applied first.  The layout returned here stacks the factors'
 * supports on the diagonal of an (L nb) x (L nb) block grid (L = log2
 * max_stride, nb = n / b): block row f nb + p keeps columns f nb + p and
 * f nb + (p XOR 2^f).  Its block-CSR order is the packing of the factors:
 * F (and dF) = [L][nb][2][b][b], factor f's block row p holding its two kept
 * blocks in ascending column order, element (r, c) of block (p, q) being
 * F_f[p b + r][q b + c].  Requires b >= 1 dividing n, max_stride a power of
 * two >= 2 dividing n / b.  Host only.  Errors: INVALID_ARG, NOMEM.
 */
pf_status pf_layout_create_butterfly(int64_t n, int32_t b, int32_t max_stride,
                                     pf_layout **out);

/*
 * One launch: the whole product on T token rows (bf16; b = 32 and
 * max_stride <= 32 in this build, else UNSUPPORTED).  Each workgroup holds a
 * 32-token x (max_stride * 32)-feature tile of the activation in LDS and
 * applies every factor to it in place.
 *   pf_butterfly_fwd:       Y = X (F_L ... F_1)^T; with acts non-NULL it also
 *                           writes the input of every factor, acts[t][f][:] =
 *                           x_f (x_0 = X, x_f = x_{f-1} F_{f+1}^T), T x (L n).
 *   pf_butterfly_bwd_data:  dX = dY F_L ... F_1; with grads non-NULL it also
 *                           writes the gradient at every factor's output,
 *                           grads[t][f][:] = g_{f+1} (g_L = dY, g_f = g_{f+1} F_{f+1}).
 * The factors' gradients, dF_f = (g_f^T x_{f-1}) on the support of F_f, are
 * one masked product on the same layout:
 *   pf_linear_bwd_weight(layout, PF_BF16, T, 0, grads, acts, NULL, NULL, dF,
 *                        NULL, NULL, workspace, ws_bytes, stream)
 * (that call needs pf_layout_upload; these two do not).  X, Y, dY, dX are
 * T x n row-major; pointers 16-byte aligned.  Errors: INVALID_ARG (not a
 * butterfly layout, bad sizes or pointers), UNSUPPORTED, HIP.
 */
pf_status pf_butterfly_fwd(const pf_layout *layout, int64_t T, const void *X,
                           const void *F, void *Y, void *acts, void *stream);
pf_status pf_butterfly_bwd_data(const pf_layout *layout, int64_t T, const void *dY,
                                const void *F, void *dX, void *grads, void *stream);

/*
 * Mask selection for one layer from a compute budget (Section 3.3, step 2):
 * a share lowrank_share of the budget (the paper's rule of thumb: one
 * quarter to one third) goes to the low-rank part, whose rank is the largest
 * multiple of the block size b within that share (and at most min(n_out,
 * n_in)); the rest selects the maximum stride of the flat block butterfly:
 * the largest power of two whose kept entries plus the low-rank entries
 * stay within the budget ("fill up the budget"), at least 1 (block
 * diagonal), at most the next power of two of s = min(n_out, n_in) / b.
 * Cost unit: weight entries, kept b x b blocks plus r (n_out + n_in),
 * against budget * n_out * n_in (per-token FLOPs are twice the entries).
 * budget in (0, 1], lowrank_share in [0, 1]; b >= 1 must divide n_out and
 * n_in.  Outputs: *r_out (rank), *max_stride_out, and (if not NULL)
 * *params_out, the entries of the chosen configuration (which exceed the
 * budget only when even the block diagonal does).  Host only.
 * Errors: INVALID_ARG, NOMEM.
 */
pf_status pf_select_mask(int64_t n_out, int64_t n_in, int32_t b, double budget,
                         double lowrank_share, int32_t *r_out, int32_t *max_stride_out,
                         int64_t *params_out);

/* Fill *out with host views of the layout.  Errors: INVALID_ARG. */
pf_status pf_layout_info_get(const pf_layout *layout, pf_layout_info *out);

/* Diagnostic: re-verify that the layout's kernel work lists (forward tiles,
 * backward-data tiles, weight-gradient items) cover every kept block exactly
 * once with the right packed index.  Host only.  Errors: INVALID_ARG with
 * the first violation in pf_last_error(). */
pf_status pf_layout_check(const pf_layout *layout);

/* Diagnostic: work-list statistics, n >= 6 entries written to stats:
 * [0] forward tile rows G, [1] forward tiles, [2] backward-data tile
 * columns G, [3] backward-data tiles, [4] weight-gradient items,
 * [5] kept blocks covered by those items; with n >= 10 also [6..9], the
 * same four figures of the wide (256-column) tile lists.  n >= 6.  Host
 * only. */
pf_status pf_layout_plan_get(const pf_layout *layout, int32_t *stats,
                             int32_t n);

/*
 * Diagnostic: the kernels and work split a forward + backward step of T
 * tokens at rank r runs on this layout (host only; the layout need not be
 * uploaded).  The rank-r products T_lr = X V^T and S = dY U report kernel 0
 * (r = 0, not run), 1 (the rank-r kernel: 32-token x 64-column workgroups)
 * or 2 (the tile kernel in dense mode), the number of workgroups that split
 * one output tile's K range (fp32 partials summed by a second pass when
 * above 1) and the output tile (tokens x columns).  The block-sparse
 * products report their output tile and kernel family (1: operands copied
 * global -> LDS directly; 0: staged through registers).  The weight
 * gradient reports its work items (kept-block tiles plus the dU and dV
 * tiles), the token split and the tokens per split, its tile side (128, or
 * 256 for the bf16 kernel whose 256 workgroups first run whole items and
 * then share the remaining items' tokens evenly) and, for the 256 tiles,
 * how many items are shared by several workgroups (their fp32 partial sums
 * added in token order by a second pass).  Errors as the compute calls'
 * argument checks: INVALID_ARG, UNSUPPORTED.
 */
typedef struct {
  int32_t lowrank_t_kernel, lowrank_t_split, lowrank_t_tile_m, lowrank_t_tile_n;
  int32_t lowrank_s_kernel, lowrank_s_split, lowrank_s_tile_m, lowrank_s_tile_n;
  int32_t fwd_tile_m, fwd_tile_n, fwd_direct_lds;
  int32_t bwd_tile_m, bwd_tile_n, bwd_direct_lds;
  int32_t tn_items, tn_split;
  int64_t tn_chunk;
  uint64_t workspace_bytes; /* pf_workspace_bytes of the same arguments */
  int32_t tn_tile, tn_shared;
} pf_linear_plan;

pf_status pf_linear_plan_get(const pf_layout *layout, pf_dtype dtype, int64_t T,
                             int32_t r, pf_linear_plan *out);

/*
 * Copy the layout's index arrays and kernel work lists to the current HIP
 * device (one-time, synchronous on `stream`).  Must precede compute calls;
 * the layout then serves that device only.  Errors: INVALID_ARG, HIP, NOMEM,
 * UNSUPPORTED (b not in {32, 64, 128}).
 */
pf_status pf_layout_upload(pf_layout *layout, void *stream);

/* Free host and device memory of the layout (NULL is a no-op).  The caller
 * must make sure no enqueued work still uses it. */
void pf_layout_destroy(pf_layout *layout);

/* Workspace bytes needed by pf_linear_fwd, pf_linear_bwd_data and
 * pf_linear_bwd_weight (the largest of the three) for T tokens and rank r;
 * 0 when none is needed or on invalid arguments. */
size_t pf_workspace_bytes(const pf_layout *layout, int64_t T, int32_t r,
                          pf_dtype dtype);

/*
 * Forward (Section 3.3; low-rank applied as U (V^T x), appendix on
 * efficient implementation):
 *     T_lr = X V^T                     (T x r, saved for the backward)
 *     Y    = X (M o W)^T + T_lr U^T    (T x N)
 * X: T x K, Wblk: packed [nnzb][b][b], U: N x r, V: r x K, Y: T x N,
 * T_lr: T x r.  r = 0 drops the low-rank term (U, V, T_lr may be NULL).
 * r must be a multiple of b (rank block-aligned, Section 3.3 step 2).
 * epi = PF_EPI_GELU writes Y_pre (T x N) = the pre-activation and
 * Y = gelu(Y_pre); with PF_EPI_NONE Y_pre must be NULL.
 * Tokens T >= 1 is arbitrary (ragged last tile handled).
 * Errors: INVALID_ARG, UNSUPPORTED, STATE, WORKSPACE, HIP.
 */
pf_status pf_linear_fwd(const pf_layout *layout, pf_dtype dtype, int64_t T,
                        int32_t r, const void *X, const void *Wblk,
                        const void *U, const void *V, void *Y, void *T_lr,
                        pf_epilogue epi, void *Y_pre, void *workspace,
                        size_t ws_bytes, void *stream);

/*
 * Backward-data (gradient of the layer w.r.t. its input):
 *     S  = dY U                         (T x r, saved for bwd_weight)
 *     dX = dY (M o W) + S V             (T x K)
 * dY: T x N.  With epi = PF_EPI_GELU, aux is a T x K tensor (the previous
 * layer's Y_pre) and dX = (dY (M o W) + S V) * gelu'(aux).
 * Errors: INVALID_ARG, UNSUPPORTED, STATE, WORKSPACE, HIP.
 */
pf_status pf_linear_bwd_data(const pf_layout *layout, pf_dtype dtype,
                             int64_t T, int32_t r, const void *dY,
                             const void *Wblk, const void *U, const void *V,
                             void *S, void *dX, pf_epilogue epi,
                             const void *aux, void *workspace,
                             size_t ws_bytes, void *stream);

/*
 * Backward-weight, restricted to the mask (gradient Lemma and sparse
 * training algorithm of the appendix on gradient computation):
 *     dW = (dY^T X) o M   stored packed like Wblk: only kept blocks
 *     dU = dY^T T_lr      (N x r)
 *     dV = S^T X          (r x K)
 * Reductions run over the T tokens.
 * Errors: INVALID_ARG, UNSUPPORTED, STATE, WORKSPACE, HIP.
 */
pf_status pf_linear_bwd_weight(const pf_layout *layout, pf_dtype dtype,
                               int64_t T, int32_t r, const void *dY,
                               const void *X, const void *T_lr, const void *S,
                               void *dWblk, void *dU, void *dV,
                               void *workspace, size_t ws_bytes, void *stream);

/*
 * The layer with the learnable mixing weight of Section 3.3 (model
 * sparsification): W = gamma B + (1 - gamma) (low-rank product), B the
 * block-sparse matrix on the mask, evaluated as the method does it:
 *
 *   pf_linear_fwd_mixed:       Y  = gamma X B^T + (1 - gamma) T_lr U^T,
 *                              T_lr = X V^T (stored unscaled);
 *   pf_linear_bwd_data_mixed:  dX = gamma dY B + (1 - gamma) S V,
 *                              S = dY U (stored unscaled);
 *   pf_linear_bwd_weight_mixed:
 *                              dW = gamma (dY^T X) o M (packed),
 *                              dU = (1 - gamma) dY^T T_lr,
 *                              dV = (1 - gamma) S^T X,
 *                              *dgamma = <(dY^T X) o M, B> - <S, T_lr>
 *                              = <dY, X B^T - T_lr U^T> (one fp32 scalar,
 *                              device memory, 4-byte aligned; summed in a
 *                              fixed order, so repeat calls agree bitwise).
 *
 * Arguments, layouts, epilogues, workspace and errors as the unmixed calls;
 * gamma must be finite (INVALID_ARG otherwise).  The kept-block sums are
 * scaled once in fp32 before the low-rank K-blocks join the same
 * accumulator, so each output is rounded once.  gamma = 1 skips the
 * low-rank K-blocks of the forward and backward-data products (T_lr and S
 * are still produced, dgamma needs them).  pf_linear_bwd_weight_mixed also
 * reads Wblk (the dgamma term) and needs pf_workspace_bytes of workspace
 * (it always includes room for the dgamma partials).
 */
pf_status pf_linear_fwd_mixed(const pf_layout *layout, pf_dtype dtype, int64_t T, int32_t r,
                              float gamma, const void *X, const void *Wblk, const void *U,
                              const void *V, void *Y, void *T_lr, pf_epilogue epi, void *Y_pre,
                              void *workspace, size_t ws_bytes, void *stream);
pf_status pf_linear_bwd_data_mixed(const pf_layout *layout, pf_dtype dtype, int64_t T, int32_t r,
                                   float gamma, const void *dY, const void *Wblk, const void *U,
                                   const void *V, void *S, void *dX, pf_epilogue epi,
                                   const void *aux, void *workspace, size_t ws_bytes,
                                   void *stream);
pf_status pf_linear_bwd_weight_mixed(const pf_layout *layout, pf_dtype dtype, int64_t T,
                                     int32_t r, float gamma, const void *dY, const void *X,
                                     const void *Wblk, const void *T_lr, const void *S,
                                     void *dWblk, void *dU, void *dV, float *dgamma,
                                     void *workspace, size_t ws_bytes, void *stream);

/* dH_pre = dH * gelu'(H_pre), n elements (exact erf GELU).  Standalone form
 * of the GELU epilogue.  Errors: INVALID_ARG, UNSUPPORTED, HIP. */
pf_status pf_gelu_bwd(pf_dtype dtype, int64_t n, const void *dH,
                      const void *H_pre, void *dH_pre, void *stream);

/*
 * Block-sparse attention forward, bf16, one mask shared by all B*H heads:
 *     S = Q K^T * scale on the kept b x b blocks only, softmax over each
 *     row's kept entries, O = P V, lse = log(sum exp S) per row (fp32).
 * Q, K, V, O: [B][H][Sq][d] bf16; lse: [B][H][Sq] fp32.  The layout must be
 * square (n_out = n_in = Sq) with b = 64; d = 64.  Non-causal, no dropout.
 * Errors: INVALID_ARG, UNSUPPORTED, STATE, HIP.
 */
pf_status pf_attn_fwd(const pf_layout *layout, int32_t B, int32_t H,
                      int32_t Sq, int32_t d, float scale, const void *Q,
                      const void *K, const void *V, void *O, float *lse,
                      void *stream);

/*
 * Block-sparse attention backward for L = <dO, O>:
 *     delta = rowsum(dO o O), P = exp(S - lse), dV = P^T dO,
 *     dS = P o (dO V^T - delta), dQ = dS K * scale, dK = dS^T Q * scale.
 * Same shapes as pf_attn_fwd; dQ, dK, dV bf16.  Needs a workspace of
 * B*H*Sq floats (pf_attn_workspace_bytes).
 * Errors: INVALID_ARG, UNSUPPORTED, STATE, WORKSPACE, HIP.
 */
pf_status pf_attn_bwd(const pf_layout *layout, int32_t B, int32_t H,
                      int32_t Sq, int32_t d, float scale, const void *Q,
                      const void *K, const void *V, const void *O,
                      const float *lse, const void *dO, void *dQ, void *dK,
                      void *dV, void *workspace, size_t ws_bytes,
                      void *stream);

/* Workspace bytes of pf_attn_bwd. */
size_t pf_attn_workspace_bytes(int32_t B, int32_t H, int32_t Sq);

/*
 * pf_attn_bwd without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, serving loops that
 * forbid allocation).  Same arguments, results and errors as pf_attn_bwd
 * minus the workspace; it allocates nothing.  The row terms delta live in a
 * library-owned device array of 2^22 floats (16 MiB) per GPU, held until the
 * process ends: calls with B*H*Sq above 2^22 fail with UNSUPPORTED.  Every
 * call on a GPU uses that GPU's one array, so calls that may overlap on one
 * GPU (other streams, other threads) race and must be serialised by the
 * caller.  The array's device address is looked up on the first call on
 * each device.
 */
pf_status pf_attn_bwd_noalloc(const pf_layout *layout, int32_t B, int32_t H,
                              int32_t Sq, int32_t d, float scale, const void *Q,
                              const void *K, const void *V, const void *O,
                              const float *lse, const void *dO, void *dQ,
                              void *dK, void *dV, void *stream);

/*
 * Dense comparator GEMM built from the same MFMA tiles as the sparse
 * kernels (the speedup baseline: an equally shaped dense layer):
 *   PF_OP_NT: C[M][N] = A[M][K] . B[N][K]^T   (forward,  X W^T)
 *   PF_OP_NN: C[M][N] = A[M][K] . B[K][N]     (backward-data, dY W)
 *   PF_OP_TN: C[M][N] = A[K][M]^T . B[K][N]   (backward-weight, dY^T X)
 * M, N multiples of 64; K a multiple of 64 (NT, NN) or >= 1 (TN, where K is
 * the reduction over tokens).  For TN a workspace of
 * pf_dense_workspace_bytes is needed.
 * Errors: INVALID_ARG, UNSUPPORTED, WORKSPACE, HIP.
 */
pf_status pf_dense_gemm(pf_dtype dtype, pf_gemm_op op, int64_t M, int64_t N,
                        int64_t K, const void *A, const void *B, void *C,
                        void *workspace, size_t ws_bytes, void *stream);

size_t pf_dense_workspace_bytes(pf_dtype dtype, pf_gemm_op op, int64_t M,
                                int64_t N, int64_t K);

/*
 * Kernel timing (a measurement aid, not part of the compute path).
 *
 * Every kernel the library launches belongs to one class below.  After
 * pf_timing_begin(n), the library records a HIP event pair on the launch
 * stream immediately before and after each of the next n launches of every
 * class (the events are created here, so the compute calls still allocate
 * nothing).  pf_timing_end waits for the recorded events, writes for each
 * class the number of timed launches and their mean duration in ms into
 * counts[PF_KERNEL_COUNT] / avg_ms[PF_KERNEL_COUNT] (either may be NULL),
 * and disarms the hook.  Recording is process-wide; timing calls must not
 * overlap compute calls issued from other threads.
 * Errors: INVALID_ARG (n < 1 or n > 2^20), STATE (end without begin),
 * NOMEM, HIP.
 */
typedef enum {
  PF_KERNEL_SPMM_FWD = 0,       /* forward block-sparse product (+ low-rank) */
  PF_KERNEL_SPMM_BWD_DATA = 1,  /* backward-data block-sparse product (+ low-rank) */
  PF_KERNEL_SDDMM = 2,          /* weight gradient on the mask, dU, dV */
  PF_KERNEL_LOWRANK_T = 3,      /* rank-r product T_lr = X V^T */
  PF_KERNEL_LOWRANK_S = 4,      /* rank-r product S = dY U */
  PF_KERNEL_REDUCE = 5,         /* sums of split partial results; the b = 32
                                   backward-data pair-block gather */
  PF_KERNEL_GELU_BWD = 6,       /* standalone GELU backward */
  PF_KERNEL_ATTN_FWD = 7,
  PF_KERNEL_ATTN_BWD_DQ = 8,    /* dQ (and the row terms delta) */
  PF_KERNEL_ATTN_BWD_DKV = 9,   /* dK, dV */
  PF_KERNEL_DENSE = 10,         /* dense comparator GEMM */
  PF_KERNEL_BUTTERFLY = 11,     /* product-form butterfly (forward, backward-data) */
  PF_KERNEL_COUNT = 12
} pf_kernel_class;

pf_status pf_timing_begin(int32_t max_launches_per_class);
pf_status pf_timing_end(int32_t *counts, double *avg_ms);

/* Static text of a status code. */
const char *pf_status_string(pf_status s);

/* Detail of the calling thread's last error ("" if none). */
const char *pf_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* PIXELFLY_H */
