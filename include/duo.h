/*
 * duo.h - C ABI of the MI355X (gfx950) DuoGPT layer solver.
 *
 * The library computes, for one linear layer, the activation-sparsity-aware
 * OBC pruning of DuoGPT (arXiv 2506.20194):
 *
 *   stage 1  duo_hessian_accum / duo_residual_term
 *            per-token magnitude sparsification of the calibration input and
 *            accumulation of H = Xh Xh^T, G = dX Xh^T and a = diag(dX dX^T)
 *            (Sec. 4.2-4.3, Algorithm 1 first two lines);
 *   stage 2  duo_chol_inv
 *            damping and the lower Cholesky factor L of the inverse Hessian,
 *            (H + lambda I)^-1 = L L^T (Sec. 4.3, "Inverse_Cholesky");
 *   stage 3  duo_score_terms + duo_sweep (together: duo_prune_layer)
 *            Q = G L, b, c, D = U L^T and the score factor of Eq. 7, then the
 *            blocked column sweep of Algorithm 1 with lazy batch updates.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Orientation.  The paper's calibration matrix X is k x m (channels x tokens).
 *   In memory activations are token-major: an m x k row-major array with row
 *   stride ldx >= k elements (PyTorch's activation layout), i.e. X^T.
 *   W is n x k row-major (out x in, PyTorch's Linear layout).  H, G, L and D are
 *   k x k row-major fp32 with a row stride >= k.  H[p][q] = sum_t Xh[t][p] Xh[t][q];
 *   G[p][q] = sum_t dX[t][p] Xh[t][q] (paper: dX Xh^T).
 * Streams X_src / X_dense.  X_src is the stream that is sparsified (the pruned
 *   model's input); X_dense is the dense model's input (the paper's X-tilde).
 *   For a single layer they are the same array; pass X_dense = NULL.
 * Pointers.  Every array argument is a DEVICE pointer owned by the caller,
 *   except where a comment says "host".  The library never allocates or frees
 *   device memory: scratch memory comes from the caller's workspace (ws,
 *   ws_bytes), sized by duo_workspace_size() and aligned to 256 bytes.
 * Streams.  `stream` is a hipStream_t (NULL = the default stream).  Work is
 *   enqueued on it in order; a call returns before the work finishes unless
 *   stated otherwise.  Calls that share a workspace must not overlap.
 * Errors.  Each call returns a duo_status.  Argument errors are detected on
 *   the host before anything is enqueued; nothing is written then.  Numerical
 *   failures detected on the device (non-positive pivot, non-finite input)
 *   are reported by duo_chol_inv.  No C++ exception crosses this interface.
 * Precision.  Inputs are fp32 or bf16; every product of two inputs is formed
 *   exactly (bf16) or in fp32, and every accumulation is fp32.  Results are
 *   deterministic: the same inputs give bitwise identical outputs.
 * Limits.  1 <= k <= 32768 (per-token selection keeps a token in registers),
 *   n >= 1, m >= 0, block in [1, 128].
 */
#ifndef DUO_H
#define DUO_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t duo_status;
enum {
  DUO_OK = 0,
  DUO_ERR_INVALID_ARG = 1,  /* null pointer, bad size/stride/ratio/dtype */
  DUO_ERR_UNSUPPORTED = 2,  /* valid but outside the library's limits    */
  DUO_ERR_WORKSPACE = 3,    /* workspace missing, too small or misaligned  */
  DUO_ERR_NOT_PD = 4,       /* damped Hessian not positive definite        */
  DUO_ERR_NONFINITE = 5,    /* NaN/Inf met where a finite value is needed  */
  DUO_ERR_HIP = 6,          /* a HIP runtime call failed                   */
  DUO_ERR_NO_DEVICE = 7     /* no gfx950 device is current                 */
};

/* element types of X and W */
enum { DUO_F32 = 0, DUO_BF16 = 1 };

/* Activation sparsification rule (Preliminaries, "Activation Sparsity").
 * DUO_ACT_TOPK_MAG_PER_TOKEN: every token keeps all but z = floor(p*k + 0.5)
 * of its k entries; the entries zeroed are those with the smallest key
 * (|x|, channel index), so on equal magnitude the lower channel goes first and
 * -0.0 counts as 0.  DUO_ACT_NONE keeps everything (p ignored). */
enum { DUO_ACT_NONE = 0, DUO_ACT_TOPK_MAG_PER_TOKEN = 1 };
typedef struct {
  int32_t kind;
  double sparsity; /* p^x in [0, 1] */
} duo_act_rule;

/* Which part of G stage 1 accumulates (duo_hessian_accum, duo_residual_term).
 * The solver reads only G's upper triangle, diagonal included: Eq. 7 uses
 * Q = G L only on and above its diagonal (U = strict upper(Q), c = diag(Q) /
 * diag(L)), and with L lower triangular Q[p][i], i >= p, involves G[p][l]
 * for l >= i >= p alone.  DUO_G_UPPER accumulates those entries (about half
 * of G's work): G[p][q] for p / 256 <= q / 256, i.e. the upper triangle plus
 * the lower halves of the 256 x 256 diagonal tiles, and leaves every other
 * entry as it was; DUO_G_FULL accumulates all of G (needed when the channels
 * are permuted afterwards, as for act_order). */
enum { DUO_G_UPPER = 0, DUO_G_FULL = 1 };

/* operations, for duo_workspace_size */
enum {
  DUO_OP_HESSIAN = 0,     /* duo_hessian_accum and duo_residual_term (uses m, k) */
  DUO_OP_CHOL_INV = 1,    /* duo_chol_inv (uses k)                               */
  DUO_OP_SCORE_TERMS = 2, /* duo_score_terms (uses k)                            */
  DUO_OP_SWEEP = 3,       /* duo_sweep (uses n, k, block)                        */
  DUO_OP_PRUNE_LAYER = 4  /* duo_prune_layer (uses n, k, block)                  */
};

/* Result record of duo_chol_inv (host memory). */
typedef struct {
  double lambda;      /* damping added to the diagonal                        */
  int64_t fail_index; /* a column whose pivot was not positive, else -1      */
  int32_t status;     /* DUO_OK, DUO_ERR_NOT_PD or DUO_ERR_NONFINITE          */
} duo_chol_info;

/* Bytes of workspace an operation needs (0 for a bad op).  Pure host
 * arithmetic; safe to call without a device. */
size_t duo_workspace_size(int32_t op, int64_t n, int64_t k, int64_t m, int32_t block);

/* Human-readable text of a status code (static storage). */
const char* duo_status_string(duo_status s);

/* Library version string, e.g. "duo 0.1.0 gfx950". */
const char* duo_version(void);

/*
 * duo_act_sparsify_mask - the activation mask alone (test and inspection hook).
 *   X (m x k, ldx, x_dtype) is sparsified per token with `rule`; bit c of
 *   token t is written to mask_out[t * ceil(k/32) + c/32] bit (c % 32),
 *   1 = kept.  mask_out must hold m * ceil(k/32) uint32 words.
 *   Workspace: DUO_OP_HESSIAN with the same m and k.
 */
duo_status duo_act_sparsify_mask(const void* X, int32_t x_dtype, int64_t m, int64_t k, int64_t ldx,
                                 duo_act_rule rule, uint32_t* mask_out, void* ws, size_t ws_bytes,
                                 void* stream);

/*
 * duo_hessian_accum - stage 1 (Algorithm 1, H <- Xh Xh^T; Sec. 4.3 a-term).
 *   X_src    m x k, ldx, x_dtype: the input to sparsify (Xh = sparsify(X_src)).
 *   X_dense  m x k, ldx, x_dtype, or NULL (= X_src): the dense stream.
 *   H        k x k fp32, ldh: H += Xh^T Xh over the m tokens; the sums are
 *            added to the upper triangle (diagonal included), and the lower
 *            triangle is then set to its mirror image, so H is returned
 *            exactly symmetric.
 *   G, a     optional (both NULL or both set): G += dX^T Xh with dX = X_dense - Xh,
 *            a[p] += sum_t dX[t][p]^2.  G is k x k fp32 with row stride ldg.
 *   g_part   DUO_G_UPPER: G[p][q] for p / 256 <= q / 256 (the upper triangle
 *            the solver reads, plus the rest of the diagonal 256 x 256 tiles);
 *            DUO_G_FULL: all of G.
 *   hdiag    NULL or k doubles: hdiag[p] += sum_t Xh[t][p]^2 summed in fp64
 *            (each square exact), the diagonal of H at the precision that
 *            decides the act_order channel order (duo_act_order).
 *   The caller zeroes H, G, a and hdiag before the first token chunk; further
 *   calls add more tokens (raw sums, no 1/m scaling).  For X_src != X_dense, dX is
 *   represented to ~16 significant bits inside the product (exact when the
 *   two streams' values are within a factor of 2^7 of each other or the entry
 *   is dropped); a is accumulated from exact fp32 differences.
 *   Workspace: DUO_OP_HESSIAN with the same m and k.
 */
duo_status duo_hessian_accum(const void* X_src, const void* X_dense, int32_t x_dtype, int64_t m,
                             int64_t k, int64_t ldx, duo_act_rule rule, float* H, int64_t ldh,
                             float* G, int64_t ldg, int32_t g_part, float* a, double* hdiag, void* ws,
                             size_t ws_bytes, void* stream);

/*
 * duo_hessian_status - non-finite input check of stage 1 (the calibration
 *   input must be finite for the sums of Sec. 4.2-4.3 to mean anything).
 *   Every duo_hessian_accum, duo_residual_term and duo_act_sparsify_mask call
 *   records in its workspace whether any entry of X_src or X_dense was NaN or
 *   +-inf (such entries are still selected by their magnitude bits, NaN above
 *   inf above every finite value, so H and G then hold non-finite sums).
 *   This call waits for `stream` and returns DUO_ERR_NONFINITE if the last
 *   such call on workspace `ws` met one, else DUO_OK; ws and ws_bytes are the
 *   workspace that call used (ws_bytes >= 256).
 */
duo_status duo_hessian_status(const void* ws, size_t ws_bytes, void* stream);

/*
 * duo_residual_term - stage 1, residual part only (Sec. 4.3: G = dX Xh^T,
 *   a = diag(dX dX^T)).  Same arguments and accumulation as duo_hessian_accum
 *   without H; X_src = NULL means X_src = X_dense (single-layer case).
 */
duo_status duo_residual_term(const void* X_dense, const void* X_src, int32_t x_dtype, int64_t m,
                             int64_t k, int64_t ldx, duo_act_rule rule, float* G, int64_t ldg,
                             int32_t g_part, float* a, void* ws, size_t ws_bytes, void* stream);

/*
 * duo_chol_inv - stage 2 (Sec. 4.3 Hessian synchronisation; Algorithm 1
 *   "Inverse_Cholesky"; App. A.2).
 *   H_inout  k x k fp32, ldh, symmetric (both triangles read as written by
 *            duo_hessian_accum; only the upper triangle is used).  On return
 *            it holds L: lower triangular with a positive diagonal and
 *            L L^T = (H + lambda I)^-1, lambda = damp_ratio * mean(diag H);
 *            the strictly upper triangle is set to 0.
 *   info     host pointer or NULL.  NULL: fully asynchronous, device-side
 *            failures are not reported.  Non-NULL: the call waits for the
 *            stream, fills *info and returns its status (DUO_ERR_NOT_PD when a
 *            pivot was not positive, DUO_ERR_NONFINITE when mean(diag H) is
 *            not finite or not positive).
 *   Workspace: DUO_OP_CHOL_INV with the same k.
 */
duo_status duo_chol_inv(float* H_inout, int64_t k, int64_t ldh, double damp_ratio,
                        duo_chol_info* info, void* ws, size_t ws_bytes, void* stream);

/*
 * duo_score_terms - stage 3 precompute (Eq. 7; App. A.3-A.4; Algorithm 1
 *   lines Q, U, a, b, c, D).
 *   L (ldl, strictly upper triangle zero), G (ldg; only its upper triangle,
 *   diagonal included, is read), a (k) -> D (k x k, ldd)
 *   and fac (k):  Q = G L, U = strict upper(Q), b = diag(U U^T),
 *   c = diag(Q) / diag(L), D = U L^T (strictly upper; its lower triangle and
 *   diagonal are written as 0 inside the diagonal 128 x 128 tiles and are not
 *   written elsewhere), fac = 1/diag(L)^2 + a - b + 2c.  The score of weight
 *   W[r][p] is S = W[r][p]^2 * fac[p].
 *   Workspace: DUO_OP_SCORE_TERMS with the same k.
 */
duo_status duo_score_terms(const float* L, int64_t ldl, const float* G, int64_t ldg, const float* a,
                           int64_t k, float* D, int64_t ldd, float* fac, void* ws, size_t ws_bytes,
                           void* stream);

/*
 * Options of the sweep (duo_sweep, duo_prune_layer).  A NULL pointer means
 * all fields 0.
 *   nm_n     0: the unstructured block mask (w_sparsity).  1..4: the N:4
 *            variant (App. B: mask selection and pruning over every group of 4
 *            consecutive columns): in each row, nm_n of every group of 4
 *            columns are pruned, those with the smallest (S, column) when the
 *            sweep reaches the group's first column (S from the values at that
 *            moment); w_sparsity is then not used (still range-checked).
 *            Needs k % 4 == 0 and block % 4 == 0.
 *   q_bits   0: no quantisation.  2..8: joint pruning and round-to-nearest
 *            quantisation (Table 4: uniform integer, channel-wise, in groups):
 *            when the sweep reaches a group of q_group columns, every row's
 *            grid is fixed from the group's current values: range
 *            [min(0, min w), max(0, max w)] ([-1, 1] if empty), step
 *            s = range / (2^q_bits - 1), zero code z = rint(-min / s).  A kept
 *            weight becomes s * (clamp(rint(w / s) + z, 0, 2^q_bits - 1) - z)
 *            (its value is exactly that fp32 product), a pruned one 0, and the
 *            later columns compensate both errors.
 *   q_group  16, 32, 64 or 128 columns per grid, dividing block.
 *   q_scale_out, q_zero_out  NULL or n x ceil(k / q_group) fp32 each: s and z
 *            per row and group (row-major), so that the integer code of a kept
 *            weight is rint(W_out / s) + z.
 */
typedef struct {
  int32_t nm_n;
  int32_t q_bits;
  int32_t q_group;
  float* q_scale_out;
  float* q_zero_out;
  int32_t residual_form;
} duo_sweep_opts;

/*
 * residual_form (duo_prune_layer only; duo_sweep, given D, accepts AUTO and
 * D): how the residual term of Algorithm 1's updates (W0 D, D = U L^T) is
 * carried.  Both forms give the same weights up to fp32 rounding order.
 *   DUO_FORM_D  D is formed (k^3 / 3 multiply-adds) and the lazy update is one
 *               product with the two terms E L^T and W0 D.
 *   DUO_FORM_Y  no D: the sweep carries Y = W0 U (W0: the values the columns
 *               had when processed) beside W, since W0 D = Y L^T with the
 *               terms of each column's own block added at the block's start;
 *               two lazy products (W += (Y - E) L^T, Y += W0 U) of the same
 *               total size.  Uses the workspace's D space for Y.  With
 *               q_bits only if q_group == block (grids fixed at a block's
 *               first column), else DUO_ERR_UNSUPPORTED.
 *   DUO_FORM_AUTO  Y when k >= 6144 and the Y form applies, else D.
 */
enum { DUO_FORM_AUTO = 0, DUO_FORM_D = 1, DUO_FORM_Y = 2 };

/*
 * duo_sweep - stage 3 sweep (Algorithm 1 outer/inner loops, lazy updates).
 *   W        n x k, ldw, w_dtype: dense weights (not modified).
 *   L, D     from duo_chol_inv / duo_score_terms; fac from duo_score_terms.
 *   w_sparsity  p^w in [0, 1].  Blocks are columns [j0, j0+B_b), B_b =
 *            min(block, k - j0); blocks 0..b hold floor(p^w*n*(j0+B_b) + 0.5)
 *            zeros in total.  Within a block the weights with the smallest key
 *            (S, column, row) are pruned.
 *   opts     NULL (defaults: unstructured mask, no quantisation) or the
 *            options of duo_sweep_opts below.
 *   The correction term of the lazy batch update uses each column's value at
 *   the moment it is processed (before pruning), so the blocked sweep equals
 *   the column-by-column sweep.
 *   mask_in  NULL, or an n x ceil(k/32) bit mask (1 = keep) that replaces the
 *            selection (forced-mask mode; counts are then not enforced).
 *   W_out    n x k fp32, row stride k: the pruned, compensated weights.
 *   W_out_lowp  NULL or n x k (row stride k) in w_dtype (round to nearest even).
 *   mask_out NULL or n x ceil(k/32) uint32 words, 1 = kept.
 *   block_scores_out  NULL or n x k fp32: each weight's score S at the time
 *            its block (N:4: its group) was selected.
 *   Workspace: DUO_OP_SWEEP with the same n, k, block.
 */
duo_status duo_sweep(const void* W, int32_t w_dtype, int64_t n, int64_t k, int64_t ldw,
                     const float* L, int64_t ldl, const float* D, int64_t ldd, const float* fac,
                     double w_sparsity, const duo_sweep_opts* opts, int32_t block, const uint32_t* mask_in,
                     float* W_out,
                     void* W_out_lowp, uint32_t* mask_out, float* block_scores_out, void* ws,
                     size_t ws_bytes, void* stream);

/*
 * act_order (App. B, calibration settings: the weight columns are processed
 * in the order of decreasing Hessian diagonal; off in Algorithm 1 as printed).
 * A layer is pruned with act_order by running the stages on its channels in
 * that order: H and G permuted on both sides, a, the columns of W and of a
 * forced mask permuted, then W_out, W_out_lowp and mask_out permuted back.
 *
 * duo_act_order - the order.
 *   hdiag    k doubles from duo_hessian_accum.
 *   perm     k int32: perm[i] = the channel processed i-th (decreasing
 *            hdiag, equal values in channel order; NaN and +inf first).
 *   inv_perm NULL or k int32: inv_perm[perm[i]] = i.
 */
duo_status duo_act_order(const double* hdiag, int64_t k, int32_t* perm, int32_t* inv_perm, void* stream);

/*
 * duo_permute - gather: dst[i][j] = src[r][c], r = row_idx ? row_idx[i] : i,
 *   c = col_idx ? col_idx[j] : j, for i < rows, j < cols.
 *   src      src_rows x src_cols, row stride lds, dtype DUO_F32 or DUO_BF16.
 *   row_idx  NULL or rows int32; col_idx NULL or cols int32.  An index
 *            outside the source writes 0 (no access outside src is made).
 *   dst      rows x cols, row stride ldd, same dtype; must not alias src.
 *   rows <= 65535.
 */
duo_status duo_permute(const void* src, int32_t dtype, int64_t src_rows, int64_t src_cols, int64_t lds,
                       const int32_t* row_idx, const int32_t* col_idx, int64_t rows, int64_t cols, void* dst,
                       int64_t ldd, void* stream);

/*
 * duo_permute_mask - column gather of a bit-packed mask (n x ceil(k/32)
 *   uint32 words, bit c of word c/32 = column c): bit j of dst row r = bit
 *   col_idx[j] of src row r (0 for an index outside [0, k)).  col_idx holds
 *   k int32; dst must not alias src.
 */
duo_status duo_permute_mask(const uint32_t* src, int64_t n, int64_t k, const int32_t* col_idx, uint32_t* dst,
                            void* stream);

/*
 * duo_prune_layer - stage 3 in one call: duo_score_terms then duo_sweep, with
 *   D and fac kept in the workspace.  Arguments as in those two calls.
 *   Workspace: DUO_OP_PRUNE_LAYER with the same n, k, block.
 */
duo_status duo_prune_layer(const void* W, int32_t w_dtype, int64_t n, int64_t k, int64_t ldw,
                           const float* L, int64_t ldl, const float* G, int64_t ldg, const float* a,
                           double w_sparsity, const duo_sweep_opts* opts, int32_t block, const uint32_t* mask_in,
                           float* W_out,
                           void* W_out_lowp, uint32_t* mask_out, float* block_scores_out, void* ws,
                           size_t ws_bytes, void* stream);

/*
 * Kernel timing for benchmarks (not part of the method).  With profiling on,
 * every launch of the tracked kernels is bracketed by HIP events on the
 * stream it runs on.  duo_profile_read waits for the recorded events and
 * returns the summed time (milliseconds) and the number of launches since the
 * last read, then resets them.  A launch whose events could not be recorded
 * is left out of both; DUO_ERR_HIP if a recorded pair could not be read
 * (the others are still summed).  Single-threaded use only.
 */
enum {
  DUO_PROF_GRAM = 0,     /* stage 1: MFMA Gram kernel (H, G)                   */
  DUO_PROF_HESSIAN = 1,  /* stage 1: whole duo_hessian_accum call              */
  DUO_PROF_CHOL = 2,     /* stage 2: whole duo_chol_inv call                   */
  DUO_PROF_SCORE = 3,    /* stage 3: Q, fac, D                                 */
  DUO_PROF_SWEEP = 4,    /* stage 3: whole sweep (select, in-block, lazy)      */
  DUO_PROF_INBLOCK = 5,  /* stage 3: in-block kernel, one launch per block     */
  DUO_PROF_TRAIL = 6,    /* stage 3: lazy trailing-update GEMM, one per block  */
  DUO_PROF_SELECT = 7,   /* stage 3: mask selection passes of one block        */
  DUO_PROF_DECODE = 8,   /* decode: the dual-sparse GEMV kernel                */
  DUO_PROF_COUNT = 9
};
duo_status duo_profile_enable(int32_t on);
duo_status duo_profile_read(int32_t kernel, double* total_ms, int64_t* launches);

/*
 * Dual-sparse decode (Preliminaries "Activation Sparsity", Sec. 4.1): at
 * decoding time a pruned linear layer computes y = W (x * m^x), the sum over
 * the input channels i whose activation survives of W[:, i] x_i, so only
 * those weight columns are read, each stored compressed (the paper leaves this
 * kernel to future work; the storage is this library's own):
 *   col_ptr    k + 1 int64: channel i's kept values are values[col_ptr[i] ..
 *              col_ptr[i + 1]);
 *   maskT      k x ceil(n/32) uint32, channel-major: bit r % 32 of word r / 32
 *              of channel i set when W[r][i] is kept;
 *   chunk_off  k x ceil(n/256) uint16: kept weights of channel i in rows
 *              [0, 256 c);
 *   values     col_ptr[k] bf16 (bit patterns): each channel's kept weights in
 *              row order; the allocation holds col_ptr[k] + 8 elements and is
 *              16-byte aligned (the GEMV reads aligned 16-byte windows).
 * Limits: n <= 65535 (duo_dsc_gemv: n <= 32768), k <= 32768.  Workspace:
 * duo_dsc_workspace_size(n, k).
 *
 * duo_dsc_layout - col_ptr, maskT and chunk_off from a pruned layer's mask
 *   (n x ceil(k/32) words as duo_sweep writes it).  The caller then reads
 *   col_ptr[k] (the number of kept weights) to size values.
 * duo_dsc_pack - values from the pruned weights W (n x k, ldw, fp32 rounded to
 *   nearest even bf16, or bf16 copied) and the layout.
 * duo_dsc_gemv - one decode step: x (k, x_dtype) is sparsified with `rule`
 *   (the calibration rule: the smallest (|x|, channel) entries zeroed), then
 *   y (n fp32) = sum over kept channels of W[:, i] x_i, products of bf16
 *   weights and activations in fp32, summed in a fixed order (deterministic).
 */
size_t duo_dsc_workspace_size(int64_t n, int64_t k);
duo_status duo_dsc_layout(const uint32_t* mask, int64_t n, int64_t k, int64_t* col_ptr, uint32_t* maskT,
                          uint16_t* chunk_off, void* ws, size_t ws_bytes, void* stream);
duo_status duo_dsc_pack(const void* W, int32_t w_dtype, int64_t n, int64_t k, int64_t ldw, const int64_t* col_ptr,
                        const uint32_t* maskT, const uint16_t* chunk_off, uint16_t* values, void* stream);
duo_status duo_dsc_gemv(const void* x, int32_t x_dtype, int64_t n, int64_t k, duo_act_rule rule,
                        const int64_t* col_ptr, const uint32_t* maskT, const uint16_t* chunk_off,
                        const uint16_t* values, float* y, void* ws, size_t ws_bytes, void* stream);

/*
 * duo_dsc_gemv_noalloc - duo_dsc_gemv for callers that cannot allocate device
 *   memory or pass a workspace (code under HIP graph capture, tight serving
 *   loops, harnesses that forbid allocation).  Same arguments, kernels and
 *   results as duo_dsc_gemv, bit for bit, without ws / ws_bytes: the partial
 *   rows live in a 2 MiB array inside the library, one per GPU, held until
 *   the process ends; its device address is looked up on the first call on a
 *   device (with that device current).  The call allocates nothing and calls
 *   no allocating routine.  Limits: n <= 32768 and k <= 32768
 *   (DUO_ERR_UNSUPPORTED beyond; the partial rows never exceed 256 x 2048
 *   floats inside those limits).  Every call on a GPU uses that GPU's one
 *   array: calls that overlap on one GPU (other streams, other threads) race
 *   and give undefined results; calls ordered on one stream are safe.  The
 *   array needs no clearing: each call writes every partial it reads.
 */
duo_status duo_dsc_gemv_noalloc(const void* x, int32_t x_dtype, int64_t n, int64_t k, duo_act_rule rule,
                                const int64_t* col_ptr, const uint32_t* maskT, const uint16_t* chunk_off,
                                const uint16_t* values, float* y, void* stream);

/*
 * Decoder-block harness.  When a whole decoder block is pruned group by group,
 * each group's solver input comes from two streams (the multi-layer case of
 * Sec. 4.2): the dense model's activations (X-tilde, dense weights, no
 * activation sparsity) and the pruned model's own activations (pruned
 * weights, every linear input sparsified per token with the rule above).
 * These calls carry both streams through a LLaMA-style block (Sec. 5 models:
 * RMSNorm, rotary attention, SiLU-gated MLP).  Activations are bf16,
 * token-major (row t = token t), arithmetic fp32, device pointers, stream
 * ordered; argument errors return before anything is enqueued.
 */
enum {
  DUO_BOP_ACT_SPARSIFY = 0, /* duo_act_sparsify (uses m)                 */
  DUO_BOP_LINEAR = 1,       /* duo_linear (fixed size)                   */
  DUO_BOP_ATTENTION = 2     /* duo_attention (uses seq_len, heads)       */
};
/* Bytes of workspace a harness call needs (0 for a bad op or size). */
size_t duo_block_workspace_size(int32_t op, int64_t m, int64_t seq_len, int64_t heads);

/* duo_rmsnorm - Y[t] = X[t] / sqrt(mean_c X[t][c]^2 + eps) (unit gain).
 *   X, Y: m x d bf16 with row strides ldx, ldy >= d (Y may equal X). */
duo_status duo_rmsnorm(const void* X, int64_t m, int64_t d, int64_t ldx, double eps, void* Y, int64_t ldy,
                       void* stream);

/* duo_act_sparsify - Y = X-hat: X (m x k bf16, ldx) with the per-token rule
 *   of duo_act_rule applied (z = floor(p*k + 0.5) smallest (|x|, channel)
 *   entries of each token set to +0); Y is m x k bf16 (ldy), not aliasing X.
 *   The kept set is the one duo_hessian_accum uses.
 *   Workspace: DUO_BOP_ACT_SPARSIFY with the same m.  1 <= k <= 32768. */
duo_status duo_act_sparsify(const void* X, int64_t m, int64_t k, int64_t ldx, duo_act_rule rule, void* Y,
                            int64_t ldy, void* ws, size_t ws_bytes, void* stream);

/* duo_linear - Y = X W^T (+ R): X m x k (ldx), W n x k (ldw, a Linear's
 *   out x in weights), optional residual R m x n (ldr; NULL for none), Y m x n
 *   (ldy; may equal R).  bf16 in and out, fp32 accumulation, one rounding
 *   (of the fp32 sum plus R).  bf16 MFMA tiles of this library; rows that are
 *   not 16-byte aligned or k % 8 != 0 take a slower per-element path.  Needs
 *   no scratch memory: ws may be NULL (DUO_BOP_LINEAR is 0 bytes). */
duo_status duo_linear(const void* X, int64_t m, int64_t k, int64_t ldx, const void* W, int64_t n, int64_t ldw,
                      const void* R, int64_t ldr, void* Y, int64_t ldy, void* ws, size_t ws_bytes, void* stream);

/* duo_rope - in place rotary position embedding of X (m x heads*head_dim bf16,
 *   ldx): in every head the pair (i, i + head_dim/2) of token t is rotated by
 *   the angle (t mod seq_len) * theta^(-2i/head_dim) (angles in fp64). */
duo_status duo_rope(void* X, int64_t m, int64_t heads, int64_t head_dim, int64_t ldx, int64_t seq_len, double theta,
                    void* stream);

/* duo_attention - causal attention of nseq sequences of seq_len tokens:
 *   for each sequence and head h, O_h = softmax(Q_h K_h^T / sqrt(head_dim)
 *   with positions j > i masked) V_h, where Q_h is columns
 *   [h*head_dim, (h+1)*head_dim) of the sequence's rows of Q.  Q, K, V share
 *   the row stride ld; O has ldo.  Scores, row maxima and sums are fp32 (two
 *   passes over the key blocks), the normalised probabilities are rounded to
 *   bf16 before the product with V, and O is accumulated in fp32.  head_dim
 *   64 or 128, ld % 8 == 0 and 16-byte aligned Q, K, V (else
 *   DUO_ERR_UNSUPPORTED).  Needs no scratch memory: ws may be NULL
 *   (DUO_BOP_ATTENTION is 0 bytes). */
duo_status duo_attention(const void* Q, const void* K, const void* V, int64_t ld, int64_t nseq, int64_t seq_len,
                         int64_t heads, int64_t head_dim, void* O, int64_t ldo, void* ws, size_t ws_bytes,
                         void* stream);

/* duo_silu_mul - Y = SiLU(G) * U elementwise, SiLU(g) = g / (1 + exp(-g));
 *   G, U m x n bf16 with row stride ld, Y m x n (ldy). */
duo_status duo_silu_mul(const void* G, const void* U, int64_t m, int64_t n, int64_t ld, void* Y, int64_t ldy,
                        void* stream);

#ifdef __cplusplus
}
#endif

#endif /* DUO_H */
