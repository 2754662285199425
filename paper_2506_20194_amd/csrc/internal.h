// Declarations shared between the translation units of the library.
#pragma once

#include "common.h"

namespace duo {

// ---- optional event timing (profile.hip) ----
void prof_begin(int id, hipStream_t s);
void prof_end(int id, hipStream_t s);

// ---- stage 1 (hessian.hip) ----
int64_t hessian_chunk_tokens(int64_t m, int64_t k);
int gram_split(int64_t ntiles, int64_t ch, int64_t kp);
size_t hessian_ws_bytes(int64_t m, int64_t k);
duo_status hessian_run(const void* Xs, const void* Xd, int32_t dtype, int64_t m, int64_t k, int64_t ldx, int z,
                       float* H, int64_t ldh, float* G, int64_t ldg, int g_full, float* a, double* hdiag, void* ws,
                       bool want_h, hipStream_t s);
// DUO_ERR_NONFINITE when the last stage-1 call on this workspace met a NaN or
// inf input (waits for the stream), else DUO_OK.
duo_status hessian_status_run(const void* ws, hipStream_t s);
// DUO_OK when the current device is a gfx950 (cached per device), else
// DUO_ERR_NO_DEVICE (or DUO_ERR_UNSUPPORTED for a device index >= 64).
duo_status device_ok();
// raise a kernel's dynamic LDS limit on the current device (cached)
duo_status set_max_lds(const void* fn, size_t bytes);

// Per-token threshold keys of the (|x|, channel) rule: entry c of token t is
// kept iff ((magnitude bits of x) << 32 | c) > thr[t]; z entries are zeroed.
duo_status act_threshold_run(const void* X, int32_t dtype, int64_t m, int64_t k, int64_t ldx, int z, int64_t* thr,
                             hipStream_t s);
duo_status act_mask_run(const void* X, int32_t dtype, int64_t m, int64_t k, int64_t ldx, int z, uint32_t* mask,
                        void* ws, hipStream_t s);

// ---- fp32 MFMA GEMM (gemm_f32.hip) ----
// C[i][j] = beta * C[i][j] + sum_terms alpha * sum_{l in range} A(i, l) B(l, j)
// over the tiles selected by `tri`.
enum { KLO_ZERO = 0, KLO_ROW = 1, KLO_COL = 2 };  // range start: 0 / tile-row start / tile-col start
enum { KHI_FULL = 0, KHI_ROW = 1, KHI_COL = 2 };  // range end: K / tile-row end / tile-col end
enum { TRI_ALL = 0, TRI_LOWER = 1, TRI_UPPER = 2 };

struct GemmTerm {
  const float* A;
  int64_t lda;
  int a_row;  // 1: A(i,l) = A[i*lda + l]; 0: A(i,l) = A[l*lda + i]
  const float* B;
  int64_t ldb;
  int b_row;  // 1: B(l,j) = B[l*ldb + j]; 0: B(l,j) = B[j*ldb + l]
  int K;
  float alpha;
  int klo, khi;
};

struct GemmDesc {
  int M, N;
  float* C;
  int64_t ldc;
  float beta;
  int tri;
  int nterms;
  GemmTerm t[2];
  // batched launches: problem z (blockIdx.y) uses C + z*sC, A_i + z*sA[i], B_i + z*sB[i]
  int batch;  // 0 or 1: a single problem
  int64_t sC, sA[2], sB[2];
  // tile order: ORDER_XCD gives each XCD a contiguous range of tiles (operand
  // reuse in its L2; for tiles of equal cost); ORDER_PLAIN deals tiles to the
  // XCDs round-robin in enumeration order (for upper tiles: by column, i.e.
  // the longest first when the K range shrinks with the column; for all tiles
  // with a K range that grows with the column: by column from the last, else
  // by row); ORDER_DIAG
  // (upper tiles only) deals them by decreasing distance from the diagonal
  // (the longest first when the K range grows with that distance)
  int order;
  // C is the first term's A operand, overwritten in place (N <= 128): every
  // workgroup must then own whole rows of C, so the launch uses 128-wide
  // tiles (a quarter tile would overwrite columns its row neighbour still reads)
  int inplace;
  // two independent one-term products in one launch (two terms, batch 0):
  // C = beta C + alpha0 A0 B0 and C2 = beta C2 + alpha1 A1 B1, C2 with the
  // row stride ldc (for two products that would otherwise be two launches)
  int dual;
  float* C2;
};
enum { ORDER_XCD = 0, ORDER_PLAIN = 1, ORDER_DIAG = 2 };

duo_status gemm_f32(const GemmDesc& d, hipStream_t s);

// ---- stage 2 (chol.hip) ----
struct CholStatus {
  double lambda;
  long long fail;
  int status;
  int pad;
};
size_t chol_ws_bytes(int64_t k);
duo_status chol_run(float* H, int64_t k, int64_t ldh, double damp, void* ws, hipStream_t s,
                    CholStatus** status_dev);

// ---- stage 3 (score.hip, sweep.hip) ----
size_t score_ws_bytes(int64_t k);
// D = NULL: Q, fac only (no D = U L^T); U (the upper 128-tiles of Q with the
// entries on and below the diagonal zeroed, k x k, ld k) stays in the
// workspace, at score_u(ws, k).
duo_status score_run(const float* L, int64_t ldl, const float* G, int64_t ldg, const float* a, int64_t k,
                     float* D, int64_t ldd, float* fac, void* ws, hipStream_t s);
const float* score_u(const void* ws, int64_t k);

size_t sweep_ws_bytes(int64_t n, int64_t k, int B);
// Sweep options (validated by the caller).  nm_n > 0: the N:4 variant (nm_n
// of every 4 consecutive columns of a row pruned, chosen when the sweep reaches
// the group; p_w unused).  q_bits > 0: joint RTN quantisation with one grid per
// row and group of q_group columns (q_group in {16, 32, 64, 128}, dividing B);
// q_scale / q_zero (NULL or n x ceil(k / q_group)) receive the grids.
struct SweepOpts {
  int nm_n = 0;
  int q_bits = 0;
  int q_group = 0;
  float* q_scale = nullptr;
  float* q_zero = nullptr;
  int form = 0;  // DUO_FORM_*
};
// U != NULL: the Y form (no D; D ignored): U is the strictly upper part of Q
// (only entries U[i][j] with j > i are read, on 128-tiles at or above the
// diagonal) and Y an n x k fp32 scratch matrix; not with nm_n or q_bits.
duo_status sweep_run(const void* W, int32_t w_dtype, int64_t n, int64_t k, int64_t ldw, const float* L,
                     int64_t ldl, const float* D, int64_t ldd, const float* fac, double p_w, const SweepOpts& o, int B,
                     const uint32_t* mask_in, float* W_out, void* W_out_lowp, uint32_t* mask_out,
                     float* scores_out, void* ws, hipStream_t s, const float* U = nullptr, int64_t ldu = 0,
                     float* Y = nullptr);

}  // namespace duo
