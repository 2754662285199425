// Stage 2 of the DuoGPT layer solver on gfx950: damping and the lower
// Cholesky factor of the inverse Hessian (paper Sec. 4.3, Algorithm 1
// "Inverse_Cholesky"; App. A.2).
//
// Route.  If (H + lambda I) = V V^T with V upper triangular (a Cholesky
// factorisation that eliminates from the last column backwards), then
// (H + lambda I)^-1 = V^-T V^-1, so L = V^-T is lower triangular with
// L L^T = (H + lambda I)^-1.  This needs one factorisation (k^3/3) and one
// triangular inverse (k^3/3) instead of an explicit inverse followed by a
// second factorisation.
//
//   1. damp: lambda = damp * mean(diag H) (fixed-order double sum), H += lambda I.
//   2. blocked factorisation from the bottom-right, 128 columns at a time:
//      diagonal block V_bb and its inverse in one workgroup (LDS), panel
//      V[0:r0, b] = H[0:r0, b] V_bb^-T and symmetric update of the leading
//      block, both on the fp32 MFMA GEMM.  V lives in the upper triangle.
//   3. N = V^-1 by recursive halving: N12 = -N11 V12 N22 (two GEMMs per node).
//   4. L = N^T written to the lower triangle; the strict upper set to zero.
#include <hip/hip_runtime.h>

#include <utility>

#include "internal.h"

namespace duo {

namespace {

__global__ __launch_bounds__(256) void damp_kernel(float* H, int64_t ldh, int k, double damp, CholStatus* st) {
  __shared__ double red[256];
  double s = 0.0;
  for (int i = threadIdx.x; i < k; i += 256) s += (double)H[(int64_t)i * ldh + i];
  red[threadIdx.x] = s;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  const double mean = red[0] / (double)k;
  const double lam = damp * mean;
  if (threadIdx.x == 0) {
    st->lambda = lam;
    st->fail = -1;
    st->status = DUO_OK;
    if (!(mean == mean) || mean > 1e300 || mean < -1e300)
      st->status = DUO_ERR_NONFINITE;
    else if (!(mean > 0.0))
      st->status = DUO_ERR_NOT_PD;
  }
  const float lf = (float)lam;
  for (int i = threadIdx.x; i < k; i += 256) H[(int64_t)i * ldh + i] += lf;
}

// Factor the s x s diagonal block at (r0, r0), s <= 128, read from its upper
// triangle: A = V V^T with V upper, eliminating the last column first, and
// return N = V^-1 (upper; zeros below the diagonal) in `vinv` (128 x 128,
// row-major).  V itself is not needed by the callers and is not stored.
//
// 192 threads; thread (h, q) keeps rows 64h..64h+63 of column q in registers
// (h = 0 for q < 64; h = 0, 1 for q >= 64: the lower-left quadrant is never
// needed).  Step c (c = s-1 .. 0) broadcasts column c of the working matrix
// and row c of N through LDS (one barrier per step):
//   columns q < c:  A[r][q] -= A[r][c] A[q][c] / A[c][c]       (factorisation)
//   column  q = c:  N[r][c]  = -A[r][c] / A[c][c], N[c][c] = 1 / sqrt(A[c][c])
//   columns q > c:  N[c][q] /= V[c][c]; N[r][q] -= V[r][c] N[c][q]  (r < c)
// The last two are back substitution of V N = I, driven by the same column c.
// Padding rows/columns beyond s are an identity block.
struct DiagCtx {
  float* colbuf;  // [2][128]
  float* rowbuf;  // [2][128]
  float* pivbuf;  // [2]
  int tid, h, q, hh, buf;
  int fail;  // first column (from the bottom) with a non-positive pivot, or -1
};

// One elimination step for column c = 64*hh + I0 (I0 a compile-time constant so
// that every register index below is static).
template <int I0>
__device__ __forceinline__ void diag_step(float (&x)[64], DiagCtx& d) {
  const int hh = d.hh, h = d.h, q = d.q;
  const int c = 64 * hh + I0;
  float* colbuf = d.colbuf + d.buf * kTile;
  float* rowbuf = d.rowbuf + d.buf * kTile;
  if (q == c) {
    float4* cb = (float4*)&colbuf[64 * h];
    if (h < hh) {
#pragma unroll
      for (int i = 0; i < 64; i += 4) cb[i / 4] = make_float4(x[i], x[i + 1], x[i + 2], x[i + 3]);
    } else if (h > hh) {
#pragma unroll
      for (int i = 0; i < 64; i += 4) cb[i / 4] = make_float4(0.f, 0.f, 0.f, 0.f);
    } else {
#pragma unroll
      for (int i = 0; i < 64; ++i) colbuf[64 * h + i] = i < I0 ? x[i] : 0.f;
      d.pivbuf[d.buf] = x[I0];
    }
  }
  if (h == hh && q > c) rowbuf[q] = x[I0];
  __syncthreads();
  const float piv = d.pivbuf[d.buf];
  if (!(piv > 0.f) && d.fail < 0) d.fail = c;  // uniform: every thread sees the same pivot
  const float inv = 1.0f / sqrtf(piv);
  const float inv2 = inv * inv;
  if (q == c) {
    // column c of N: N[r][c] = -A[r][c] / A[c][c] for r < c (x[i] holds A[r][c])
    if (h < hh) {
#pragma unroll
      for (int i = 0; i < 64; ++i) x[i] = -x[i] * inv2;
    } else if (h == hh) {
#pragma unroll
      for (int i = 0; i < I0; ++i) x[i] = -x[i] * inv2;
    }
  } else if (64 * h < c) {
    // columns q < c (factorisation) and q > c (back substitution) share one
    // FMA stream; colbuf rows >= c are zero
    const float coef = q < c ? inv2 * colbuf[q] : inv2 * rowbuf[q];
    const float4* cb = (const float4*)&colbuf[64 * h];
#pragma unroll
    for (int i = 0; i < 64; i += 4) {
      const float4 v = cb[i / 4];
      x[i] = fmaf(-v.x, coef, x[i]);
      x[i + 1] = fmaf(-v.y, coef, x[i + 1]);
      x[i + 2] = fmaf(-v.z, coef, x[i + 2]);
      x[i + 3] = fmaf(-v.w, coef, x[i + 3]);
    }
  }
  if (h == hh) {
    if (q > c) x[I0] = x[I0] * inv;
    if (q == c) x[I0] = inv;
  }
  d.buf ^= 1;
}

template <int... Is>
__device__ __forceinline__ void diag_steps(float (&x)[64], DiagCtx& d, std::integer_sequence<int, Is...>) {
  (diag_step<63 - Is>(x, d), ...);  // columns 64*hh + 63 down to 64*hh
}

__global__ __launch_bounds__(192) void diag_factor_kernel(const float* H, int64_t ldh, int r0, int s, float* vinv,
                                                          CholStatus* st) {
  __shared__ __attribute__((aligned(16))) float colbuf[2][kTile];
  __shared__ float rowbuf[2][kTile];
  __shared__ float pivbuf[2];
  const int tid = threadIdx.x;
  const int w = tid >> 6, lane = tid & 63;
  const int h = w == 2 ? 1 : 0;
  const int q = w == 0 ? lane : 64 + lane;
  float x[64];
#pragma unroll
  for (int i = 0; i < 64; ++i) {
    const int r = 64 * h + i;
    float v = 0.f;
    if (r < s && q < s)
      v = r <= q ? H[(int64_t)(r0 + r) * ldh + r0 + q] : H[(int64_t)(r0 + q) * ldh + r0 + r];
    else if (r == q)
      v = 1.f;
    x[i] = v;
  }
  DiagCtx d{&colbuf[0][0], &rowbuf[0][0], pivbuf, tid, h, q, 1, 0, -1};
  diag_steps(x, d, std::make_integer_sequence<int, 64>{});
  d.hh = 0;
  diag_steps(x, d, std::make_integer_sequence<int, 64>{});
  if (tid == 0 && d.fail >= 0 && d.fail < s && st->status == DUO_OK) {
    st->status = DUO_ERR_NOT_PD;
    st->fail = r0 + d.fail;
  }
  // N (upper, rows <= q) to vinv; everything else 0
#pragma unroll
  for (int i = 0; i < 64; ++i) {
    const int r = 64 * h + i;
    vinv[r * kTile + q] = (r <= q && r < s && q < s) ? x[i] : 0.f;
  }
  for (int e = tid; e < 64 * 64; e += 192) vinv[(64 + e / 64) * kTile + (e % 64)] = 0.f;  // lower-left quadrant
}

// Copy the inverted diagonal blocks into place (full 128 x 128 incl. zeros).
__global__ __launch_bounds__(256) void place_diag_kernel(float* H, int64_t ldh, int k, const float* vinv) {
  const int b = blockIdx.x;
  const float* src = vinv + (int64_t)b * kTile * kTile;
  for (int e = threadIdx.x; e < kTile * kTile; e += 256) {
    const int r = b * kTile + e / kTile, c = b * kTile + e % kTile;
    if (r < k && c < k) H[(int64_t)r * ldh + c] = src[e];
  }
}

// L = N^T: tile pair (ti <= tj): upper tile (ti, tj) -> lower tile (tj, ti); upper zeroed.
__global__ __launch_bounds__(256) void transpose_upper_kernel(float* H, int64_t ldh, int k) {
  __shared__ float t[64][65];
  int ti, tj;
  tri_pair(blockIdx.x, &tj, &ti);  // ti <= tj, tiles of 64
  const int i0 = ti * 64, j0 = tj * 64;
  for (int e = threadIdx.x; e < 64 * 64; e += 256) {
    const int r = e / 64, c = e % 64;
    const int gi = i0 + r, gj = j0 + c;
    float v = 0.f;
    if (gi < k && gj < k && gi <= gj) v = H[(int64_t)gi * ldh + gj];
    t[r][c] = v;
  }
  __syncthreads();
  for (int e = threadIdx.x; e < 64 * 64; e += 256) {
    const int r = e / 64, c = e % 64;
    // destination (j0 + r, i0 + c) takes source (i0 + c, j0 + r)
    const int gi = j0 + r, gj = i0 + c;
    if (gi < k && gj < k) {
      if (gi >= gj)
        H[(int64_t)gi * ldh + gj] = t[c][r];
      else
        H[(int64_t)gi * ldh + gj] = 0.f;
    }
    // zero the strictly upper source entries of off-diagonal tiles
    const int si = i0 + r, sj = j0 + c;
    if (ti != tj && si < k && sj < k) H[(int64_t)si * ldh + sj] = 0.f;
  }
}

struct CholWs {
  CholStatus* st;
  float* vinv;
  float* X;
  size_t bytes;
};

CholWs carve(void* ws, int64_t k) {
  const int64_t T = cdiv(k, kTile);
  const int64_t half = cdiv(T, 2) * kTile;
  Carver c(ws);
  CholWs w;
  w.st = c.take<CholStatus>(1);
  w.vinv = c.take<float>((size_t)T * kTile * kTile);
  w.X = c.take<float>((size_t)half * half);
  w.bytes = c.off;
  return w;
}

// N = V^-1 by bottom-up merging (units of 128 columns; the diagonal blocks
// already hold their inverses).  At level L every node [lo, lo + 2^L) whose
// halves [lo, mid) and [mid, hi) are inverted becomes
//   N12 = -N11 V12 N22,  as X = V12 N22 then N12 = -N11 X.
// All complete nodes of a level share one batched launch per product; a node
// containing the ragged last block gets its own.
duo_status merge_nodes(float* H, int64_t ldh, int64_t k, int64_t span, int64_t half, int64_t q0, int nodes,
                       float* X, hipStream_t s) {
  const int64_t r_lo = q0 * span * kTile, r_mid = r_lo + half * kTile;
  const int64_t r_hi = r_lo + span * kTile < k ? r_lo + span * kTile : k;
  const int m1 = (int)(r_mid - r_lo), m2 = (int)(r_hi - r_mid);
  const int64_t diag_step = span * kTile * (ldh + 1);  // next node along the diagonal
  // X = V12 N22 (N22 upper: for output column tile j only l < j-tile end)
  GemmDesc a{};
  a.M = m1;
  a.N = m2;
  a.C = X;
  a.ldc = m2;
  a.beta = 0.f;
  a.tri = TRI_ALL;
  a.nterms = 1;
  a.t[0] = GemmTerm{H + r_lo * ldh + r_mid, ldh, 1, H + r_mid * ldh + r_mid, ldh, 1, m2, 1.f, KLO_ZERO, KHI_COL};
  a.batch = nodes;
  a.sC = (int64_t)m1 * m2;
  a.sA[0] = diag_step;
  a.sB[0] = diag_step;
  duo_status st = gemm_f32(a, s);
  if (st != DUO_OK) return st;
  // V12 <- -N11 X (N11 upper: for output row tile i only l >= i-tile start)
  GemmDesc b{};
  b.M = m1;
  b.N = m2;
  b.C = H + r_lo * ldh + r_mid;
  b.ldc = ldh;
  b.beta = 0.f;
  b.tri = TRI_ALL;
  b.nterms = 1;
  b.t[0] = GemmTerm{H + r_lo * ldh + r_lo, ldh, 1, X, m2, 1, m1, -1.f, KLO_ROW, KHI_FULL};
  b.batch = nodes;
  b.sC = diag_step;
  b.sA[0] = diag_step;
  b.sB[0] = (int64_t)m1 * m2;
  return gemm_f32(b, s);
}

duo_status trinv(float* H, int64_t ldh, int64_t k, int T, float* X, hipStream_t s) {
  for (int64_t half = 1; half < T; half *= 2) {
    const int64_t span = 2 * half;
    const int64_t full = k / (span * kTile);  // nodes with both halves complete (no ragged block)
    if (full > 0) {
      duo_status st = merge_nodes(H, ldh, k, span, half, 0, (int)full, X, s);
      if (st != DUO_OK) return st;
    }
    if (full * span + half < T) {  // the node holding the tail
      duo_status st = merge_nodes(H, ldh, k, span, half, full, 1, X, s);
      if (st != DUO_OK) return st;
    }
  }
  return DUO_OK;
}

}  // namespace

size_t chol_ws_bytes(int64_t k) { return carve(nullptr, k).bytes; }

duo_status chol_run(float* H, int64_t k, int64_t ldh, double damp, void* ws, hipStream_t s, CholStatus** status_dev) {
  const CholWs w = carve(ws, k);
  *status_dev = w.st;
  const int T = (int)cdiv(k, kTile);
  hipLaunchKernelGGL(damp_kernel, dim3(1), dim3(256), 0, s, H, ldh, (int)k, damp, w.st);
  DUO_LAUNCH_CHECK();
  for (int b = T - 1; b >= 0; --b) {
    const int r0 = b * kTile;
    const int sz = (int)((int64_t)r0 + kTile <= k ? kTile : k - r0);
    hipLaunchKernelGGL(diag_factor_kernel, dim3(1), dim3(192), 0, s, (const float*)H, ldh, r0, sz,
                       w.vinv + (int64_t)b * kTile * kTile, w.st);
    DUO_LAUNCH_CHECK();
    if (r0 == 0) break;
    // panel: H[0:r0, r0:r0+sz] <- H[0:r0, r0:r0+sz] * Vinv_bb^T   (in place: one tile column)
    GemmDesc p{};
    p.M = r0;
    p.N = sz;
    p.C = H + r0;
    p.ldc = ldh;
    p.beta = 0.f;
    p.tri = TRI_ALL;
    p.nterms = 1;
    p.t[0] = GemmTerm{H + r0, ldh, 1, w.vinv + (int64_t)b * kTile * kTile, kTile, 0, sz, 1.f, KLO_ZERO, KHI_FULL};
    duo_status st = gemm_f32(p, s);
    if (st != DUO_OK) return st;
    // leading block (upper tiles): H[0:r0, 0:r0] -= P P^T
    GemmDesc u{};
    u.M = r0;
    u.N = r0;
    u.C = H;
    u.ldc = ldh;
    u.beta = 1.f;
    u.tri = TRI_UPPER;
    u.nterms = 1;
    u.t[0] = GemmTerm{H + r0, ldh, 1, H + r0, ldh, 0, sz, -1.f, KLO_ZERO, KHI_FULL};
    st = gemm_f32(u, s);
    if (st != DUO_OK) return st;
  }
  hipLaunchKernelGGL(place_diag_kernel, dim3(T), dim3(256), 0, s, H, ldh, (int)k, (const float*)w.vinv);
  DUO_LAUNCH_CHECK();
  duo_status st = trinv(H, ldh, k, T, w.X, s);
  if (st != DUO_OK) return st;
  const int T64 = (int)cdiv(k, 64);
  hipLaunchKernelGGL(transpose_upper_kernel, dim3(T64 * (T64 + 1) / 2), dim3(256), 0, s, H, ldh, (int)k);
  DUO_LAUNCH_CHECK();
  return DUO_OK;
}

}  // namespace duo
