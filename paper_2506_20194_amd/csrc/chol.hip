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
  // 16 diagonal loads per thread in flight at a time (clamped, masked)
  for (int i0 = 0; i0 < k; i0 += 256 * 16) {
    float v[16];
#pragma unroll
    for (int u = 0; u < 16; ++u) {
      const int i = min(i0 + 256 * u + (int)threadIdx.x, k - 1);
      v[u] = H[(int64_t)i * ldh + i];
    }
#pragma unroll
    for (int u = 0; u < 16; ++u)
      if (i0 + 256 * u + (int)threadIdx.x < k) s += (double)v[u];
  }
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
// triangle: A = V V^T with V upper, eliminating from the last column, and
// return N = V^-1 (upper; zeros below the diagonal) in `vinv` (128 x 128,
// row-major).  V itself is not needed by the callers and is not stored.
//
// The block is split into four 32-column leaves J = 3..0 (bottom-up, like the
// whole factorisation):
//   leaf     one wave factors A_JJ = V_JJ V_JJ^T and inverts it in the same
//            sweep (column c of the working matrix drives both the rank-1
//            update of the columns before it and the back substitution
//            V N = I of the columns after it); column c reaches the wave's
//            lanes as scalars read from its lane, so the 32 steps need no
//            LDS round trip and no workgroup barrier;
//   panel    V_IJ = A_IJ N_JJ^T for the leaves I < J, and beside it the
//            finished inverse blocks N_JK = -N_JJ T_JK for K > J;
//   update   A_II' -= V_IJ V_I'J^T for I <= I' < J, and beside it
//            T_IK += V_IJ N_JK for I < J <= K; wave 0 takes the update of
//            the next leaf's own block and then factors that leaf while the
//            other three waves do the rest of the update,
// so that T_JK = sum_{L=J+1..K} V_JL N_LK is complete when leaf J is done
// (block back substitution N_JK = -N_JJ T_JK folded into the factorisation's
// own steps).  T_IK lives in the block (K, I) below the diagonal, which the
// factorisation never reads.  The small products run on all four waves with
// fp32 MFMA, one 32 x 32 block per wave and task.
// Padding rows/columns beyond s are an identity block.
constexpr int DS = kTile + 2;  // LDS row stride of the working matrices (rows 2 banks apart)
constexpr int LF = 32;         // leaf width

// acc(32x32) += A(32x32) * op(B)(32x32) for one wave on fp32 MFMA
// (16x16x4): lane l supplies A[16a + l%16][k + l/16] and op(B)[k + l/16][16b +
// l%16]; acc[a][b][r] is out[16a + 4(l/16) + r][16b + l%16].
template <bool BT>
__device__ inline void wave_gemm32(const float* A, const float* B, f4 (&acc)[2][2], int lane) {
  const int l16 = lane & 15, kq = lane >> 4;
  {
#pragma unroll
    for (int k0 = 0; k0 < LF; k0 += 4) {
      const int k = k0 + kq;
      float av[2], bv[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        av[i] = A[(16 * i + l16) * DS + k];
        bv[i] = BT ? B[(16 * i + l16) * DS + k] : B[k * DS + 16 * i + l16];
      }
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[i], bv[j], acc[i][j], 0, 0, 0);
    }
  }
}

__device__ inline void store32(float* C, const f4 (&acc)[2][2], int lane, float scale, bool add) {
  const int l16 = lane & 15, rq = 4 * (lane >> 4);
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        float* p = &C[(16 * i + rq + r) * DS + 16 * j + l16];
        *p = add ? *p + scale * acc[i][j][r] : scale * acc[i][j][r];
      }
}

// Step c of the leaf sweep.  Lane q (and its twin q + 32, which repeats the
// same work) holds column q of the 32 x 32 working matrix in x[0..31].  Column
// c reaches every lane as scalars read from lane c, so a step needs no LDS
// round trip and no barrier.  The leading c x c block stays symmetric (every
// update to it is a symmetric rank-1 term), so the coefficient W[q][c] of a
// column q < c is the lane's own W[c][q]; for q > c (the columns that become
// the inverse) it is W[c][q] by definition.
template <int C>
__device__ __forceinline__ void leaf_step(float (&x)[LF], int q, int& fail) {
  // the lane's column made opaque per step, so that the compiler evaluates
  // the lane tests where they are used instead of hoisting (and spilling)
  // the masks of every step out of the leaf loop
  asm volatile("" : "+v"(q));
  float cv[C > 0 ? C : 1];
#pragma unroll
  for (int i = 0; i < C; ++i)
    cv[i] = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, x[i]), C));
  const float piv = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, x[C]), C));
  if (!(piv > 0.f) && fail < 0) fail = C;  // uniform
  const float inv = __builtin_amdgcn_rsqf(piv);
  const float inv2 = inv * inv;
  const float xc = x[C];
  const float coef = xc * inv2;
#pragma unroll
  for (int i = 0; i < C; ++i) x[i] = fmaf(-cv[i], coef, x[i]);
  if (q == C) {
    // the pivot column: rows below the diagonal are never read again
#pragma unroll
    for (int i = 0; i < C; ++i) x[i] = -cv[i] * inv2;
  }
  x[C] = q == C ? inv : (q > C ? xc * inv : xc);
}

template <int... Cs>
__device__ __forceinline__ void leaf_steps(float (&x)[LF], int q, int& fail, std::integer_sequence<int, Cs...>) {
  (leaf_step<LF - 1 - Cs>(x, q, fail), ...);
}

__global__ __launch_bounds__(256) void diag_factor_kernel(const float* H, int64_t ldh, int r0, int s, float* vinv,
                                                          CholStatus* st) {
  extern __shared__ __attribute__((aligned(16))) float dsm[];
  float* A = dsm;                  // [128][DS] working matrix (both triangles); then V's upper off-diagonal
                                   // blocks, and the back substitution's products in blocks (1..3, 0)
  float* N = A + kTile * DS;       // [128][DS] the inverse
  int* fail_sh = (int*)(N + kTile * DS);  // [1]
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // load the upper triangle, mirror it; identity outside the s x s block.
  // Every load is issued before the first is used (addresses clamped into
  // the block, so none is conditional): one memory latency, not one per row
  // group.
  {
    constexpr int NU = kTile * kTile / 256;
    const int c = tid % kTile, cc = min(c, s - 1);
    const float* Hb = H + (int64_t)r0 * ldh + r0;
    float v[NU];
#pragma unroll
    for (int u = 0; u < NU; ++u) {
      // 32-bit lane offsets within the block (128 rows of at most 2^24
      // columns); kept in vector registers rather than 64 scalar pairs
      int off = min(2 * u + tid / kTile, s - 1) * (int)ldh + cc;
      asm volatile("" : "+v"(off));
      v[u] = Hb[off];
    }
#pragma unroll
    for (int u = 0; u < NU; ++u) {
      const int r = 2 * u + tid / kTile;
      const float w = (c < s) ? v[u] : (r == c ? 1.f : 0.f);
      if (r <= c) {
        A[r * DS + c] = w;
        A[c * DS + r] = r / LF == c / LF ? w : 0.f;  // below the diagonal blocks: T accumulators
      }
    }
  }
  if (tid == 0) *fail_sh = -1;
  __syncthreads();
  constexpr int NB = kTile / LF;
  // leaf J: wave 0 factors and inverts the diagonal block J in registers
  auto leaf = [&](int J) {
    const int j0 = J * LF;
    const int q = lane & (LF - 1);
    int fail = -1;
    float x[LF];
#pragma unroll
    for (int i = 0; i < LF; ++i) x[i] = A[(j0 + i) * DS + j0 + q];
    leaf_steps(x, q, fail, std::make_integer_sequence<int, LF>{});
    if (lane < LF) {
      int qs = q;
      asm volatile("" : "+v"(qs));  // no hoisted per-row masks
#pragma unroll
      for (int i = 0; i < LF; ++i) N[(j0 + i) * DS + j0 + qs] = i <= qs ? x[i] : 0.f;
    }
    if (lane == 0 && fail >= 0 && *fail_sh < 0) *fail_sh = j0 + fail;
  };
  if (wave == 0) leaf(NB - 1);
  __syncthreads();
  for (int J = NB - 1; J >= 0; --J) {
    const int j0 = J * LF;
    // NB - 1 products, one per wave: the panel V_IJ = A_IJ N_JJ^T for I < J
    // (in place: only this wave reads A_IJ at this step), and the finished
    // blocks N_JK = -N_JJ T_JK for K > J
    if (wave < NB - 1) {
      f4 acc[2][2] = {};
      if (wave < J) {
        wave_gemm32<true>(&A[wave * LF * DS + j0], &N[j0 * DS + j0], acc, lane);
        store32(&A[wave * LF * DS + j0], acc, lane, 1.f, false);
      } else {
        const int K = wave + 1;
        wave_gemm32<false>(&N[j0 * DS + j0], &A[K * LF * DS + j0], acc, lane);
        store32(&N[j0 * DS + K * LF], acc, lane, -1.f, false);
      }
    }
    __syncthreads();
    if (J == 0) break;
    // Schur update A_II' -= V_IJ V_I'J^T for I <= I' < J, and T_IK += V_IJ N_JK
    // for I < J <= K (T_IK sits in the free block (K, I) below the diagonal).
    // Wave 0 updates the next leaf's own block (J - 1, J - 1), the last Schur
    // task, and goes straight on to that leaf; the other waves share the rest,
    // which no leaf step reads, so they run beside it.
    const int nsch = J * (J + 1) / 2, ntot = nsch + J * (NB - J);
    if (wave == 0) {
      f4 u[2][2] = {};
      const int I = J - 1;
      wave_gemm32<true>(&A[I * LF * DS + j0], &A[I * LF * DS + j0], u, lane);
      store32(&A[I * LF * DS + I * LF], u, lane, -1.f, true);
      leaf(I);
    } else {
      for (int task = wave - 1; task < ntot; task += 3) {
        if (task == nsch - 1) continue;  // wave 0's
        f4 u[2][2] = {};
        if (task < nsch) {
          int I = 0, r = task;
          while (r >= J - I) {
            r -= J - I;
            ++I;
          }
          const int I2 = I + r;
          wave_gemm32<true>(&A[I * LF * DS + j0], &A[I2 * LF * DS + j0], u, lane);
          store32(&A[I * LF * DS + I2 * LF], u, lane, -1.f, true);
        } else {
          const int r = task - nsch, I = r / (NB - J), K = J + r % (NB - J);
          wave_gemm32<false>(&A[I * LF * DS + j0], &N[j0 * DS + K * LF], u, lane);
          store32(&A[K * LF * DS + I * LF], u, lane, 1.f, true);
        }
      }
    }
    __syncthreads();
  }
  if (tid == 0 && *fail_sh >= 0 && *fail_sh < s && st->status == DUO_OK) {
    st->status = DUO_ERR_NOT_PD;
    st->fail = r0 + *fail_sh;
  }
#pragma unroll 4
  for (int e4 = tid; e4 < kTile * kTile / 4; e4 += 256) {
    const int r = e4 / (kTile / 4), c0 = 4 * (e4 % (kTile / 4));
    float o[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int c = c0 + i;
      o[i] = (r <= c && r < s && c < s) ? N[r * DS + c] : 0.f;
    }
    ((float4*)vinv)[e4] = make_float4(o[0], o[1], o[2], o[3]);
  }
}

// Copy the inverted diagonal blocks into place (full 128 x 128 incl. zeros).
// Workgroup (b, y) copies rows 16y .. 16y + 15 of block b; with k and ldh
// multiples of 4 and H 16-byte aligned, as 16-byte vectors.
__global__ __launch_bounds__(256) void place_diag_kernel(float* H, int64_t ldh, int k, const float* vinv, int vec) {
  const int b = blockIdx.x;
  const float* src = vinv + (int64_t)b * kTile * kTile;
  if (vec) {
    const int rl = 16 * blockIdx.y + (threadIdx.x >> 4), c4 = 4 * (threadIdx.x & 15);
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int r = b * kTile + rl, c = b * kTile + c4 + 64 * h;
      if (r < k && c < k) *(float4*)(H + (int64_t)r * ldh + c) = *(const float4*)(src + rl * kTile + c4 + 64 * h);
    }
    return;
  }
  if (blockIdx.y) return;
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
  a.order = ORDER_PLAIN;  // K ranges grow with the column: deal the tiles round-robin
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
  b.order = ORDER_PLAIN;  // K ranges shrink with the row: deal the tiles round-robin
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

constexpr size_t kDiagLds = (size_t)(2 * kTile * DS + 4) * sizeof(float);

duo_status chol_run(float* H, int64_t k, int64_t ldh, double damp, void* ws, hipStream_t s, CholStatus** status_dev) {
  const CholWs w = carve(ws, k);
  if (duo_status d = set_max_lds((const void*)diag_factor_kernel, kDiagLds); d != DUO_OK) return d;
  *status_dev = w.st;
  const int T = (int)cdiv(k, kTile);
  hipLaunchKernelGGL(damp_kernel, dim3(1), dim3(256), 0, s, H, ldh, (int)k, damp, w.st);
  DUO_LAUNCH_CHECK();
  auto factor = [&](int b, int sz) -> duo_status {
    const int r0 = b * kTile;
    hipLaunchKernelGGL(diag_factor_kernel, dim3(1), dim3(256), kDiagLds, s, (const float*)H, ldh, r0, sz,
                       w.vinv + (int64_t)b * kTile * kTile, w.st);
    DUO_LAUNCH_CHECK();
    if (r0 == 0) return DUO_OK;
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
    p.inplace = 1;
    return gemm_f32(p, s);
  };
  // Groups of kGroup blocks, from the last one.  Inside a group, before block
  // b is factored its own block column (rows 0 .. r_b + 128) takes the rank
  // updates of the group's blocks already factored (one product: their
  // panels are adjacent columns of H, so K = 128 per block); after the group,
  // the leading matrix takes all of the group's updates in one product with
  // K = 128 kGroup.  Every column still receives every update before its own
  // block is factored; only the fp32 summation order changes.
  // (8 blocks per group from 128 blocks up: measured 170 -> 159 ms at
  // k = 28672, while at k = 4096 the longer strips cost more than they save)
  const int kGroup = T >= 128 ? 8 : 4;
  for (int top = T - 1; top >= 0;) {
    const int lo = top - kGroup + 1 > 0 ? top - kGroup + 1 : 0;
    const int64_t top_end = (int64_t)top * kTile + kTile <= k ? (int64_t)top * kTile + kTile : k;
    for (int b = top; b >= lo; --b) {
      const int rb = b * kTile;
      const int sz = (int)((int64_t)rb + kTile <= k ? kTile : k - rb);
      if (b < top) {
        // strip: H[0:rb+128, rb:rb+128] -= Pp Pp[rb:rb+128]^T, Pp = H[:, rb+128 : top_end]
        const int rp = rb + kTile;
        GemmDesc g{};
        g.M = rp;
        g.N = kTile;
        g.C = H + rb;
        g.ldc = ldh;
        g.beta = 1.f;
        g.tri = TRI_ALL;
        g.nterms = 1;
        g.t[0] = GemmTerm{H + rp, ldh, 1, H + (int64_t)rb * ldh + rp, ldh, 0, (int)(top_end - rp), -1.f, KLO_ZERO,
                          KHI_FULL};
        duo_status st = gemm_f32(g, s);
        if (st != DUO_OK) return st;
      }
      duo_status st = factor(b, sz);
      if (st != DUO_OK) return st;
    }
    if (lo == 0) break;
    // leading block (upper tiles): H[0:r, 0:r] -= Pg Pg^T, Pg = H[0:r, r : top_end], r = lo * 128
    const int r = lo * kTile;
    GemmDesc u{};
    u.M = r;
    u.N = r;
    u.C = H;
    u.ldc = ldh;
    u.beta = 1.f;
    u.tri = TRI_UPPER;
    u.nterms = 1;
    u.t[0] = GemmTerm{H + r, ldh, 1, H + r, ldh, 0, (int)(top_end - r), -1.f, KLO_ZERO, KHI_FULL};
    duo_status st = gemm_f32(u, s);
    if (st != DUO_OK) return st;
    top = lo - 1;
  }
  const int pvec = k % 4 == 0 && ldh % 4 == 0 && (reinterpret_cast<uintptr_t>(H) & 15) == 0;
  hipLaunchKernelGGL(place_diag_kernel, dim3(T, kTile / 16), dim3(256), 0, s, H, ldh, (int)k, (const float*)w.vinv,
                     pvec);
  DUO_LAUNCH_CHECK();
  duo_status st = trinv(H, ldh, k, T, w.X, s);
  if (st != DUO_OK) return st;
  const int T64 = (int)cdiv(k, 64);
  hipLaunchKernelGGL(transpose_upper_kernel, dim3(T64 * (T64 + 1) / 2), dim3(256), 0, s, H, ldh, (int)k);
  DUO_LAUNCH_CHECK();
  return DUO_OK;
}

}  // namespace duo
