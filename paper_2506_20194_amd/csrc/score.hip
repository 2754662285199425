// Stage 3 precompute of the DuoGPT layer solver on gfx950 (paper Eq. 7;
// App. A.3-A.4; Algorithm 1 lines Q, U, a, b, c, D):
//   Q = G L            only the upper triangle (incl. diagonal) is needed;
//   b_p = sum_{i>p} Q_pi^2, c_p = Q_pp / L_pp, fac_p = 1/L_pp^2 + a_p - b_p + 2 c_p;
//   U = strict upper(Q); D = U L^T (strictly upper).
// Both products run on the fp32 MFMA GEMM with tile-granular triangular K
// ranges; fac uses fixed-order double sums.
#include <hip/hip_runtime.h>

#include "internal.h"

namespace duo {

namespace {

// One workgroup per row p: b, c, fac, then turn row p of Q into row p of U
// inside its diagonal tile (zero the entries at columns tile_start(p)..p).
__global__ __launch_bounds__(256) void fac_kernel(float* Q, int64_t ldq, const float* L, int64_t ldl, const float* a,
                                                  int k, float* fac) {
  __shared__ double red[256];
  const int p = blockIdx.x;
  const float* q = Q + (int64_t)p * ldq;
  double s = 0.0;
  for (int i = p + 1 + threadIdx.x; i < k; i += 256) {
    const double v = q[i];
    s += v * v;
  }
  red[threadIdx.x] = s;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    const double lpp = L[(int64_t)p * ldl + p];
    const double b = red[0];
    const double c = (double)q[p] / lpp;
    fac[p] = (float)(1.0 / (lpp * lpp) + (double)a[p] - b + 2.0 * c);
  }
  __syncthreads();
  const int t0 = p / kTile * kTile;
  for (int i = t0 + threadIdx.x; i <= p; i += 256) Q[(int64_t)p * ldq + i] = 0.f;
}

struct ScoreWs {
  float* Q;
  size_t bytes;
};

ScoreWs carve(void* ws, int64_t k) {
  Carver c(ws);
  ScoreWs w;
  w.Q = c.take<float>((size_t)k * k);
  w.bytes = c.off;
  return w;
}

}  // namespace

size_t score_ws_bytes(int64_t k) { return carve(nullptr, k).bytes; }

const float* score_u(const void* ws, int64_t k) { return carve(const_cast<void*>(ws), k).Q; }

duo_status score_run(const float* L, int64_t ldl, const float* G, int64_t ldg, const float* a, int64_t k, float* D,
                     int64_t ldd, float* fac, void* ws, hipStream_t s) {
  const ScoreWs w = carve(ws, k);
  // Q = G L on upper tiles; L[l][i] = 0 for l < i, so l starts at the tile column
  GemmDesc q{};
  q.M = (int)k;
  q.N = (int)k;
  q.C = w.Q;
  q.ldc = k;
  q.beta = 0.f;
  q.tri = TRI_UPPER;
  q.order = ORDER_PLAIN;  // K range [j0, k): the first columns are the longest
  q.nterms = 1;
  q.t[0] = GemmTerm{G, ldg, 1, L, ldl, 1, (int)k, 1.f, KLO_COL, KHI_FULL};
  duo_status st = gemm_f32(q, s);
  if (st != DUO_OK) return st;
  hipLaunchKernelGGL(fac_kernel, dim3((unsigned)k), dim3(256), 0, s, w.Q, (int64_t)k, L, ldl, a, (int)k, fac);
  DUO_LAUNCH_CHECK();
  if (!D) return DUO_OK;  // the Y form of the sweep reads U (score_u) instead
  // D = U L^T on upper tiles: D[p][j] = sum_{p < i <= j} U[p][i] L[j][i]
  GemmDesc d{};
  d.M = (int)k;
  d.N = (int)k;
  d.C = D;
  d.ldc = ldd;
  d.beta = 0.f;
  d.tri = TRI_UPPER;
  d.order = ORDER_DIAG;  // K range [i0, j0 + 128): grows with the distance from the diagonal
  d.nterms = 1;
  d.t[0] = GemmTerm{w.Q, k, 1, L, ldl, 0, (int)k, 1.f, KLO_ROW, KHI_COL};
  return gemm_f32(d, s);
}

}  // namespace duo
