// Stage 3 column sweep of the DuoGPT layer solver on gfx950 (paper
// Algorithm 1, inner and outer loops; scores from Eq. 7).
//
// Per block of B columns [j0, j0+Bb):
//   select   S = W[:, blk]^2 * fac[blk]; the z lowest by (S, column, row)
//            are pruned.  Three radix passes (11/11/10 bits) over the
//            order-preserving bits of S find the threshold value; the last
//            workgroup of each pass resolves the bucket (integer atomics
//            only, so the result is deterministic); exact ties at the
//            threshold are ordered by (column, row).
//   in-block one row per 8 lanes, each lane owning 16 columns (c = lane%8 +
//            8i); L[blk, blk] and D[blk, blk] sit in LDS.  Column j: w0 =
//            W[:, j], p = w0 * m_j, e = (w0 - p) / L_jj; later columns get
//            w -= e L[c][j] - w0 D[j][c].  E and W0 are kept for the lazy
//            update.
//   lazy     W[:, rest] += -E L[rest, blk]^T + W0 D[blk, rest] as one two-term
//            fp32 MFMA GEMM (W0 = the columns' values before pruning).
#include <hip/hip_runtime.h>

#include "internal.h"

namespace duo {

namespace {

enum { MODE_SELECT = 0, MODE_FORCED = 1, MODE_KEEP_ALL = 2, MODE_PRUNE_ALL = 3 };
constexpr int kBins = 2048;

struct SelState {
  uint32_t prefix;   // key bits found so far (the full threshold key after pass 2)
  uint32_t rank;     // rank of the z-th key inside the current bucket (1-based)
  uint32_t counter;  // workgroups finished in the current pass
  uint32_t cnt_eq;   // number of keys equal to the threshold
  long long tie_idx; // ties with (column*n + row) <= tie_idx are pruned
};

__global__ void sel_init_kernel(SelState* st, uint32_t* hist, uint32_t z) {
  for (int i = threadIdx.x; i < kBins; i += blockDim.x) hist[i] = 0;
  if (threadIdx.x == 0) {
    st->prefix = 0;
    st->rank = z;
    st->counter = 0;
    st->cnt_eq = 0;
    st->tie_idx = -1;
  }
}

__device__ inline uint32_t atomic_ld(const uint32_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// One radix pass.  pass 0 also writes the scores when requested; with
// do_hist == 0 it only writes scores.
__global__ __launch_bounds__(256) void sel_pass_kernel(const float* __restrict__ W, int64_t ldw, int n, int Bb, int j0,
                                                       const float* __restrict__ fac, SelState* st, uint32_t* hist,
                                                       int pass, int do_hist, float* scores_out) {
  __shared__ uint32_t lh[kBins];
  __shared__ uint32_t wsum[4];
  __shared__ int last;
  const int shift = pass == 0 ? 21 : pass == 1 ? 10 : 0;
  const uint32_t nb = pass == 2 ? 1024u : 2048u;
  const uint32_t pmask = pass == 0 ? 0u : pass == 1 ? 0xffe00000u : 0xfffffc00u;
  const uint32_t prefix = do_hist ? st->prefix : 0u;
  for (int i = threadIdx.x; i < kBins; i += 256) lh[i] = 0;
  __syncthreads();
  const int64_t total = (int64_t)n * Bb;
  for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < total; e += (int64_t)gridDim.x * 256) {
    const int r = (int)(e / Bb), c = (int)(e % Bb);
    const float S = weight_score(W[(int64_t)r * ldw + j0 + c], fac[j0 + c]);
    if (scores_out && pass == 0) scores_out[(int64_t)r * ldw + j0 + c] = S;
    if (do_hist) {
      const uint32_t key = orderable(S);
      if ((key & pmask) == prefix) atomicAdd(&lh[(key >> shift) & (nb - 1)], 1u);
    }
  }
  if (!do_hist) return;
  __syncthreads();
  for (int i = threadIdx.x; i < (int)nb; i += 256)
    if (lh[i]) atomicAdd(&hist[i], lh[i]);
  __threadfence();
  __syncthreads();
  if (threadIdx.x == 0) last = atomicAdd(&st->counter, 1u) == gridDim.x - 1;
  __syncthreads();
  if (!last) return;
  __threadfence();
  // last workgroup: locate the bucket holding the rank-th key
  const uint32_t rank = st->rank;
  const int per = (int)nb / 256;
  uint32_t h[8];
  uint32_t mine = 0;
  for (int q = 0; q < per; ++q) {
    h[q] = atomic_ld(&hist[threadIdx.x * per + q]);
    mine += h[q];
  }
  // exclusive scan of `mine` over the 256 threads (bins in ascending order)
  uint32_t incl = mine;
  const int lane = threadIdx.x & 63;
  for (int o = 1; o < 64; o <<= 1) {
    const uint32_t y = __shfl_up(incl, o);
    if (lane >= o) incl += y;
  }
  if (lane == 63) wsum[threadIdx.x >> 6] = incl;
  __syncthreads();
  uint32_t base = 0;
  for (int w = 0; w < (int)(threadIdx.x >> 6); ++w) base += wsum[w];
  const uint32_t excl = base + incl - mine;
  if (excl < rank && rank <= excl + mine) {
    uint32_t cum = excl;
    for (int q = 0; q < per; ++q) {
      if (rank <= cum + h[q]) {
        const uint32_t bin = (uint32_t)(threadIdx.x * per + q);
        st->prefix = prefix | (bin << shift);
        st->rank = rank - cum;
        st->cnt_eq = h[q];
        break;
      }
      cum += h[q];
    }
  }
  __syncthreads();
  for (int i = threadIdx.x; i < kBins; i += 256) hist[i] = 0;
  if (threadIdx.x == 0) st->counter = 0;
  if (pass != 2) return;
  __threadfence();
  __syncthreads();
  // ties at the threshold: prune the first `rank` of them in (column, row) order
  const uint32_t T = atomic_ld(&st->prefix);
  const uint32_t need = atomic_ld(&st->rank);
  const uint32_t eq = atomic_ld(&st->cnt_eq);
  if (need >= eq) {
    if (threadIdx.x == 0) st->tie_idx = 0x7fffffffffffffffLL;
    return;
  }
  __shared__ uint32_t found;
  uint32_t seen = 0;
  for (int64_t b0 = 0; b0 < total; b0 += 256) {
    const int64_t idx = b0 + threadIdx.x;  // idx = column * n + row
    uint32_t is = 0;
    if (idx < total) {
      const int c = (int)(idx / n), r = (int)(idx % n);
      is = orderable(weight_score(W[(int64_t)r * ldw + j0 + c], fac[j0 + c])) == T;
    }
    uint32_t inc = is;
    for (int o = 1; o < 64; o <<= 1) {
      const uint32_t y = __shfl_up(inc, o);
      if (lane >= o) inc += y;
    }
    __syncthreads();
    if (lane == 63) wsum[threadIdx.x >> 6] = inc;
    __syncthreads();
    uint32_t bb = 0, tot = 0;
    for (int w = 0; w < 4; ++w) {
      if (w < (int)(threadIdx.x >> 6)) bb += wsum[w];
      tot += wsum[w];
    }
    if (is && seen + bb + inc == need) st->tie_idx = idx;
    seen += tot;
    if (seen >= need) break;  // uniform
  }
  (void)found;
}

// ---------------------------------------------------------------------------
// in-block sweep
// ---------------------------------------------------------------------------
constexpr int GS = 8;    // lanes per row
constexpr int NPT = 16;  // columns per lane
constexpr int RPB = 32;  // rows per workgroup

__global__ __launch_bounds__(256) void inblock_kernel(float* __restrict__ Wo, int n, int k, int j0, int Bb, int B,
                                                      const float* __restrict__ L, int64_t ldl,
                                                      const float* __restrict__ D, int64_t ldd,
                                                      const float* __restrict__ fac, const SelState* st, int mode,
                                                      const uint32_t* __restrict__ mask_in, float* __restrict__ EW,
                                                      uint8_t* __restrict__ bmask) {
  extern __shared__ __attribute__((aligned(16))) float sm[];
  float* Lq = sm;                           // [128][8][16]: L[j0+q+8i][j0+j] for q+8i > j
  float* Dq = sm + kMaxBlock * GS * NPT;    // [128][8][16]: D[j0+j][j0+q+8i] for q+8i > j
  float* Ld = Dq + kMaxBlock * GS * NPT;    // [128]: L[j0+j][j0+j]
  const int tid = threadIdx.x;
  for (int p = tid; p < kMaxBlock * GS; p += 256) {
    {  // L: j fastest so that global reads are contiguous
      const int j = p % kMaxBlock, q = p / kMaxBlock;
      float v[NPT];
#pragma unroll
      for (int i = 0; i < NPT; ++i) {
        const int c = q + GS * i;
        v[i] = (c > j && c < Bb && j < Bb) ? L[(int64_t)(j0 + c) * ldl + j0 + j] : 0.f;
      }
      float4* dst = (float4*)&Lq[(j * GS + q) * NPT];
#pragma unroll
      for (int i = 0; i < NPT / 4; ++i) dst[i] = make_float4(v[4 * i], v[4 * i + 1], v[4 * i + 2], v[4 * i + 3]);
    }
    {  // D: q fastest
      const int q = p % GS, j = p / GS;
      float v[NPT];
#pragma unroll
      for (int i = 0; i < NPT; ++i) {
        const int c = q + GS * i;
        v[i] = (c > j && c < Bb && j < Bb) ? D[(int64_t)(j0 + j) * ldd + j0 + c] : 0.f;
      }
      float4* dst = (float4*)&Dq[(j * GS + q) * NPT];
#pragma unroll
      for (int i = 0; i < NPT / 4; ++i) dst[i] = make_float4(v[4 * i], v[4 * i + 1], v[4 * i + 2], v[4 * i + 3]);
    }
  }
  if (tid < kMaxBlock) Ld[tid] = tid < Bb ? L[(int64_t)(j0 + tid) * ldl + j0 + tid] : 1.f;
  __syncthreads();

  const int row = blockIdx.x * RPB + (tid >> 3);
  const int q = tid & 7;
  const bool rv = row < n;
  float w[NPT];
  uint32_t my = 0;  // bit i: column q + 8i kept
  uint32_t T = 0;
  long long tie = -1;
  if (mode == MODE_SELECT) {
    T = st->prefix;
    tie = st->tie_idx;
  }
  const int words = (k + 31) / 32;
#pragma unroll
  for (int i = 0; i < NPT; ++i) {
    const int c = q + GS * i;
    const bool cv = rv && c < Bb;
    w[i] = cv ? Wo[(int64_t)row * k + j0 + c] : 0.f;
    bool keep = true;
    if (cv) {
      if (mode == MODE_SELECT) {
        const uint32_t key = orderable(weight_score(w[i], fac[j0 + c]));
        const long long idx = (long long)c * n + row;
        keep = !(key < T || (key == T && idx <= tie));
      } else if (mode == MODE_FORCED) {
        const int gc = j0 + c;
        keep = (mask_in[(int64_t)row * words + gc / 32] >> (gc % 32)) & 1u;
      } else {
        keep = mode == MODE_KEEP_ALL;
      }
    }
    my |= (keep ? 1u : 0u) << i;
  }
  uint32_t m[GS];  // keep bits of the 8 lanes of this row (bit i: group g + i)
#pragma unroll
  for (int o = 0; o < GS; ++o) m[o] = __shfl(my, o, GS);
  const int ngroups = (Bb + GS - 1) / GS;

  // Group g holds columns 8g..8g+7 (column 8g+o belongs to lane o).  After each
  // group the register arrays shift down by one so that the current group is
  // always w[0] and every register index is a compile-time constant.
  for (int g = 0; g < ngroups; ++g) {
    float e_own = 0.f, w0_own = 0.f;
#pragma unroll
    for (int o = 0; o < GS; ++o) {
      const int j = g * GS + o;
      if (j < Bb) {  // uniform
        const float wj = __shfl(w[0], o, GS);
        const bool kj = m[o] & 1u;
        const float p = kj ? wj : 0.f;
        const float e = (wj - p) / Ld[j];
        if (q == o) {
          w[0] = p;
          e_own = e;
          w0_own = wj;
        }
        const float* lq = &Lq[(j * GS + q) * NPT + g];
        const float* dq = &Dq[(j * GS + q) * NPT + g];
#pragma unroll
        for (int i = 0; i < NPT; ++i) {
          if (i < NPT - g && (i > 0 || q > o)) w[i] -= fmaf(e, lq[i], -(wj * dq[i]));
        }
      }
    }
    const int c = q + GS * g;
    if (rv && c < Bb) {
      Wo[(int64_t)row * k + j0 + c] = w[0];
      EW[(int64_t)row * 2 * B + c] = e_own;
      EW[(int64_t)row * 2 * B + B + c] = w0_own;
      bmask[(int64_t)row * k + j0 + c] = (uint8_t)((my >> g) & 1u);
    }
#pragma unroll
    for (int i = 0; i < NPT - 1; ++i) w[i] = w[i + 1];
    w[NPT - 1] = 0.f;
#pragma unroll
    for (int o = 0; o < GS; ++o) m[o] >>= 1;
  }
}

__global__ void init_w_kernel(const void* W, int dtype, int64_t ldw, int n, int k, float* Wo) {
  const int64_t id = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (id >= (int64_t)n * k) return;
  const int64_t r = id / k, c = id % k;
  Wo[id] = dtype == DUO_BF16 ? bf16_bits_to_f32(((const uint16_t*)W)[r * ldw + c]) : ((const float*)W)[r * ldw + c];
}

__global__ void finalize_kernel(const float* Wo, const uint8_t* bmask, int n, int k, int dtype, void* lowp,
                                uint32_t* mask_out) {
  const int64_t id = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int words = (k + 31) / 32;
  if (mask_out && id < (int64_t)n * words) {
    const int64_t r = id / words, w = id % words;
    uint32_t bits = 0;
    for (int e = 0; e < 32; ++e) {
      const int64_t c = w * 32 + e;
      if (c < k && bmask[r * k + c]) bits |= 1u << e;
    }
    mask_out[id] = bits;
  }
  if (lowp && id < (int64_t)n * k) {
    if (dtype == DUO_BF16)
      ((uint16_t*)lowp)[id] = f32_to_bf16_bits(Wo[id]);
    else
      ((float*)lowp)[id] = Wo[id];
  }
}

struct SweepWs {
  SelState* st;
  uint32_t* hist;
  float* EW;
  uint8_t* bmask;
  size_t bytes;
};

SweepWs carve(void* ws, int64_t n, int64_t k, int B) {
  Carver c(ws);
  SweepWs w;
  w.st = c.take<SelState>(1);
  w.hist = c.take<uint32_t>(kBins);
  w.EW = c.take<float>((size_t)n * 2 * B);
  w.bmask = c.take<uint8_t>((size_t)n * k);
  w.bytes = c.off;
  return w;
}

}  // namespace

size_t sweep_ws_bytes(int64_t n, int64_t k, int B) { return carve(nullptr, n, k, B).bytes; }

duo_status sweep_run(const void* W, int32_t w_dtype, int64_t n, int64_t k, int64_t ldw, const float* L, int64_t ldl,
                     const float* D, int64_t ldd, const float* fac, double p_w, int B, const uint32_t* mask_in,
                     float* W_out, void* W_out_lowp, uint32_t* mask_out, float* scores_out, void* ws,
                     hipStream_t s) {
  const SweepWs w = carve(ws, n, k, B);
  const int64_t nk = n * k;
  hipLaunchKernelGGL(init_w_kernel, dim3((unsigned)cdiv(nk, 256)), dim3(256), 0, s, W, (int)w_dtype, ldw, (int)n,
                     (int)k, W_out);
  DUO_LAUNCH_CHECK();
  const size_t lds = (size_t)(2 * kMaxBlock * GS * NPT + kMaxBlock) * sizeof(float);
  DUO_HIP_TRY(hipFuncSetAttribute((const void*)inblock_kernel, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds));
  int64_t prev = 0;
  for (int64_t j0 = 0; j0 < k; j0 += B) {
    const int Bb = (int)(k - j0 < B ? k - j0 : B);
    const int64_t j1 = j0 + Bb;
    const int64_t cum = (int64_t)floor(p_w * (double)n * (double)j1 + 0.5);
    const int64_t z = cum - prev;
    prev = cum;
    const int64_t total = n * Bb;
    int mode = MODE_SELECT;
    if (mask_in)
      mode = MODE_FORCED;
    else if (z <= 0)
      mode = MODE_KEEP_ALL;
    else if (z >= total)
      mode = MODE_PRUNE_ALL;
    // few workgroups: each pushes its local histogram to the global one with
    // integer atomics, and hot bins serialise across workgroups
    const int pgrid = (int)(cdiv(total, 8192) < 128 ? cdiv(total, 8192) : 128);
    prof_begin(DUO_PROF_SELECT, s);
    if (mode == MODE_SELECT) {
      hipLaunchKernelGGL(sel_init_kernel, dim3(1), dim3(256), 0, s, w.st, w.hist, (uint32_t)z);
      DUO_LAUNCH_CHECK();
      for (int pass = 0; pass < 3; ++pass) {
        hipLaunchKernelGGL(sel_pass_kernel, dim3(pgrid), dim3(256), 0, s, (const float*)W_out, k, (int)n, Bb, (int)j0,
                           fac, w.st, w.hist, pass, 1, scores_out);
        DUO_LAUNCH_CHECK();
      }
    } else if (scores_out) {
      hipLaunchKernelGGL(sel_pass_kernel, dim3(pgrid), dim3(256), 0, s, (const float*)W_out, k, (int)n, Bb, (int)j0,
                         fac, w.st, w.hist, 0, 0, scores_out);
      DUO_LAUNCH_CHECK();
    }
    prof_end(DUO_PROF_SELECT, s);
    prof_begin(DUO_PROF_INBLOCK, s);
    hipLaunchKernelGGL(inblock_kernel, dim3((unsigned)cdiv(n, RPB)), dim3(256), lds, s, W_out, (int)n, (int)k, (int)j0,
                       Bb, B, L, ldl, D, ldd, fac, (const SelState*)w.st, mode, mask_in, w.EW, w.bmask);
    DUO_LAUNCH_CHECK();
    prof_end(DUO_PROF_INBLOCK, s);
    if (j1 < k) {
      GemmDesc g{};
      g.M = (int)n;
      g.N = (int)(k - j1);
      g.C = W_out + j1;
      g.ldc = k;
      g.beta = 1.f;
      g.tri = TRI_ALL;
      g.nterms = 2;
      g.t[0] = GemmTerm{w.EW, 2 * B, 1, L + j1 * ldl + j0, ldl, 0, Bb, -1.f, KLO_ZERO, KHI_FULL};
      g.t[1] = GemmTerm{w.EW + B, 2 * B, 1, D + j0 * ldd + j1, ldd, 1, Bb, 1.f, KLO_ZERO, KHI_FULL};
      prof_begin(DUO_PROF_TRAIL, s);
      duo_status st = gemm_f32(g, s);
      prof_end(DUO_PROF_TRAIL, s);
      if (st != DUO_OK) return st;
    }
  }
  if (mask_out || W_out_lowp) {
    const int64_t words = cdiv(k, 32);
    const int64_t cnt = nk > n * words ? nk : n * words;
    hipLaunchKernelGGL(finalize_kernel, dim3((unsigned)cdiv(cnt, 256)), dim3(256), 0, s, (const float*)W_out,
                       (const uint8_t*)w.bmask, (int)n, (int)k, (int)w_dtype, W_out_lowp, mask_out);
    DUO_LAUNCH_CHECK();
  }
  return DUO_OK;
}

}  // namespace duo
