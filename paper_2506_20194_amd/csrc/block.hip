// Decoder-block harness: the operations that carry the two activation streams
// of a LLaMA-style decoder block between the solver's groups (the multi-layer
// case of Sec. 4.2: the dense model sees X-tilde, the pruned model sees its
// own, sparsified input).  All activations are bf16 row-major token x feature
// arrays; arithmetic is fp32.
//
//   duo_rmsnorm       y = x / sqrt(mean(x^2) + eps)          (unit gain)
//   duo_act_sparsify  y = x with the per-token (|x|, channel) rule applied
//   duo_linear        Y = X W^T (+ R)       (bf16 MFMA tiles, fp32 accumulate)
//   duo_rope          rotary position embedding, rotate-half pairs (i, i + d/2)
//   duo_attention     causal softmax(Q K^T / sqrt(d)) V per sequence and head
//                     (two passes over the key blocks with bf16 MFMA: row
//                     maxima and sums, then the probabilities, rounded to bf16
//                     after normalisation, times V)
//   duo_silu_mul      y = SiLU(g) * u
#include <hip/hip_runtime.h>

#include <cmath>
#include <mutex>

#include "internal.h"

using namespace duo;

namespace {

__device__ inline float ld_bf16(const uint16_t* p) { return bf16_bits_to_f32(*p); }

// ---------------------------------------------------------------------------
// kernels
// ---------------------------------------------------------------------------

// One 256-thread workgroup per token.
__global__ __launch_bounds__(256) void rmsnorm_kernel(const uint16_t* __restrict__ X, int64_t ldx, int d, float eps,
                                                      uint16_t* __restrict__ Y, int64_t ldy) {
  __shared__ float red[4];
  const uint16_t* x = X + (int64_t)blockIdx.x * ldx;
  uint16_t* y = Y + (int64_t)blockIdx.x * ldy;
  float ss = 0.f;
  for (int c = threadIdx.x; c < d; c += 256) {
    const float v = ld_bf16(x + c);
    ss = fmaf(v, v, ss);
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) ss += __shfl_xor(ss, o);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
  __syncthreads();
  const float tot = (red[0] + red[1]) + (red[2] + red[3]);
  const float inv = 1.0f / sqrtf(tot / (float)d + eps);
  for (int c = threadIdx.x; c < d; c += 256) y[c] = f32_to_bf16_bits(ld_bf16(x + c) * inv);
}

// 16-byte form (k, ldx, ldy multiples of 8, aligned rows): one workgroup row
// of threads per token, 8 channels per thread.
__global__ __launch_bounds__(256) void act_apply8_kernel(const uint16_t* __restrict__ X, int64_t ldx, int k,
                                                         const int64_t* __restrict__ thr, uint16_t* __restrict__ Y,
                                                         int64_t ldy) {
  const int cpr = (k + 2047) / 2048;  // workgroups per token
  const int t = (int)(blockIdx.x / cpr);
  const int c0 = ((int)(blockIdx.x % cpr) * 256 + threadIdx.x) * 8;
  if (c0 >= k) return;
  const int64_t th = thr[t];
  const u32x4 x = *(const u32x4*)(X + (int64_t)t * ldx + c0);
  u32x4 y;
#pragma unroll
  for (int h = 0; h < 4; ++h) {
    uint32_t o = 0;
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const uint32_t v = (x[h] >> (16 * j)) & 0xFFFFu;
      const int64_t key = ((int64_t)(v & 0x7fffu) << 32) | (c0 + 2 * h + j);
      o |= (key > th ? v : 0u) << (16 * j);
    }
    y[h] = o;
  }
  *(u32x4*)(Y + (int64_t)t * ldy + c0) = y;
}

__global__ void act_apply_kernel(const uint16_t* __restrict__ X, int64_t ldx, int m, int k,
                                 const int64_t* __restrict__ thr, uint16_t* __restrict__ Y, int64_t ldy) {
  const int64_t id = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (id >= (int64_t)m * k) return;
  const int t = (int)(id / k), c = (int)(id % k);
  const uint16_t x = X[(int64_t)t * ldx + c];
  const int64_t key = ((int64_t)(x & 0x7fffu) << 32) | c;
  Y[(int64_t)t * ldy + c] = key > thr[t] ? x : (uint16_t)0;
}

// One workgroup per token: the half = head_dim / 2 rotation angles
// pos * theta^(-2i/head_dim) (pos = token % seq_len) and their cosines and
// sines are computed once in fp64 and shared by every head; each thread then
// rotates pairs (i, i + half) of the token's heads in fp32.
__global__ __launch_bounds__(256) void rope_kernel(uint16_t* __restrict__ X, int64_t ldx, int heads, int hd,
                                                   int seq_len, double theta) {
  __shared__ float cs[2][256];
  const int half = hd / 2;
  const int t = blockIdx.x;
  for (int i = threadIdx.x; i < half; i += 256) {
    const double ang = (double)(t % seq_len) * pow(theta, -2.0 * (double)i / (double)hd);
    double sd, cd;
    sincos(ang, &sd, &cd);
    cs[0][i] = (float)cd;
    cs[1][i] = (float)sd;
  }
  __syncthreads();
  uint16_t* row = X + (int64_t)t * ldx;
  for (int e = threadIdx.x; e < heads * half; e += 256) {
    const int h = e / half, i = e % half;
    uint16_t* p = row + (int64_t)h * hd;
    const float c = cs[0][i], s = cs[1][i];
    const float x1 = bf16_bits_to_f32(p[i]), x2 = bf16_bits_to_f32(p[i + half]);
    p[i] = f32_to_bf16_bits(x1 * c - x2 * s);
    p[i + half] = f32_to_bf16_bits(x2 * c + x1 * s);
  }
}

// 16-byte form of silu_mul_kernel (n, ld, ldy multiples of 8, aligned rows).
__global__ __launch_bounds__(256) void silu_mul8_kernel(const uint16_t* __restrict__ G, const uint16_t* __restrict__ U,
                                                        int64_t ld, int n, uint16_t* __restrict__ Y, int64_t ldy) {
  const int cpr = (n + 2047) / 2048;  // workgroups per token
  const int t = (int)(blockIdx.x / cpr);
  const int c0 = ((int)(blockIdx.x % cpr) * 256 + threadIdx.x) * 8;
  if (c0 >= n) return;
  const u32x4 g = *(const u32x4*)(G + (int64_t)t * ld + c0);
  const u32x4 u = *(const u32x4*)(U + (int64_t)t * ld + c0);
  u32x4 y;
#pragma unroll
  for (int h = 0; h < 4; ++h) {
    uint32_t o = 0;
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const float gv = bf16_bits_to_f32((uint16_t)(g[h] >> (16 * j))), uv = bf16_bits_to_f32((uint16_t)(u[h] >> (16 * j)));
      o |= (uint32_t)f32_to_bf16_bits(gv / (1.0f + expf(-gv)) * uv) << (16 * j);
    }
    y[h] = o;
  }
  *(u32x4*)(Y + (int64_t)t * ldy + c0) = y;
}

__global__ void silu_mul_kernel(const uint16_t* __restrict__ G, const uint16_t* __restrict__ U, int64_t ld, int m,
                                int n, uint16_t* __restrict__ Y, int64_t ldy) {
  const int64_t id = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (id >= (int64_t)m * n) return;
  const int64_t t = id / n, c = id % n;
  const float g = bf16_bits_to_f32(G[t * ld + c]), u = bf16_bits_to_f32(U[t * ld + c]);
  Y[t * ldy + c] = f32_to_bf16_bits(g / (1.0f + expf(-g)) * u);
}

// ---------------------------------------------------------------------------
// bf16 MFMA building blocks (v_mfma_f32_16x16x32_bf16: lane l holds row l % 16
// of A and column l % 16 of B, each as the 8 consecutive k of group l / 16; the
// accumulator's element r sits at row 4 (l / 16) + r, column l % 16)
// ---------------------------------------------------------------------------
__device__ __forceinline__ f4 mma_bf16(const u32x4& a, const u32x4& b, f4 c) {
  bf16x8 av, bv;
  __builtin_memcpy(&av, &a, 16);
  __builtin_memcpy(&bv, &b, 16);
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, bv, c, 0, 0, 0);
}

// Workgroup barrier without the memory fence of __syncthreads, whose fence
// would wait for the global prefetches in flight; this wave's LDS traffic is
// drained first.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0)
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// A row of 8 16-byte chunks stored at chunk position c ^ ((r >> 1) & 7): the 16
// rows one fragment read touches (one chunk each) cover the 64 LDS banks once.
__device__ __forceinline__ int swz8(int r, int c) { return r * 8 + (c ^ ((r >> 1) & 7)); }

// ---------------------------------------------------------------------------
// Linear: Y = X W^T (+ R).  One 256-thread workgroup per 128 x 128 tile of Y,
// 2 x 2 waves of 64 x 64 (4 x 4 accumulator blocks); K staged 64 at a time
// through two LDS buffers with the global loads of the stage after next held
// in registers (zero-filled past K).  Needs 16-byte aligned rows and K % 8 == 0.
// ---------------------------------------------------------------------------
constexpr int kLinT = 128, kLinK = 64;

__global__ __launch_bounds__(256, 2) void lin_kernel(const uint16_t* __restrict__ X, int64_t ldx,
                                                     const uint16_t* __restrict__ W, int64_t ldw,
                                                     const uint16_t* R, int64_t ldr, uint16_t* Y, int64_t ldy,
                                                     int M, int N, int K) {
  __shared__ u32x4 sm[2][2][kLinT * 8];  // [buffer][X, W][swizzled rows of 8 chunks]: 64 KB
  const int tn = (N + kLinT - 1) / kLinT;
  const int per = (int)((gridDim.x + 7) / 8);
  const int id = (int)(blockIdx.x % 8) * per + (int)(blockIdx.x / 8);  // contiguous tile ranges per XCD
  if (id >= (int)cdiv((int64_t)M, kLinT) * tn) return;
  const int i0 = (id / tn) * kLinT, j0 = (id % tn) * kLinT;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wi = wave >> 1, wj = wave & 1;
  const u32x4 zero = {0u, 0u, 0u, 0u};
  // this thread's loads: rows (tid / 8) + 32 q, chunk tid % 8 (8 threads per 128-byte row segment)
  const int lc = tid & 7;
  const uint16_t* xa[4];
  const uint16_t* wb[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int r = (tid >> 3) + 32 * q;
    xa[q] = X + (int64_t)min(i0 + r, M - 1) * ldx + 8 * lc;
    wb[q] = W + (int64_t)min(j0 + r, N - 1) * ldw + 8 * lc;
  }
  auto load = [&](int k0, u32x4 (&ra)[4], u32x4 (&rb)[4]) {
    const bool ok = k0 + 8 * lc < K;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      ra[q] = ok ? *(const u32x4*)(xa[q] + k0) : zero;
      rb[q] = ok ? *(const u32x4*)(wb[q] + k0) : zero;
    }
  };
  auto store = [&](int buf, const u32x4 (&ra)[4], const u32x4 (&rb)[4]) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int r = (tid >> 3) + 32 * q;
      sm[buf][0][swz8(r, lc)] = ra[q];
      sm[buf][1][swz8(r, lc)] = rb[q];
    }
  };
  f4 acc[4][4];
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int b = 0; b < 4; ++b) acc[a][b] = f4{0.f, 0.f, 0.f, 0.f};
  auto compute = [&](int buf) {
#pragma unroll
    for (int s2 = 0; s2 < kLinK / 32; ++s2) {
      const int c = 4 * s2 + (lane >> 4);
      u32x4 fa[4], fb[4];
#pragma unroll
      for (int a = 0; a < 4; ++a) fa[a] = sm[buf][0][swz8(wi * 64 + a * 16 + (lane & 15), c)];
#pragma unroll
      for (int b = 0; b < 4; ++b) fb[b] = sm[buf][1][swz8(wj * 64 + b * 16 + (lane & 15), c)];
#pragma unroll
      for (int a = 0; a < 4; ++a)
#pragma unroll
        for (int b = 0; b < 4; ++b) acc[a][b] = mma_bf16(fa[a], fb[b], acc[a][b]);
    }
  };
  const int nst = (K + kLinK - 1) / kLinK;
  u32x4 ra0[4], rb0[4], ra1[4], rb1[4];
  load(0, ra0, rb0);
  if (nst > 1) load(kLinK, ra1, rb1);
  store(0, ra0, rb0);
  lds_barrier();
#pragma nounroll
  for (int s = 0; s < nst; s += 2) {
    if (s + 2 < nst) load((s + 2) * kLinK, ra0, rb0);
    compute(0);
    if (s + 1 < nst) store(1, ra1, rb1);
    lds_barrier();
    if (s + 1 >= nst) break;
    if (s + 3 < nst) load((s + 3) * kLinK, ra1, rb1);
    compute(1);
    if (s + 2 < nst) store(0, ra0, rb0);
    lds_barrier();
  }
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int b = 0; b < 4; ++b)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int i = i0 + wi * 64 + a * 16 + (lane >> 4) * 4 + r, j = j0 + wj * 64 + b * 16 + (lane & 15);
        if (i < M && j < N) {
          float v = acc[a][b][r];
          if (R) v += bf16_bits_to_f32(R[(int64_t)i * ldr + j]);
          Y[(int64_t)i * ldy + j] = f32_to_bf16_bits(v);
        }
      }
}

// Linear for rows that are not 16-byte aligned or K % 8 != 0: one thread per
// output, fp32 sum in k order.
__global__ void lin_plain_kernel(const uint16_t* __restrict__ X, int64_t ldx, const uint16_t* __restrict__ W,
                                 int64_t ldw, const uint16_t* R, int64_t ldr, uint16_t* Y, int64_t ldy, int M, int N,
                                 int K) {
  const int64_t id = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (id >= (int64_t)M * N) return;
  const int i = (int)(id / N), j = (int)(id % N);
  float v = 0.f;
  for (int k = 0; k < K; ++k) v = fmaf(bf16_bits_to_f32(X[(int64_t)i * ldx + k]), bf16_bits_to_f32(W[(int64_t)j * ldw + k]), v);
  if (R) v += bf16_bits_to_f32(R[(int64_t)i * ldr + j]);
  Y[(int64_t)i * ldy + j] = f32_to_bf16_bits(v);
}

// ---------------------------------------------------------------------------
// Causal attention, one 256-thread workgroup per (sequence, head, block of 64
// queries); wave w owns queries 16 w .. 16 w + 15 of the block, its Q rows held
// in registers as MFMA fragments.  Key blocks of 64 are staged in LDS.
//   pass 1: S = Q K^T / sqrt(d) per key block; each row's running maximum m and
//           sum l of exp(s - m) (rescaled when m grows);
//   pass 2: S again, P = bf16(exp(s - m) / l) (the rounding point of the
//           reference: normalised probabilities in bf16), O += P V with V
//           staged transposed so that its fragments are 16-byte reads.
// Keys above the query (and past the sequence) are masked.  HD = head_dim.
// ---------------------------------------------------------------------------
template <int HD>
__global__ __launch_bounds__(256) void attn_kernel(const uint16_t* __restrict__ Q, const uint16_t* __restrict__ Kx,
                                                   const uint16_t* __restrict__ V, int64_t ld, int L, int heads,
                                                   float scale, uint16_t* __restrict__ O, int64_t ldo, int nqb) {
  constexpr int CH = HD / 8;       // 16-byte chunks per key row
  constexpr int KC = HD / 32;      // MFMA k-steps over head_dim
  constexpr int DB = HD / 16;      // 16-wide blocks of the output row
  __shared__ u32x4 sK[64 * CH];            // [64 keys][CH chunks], swizzled
  __shared__ __attribute__((aligned(16))) uint16_t sV[HD * 64];     // [HD][64 keys]: rows of 8 chunks, swizzled
  __shared__ __attribute__((aligned(16))) uint16_t sP[4][16 * 64];  // per wave [16 queries][64 keys], swizzled
  const int qb = nqb - 1 - (int)(blockIdx.x % nqb);   // the longest query blocks first
  const int sh = (int)(blockIdx.x / nqb);
  const int h = sh % heads;
  const int64_t row0 = (int64_t)(sh / heads) * L;     // the sequence's first token
  const int col0 = h * HD;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int q0 = qb * 64;
  auto kswz = [](int key, int c) { return CH == 16 ? key * 16 + (c ^ (key & 15)) : swz8(key, c); };

  u32x4 qa[KC];
  {
    const int qr = min(q0 + wave * 16 + (lane & 15), L - 1);
#pragma unroll
    for (int c = 0; c < KC; ++c) qa[c] = *(const u32x4*)(Q + (row0 + qr) * ld + col0 + 8 * ((lane >> 4) + 4 * c));
  }
  const int qrow = q0 + wave * 16 + (lane >> 4) * 4;  // + r: this lane's accumulator rows
  const int nkb = min(qb + 1, (L + 63) / 64);

  auto load_k = [&](int kb) {
#pragma unroll
    for (int i = 0; i < 64 * CH / 256; ++i) {
      const int e = tid + 256 * i, key = e / CH, c = e % CH;
      const int kr = min(kb * 64 + key, L - 1);
      sK[kswz(key, c)] = *(const u32x4*)(Kx + (row0 + kr) * ld + col0 + 8 * c);
    }
  };
  auto scores = [&](int kb, f4 (&sc)[4]) {
#pragma unroll
    for (int b = 0; b < 4; ++b) sc[b] = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int c = 0; c < KC; ++c)
#pragma unroll
      for (int b = 0; b < 4; ++b) sc[b] = mma_bf16(qa[c], sK[kswz(b * 16 + (lane & 15), (lane >> 4) + 4 * c)], sc[b]);
#pragma unroll
    for (int b = 0; b < 4; ++b)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int key = kb * 64 + b * 16 + (lane & 15);
        sc[b][r] = (key <= qrow + r && key < L) ? sc[b][r] * scale : -INFINITY;
      }
  };
  auto row_max16 = [](float v) {
#pragma unroll
    for (int o = 1; o < 16; o <<= 1) v = fmaxf(v, __shfl_xor(v, o));
    return v;
  };
  auto row_sum16 = [](float v) {
#pragma unroll
    for (int o = 1; o < 16; o <<= 1) v += __shfl_xor(v, o);
    return v;
  };

  // pass 1: row maxima and sums
  float mrow[4], lrow[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    mrow[r] = -INFINITY;
    lrow[r] = 0.f;
  }
  for (int kb = 0; kb < nkb; ++kb) {
    load_k(kb);
    __syncthreads();
    f4 sc[4];
    scores(kb, sc);
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const float mb = row_max16(fmaxf(fmaxf(sc[0][r], sc[1][r]), fmaxf(sc[2][r], sc[3][r])));
      const float mn = fmaxf(mrow[r], mb);
      float e = 0.f;
#pragma unroll
      for (int b = 0; b < 4; ++b) e += expf(sc[b][r] - mn);
      lrow[r] = lrow[r] * expf(mrow[r] - mn) + row_sum16(e);
      mrow[r] = mn;
    }
    __syncthreads();
  }
  float inv[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) inv[r] = 1.0f / lrow[r];

  // pass 2: normalised bf16 probabilities times V
  f4 o[DB];
#pragma unroll
  for (int d = 0; d < DB; ++d) o[d] = f4{0.f, 0.f, 0.f, 0.f};
  uint16_t* p = sP[wave];
  for (int kb = 0; kb < nkb; ++kb) {
    load_k(kb);
#pragma unroll
    for (int i = 0; i < 64 * CH / 256; ++i) {  // V block transposed: 8 d values of one key per load
      const int e = tid + 256 * i, key = e / CH, c = e % CH;
      const int kr = min(kb * 64 + key, L - 1);
      const u32x4 v8 = *(const u32x4*)(V + (row0 + kr) * ld + col0 + 8 * c);
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int d = 8 * c + j;
        sV[swz8(d, key >> 3) * 8 + (key & 7)] = (uint16_t)(v8[j >> 1] >> (16 * (j & 1)));
      }
    }
    __syncthreads();
    f4 sc[4];
    scores(kb, sc);
#pragma unroll
    for (int b = 0; b < 4; ++b)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int qr = (lane >> 4) * 4 + r, key = b * 16 + (lane & 15);
        p[swz8(qr, key >> 3) * 8 + (key & 7)] = f32_to_bf16_bits(expf(sc[b][r] - mrow[r]) * inv[r]);
      }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      const u32x4 pa = *(const u32x4*)&p[swz8(lane & 15, (lane >> 4) + 4 * c) * 8];
#pragma unroll
      for (int d = 0; d < DB; ++d)
        o[d] = mma_bf16(pa, *(const u32x4*)&sV[swz8(d * 16 + (lane & 15), (lane >> 4) + 4 * c) * 8], o[d]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int d = 0; d < DB; ++d)
#pragma unroll
    for (int r = 0; r < 4; ++r)
      if (qrow + r < L) O[(row0 + qrow + r) * ldo + col0 + d * 16 + (lane & 15)] = f32_to_bf16_bits(o[d][r]);
}

bool aligned(const void* ws) { return (reinterpret_cast<uintptr_t>(ws) % kAlign) == 0; }
bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) % 16) == 0; }

int act_zeros(const duo_act_rule& r, int64_t k) {
  if (r.kind == DUO_ACT_NONE) return 0;
  return (int)std::floor(r.sparsity * (double)k + 0.5);
}

}  // namespace

extern "C" {

size_t duo_block_workspace_size(int32_t op, int64_t m, int64_t seq_len, int64_t heads) {
  switch (op) {
    case DUO_BOP_ACT_SPARSIFY: return m < 1 ? 0 : (size_t)rup(m * (int64_t)sizeof(int64_t), kAlign);
    case DUO_BOP_LINEAR: return 0;  // no scratch memory
    case DUO_BOP_ATTENTION: return 0;  // no scratch memory
    default: return 0;
  }
}

duo_status duo_rmsnorm(const void* X, int64_t m, int64_t d, int64_t ldx, double eps, void* Y, int64_t ldy,
                       void* stream) {
  if (m < 0 || d < 1 || ldx < d || ldy < d || !(eps >= 0.0) || !std::isfinite(eps)) return DUO_ERR_INVALID_ARG;
  if (m == 0) return DUO_OK;
  if (!X || !Y || m > INT32_MAX) return DUO_ERR_INVALID_ARG;
  if (duo_status d = device_ok(); d != DUO_OK) return d;
  hipLaunchKernelGGL(rmsnorm_kernel, dim3((unsigned)m), dim3(256), 0, (hipStream_t)stream, (const uint16_t*)X, ldx,
                     (int)d, (float)eps, (uint16_t*)Y, ldy);
  DUO_LAUNCH_CHECK();
  return DUO_OK;
}

duo_status duo_act_sparsify(const void* X, int64_t m, int64_t k, int64_t ldx, duo_act_rule rule, void* Y, int64_t ldy,
                            void* ws, size_t ws_bytes, void* stream) {
  if (m < 0 || k < 1 || k > kMaxK || ldx < k || ldy < k) return DUO_ERR_INVALID_ARG;
  if (rule.kind != DUO_ACT_NONE &&
      !(rule.kind == DUO_ACT_TOPK_MAG_PER_TOKEN && std::isfinite(rule.sparsity) && rule.sparsity >= 0.0 &&
        rule.sparsity <= 1.0))
    return DUO_ERR_INVALID_ARG;
  if (m == 0) return DUO_OK;
  if (!X || !Y || m > INT32_MAX) return DUO_ERR_INVALID_ARG;
  const size_t need = duo_block_workspace_size(DUO_BOP_ACT_SPARSIFY, m, 0, 0);
  if (!ws || ws_bytes < need || !aligned(ws)) return DUO_ERR_WORKSPACE;
  if (duo_status d = device_ok(); d != DUO_OK) return d;
  hipStream_t s = (hipStream_t)stream;
  int64_t* thr = (int64_t*)ws;
  duo_status st = act_threshold_run(X, DUO_BF16, m, k, ldx, act_zeros(rule, k), thr, s);
  if (st != DUO_OK) return st;
  const int64_t tot = m * k;
  if (k % 8 == 0 && ldx % 8 == 0 && ldy % 8 == 0 && aligned16(X) && aligned16(Y) && m * cdiv(k, 2048) <= INT32_MAX)
    hipLaunchKernelGGL(act_apply8_kernel, dim3((unsigned)(m * cdiv(k, 2048))), dim3(256), 0, s,
                       (const uint16_t*)X, ldx, (int)k, (const int64_t*)thr, (uint16_t*)Y, ldy);
  else
    hipLaunchKernelGGL(act_apply_kernel, dim3((unsigned)cdiv(tot, 256)), dim3(256), 0, s, (const uint16_t*)X, ldx,
                       (int)m, (int)k, (const int64_t*)thr, (uint16_t*)Y, ldy);
  DUO_LAUNCH_CHECK();
  return DUO_OK;
}

duo_status duo_linear(const void* X, int64_t m, int64_t k, int64_t ldx, const void* W, int64_t n, int64_t ldw,
                      const void* R, int64_t ldr, void* Y, int64_t ldy, void* ws, size_t ws_bytes, void* stream) {
  (void)ws;
  (void)ws_bytes;
  if (m < 0 || k < 1 || n < 1 || ldx < k || ldw < k || ldy < n || (R && ldr < n)) return DUO_ERR_INVALID_ARG;
  if (m > INT32_MAX || n > INT32_MAX || k > INT32_MAX || m * n > ((int64_t)1 << 40)) return DUO_ERR_UNSUPPORTED;
  if (m == 0) return DUO_OK;
  if (!X || !W || !Y) return DUO_ERR_INVALID_ARG;
  if (duo_status d = device_ok(); d != DUO_OK) return d;
  const hipStream_t s = (hipStream_t)stream;
  const bool vec = k % 8 == 0 && ldx % 8 == 0 && ldw % 8 == 0 && aligned16(X) && aligned16(W);
  if (vec) {
    const int64_t tiles = cdiv(m, kLinT) * cdiv(n, kLinT);
    if (tiles > INT32_MAX) return DUO_ERR_UNSUPPORTED;
    hipLaunchKernelGGL(lin_kernel, dim3((unsigned)rup(tiles, 8)), dim3(256), 0, s, (const uint16_t*)X, ldx,
                       (const uint16_t*)W, ldw, (const uint16_t*)R, ldr, (uint16_t*)Y, ldy, (int)m, (int)n, (int)k);
  } else {
    hipLaunchKernelGGL(lin_plain_kernel, dim3((unsigned)cdiv(m * n, 256)), dim3(256), 0, s, (const uint16_t*)X, ldx,
                       (const uint16_t*)W, ldw, (const uint16_t*)R, ldr, (uint16_t*)Y, ldy, (int)m, (int)n, (int)k);
  }
  DUO_LAUNCH_CHECK();
  return DUO_OK;
}

duo_status duo_rope(void* X, int64_t m, int64_t heads, int64_t head_dim, int64_t ldx, int64_t seq_len, double theta,
                    void* stream) {
  if (m < 0 || heads < 1 || head_dim < 2 || (head_dim & 1) || ldx < heads * head_dim || seq_len < 1 ||
      !(theta > 0.0) || !std::isfinite(theta))
    return DUO_ERR_INVALID_ARG;
  if (m == 0) return DUO_OK;
  if (!X || m > INT32_MAX) return DUO_ERR_INVALID_ARG;
  if (duo_status d = device_ok(); d != DUO_OK) return d;
  hipLaunchKernelGGL(rope_kernel, dim3((unsigned)m), dim3(256), 0, (hipStream_t)stream, (uint16_t*)X, ldx, (int)heads,
                     (int)head_dim, (int)seq_len, theta);
  DUO_LAUNCH_CHECK();
  return DUO_OK;
}

duo_status duo_attention(const void* Q, const void* K, const void* V, int64_t ld, int64_t nseq, int64_t seq_len,
                         int64_t heads, int64_t head_dim, void* O, int64_t ldo, void* ws, size_t ws_bytes,
                         void* stream) {
  (void)ws;
  (void)ws_bytes;
  if (nseq < 0 || seq_len < 1 || heads < 1 || head_dim < 1 || ld < heads * head_dim || ldo < heads * head_dim)
    return DUO_ERR_INVALID_ARG;
  if (head_dim != 64 && head_dim != 128) return DUO_ERR_UNSUPPORTED;
  if (seq_len > INT32_MAX || ld > INT32_MAX || ldo > INT32_MAX || nseq * heads * cdiv(seq_len, 64) > INT32_MAX)
    return DUO_ERR_UNSUPPORTED;
  if (nseq == 0) return DUO_OK;
  if (!Q || !K || !V || !O) return DUO_ERR_INVALID_ARG;
  if (ld % 8 != 0 || !aligned16(Q) || !aligned16(K) || !aligned16(V)) return DUO_ERR_UNSUPPORTED;
  if (duo_status d = device_ok(); d != DUO_OK) return d;
  const hipStream_t s = (hipStream_t)stream;
  const float scale = 1.0f / std::sqrt((float)head_dim);
  const int nqb = (int)cdiv(seq_len, 64);
  const dim3 grid((unsigned)(nseq * heads * nqb));
  if (head_dim == 128)
    hipLaunchKernelGGL(attn_kernel<128>, grid, dim3(256), 0, s, (const uint16_t*)Q, (const uint16_t*)K,
                       (const uint16_t*)V, ld, (int)seq_len, (int)heads, scale, (uint16_t*)O, ldo, nqb);
  else
    hipLaunchKernelGGL(attn_kernel<64>, grid, dim3(256), 0, s, (const uint16_t*)Q, (const uint16_t*)K,
                       (const uint16_t*)V, ld, (int)seq_len, (int)heads, scale, (uint16_t*)O, ldo, nqb);
  DUO_LAUNCH_CHECK();
  return DUO_OK;
}

duo_status duo_silu_mul(const void* G, const void* U, int64_t m, int64_t n, int64_t ld, void* Y, int64_t ldy,
                        void* stream) {
  if (m < 0 || n < 1 || ld < n || ldy < n) return DUO_ERR_INVALID_ARG;
  if (m == 0) return DUO_OK;
  if (!G || !U || !Y) return DUO_ERR_INVALID_ARG;
  if (duo_status d = device_ok(); d != DUO_OK) return d;
  const int64_t tot = m * n;
  if (n % 8 == 0 && ld % 8 == 0 && ldy % 8 == 0 && aligned16(G) && aligned16(U) && aligned16(Y) &&
      m * cdiv(n, 2048) <= INT32_MAX)
    hipLaunchKernelGGL(silu_mul8_kernel, dim3((unsigned)(m * cdiv(n, 2048))), dim3(256), 0,
                       (hipStream_t)stream, (const uint16_t*)G, (const uint16_t*)U, ld, (int)n, (uint16_t*)Y, ldy);
  else
    hipLaunchKernelGGL(silu_mul_kernel, dim3((unsigned)cdiv(tot, 256)), dim3(256), 0, (hipStream_t)stream,
                       (const uint16_t*)G, (const uint16_t*)U, ld, (int)m, (int)n, (uint16_t*)Y, ldy);
  DUO_LAUNCH_CHECK();
  return DUO_OK;
}

}  // extern "C"
