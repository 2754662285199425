// Stage 1 of the DuoGPT layer solver on gfx950: per-token activation
// sparsification and accumulation of H = Xh Xh^T, G = dX Xh^T and
// a = diag(dX dX^T) (paper Sec. 4.2-4.3, Algorithm 1 first lines).
//
// Pipeline per chunk of tokens:
//   act_select  one workgroup per token finds the largest dropped key
//               (|x|, channel) by bisection on the magnitude bits;
//   pack        applies the per-token threshold and writes Xh and dX (and,
//               for two input streams, the low part of dX) in an MFMA-ready
//               token-blocked layout [token block][group][channel][16 bytes];
//               also sums dX^2 per channel;
//   gram        MFMA kernel over pairs of 128-channel tiles (i >= j): one
//               pass over the tokens yields H_ij, G_ij and G_ji;
//   reductions  fixed-order sums of per-segment partials (deterministic).
#include <hip/hip_runtime.h>

#include "common.h"
#include "internal.h"

namespace duo {

// ---------------------------------------------------------------------------
// element traits
// ---------------------------------------------------------------------------
template <typename T>
struct Elem;
template <>
struct Elem<uint16_t> {  // bf16 stored as raw bits
  static constexpr int kMagBits = 15;
  __device__ static inline uint32_t mag(uint16_t v) { return v & 0x7fffu; }
  __device__ static inline float to_f32(uint16_t v) { return bf16_bits_to_f32(v); }
  __device__ static inline uint16_t from_f32(float f) { return f32_to_bf16_bits(f); }
};
template <>
struct Elem<float> {
  static constexpr int kMagBits = 31;
  __device__ static inline uint32_t mag(float v) { return __float_as_uint(v) & 0x7fffffffu; }
  __device__ static inline float to_f32(float v) { return v; }
  __device__ static inline float from_f32(float f) { return f; }
};

// ---------------------------------------------------------------------------
// block-wide helpers for 256 threads
// ---------------------------------------------------------------------------
__device__ inline int wave_sum(int v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// Sum over the 256 threads; `red` is LDS int[8], `slot` alternates 0/1 so a
// single barrier per call is enough.
__device__ inline int block_sum256(int v, int* red, int slot) {
  v = wave_sum(v);
  if ((threadIdx.x & 63) == 0) red[slot * 4 + (threadIdx.x >> 6)] = v;
  __syncthreads();
  return red[slot * 4] + red[slot * 4 + 1] + red[slot * 4 + 2] + red[slot * 4 + 3];
}

// ---------------------------------------------------------------------------
// act_select: per-token threshold key.  Element (t, c) is kept iff
// (mag(x) << 32 | c) > thr[t] (signed compare).  thr = -1 keeps everything,
// INT64_MAX drops everything.
// ---------------------------------------------------------------------------
template <typename T, int C>
__global__ __launch_bounds__(256) void act_select_kernel(const T* __restrict__ X, int64_t ldx, int m,
                                                         int k, int z, int64_t* __restrict__ thr) {
  __shared__ int red[8];
  __shared__ int scan[4];
  const int t = blockIdx.x;
  if (t >= m) return;
  if (z <= 0 || z >= k) {
    if (threadIdx.x == 0) thr[t] = z <= 0 ? (int64_t)-1 : INT64_MAX;
    return;
  }
  const T* row = X + (int64_t)t * ldx;
  const int c0 = threadIdx.x * C;
  uint32_t mag[C];
#pragma unroll
  for (int e = 0; e < C; ++e) {
    const int c = c0 + e;
    mag[e] = c < k ? Elem<T>::mag(row[c]) : 0xffffffffu;
  }
  // smallest v with count(mag <= v) >= z
  uint32_t lo = 0, hi = (1u << Elem<T>::kMagBits) - 1u;
  int slot = 0;
  while (lo < hi) {
    const uint32_t mid = lo + ((hi - lo) >> 1);
    int cnt = 0;
#pragma unroll
    for (int e = 0; e < C; ++e) cnt += mag[e] <= mid;
    cnt = block_sum256(cnt, red, slot);
    slot ^= 1;
    if (cnt >= z)
      hi = mid;
    else
      lo = mid + 1;
  }
  const uint32_t v = lo;
  int lt = 0, eq = 0;
#pragma unroll
  for (int e = 0; e < C; ++e) {
    lt += mag[e] < v;
    eq += mag[e] == v;
  }
  lt = block_sum256(lt, red, slot);
  const int r = z - lt;  // 1 <= r <= (number of ties)
  // exclusive prefix of tie counts in channel order
  int incl = eq;
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(incl, o);
    if (lane >= o) incl += y;
  }
  if (lane == 63) scan[threadIdx.x >> 6] = incl;
  __syncthreads();
  int base = 0;
  for (int w = 0; w < (int)(threadIdx.x >> 6); ++w) base += scan[w];
  const int excl = base + incl - eq;
  if (eq > 0 && excl < r && r <= excl + eq) {
    int need = r - excl;
#pragma unroll
    for (int e = 0; e < C; ++e) {
      if (mag[e] == v) {
        if (--need == 0) thr[t] = ((int64_t)v << 32) | (int64_t)(c0 + e);
      }
    }
  }
}

template <typename T>
static duo_status launch_act_select(const T* X, int64_t ldx, int m, int k, int z, int64_t* thr,
                                    hipStream_t s) {
  if (m <= 0) return DUO_OK;
  const int per = (int)cdiv(k, 256);
  dim3 g(m), b(256);
#define DUO_SEL(CC) hipLaunchKernelGGL((act_select_kernel<T, CC>), g, b, 0, s, X, ldx, m, k, z, thr)
  if (per <= 1)
    DUO_SEL(1);
  else if (per <= 2)
    DUO_SEL(2);
  else if (per <= 4)
    DUO_SEL(4);
  else if (per <= 8)
    DUO_SEL(8);
  else if (per <= 16)
    DUO_SEL(16);
  else if (per <= 32)
    DUO_SEL(32);
  else if (per <= 64)
    DUO_SEL(64);
  else
    DUO_SEL(128);
#undef DUO_SEL
  DUO_LAUNCH_CHECK();
  return DUO_OK;
}

// ---------------------------------------------------------------------------
// mask export (test hook): bit c of token t = kept
// ---------------------------------------------------------------------------
template <typename T>
__global__ void act_mask_kernel(const T* __restrict__ X, int64_t ldx, int m, int k,
                                const int64_t* __restrict__ thr, uint32_t* __restrict__ mask) {
  const int words = (int)cdiv(k, 32);
  const int64_t id = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (id >= (int64_t)m * words) return;
  const int t = (int)(id / words), w = (int)(id % words);
  const int64_t th = thr[t];
  uint32_t bits = 0;
  for (int e = 0; e < 32; ++e) {
    const int c = w * 32 + e;
    if (c >= k) break;
    const int64_t key = ((int64_t)Elem<T>::mag(X[(int64_t)t * ldx + c]) << 32) | c;
    if (key > th) bits |= 1u << e;
  }
  mask[id] = bits;
}

// ---------------------------------------------------------------------------
// pack: 256 channels x 256 tokens per workgroup, in 8 tiles of 32 tokens.
// Packed layout (EPG = 16 / sizeof(T) elements per group, NG = 32 / EPG):
//   P[((tb * NG + g) * kp + c) * EPG + e]  = value of token tb*32 + g*EPG + e.
// apart[tokens/256 block][kp] receives per-channel partial sums of dX^2.
// ---------------------------------------------------------------------------
template <typename T, bool TWO>
__global__ __launch_bounds__(256) void pack_kernel(const T* __restrict__ Xs, const T* __restrict__ Xd,
                                                   int64_t ldx, int mc, int k, int kp,
                                                   const int64_t* __restrict__ thr, T* __restrict__ Ph,
                                                   T* __restrict__ Pz, T* __restrict__ Pl,
                                                   float* __restrict__ apart) {
  constexpr int EPG = 16 / (int)sizeof(T);
  constexpr int NG = kTokBlk / EPG;
  constexpr bool LO = TWO && sizeof(T) == 2;  // bf16 two-stream: dX = hi + lo
  constexpr int RS = kTokBlk + EPG;           // LDS row stride (elements)
  constexpr int NSLOT = LO ? 3 : 2;
  constexpr int STAGE = NSLOT * 256 * RS * (int)sizeof(T);
  constexpr int RED = 32 * 257 * (int)sizeof(float);
  __shared__ __attribute__((aligned(16))) uint8_t raw[STAGE > RED ? STAGE : RED];
  T* sh = (T*)raw;
  T* sz = sh + 256 * RS;
  T* sl = sz + 256 * RS;
  float* sa = (float*)raw;  // reused after the token loop

  const int cb0 = blockIdx.x * 256;
  const int tsb = blockIdx.y * 256;
  const int tr = threadIdx.x >> 3;        // token row inside a 32-token tile
  const int cg = (threadIdx.x & 7) * 32;  // first of 32 channels
  const T zero = Elem<T>::from_f32(0.f);
  float acc[32];
#pragma unroll
  for (int e = 0; e < 32; ++e) acc[e] = 0.f;

  for (int tt = 0; tt < 8; ++tt) {
    const int tok0 = tsb + tt * kTokBlk;
    if (tok0 >= mc) break;  // uniform
    const int t = tok0 + tr;
    const bool tok_ok = t < mc;
    const int64_t th = tok_ok ? thr[t] : INT64_MAX;
#pragma unroll 8
    for (int e = 0; e < 32; ++e) {
      const int c = cb0 + cg + e;
      float d = 0.f;
      T vh = zero, vz = zero, vl = zero;
      if (tok_ok && c < k) {
        const T x = Xs[(int64_t)t * ldx + c];
        const int64_t key = ((int64_t)Elem<T>::mag(x) << 32) | c;
        const bool keep = key > th;
        vh = keep ? x : zero;
        if (TWO) {
          d = Elem<T>::to_f32(Xd[(int64_t)t * ldx + c]) - Elem<T>::to_f32(vh);
          vz = Elem<T>::from_f32(d);
          if (LO) vl = Elem<T>::from_f32(d - Elem<T>::to_f32(vz));
        } else {
          vz = keep ? zero : x;
          d = Elem<T>::to_f32(vz);
        }
      }
      acc[e] += d * d;
      sh[(cg + e) * RS + tr] = vh;
      sz[(cg + e) * RS + tr] = vz;
      if (LO) sl[(cg + e) * RS + tr] = vl;
    }
    __syncthreads();
    const int c = cb0 + threadIdx.x;
    if (c < kp) {
      const int tb = tok0 / kTokBlk;
#pragma unroll
      for (int g = 0; g < NG; ++g) {
        const int64_t off = (((int64_t)tb * NG + g) * kp + c) * EPG;
        *(uint4*)(Ph + off) = *(const uint4*)&sh[threadIdx.x * RS + g * EPG];
        *(uint4*)(Pz + off) = *(const uint4*)&sz[threadIdx.x * RS + g * EPG];
        if (LO) *(uint4*)(Pl + off) = *(const uint4*)&sl[threadIdx.x * RS + g * EPG];
      }
    }
    __syncthreads();
  }
  // per-channel sum of dX^2 over this block's tokens, fixed order
#pragma unroll
  for (int e = 0; e < 32; ++e) sa[tr * 257 + cg + e] = acc[e];
  __syncthreads();
  const int c = cb0 + threadIdx.x;
  if (apart && c < kp) {
    float s = 0.f;
    for (int r = 0; r < 32; ++r) s += sa[r * 257 + threadIdx.x];
    apart[(int64_t)blockIdx.y * kp + c] = s;
  }
}

__global__ void a_reduce_kernel(const float* __restrict__ apart, int nblk, int kp, int k,
                                float* __restrict__ a) {
  const int c = blockIdx.x * blockDim.x + threadIdx.x;
  if (c >= k) return;
  float s = 0.f;
  for (int b = 0; b < nblk; ++b) s += apart[(int64_t)b * kp + c];
  a[c] += s;
}

// ---------------------------------------------------------------------------
// gram: MFMA over a pair of 128-channel tiles (ti >= tj).
// ---------------------------------------------------------------------------
template <typename T>
struct GramArgs {
  const T* Ph;
  const T* Pz;
  const T* Pl;
  int kp, k, ntile, npairs, nseg, seg_len, ntb;
  float* H;
  int64_t ldh;
  float* G;
  int64_t ldg;
  float* part;  // [nseg][npairs][3][128*128] when nseg > 1
};

// Pair order: bands of 8 tile-rows; inside a band, column by column.  Neighbouring
// ids share operand tiles, and the XCD remap below gives each XCD a contiguous
// id range, so concurrently resident workgroups of one XCD reuse its L2.
__device__ inline void band_pair(int q, int T, int* ti, int* tj) {
  constexpr int GB = 8;
  for (int b0 = 0; b0 < T; b0 += GB) {
    const int b1 = min(T, b0 + GB), h = b1 - b0;
    const int cnt = b0 * h + h * (h + 1) / 2;  // columns < b0: h rows each; then a triangle
    if (q < cnt) {
      if (q < b0 * h) {
        *tj = q / h;
        *ti = b0 + q % h;
        return;
      }
      q -= b0 * h;
      for (int c = b0; c < b1; ++c) {
        const int nr = b1 - c;
        if (q < nr) {
          *tj = c;
          *ti = c + q;
          return;
        }
        q -= nr;
      }
    }
    q -= cnt;
  }
  *ti = *tj = 0;
}

__device__ inline int xcd_remap(int b, int nblocks) {
  const int per = (nblocks + 7) / 8;
  return (b % 8) * per + b / 8;
}

typedef unsigned int v4u __attribute__((ext_vector_type(4)));

template <typename T>
struct MfmaOp;
template <>
struct MfmaOp<uint16_t> {
  // one 16x16x32 bf16 MFMA per 16-row fragment pair per 32-token stage
  static constexpr int kFrags = 1;
  __device__ static inline f4 mma(const v4u& a, const v4u& b, f4 c) {
    bf16x8 av, bv;
    __builtin_memcpy(&av, &a, 16);
    __builtin_memcpy(&bv, &b, 16);
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, bv, c, 0, 0, 0);
  }
};
template <>
struct MfmaOp<float> {
  // eight 16x16x4 fp32 MFMAs: fragment s holds tokens of group s*4 + lane/16
  static constexpr int kFrags = 2;
  __device__ static inline f4 mma(const v4u& a, const v4u& b, f4 c) {
    const float* x = (const float*)&a;
    const float* y = (const float*)&b;
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(x[0], y[0], c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(x[1], y[1], c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(x[2], y[2], c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(x[3], y[3], c, 0, 0, 0);
    return c;
  }
};

template <typename T, bool WANT_H, bool WANT_G, bool HAS_LO>
__global__ __launch_bounds__(256, 1) void gram_kernel(GramArgs<T> A) {
  constexpr int EPG = 16 / (int)sizeof(T);
  constexpr int NG = kTokBlk / EPG;
  constexpr int TILE_B = kTile * kTokBlk * (int)sizeof(T);  // bytes of one operand tile
  constexpr int NOPS = 2 + (HAS_LO ? 1 : 0);               // Xh, Zhi, Zlo per side
  constexpr int STAGE_B = 2 * NOPS * TILE_B;
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];

  const int nunits = A.npairs * A.nseg;
  const int u = xcd_remap(blockIdx.x, gridDim.x);
  if (u >= nunits) return;
  const int seg = u / A.npairs;
  const int pair = u % A.npairs;
  int ti, tj;
  band_pair(pair, A.ntile, &ti, &tj);
  const bool diag = ti == tj;
  const int tb0 = seg * A.seg_len;
  const int tb1 = min(A.ntb, tb0 + A.seg_len);

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wi = wave >> 1, wj = wave & 1;

  // One operand tile = NG planes of 128 rows x 16 bytes; the plane stride in
  // global memory is kp * 16 bytes, in LDS 128 * 16 bytes.
  constexpr int CHUNKS = TILE_B / 16;
  constexpr int PER_T = CHUNKS / 256;
  const v4u* gbase[2][NOPS];
#pragma unroll
  for (int side = 0; side < 2; ++side)
#pragma unroll
    for (int o = 0; o < NOPS; ++o) {
      const T* b = o == 0 ? A.Ph : o == 1 ? A.Pz : A.Pl;
      gbase[side][o] = (const v4u*)(b + (int64_t)(side ? tj : ti) * kTile * EPG);
    }
  const int64_t tb_stride = (int64_t)NG * A.kp;  // v4u per token block
  int64_t goff[PER_T];
#pragma unroll
  for (int q = 0; q < PER_T; ++q) {
    const int ch = q * 256 + tid;
    goff[q] = (int64_t)(ch / kTile) * A.kp + ch % kTile;
  }
  v4u pre0[NOPS][PER_T], pre1[NOPS][PER_T];

  f4 accH[4][4], accG1[4][4], accG2[4][4];
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      accH[a][b] = f4{0.f, 0.f, 0.f, 0.f};
      accG1[a][b] = accH[a][b];
      accG2[a][b] = accH[a][b];
    }

#define DUO_LOAD_STAGE(TB)                                                          \
  {                                                                                 \
    const int64_t tbo_ = (int64_t)(TB) * tb_stride;                                 \
    _Pragma("unroll") for (int o = 0; o < NOPS; ++o)                                \
    _Pragma("unroll") for (int q = 0; q < PER_T; ++q)                               \
      pre0[o][q] = gbase[0][o][tbo_ + goff[q]];                                     \
    if (!diag) {                                                                    \
      _Pragma("unroll") for (int o = 0; o < NOPS; ++o)                              \
      _Pragma("unroll") for (int q = 0; q < PER_T; ++q)                             \
        pre1[o][q] = gbase[1][o][tbo_ + goff[q]];                                   \
    }                                                                               \
  }
#define DUO_STORE_STAGE(BUF)                                                        \
  {                                                                                 \
    v4u* dst_ = (v4u*)(smem + (BUF) * STAGE_B);                                  \
    _Pragma("unroll") for (int o = 0; o < NOPS; ++o)                                \
    _Pragma("unroll") for (int q = 0; q < PER_T; ++q)                               \
      dst_[o * CHUNKS + q * 256 + tid] = pre0[o][q];                                \
    if (!diag) {                                                                    \
      _Pragma("unroll") for (int o = 0; o < NOPS; ++o)                              \
      _Pragma("unroll") for (int q = 0; q < PER_T; ++q)                             \
        dst_[(NOPS + o) * CHUNKS + q * 256 + tid] = pre1[o][q];                     \
    }                                                                               \
  }

  const int side_j = diag ? 0 : 1;
  if (tb0 < tb1) {
    DUO_LOAD_STAGE(tb0);
    DUO_STORE_STAGE(0);
    __syncthreads();
    int buf = 0;
    for (int tb = tb0; tb < tb1; ++tb) {
      const bool more = tb + 1 < tb1;
      if (more) {
        DUO_LOAD_STAGE(tb + 1);
      }
      const v4u* lds = (const v4u*)(smem + buf * STAGE_B);
#pragma unroll
      for (int f = 0; f < MfmaOp<T>::kFrags; ++f) {
        const int fo = (f * 4 + (lane >> 4)) * kTile + (lane & 15);
        v4u hi_[4], hj_[4];
#pragma unroll
        for (int a = 0; a < 4; ++a) {
          hi_[a] = lds[(0 * NOPS + 0) * CHUNKS + fo + wi * 64 + a * 16];
          hj_[a] = lds[(side_j * NOPS + 0) * CHUNKS + fo + wj * 64 + a * 16];
        }
        if (WANT_H) {
#pragma unroll
          for (int a = 0; a < 4; ++a)
#pragma unroll
            for (int b = 0; b < 4; ++b) accH[a][b] = MfmaOp<T>::mma(hi_[a], hj_[b], accH[a][b]);
        }
        if (WANT_G) {
#pragma unroll
          for (int o = 1; o < NOPS; ++o) {
            v4u zi[4];
#pragma unroll
            for (int a = 0; a < 4; ++a) zi[a] = lds[(0 * NOPS + o) * CHUNKS + fo + wi * 64 + a * 16];
#pragma unroll
            for (int a = 0; a < 4; ++a)
#pragma unroll
              for (int b = 0; b < 4; ++b) accG1[a][b] = MfmaOp<T>::mma(zi[a], hj_[b], accG1[a][b]);
            if (!diag) {
              v4u zj[4];
#pragma unroll
              for (int a = 0; a < 4; ++a) zj[a] = lds[(1 * NOPS + o) * CHUNKS + fo + wj * 64 + a * 16];
#pragma unroll
              for (int a = 0; a < 4; ++a)
#pragma unroll
                for (int b = 0; b < 4; ++b) accG2[a][b] = MfmaOp<T>::mma(zj[a], hi_[b], accG2[a][b]);
            }
          }
        }
      }
      if (more) {
        DUO_STORE_STAGE(buf ^ 1);
        __syncthreads();
        buf ^= 1;
      }
    }
  }
#undef DUO_LOAD_STAGE
#undef DUO_STORE_STAGE

  // epilogue.  Accumulator element r of block (a, b) sits at row
  // 16a + 4*(lane/16) + r, column 16b + lane%16 of the wave's 64 x 64 sub-tile.
  const int i0 = ti * kTile, j0 = tj * kTile;
  const int rq = (lane >> 4) * 4, cc = lane & 15;
  if (A.nseg > 1) {
    float* base = A.part + ((int64_t)seg * A.npairs + pair) * 3 * kTile * kTile;
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
      for (int b = 0; b < 4; ++b)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int rowl = wi * 64 + a * 16 + rq + r, coll = wj * 64 + b * 16 + cc;
          if (WANT_H) base[rowl * kTile + coll] = accH[a][b][r];
          if (WANT_G) {
            base[kTile * kTile + rowl * kTile + coll] = accG1[a][b][r];
            // G_ji block: rows are j channels (wj half), columns i channels (wi half)
            const int rowj = wj * 64 + a * 16 + rq + r, coli = wi * 64 + b * 16 + cc;
            base[2 * kTile * kTile + rowj * kTile + coli] = accG2[a][b][r];
          }
        }
    return;
  }
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int b = 0; b < 4; ++b)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = i0 + wi * 64 + a * 16 + rq + r, col = j0 + wj * 64 + b * 16 + cc;
        if (row < A.k && col < A.k) {
          if (WANT_H) {
            A.H[(int64_t)row * A.ldh + col] += accH[a][b][r];
            if (!diag) A.H[(int64_t)col * A.ldh + row] += accH[a][b][r];
          }
          if (WANT_G) A.G[(int64_t)row * A.ldg + col] += accG1[a][b][r];
        }
        if (WANT_G && !diag) {
          const int rowj = j0 + wj * 64 + a * 16 + rq + r, coli = i0 + wi * 64 + b * 16 + cc;
          if (rowj < A.k && coli < A.k) A.G[(int64_t)rowj * A.ldg + coli] += accG2[a][b][r];
        }
      }
}

// Fixed-order sum of the per-segment partial tiles into H and G.
template <typename T>
__global__ __launch_bounds__(256) void gram_reduce_kernel(GramArgs<T> A, int want_h, int want_g) {
  const int pair = blockIdx.x / 3, which = blockIdx.x % 3;
  int ti, tj;
  band_pair(pair, A.ntile, &ti, &tj);
  const bool diag = ti == tj;
  if ((which == 0 && !want_h) || (which > 0 && !want_g) || (which == 2 && diag)) return;
  const int64_t stride = (int64_t)A.npairs * 3 * kTile * kTile;
  const float* p0 = A.part + ((int64_t)pair * 3 + which) * kTile * kTile;
  for (int e = threadIdx.x + blockIdx.y * 256 * 16; e < min(kTile * kTile, (int)(blockIdx.y + 1) * 256 * 16);
       e += 256) {
    float s = 0.f;
    for (int sg = 0; sg < A.nseg; ++sg) s += p0[sg * stride + e];
    const int rl = e / kTile, cl = e % kTile;
    if (which == 0) {
      const int row = ti * kTile + rl, col = tj * kTile + cl;
      if (row < A.k && col < A.k) {
        A.H[(int64_t)row * A.ldh + col] += s;
        if (!diag) A.H[(int64_t)col * A.ldh + row] += s;
      }
    } else if (which == 1) {
      const int row = ti * kTile + rl, col = tj * kTile + cl;
      if (row < A.k && col < A.k) A.G[(int64_t)row * A.ldg + col] += s;
    } else {
      const int row = tj * kTile + rl, col = ti * kTile + cl;
      if (row < A.k && col < A.k) A.G[(int64_t)row * A.ldg + col] += s;
    }
  }
}

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------
int64_t hessian_chunk_tokens(int64_t m, int64_t k) {
  const int64_t kp = rup(k, kTile);
  int64_t ch = (int64_t)12e9 / (kp * 8);
  ch = ch < 4096 ? 4096 : ch;
  ch = ch > 131072 ? 131072 : ch;
  ch = ch / 256 * 256;
  return m < ch ? (m < 1 ? 1 : m) : ch;
}

int gram_split(int64_t npairs) {
  int best = 1;
  double best_cost = 1e30;
  for (int s = 1; s <= 8; ++s) {
    const double cost = (double)cdiv(npairs * s, 256) / s + (s > 1 ? 0.03 * s : 0.0);
    if (cost < best_cost - 1e-12) {
      best_cost = cost;
      best = s;
    }
  }
  return best;
}

struct HessWs {
  int64_t* thr;
  uint8_t* Ph;
  uint8_t* Pz;
  uint8_t* Pl;
  float* apart;
  float* part;
  size_t bytes;
};

static HessWs carve_hessian(void* ws, int64_t m, int64_t k) {
  const int64_t ch = hessian_chunk_tokens(m, k);
  const int64_t kp = rup(k, kTile);
  const int64_t tokp = rup(ch, 256);
  const int64_t T = kp / kTile;
  const int64_t npairs = T * (T + 1) / 2;
  const int nseg = gram_split(npairs);
  Carver c(ws);
  HessWs h;
  h.thr = c.take<int64_t>(tokp);
  h.Ph = c.take<uint8_t>((size_t)tokp * kp * 4);  // sized for fp32; bf16 uses half
  h.Pz = c.take<uint8_t>((size_t)tokp * kp * 4);
  h.Pl = c.take<uint8_t>((size_t)tokp * kp * 2);  // low part exists for bf16 only
  h.apart = c.take<float>((size_t)(tokp / 256) * kp);
  h.part = c.take<float>(nseg > 1 ? (size_t)nseg * npairs * 3 * kTile * kTile : 1);
  h.bytes = c.off;
  return h;
}

size_t hessian_ws_bytes(int64_t m, int64_t k) { return carve_hessian(nullptr, m, k).bytes; }

template <typename T, bool WH, bool WG, bool LO>
static duo_status launch_gram(const GramArgs<T>& A, int nunits, hipStream_t s) {
  constexpr int NOPS = 2 + (LO ? 1 : 0);
  const size_t lds = 2 * 2 * NOPS * (size_t)kTile * kTokBlk * sizeof(T);
  auto kern = gram_kernel<T, WH, WG, LO>;
  DUO_HIP_TRY(hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds));
  const int grid = (int)rup(nunits, 8);
  hipLaunchKernelGGL(kern, dim3(grid), dim3(256), lds, s, A);
  DUO_LAUNCH_CHECK();
  return DUO_OK;
}

template <typename T>
static duo_status hessian_typed(const T* Xs, const T* Xd, int64_t m, int64_t k, int64_t ldx, int z,
                                float* H, int64_t ldh, float* G, int64_t ldg, float* a, void* ws,
                                bool want_h, hipStream_t s) {
  const bool want_g = G != nullptr;
  const bool two = Xd != nullptr && Xd != Xs;
  const bool lo = two && sizeof(T) == 2;
  const HessWs w = carve_hessian(ws, m, k);
  const int64_t ch = hessian_chunk_tokens(m, k);
  const int64_t kp = rup(k, kTile);
  const int T_ = (int)(kp / kTile);
  const int npairs = T_ * (T_ + 1) / 2;
  const int nseg = gram_split(npairs);
  for (int64_t t0 = 0; t0 < m; t0 += ch) {
    const int mc = (int)(m - t0 < ch ? m - t0 : ch);
    const T* xs = Xs + t0 * ldx;
    const T* xd = two ? Xd + t0 * ldx : nullptr;
    duo_status st = launch_act_select<T>(xs, ldx, mc, (int)k, z, w.thr, s);
    if (st != DUO_OK) return st;
    dim3 pg((unsigned)cdiv(kp, 256), (unsigned)cdiv(mc, 256));
    if (two)
      hipLaunchKernelGGL((pack_kernel<T, true>), pg, dim3(256), 0, s, xs, xd, ldx, mc, (int)k, (int)kp,
                         w.thr, (T*)w.Ph, (T*)w.Pz, (T*)w.Pl, want_g ? w.apart : nullptr);
    else
      hipLaunchKernelGGL((pack_kernel<T, false>), pg, dim3(256), 0, s, xs, xs, ldx, mc, (int)k, (int)kp,
                         w.thr, (T*)w.Ph, (T*)w.Pz, (T*)w.Pl, want_g ? w.apart : nullptr);
    DUO_LAUNCH_CHECK();
    if (want_g) {
      hipLaunchKernelGGL(a_reduce_kernel, dim3((unsigned)cdiv(k, 256)), dim3(256), 0, s, w.apart,
                         (int)cdiv(mc, 256), (int)kp, (int)k, a);
      DUO_LAUNCH_CHECK();
    }
    GramArgs<T> A;
    A.Ph = (const T*)w.Ph;
    A.Pz = (const T*)w.Pz;
    A.Pl = (const T*)w.Pl;
    A.kp = (int)kp;
    A.k = (int)k;
    A.ntile = T_;
    A.npairs = npairs;
    A.nseg = nseg;
    A.ntb = (int)cdiv(mc, kTokBlk);
    A.seg_len = (int)cdiv(A.ntb, nseg);
    A.H = H;
    A.ldh = ldh;
    A.G = G;
    A.ldg = ldg;
    A.part = w.part;
    const int nunits = npairs * nseg;
    prof_begin(DUO_PROF_GRAM, s);
    constexpr bool kLoOk = sizeof(T) == 2;  // the low part of dX exists for bf16 only
    if (want_h && want_g) {
      if constexpr (kLoOk)
        st = lo ? launch_gram<T, true, true, true>(A, nunits, s) : launch_gram<T, true, true, false>(A, nunits, s);
      else
        st = launch_gram<T, true, true, false>(A, nunits, s);
    } else if (want_h) {
      st = launch_gram<T, true, false, false>(A, nunits, s);
    } else {
      if constexpr (kLoOk)
        st = lo ? launch_gram<T, false, true, true>(A, nunits, s) : launch_gram<T, false, true, false>(A, nunits, s);
      else
        st = launch_gram<T, false, true, false>(A, nunits, s);
    }
    prof_end(DUO_PROF_GRAM, s);
    if (st != DUO_OK) return st;
    if (nseg > 1) {
      hipLaunchKernelGGL(gram_reduce_kernel<T>, dim3(npairs * 3, (kTile * kTile) / (256 * 16)), dim3(256), 0, s, A,
                         (int)want_h, (int)want_g);
      DUO_LAUNCH_CHECK();
    }
  }
  return DUO_OK;
}

duo_status hessian_run(const void* Xs, const void* Xd, int32_t dtype, int64_t m, int64_t k, int64_t ldx, int z,
                       float* H, int64_t ldh, float* G, int64_t ldg, float* a, void* ws, bool want_h,
                       hipStream_t s) {
  if (dtype == DUO_BF16)
    return hessian_typed<uint16_t>((const uint16_t*)Xs, (const uint16_t*)Xd, m, k, ldx, z, H, ldh, G, ldg, a,
                                   ws, want_h, s);
  return hessian_typed<float>((const float*)Xs, (const float*)Xd, m, k, ldx, z, H, ldh, G, ldg, a, ws, want_h,
                              s);
}

duo_status act_mask_run(const void* X, int32_t dtype, int64_t m, int64_t k, int64_t ldx, int z, uint32_t* mask,
                        void* ws, hipStream_t s) {
  const HessWs w = carve_hessian(ws, m, k);
  const int64_t ch = hessian_chunk_tokens(m, k);
  const int64_t words = cdiv(k, 32);
  for (int64_t t0 = 0; t0 < m; t0 += ch) {
    const int mc = (int)(m - t0 < ch ? m - t0 : ch);
    const int64_t n = mc * words;
    duo_status st;
    if (dtype == DUO_BF16) {
      const uint16_t* x = (const uint16_t*)X + t0 * ldx;
      st = launch_act_select<uint16_t>(x, ldx, mc, (int)k, z, w.thr, s);
      if (st != DUO_OK) return st;
      hipLaunchKernelGGL(act_mask_kernel<uint16_t>, dim3((unsigned)cdiv(n, 256)), dim3(256), 0, s, x, ldx, mc,
                         (int)k, (const int64_t*)w.thr, mask + t0 * words);
    } else {
      const float* x = (const float*)X + t0 * ldx;
      st = launch_act_select<float>(x, ldx, mc, (int)k, z, w.thr, s);
      if (st != DUO_OK) return st;
      hipLaunchKernelGGL(act_mask_kernel<float>, dim3((unsigned)cdiv(n, 256)), dim3(256), 0, s, x, ldx, mc, (int)k,
                         (const int64_t*)w.thr, mask + t0 * words);
    }
    DUO_LAUNCH_CHECK();
  }
  return DUO_OK;
}


}  // namespace duo
