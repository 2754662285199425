// fp32 MFMA GEMM for gfx950 used by the dense k^3 stages (inverse Cholesky,
// Q = G L, D = U L^T) and by the lazy trailing update of the column sweep.
//
// 128 x 128 output tile per 256-thread workgroup, 2 x 2 waves of 64 x 64
// (64 x 64 tiles for launches too small to fill the chip),
// v_mfma_f32_16x16x4_f32; K staged 32 at a time through LDS, with the global
// loads of the stage after next in flight during each multiply (fence-free
// barriers, so the prefetch is not drained at every stage).  Triangular operands are handled by restricting each
// tile's K range (tile-granular) and by tile filters (lower/upper only); the
// zeros inside diagonal tiles must be stored explicitly.
#include <hip/hip_runtime.h>

#include "internal.h"

namespace duo {

namespace {

constexpr int KT = 32;      // K per stage
constexpr int KS = KT + 2;  // stride of the k-contiguous LDS layout [row][KS] (operand loaded along k)

// Per tile edge TE (128, or 64 for launches too small to fill the chip):
// 2 x 2 waves of (TE/2)^2 outputs, NA x NA MFMA blocks of 16 x 16 per wave.
template <int TE>
struct Geo {
  static constexpr int LS = TE + 16;                            // stride of the k-major layout [k][LS]
  static constexpr int SLOT = TE * KS > KT * LS ? TE * KS : KT * LS;  // floats per operand per stage
  static constexpr int PQ = TE * KT / 1024;                    // float4 loads per thread per operand per stage
  static constexpr int TPR = TE / 4;                           // threads per k line in the k-major loads
  static constexpr int NA = TE / 32;                           // 16 x 16 blocks per wave and dimension
};

template <int TE>
struct Stage {
  float4 a[Geo<TE>::PQ];
  float4 b[Geo<TE>::PQ];
};

template <int TE>
__device__ inline int64_t lo_of(int mode, int i0, int j0) {
  return mode == KLO_ROW ? i0 : mode == KLO_COL ? j0 : 0;
}
template <int TE>
__device__ inline int64_t hi_of(int mode, int i0, int j0, int K) {
  const int64_t v = mode == KHI_ROW ? (int64_t)i0 + TE : mode == KHI_COL ? (int64_t)j0 + TE : K;
  return v < K ? v : K;
}

// Load 4 consecutive elements p[0..3] of a line whose valid index range is
// [lo, hi), starting at index `idx` (edge tiles and ragged stages only).
__device__ inline float4 load4(const float* p, int64_t idx, int64_t lo, int64_t hi, bool line_ok) {
  float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
  if (!line_ok) return v;
  if (idx + 0 >= lo && idx + 0 < hi) v.x = p[0];
  if (idx + 1 >= lo && idx + 1 < hi) v.y = p[1];
  if (idx + 2 >= lo && idx + 2 < hi) v.z = p[2];
  if (idx + 3 >= lo && idx + 3 < hi) v.w = p[3];
  return v;
}

// Workgroup barrier without the memory fence of __syncthreads: that fence
// would wait for the global prefetches in flight.  This wave's LDS traffic is
// drained first; the empty asm statements keep memory accesses on their side.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0)
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// One stage = KT values of K for TE rows of A and TE columns of B; each of
// the 256 threads moves PQ float4 of each operand.  FAST (uniform over the
// workgroup): the tile lies inside M x N, the stage inside [klo, khi) and
// both operands are 16-byte aligned, so every load is a plain 16-byte one.
template <int TE, bool AR, bool BR, bool FAST>
__device__ inline void load_stage(const GemmTerm& t, int M, int N, int i0, int j0, int64_t k0, int64_t klo,
                                  int64_t khi, Stage<TE>& st) {
  using G = Geo<TE>;
  const int tid = threadIdx.x;
#pragma unroll
  for (int q = 0; q < G::PQ; ++q) {
    if (AR) {  // A(i,l) = A[i*lda + l]: 4 consecutive l of one row
      const int row = (tid >> 3) + 32 * q, l4 = (tid & 7) * 4;
      const int64_t i = i0 + row, l = k0 + l4;
      st.a[q] = FAST ? *(const float4*)(t.A + i * t.lda + l) : load4(t.A + i * t.lda + l, l, klo, khi, i < M);
    } else {  // A(i,l) = A[l*lda + i]: 4 consecutive i of one l
      const int lr = tid / G::TPR + (256 / G::TPR) * q, i4 = (tid % G::TPR) * 4;
      const int64_t i = i0 + i4, l = k0 + lr;
      st.a[q] = FAST ? *(const float4*)(t.A + l * t.lda + i)
                     : load4(t.A + l * t.lda + i, i, 0, M, l >= klo && l < khi);
    }
    if (BR) {  // B(l,j) = B[l*ldb + j]: 4 consecutive j of one l
      const int lr = tid / G::TPR + (256 / G::TPR) * q, j4 = (tid % G::TPR) * 4;
      const int64_t j = j0 + j4, l = k0 + lr;
      st.b[q] = FAST ? *(const float4*)(t.B + l * t.ldb + j)
                     : load4(t.B + l * t.ldb + j, j, 0, N, l >= klo && l < khi);
    } else {  // B(l,j) = B[j*ldb + l]: 4 consecutive l of one column
      const int col = (tid >> 3) + 32 * q, l4 = (tid & 7) * 4;
      const int64_t j = j0 + col, l = k0 + l4;
      st.b[q] = FAST ? *(const float4*)(t.B + j * t.ldb + l) : load4(t.B + j * t.ldb + l, l, klo, khi, j < N);
    }
  }
}

template <int TE, bool AR, bool BR>
__device__ inline void load_stage_any(const GemmTerm& t, int M, int N, int i0, int j0, int64_t k0, int64_t klo,
                                      int64_t khi, bool fast_tile, Stage<TE>& st) {
  if (fast_tile && k0 + KT <= khi)
    load_stage<TE, AR, BR, true>(t, M, N, i0, j0, k0, klo, khi, st);
  else
    load_stage<TE, AR, BR, false>(t, M, N, i0, j0, k0, klo, khi, st);
}

// LDS layout per operand: an operand loaded 4 consecutive rows/columns at a
// time is stored k-major, [k][LS] (float4 stores); one loaded 4 consecutive k
// at a time is stored k-contiguous, [row][KS] (float2 stores), so that neither
// the stores nor the fragment reads meet bank conflicts (KS = 34: the 32
// lanes of a half-wave read rows 2 banks apart, at k and k+1; LS = TE + 16:
// the two k lines of a half-wave sit 16 banks apart).  alpha is folded into A.
template <int TE, bool AR, bool BR>
__device__ inline void store_stage(float* sA, float* sB, const Stage<TE>& st, float alpha) {
  using G = Geo<TE>;
  const int tid = threadIdx.x;
#pragma unroll
  for (int q = 0; q < G::PQ; ++q) {
    const float4 a = st.a[q];
    if (AR) {
      const int row = (tid >> 3) + 32 * q, l4 = (tid & 7) * 4;
      *(float2*)&sA[row * KS + l4] = make_float2(alpha * a.x, alpha * a.y);
      *(float2*)&sA[row * KS + l4 + 2] = make_float2(alpha * a.z, alpha * a.w);
    } else {
      const int lr = tid / G::TPR + (256 / G::TPR) * q, i4 = (tid % G::TPR) * 4;
      *(float4*)&sA[lr * G::LS + i4] = make_float4(alpha * a.x, alpha * a.y, alpha * a.z, alpha * a.w);
    }
    const float4 b = st.b[q];
    if (BR) {
      const int lr = tid / G::TPR + (256 / G::TPR) * q, j4 = (tid % G::TPR) * 4;
      *(float4*)&sB[lr * G::LS + j4] = b;
    } else {
      const int col = (tid >> 3) + 32 * q, l4 = (tid & 7) * 4;
      *(float2*)&sB[col * KS + l4] = make_float2(b.x, b.y);
      *(float2*)&sB[col * KS + l4 + 2] = make_float2(b.z, b.w);
    }
  }
}

template <int TE, bool AR, bool BR>
__device__ inline void compute_stage(const float* sA, const float* sB, f4 (&acc)[Geo<TE>::NA][Geo<TE>::NA]) {
  using G = Geo<TE>;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wi = wave >> 1, wj = wave & 1;
#pragma unroll
  for (int ks = 0; ks < KT / 4; ++ks) {
    const int kr = ks * 4 + (lane >> 4);
    float av[G::NA], bv[G::NA];
#pragma unroll
    for (int a = 0; a < G::NA; ++a) {
      const int r = wi * (TE / 2) + a * 16 + (lane & 15), c = wj * (TE / 2) + a * 16 + (lane & 15);
      av[a] = AR ? sA[r * KS + kr] : sA[kr * G::LS + r];
      bv[a] = BR ? sB[kr * G::LS + c] : sB[c * KS + kr];
    }
#pragma unroll
    for (int a = 0; a < G::NA; ++a)
#pragma unroll
      for (int b = 0; b < G::NA; ++b)
        acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[a], bv[b], acc[a][b], 0, 0, 0);
  }
}

// K loop of one term: stage s sits in LDS buffer s & 1; the global loads of
// stage s + 2 are in flight while stage s is multiplied (two register slots,
// the loop unrolled by two so that every slot index is static).
template <int TE, bool AR, bool BR>
__device__ inline void run_term(const GemmTerm& t, int M, int N, int i0, int j0, float* smem,
                                f4 (&acc)[Geo<TE>::NA][Geo<TE>::NA]) {
  constexpr int SLOT = Geo<TE>::SLOT;
  const int64_t klo = lo_of<TE>(t.klo, i0, j0);
  const int64_t khi = hi_of<TE>(t.khi, i0, j0, t.K);
  if (klo >= khi) return;
  const int nst = (int)((khi - klo + KT - 1) / KT);
  // klo is 0 or a tile start, so every stage start is a multiple of 4
  const bool fast_tile = i0 + TE <= M && j0 + TE <= N && ((reinterpret_cast<uintptr_t>(t.A) & 15) == 0) &&
                         ((reinterpret_cast<uintptr_t>(t.B) & 15) == 0) && (t.lda & 3) == 0 && (t.ldb & 3) == 0;
  float* sa[2] = {smem, smem + 2 * SLOT};
  float* sb[2] = {smem + SLOT, smem + 3 * SLOT};
  Stage<TE> st0, st1;
  load_stage_any<TE, AR, BR>(t, M, N, i0, j0, klo, klo, khi, fast_tile, st0);
  if (nst > 1) load_stage_any<TE, AR, BR>(t, M, N, i0, j0, klo + KT, klo, khi, fast_tile, st1);
  lds_barrier();  // earlier users of the LDS buffers are done
  store_stage<TE, AR, BR>(sa[0], sb[0], st0, t.alpha);
  lds_barrier();
#pragma nounroll
  for (int s = 0; s < nst; s += 2) {
    if (s + 2 < nst) load_stage_any<TE, AR, BR>(t, M, N, i0, j0, klo + (int64_t)(s + 2) * KT, klo, khi, fast_tile, st0);
    compute_stage<TE, AR, BR>(sa[0], sb[0], acc);
    if (s + 1 < nst) store_stage<TE, AR, BR>(sa[1], sb[1], st1, t.alpha);
    lds_barrier();
    if (s + 1 >= nst) break;
    if (s + 3 < nst) load_stage_any<TE, AR, BR>(t, M, N, i0, j0, klo + (int64_t)(s + 3) * KT, klo, khi, fast_tile, st1);
    compute_stage<TE, AR, BR>(sa[1], sb[1], acc);
    if (s + 2 < nst) store_stage<TE, AR, BR>(sa[0], sb[0], st0, t.alpha);
    lds_barrier();
  }
}

__device__ inline int xcd_remap_g(int b, int nblocks) {
  const int per = (nblocks + 7) / 8;
  return (b % 8) * per + b / 8;
}

// Tile (ti, tj) of the 128 grid with enumeration index pid (the triangular
// filters and the tile orders are defined on that grid).
__device__ inline void tile_of(const GemmDesc& d, int pid, int* ti, int* tj) {
  if (d.tri == TRI_ALL) {
    const int tn = (int)cdiv(d.N, kTile);
    if (d.order == ORDER_PLAIN && d.t[0].khi == KHI_COL && d.t[0].klo == KLO_ZERO) {
      // K range [0, j0 + 128): by columns, from the last (the longest) down.
      // (Row by row, the workgroups that share a CU in a launch of a few
      // waves, 256 ids apart, all held tiles of one column.)
      const int tm = (int)cdiv(d.M, kTile);
      *tj = tn - 1 - pid / tm;
      *ti = pid % tm;
      return;
    }
    *ti = pid / tn;
    *tj = pid % tn;
  } else if (d.tri == TRI_LOWER) {
    tri_pair(pid, ti, tj);
  } else if (d.order == ORDER_DIAG) {
    // group s holds the s + 1 tiles at distance T - 1 - s from the diagonal
    const int T = (int)cdiv(d.N, kTile);
    int sgrp, off;
    tri_pair(pid, &sgrp, &off);
    *ti = off;
    *tj = off + (T - 1 - sgrp);
  } else {
    tri_pair(pid, tj, ti);
  }
}

// Tiles are enumerated on the 128 grid (the triangular filters and the tile
// orders are defined there); with TE = 64 each 128 tile is split into its
// four quarters, which are consecutive ids.
template <int TE, bool A1R, bool B1R, bool A2R, bool B2R, bool TWO>
__global__ __launch_bounds__(256, 2) void gemm_kernel(GemmDesc d, int ntiles) {
  using G = Geo<TE>;
  constexpr int SUB = kTile / TE;  // tiles per 128 edge
  __shared__ __attribute__((aligned(16))) float smem[4 * G::SLOT];  // 2 buffers x (A, B)
  const int id = d.order == ORDER_XCD ? xcd_remap_g(blockIdx.x, gridDim.x) : (int)blockIdx.x;
  if (id >= ntiles) return;
  if (blockIdx.y) {
    const int64_t z = blockIdx.y;
    d.C += z * d.sC;
    d.t[0].A += z * d.sA[0];
    d.t[0].B += z * d.sB[0];
    d.t[1].A += z * d.sA[1];
    d.t[1].B += z * d.sB[1];
  }
  const int pid = id / (SUB * SUB), sub = id % (SUB * SUB);
  int ti, tj;  // on the 128 grid
  tile_of(d, pid, &ti, &tj);
  const int i0 = ti * kTile + (sub / SUB) * TE, j0 = tj * kTile + (sub % SUB) * TE;
  if (i0 >= d.M || j0 >= d.N) return;
  f4 acc[G::NA][G::NA];
#pragma unroll
  for (int a = 0; a < G::NA; ++a)
#pragma unroll
    for (int b = 0; b < G::NA; ++b) acc[a][b] = f4{0.f, 0.f, 0.f, 0.f};
  run_term<TE, A1R, B1R>(d.t[0], d.M, d.N, i0, j0, smem, acc);
  if (TWO) run_term<TE, A2R, B2R>(d.t[1], d.M, d.N, i0, j0, smem, acc);

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wi = wave >> 1, wj = wave & 1;
#pragma unroll
  for (int a = 0; a < G::NA; ++a)
#pragma unroll
    for (int b = 0; b < G::NA; ++b)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t i = i0 + wi * (TE / 2) + a * 16 + (lane >> 4) * 4 + r;
        const int64_t j = j0 + wj * (TE / 2) + b * 16 + (lane & 15);
        if (i < d.M && j < d.N) {
          float* c = d.C + i * d.ldc + j;
          *c = d.beta != 0.f ? d.beta * *c + acc[a][b][r] : acc[a][b][r];
        }
      }
}

// ---------------------------------------------------------------------------
// Fast path for launches whose tiles all lie inside M x N with 16-byte aligned
// operands (every DuoGPT product at k a multiple of 128): A row-major (K
// contiguous); B either K-contiguous (b_row = 0, "NT") or row-major (b_row = 1,
// "NN").  TF x TF tile (128, or 64 for launches too small to fill the chip),
// 2 x 2 waves of TF/2 x TF/2, K staged 32 at a time through two LDS stages
// filled by direct global->LDS loads (no register staging): the loads of
// stage s + 1 are in flight while stage s is multiplied.  The 128 tile needs
// about 150 VGPRs and 64 KB of LDS, so two workgroups share a CU (the 64
// tile: 32 KB, five): while one waits at a stage barrier or for its fragment
// reads, the other keeps the matrix core busy.  A stage is 128 MFMAs per
// wave on the 128 tile; 16-deep stages (a barrier every 64 MFMAs, three
// workgroups per CU) measured 1-4 % slower.
//
// K order inside a stage: MFMA step s (of 8) takes k = 8g + s in lane group g,
// so that a K-contiguous operand's fragment for all eight steps is two 16-byte
// chunks (k = 8g .. 8g + 7) per lane.  Both operands use the same order, so
// the sum is the same.  Layouts (16-byte chunks):
//   K-contiguous operand, TF lines x 8 chunks: chunk c of line r at
//     r * 8 + (c ^ ((r >> 1) & 7)), so the 16 lines of a fragment read hit 16
//     distinct bank groups (the 8 lines of each parity, 8 distinct positions);
//   row-major B, 32 k-rows x TF/4 chunks: chunk c of row k at
//     k * TF/4 + (c ^ (4 * ((k >> 3) & 3))), so the four lane groups (k eight
//     apart) read disjoint bank groups.
// ---------------------------------------------------------------------------
constexpr int FK = 32;       // K per stage
constexpr int FCH = FK / 4;  // 16-byte chunks per K-contiguous line = MFMA steps per stage
constexpr int FEP = 64;      // tile rows per epilogue pass

template <int TF>
struct FGeo {
  static constexpr int OP = TF * FK * 4;    // bytes per operand per stage
  static constexpr int STAGE = 2 * OP;
  static constexpr int Q = TF * FK / 1024;  // 16-byte chunks per thread per operand per stage
  static constexpr int NB = TF / 32;        // 16 x 16 blocks per wave and dimension
  static constexpr int HW = TF / 2;         // wave tile edge
  static constexpr int OCC = TF == kTile ? 2 : 5;  // workgroups per CU
  static constexpr size_t EPI = (size_t)FEP * (TF + 4) * 4;
  static constexpr size_t LDS = (size_t)2 * STAGE > EPI ? (size_t)2 * STAGE : EPI;
  static_assert(LDS * OCC <= 160 * 1024, "fast-path LDS");
};

// chunk positions: K-contiguous line r, row-major B row k
__device__ __forceinline__ int swa(int r) { return (r >> 1) & 7; }
__device__ __forceinline__ int swb(int k) { return 4 * ((k >> 3) & 3); }

__device__ __forceinline__ void wait_vm0() {
  // vmcnt 0; expcnt and lgkmcnt not waited for
  __builtin_amdgcn_s_waitcnt((7 << 4) | (15 << 8));
}

template <int TF, bool BR>
__device__ inline void fast_term(const GemmTerm& t, int i0, int j0, uint8_t* smem,
                                 f4 (&acc)[FGeo<TF>::NB][FGeo<TF>::NB]) {
  using G = FGeo<TF>;
  constexpr int NB = G::NB, Q = G::Q, CPR = TF / 4, CH = FCH;  // CPR: chunks per row-major B row
  const int64_t klo = lo_of<TF>(t.klo, i0, j0);
  const int64_t khi = hi_of<TF>(t.khi, i0, j0, t.K);
  if (klo >= khi) return;
  const int nst = (int)((khi - klo) / FK);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wi = wave >> 1, wj = wave & 1;
  // this lane's Q chunks of each operand per stage (wave-wide loads Q w .. Q w + Q - 1)
  const float* ga[Q];
  const float* gb[Q];
  uint32_t la[Q], lb[Q];
#pragma unroll
  for (int q = 0; q < Q; ++q) {
    const int pos = (Q * wave + q) * 64 + lane;  // 16-byte position in the operand's stage image
    {
      const int r = pos / CH, c = (pos % CH) ^ swa(r);
      ga[q] = t.A + (int64_t)(i0 + r) * t.lda + klo + 4 * c;
    }
    if (BR) {
      const int k = pos / CPR, c = (pos % CPR) ^ swb(k);
      gb[q] = t.B + (klo + k) * t.ldb + j0 + 4 * c;
    } else {
      const int r = pos / CH, c = (pos % CH) ^ swa(r);
      gb[q] = t.B + (int64_t)(j0 + r) * t.ldb + klo + 4 * c;
    }
    la[q] = (uint32_t)((Q * wave + q) * 64 * 16);
    lb[q] = (uint32_t)(G::OP + (Q * wave + q) * 64 * 16);
  }
  const int64_t da = FK, db = BR ? (int64_t)FK * t.ldb : FK;  // element step per stage
  auto issue = [&](int st) {
    uint8_t* base = smem + (st & 1) * G::STAGE;
#pragma unroll
    for (int q = 0; q < Q; ++q) {
      __builtin_amdgcn_global_load_lds((const void*)(ga[q] + st * da),
                                       (__attribute__((address_space(3))) void*)(base + la[q]), 16, 0, 0);
      __builtin_amdgcn_global_load_lds((const void*)(gb[q] + st * db),
                                       (__attribute__((address_space(3))) void*)(base + lb[q]), 16, 0, 0);
    }
  };
  const int g = lane >> 4, l16 = lane & 15;
  auto compute = [&](int st) {
    const u32x4* sa = (const u32x4*)(smem + (st & 1) * G::STAGE);
    const uint8_t* sbb = smem + (st & 1) * G::STAGE + G::OP;
    float av[NB][CH], bv[NB][CH];  // [block][step]
#pragma unroll
    for (int a = 0; a < NB; ++a) {
      const int r = wi * G::HW + a * 16 + l16;
#pragma unroll
      for (int h = 0; h < CH / 4; ++h) {
        const u32x4 v = sa[r * CH + (((CH / 4) * g + h) ^ swa(r))];
#pragma unroll
        for (int s2 = 0; s2 < 4; ++s2) av[a][4 * h + s2] = __uint_as_float(v[s2]);
      }
    }
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      const int col = wj * G::HW + b * 16 + l16;
      if (BR) {
        const float* sb = (const float*)sbb;
#pragma unroll
        for (int s2 = 0; s2 < CH; ++s2) {
          const int k = CH * g + s2;
          bv[b][s2] = sb[k * TF + (((col >> 2) ^ swb(k)) << 2) + (col & 3)];
        }
      } else {
#pragma unroll
        for (int h = 0; h < CH / 4; ++h) {
          const u32x4 v = ((const u32x4*)sbb)[col * CH + (((CH / 4) * g + h) ^ swa(col))];
#pragma unroll
          for (int s2 = 0; s2 < 4; ++s2) bv[b][4 * h + s2] = __uint_as_float(v[s2]);
        }
      }
    }
#pragma unroll
    for (int s2 = 0; s2 < CH; ++s2)
#pragma unroll
      for (int a = 0; a < NB; ++a)
#pragma unroll
        for (int b = 0; b < NB; ++b) acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[a][s2], bv[b][s2], acc[a][b], 0, 0, 0);
  };
  lds_barrier();  // the previous user of the stages (an earlier term) is done with them
  issue(0);
  for (int st = 0; st < nst; ++st) {
    wait_vm0();     // stage st landed (this wave's part)
    lds_barrier();  // every wave's part landed; every wave is done with stage st - 1
    if (st + 1 < nst) issue(st + 1);
    compute(st);
  }
}

// Tiles are enumerated on the 128 grid (the triangular filters and the tile
// orders are defined there); with TF = 64 each 128 tile is split into its
// four quarters, which are consecutive ids (a quarter outside M x N exits).
// PAIR (64 tiles, launches whose C overwrites the first term's A in place,
// N <= 128): a workgroup takes both column quarters of a row quarter, runs
// both K loops and only then writes, so no workgroup overwrites columns that
// another one of the same rows has still to read.
// DUAL: two independent one-term products (GemmDesc::dual), blockIdx.y
// selects which.
template <int TF, bool B1R, bool B2R, bool TWO, bool PAIR, bool DUAL>
__global__ __launch_bounds__(256, FGeo<TF>::OCC) void gemm_fast_kernel(GemmDesc d, int ntiles) {
  using G = FGeo<TF>;
  constexpr int NB = G::NB, SUB = kTile / TF;
  constexpr int NQ = PAIR ? 2 : 1;  // column quarters per workgroup
  static_assert(!PAIR || TF == 64, "paired quarters on 64 tiles");
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];  // the ring; reused by the epilogue
  const int id = d.order == ORDER_XCD ? xcd_remap_g(blockIdx.x, gridDim.x) : (int)blockIdx.x;
  if (id >= ntiles) return;
  const int prob = DUAL ? (int)blockIdx.y : 0;  // the product this workgroup computes
  if (DUAL) {
    if (prob) d.C = d.C2;
  } else if (blockIdx.y) {
    const int64_t z = blockIdx.y;
    d.C += z * d.sC;
    d.t[0].A += z * d.sA[0];
    d.t[0].B += z * d.sB[0];
    d.t[1].A += z * d.sA[1];
    d.t[1].B += z * d.sB[1];
  }
  const int SPT = PAIR ? SUB : SUB * SUB;  // ids per 128 tile
  const int pid = id / SPT, sub = id % SPT;
  int ti, tj;
  tile_of(d, pid, &ti, &tj);
  const int i0 = ti * kTile + (PAIR ? sub : sub / SUB) * TF;
  const int jb = tj * kTile + (PAIR ? 0 : (sub % SUB) * TF);  // first column quarter
  if (i0 >= d.M || jb >= d.N) return;
  f4 acc[NQ][NB][NB];
#pragma unroll
  for (int q = 0; q < NQ; ++q)
#pragma unroll
    for (int a = 0; a < NB; ++a)
#pragma unroll
      for (int b = 0; b < NB; ++b) acc[q][a][b] = f4{0.f, 0.f, 0.f, 0.f};
  // The terms are summed unscaled: acc = P0 (r P0 + P1 with r = alpha0 / alpha1
  // for two terms) and the epilogue multiplies by alpha0 (alpha1), so the
  // fragments go from LDS to the MFMAs untouched.  For alpha = +-1 the result
  // is bit for bit that of accumulating the scaled products.
  const float a0 = d.t[0].alpha, a1 = d.t[1].alpha;
  const bool two = TWO && !DUAL && a1 != 0.f && d.t[1].K > 0;
  const float ae = (DUAL && prob) || two ? a1 : a0, r01 = two ? a0 / a1 : 1.f;
#pragma unroll
  for (int q = 0; q < NQ; ++q) {
    const int j0 = jb + q * TF;
    if (j0 < d.N) {  // uniform
      if (DUAL && prob)
        fast_term<TF, B2R>(d.t[1], i0, j0, smem, acc[q]);
      else
        fast_term<TF, B1R>(d.t[0], i0, j0, smem, acc[q]);
      if (two) {
        if (r01 != 1.f) {
#pragma unroll
          for (int a = 0; a < NB; ++a)
#pragma unroll
            for (int b = 0; b < NB; ++b) acc[q][a][b] *= r01;
        }
        fast_term<TF, B2R>(d.t[1], i0, j0, smem, acc[q]);
      }
    }
  }

  // epilogue through LDS: C = beta C + acc with coalesced 16-byte accesses,
  // FEP rows of the tile per pass (the waves holding them stage them).  Every
  // read of C is issued before the staging starts, so the tile waits for one
  // memory latency rather than one per batch of loads.
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wi = wave >> 1, wj = wave & 1;
  constexpr int LS = TF + 4;  // FEP * LS floats: the dynamic LDS is sized for it
  constexpr int CPR = TF / 4;
  constexpr int NP = TF / FEP, QPT = FEP * TF / 4 / 256;  // passes, 16-byte pieces per thread and pass
  static_assert(QPT * 256 * 4 == FEP * TF, "epilogue split");
  const bool keep_c = d.beta != 0.f;
  float* st = (float*)smem;
#pragma unroll
  for (int q = 0; q < NQ; ++q) {
    const int j0 = jb + q * TF;
    if (j0 >= d.N) break;  // uniform
    float4 cv[NP][QPT];
    if (keep_c) {
#pragma unroll
      for (int e = 0; e < NP; ++e)
#pragma unroll
        for (int i = 0; i < QPT; ++i) {
          const int qq = tid + 256 * i, r = qq / CPR, c4 = (qq % CPR) * 4;
          cv[e][i] = *(const float4*)(d.C + (int64_t)(i0 + e * FEP + r) * d.ldc + j0 + c4);
        }
    }
#pragma unroll
    for (int e = 0; e < NP; ++e) {
      const int e0 = e * FEP;
      lds_barrier();
      if (wi * G::HW >= e0 && wi * G::HW < e0 + FEP) {
#pragma unroll
        for (int a = 0; a < NB; ++a)
#pragma unroll
          for (int b = 0; b < NB; ++b)
#pragma unroll
            for (int r = 0; r < 4; ++r)
              st[(wi * G::HW - e0 + a * 16 + (lane >> 4) * 4 + r) * LS + wj * G::HW + b * 16 + (lane & 15)] =
                  acc[q][a][b][r];
      }
      lds_barrier();
#pragma unroll
      for (int i = 0; i < QPT; ++i) {
        const int qq = tid + 256 * i, r = qq / CPR, c4 = (qq % CPR) * 4;
        float4 v = *(const float4*)&st[r * LS + c4];
        v = make_float4(ae * v.x, ae * v.y, ae * v.z, ae * v.w);
        if (keep_c) {
          const float4 c = cv[e][i];
          v = make_float4(d.beta * c.x + v.x, d.beta * c.y + v.y, d.beta * c.z + v.z, d.beta * c.w + v.w);
        }
        *(float4*)(d.C + (int64_t)(i0 + e0 + r) * d.ldc + j0 + c4) = v;
      }
    }
  }
}

// A launch with fewer 128 tiles than kSmallTiles runs on 64 tiles: four
// times the workgroups.  Short products then still cover the 256 CUs, and
// launches of a few waves of 128 tiles lose less to the last, partly filled
// wave (measured at k = 4096 and 11008: 2048 beats 512, 1024 and 4096).
constexpr int kSmallTiles = 2048;

// Whether every TF tile of a launch can take the fast path: interior tiles,
// 16-byte aligned operands and rows, K ranges in whole stages.
template <int TF>
bool fast_ok(const GemmDesc& d) {
  if (d.M % TF != 0 || d.N % TF != 0 || (d.ldc & 3) != 0 || (reinterpret_cast<uintptr_t>(d.C) & 15) != 0)
    return false;
  if (d.dual && (reinterpret_cast<uintptr_t>(d.C2) & 15) != 0) return false;
  for (int i = 0; i < d.nterms; ++i) {
    const GemmTerm& t = d.t[i];
    if (!t.a_row || t.K % FK != 0 || (t.lda & 3) != 0 || (t.ldb & 3) != 0) return false;
    if ((reinterpret_cast<uintptr_t>(t.A) & 15) != 0 || (reinterpret_cast<uintptr_t>(t.B) & 15) != 0) return false;
    if (d.batch > 1 && ((d.sA[i] & 3) != 0 || (d.sB[i] & 3) != 0)) return false;
  }
  if (d.batch > 1 && (d.sC & 3) != 0) return false;
  return true;
}

template <int TF, bool B1R, bool B2R, bool TWO, bool PAIR = false>
duo_status launch_fast(const GemmDesc& d, int ids, int nb, hipStream_t s) {
  if constexpr (!PAIR && TWO && !B1R && B2R) {
    if (d.dual) {
      auto kern = gemm_fast_kernel<TF, B1R, B2R, TWO, false, true>;
      if (duo_status st = set_max_lds((const void*)kern, FGeo<TF>::LDS); st != DUO_OK) return st;
      hipLaunchKernelGGL(kern, dim3((unsigned)rup(ids, 8), nb), dim3(256), FGeo<TF>::LDS, s, d, ids);
      DUO_LAUNCH_CHECK();
      return DUO_OK;
    }
  }
  if (d.dual) return DUO_ERR_UNSUPPORTED;
  auto kern = gemm_fast_kernel<TF, B1R, B2R, TWO, PAIR, false>;
  if (duo_status st = set_max_lds((const void*)kern, FGeo<TF>::LDS); st != DUO_OK) return st;
  hipLaunchKernelGGL(kern, dim3((unsigned)rup(ids, 8), nb), dim3(256), FGeo<TF>::LDS, s, d, ids);
  DUO_LAUNCH_CHECK();
  return DUO_OK;
}

template <bool A1R, bool B1R, bool A2R, bool B2R, bool TWO>
duo_status launch(const GemmDesc& d, hipStream_t s) {
  const int tm = (int)cdiv(d.M, kTile), tn = (int)cdiv(d.N, kTile);
  const int ntiles = d.tri == TRI_ALL ? tm * tn : tm * (tm + 1) / 2;
  if (ntiles <= 0) return DUO_OK;
  const int nb = d.dual ? 2 : (d.batch > 1 ? d.batch : 1);
  if (d.inplace) {
    if (d.N > kTile) return DUO_ERR_UNSUPPORTED;
    if constexpr (A1R && A2R && !B1R && !B2R) {
      if ((int64_t)ntiles * nb >= kSmallTiles) {
        if (fast_ok<kTile>(d)) return launch_fast<kTile, B1R, B2R, TWO>(d, ntiles, nb, s);
      } else if (fast_ok<64>(d)) {
        return launch_fast<64, B1R, B2R, TWO, true>(d, 2 * ntiles, nb, s);
      }
    }
    const int grid = (int)rup(ntiles, 8);
    hipLaunchKernelGGL((gemm_kernel<kTile, A1R, B1R, A2R, B2R, TWO>), dim3(grid, nb), dim3(256), 0, s, d, ntiles);
    DUO_LAUNCH_CHECK();
    return DUO_OK;
  }
  if constexpr (A1R && A2R) {
    if ((int64_t)ntiles * nb >= kSmallTiles && fast_ok<kTile>(d)) return launch_fast<kTile, B1R, B2R, TWO>(d, ntiles, nb, s);
    if (fast_ok<64>(d)) return launch_fast<64, B1R, B2R, TWO>(d, 4 * ntiles, nb, s);
  }
  if ((int64_t)ntiles * nb < kSmallTiles) {
    const int grid = (int)rup(4 * ntiles, 8);
    hipLaunchKernelGGL((gemm_kernel<64, A1R, B1R, A2R, B2R, TWO>), dim3(grid, nb), dim3(256), 0, s, d, 4 * ntiles);
  } else {
    const int grid = (int)rup(ntiles, 8);
    hipLaunchKernelGGL((gemm_kernel<kTile, A1R, B1R, A2R, B2R, TWO>), dim3(grid, nb), dim3(256), 0, s, d, ntiles);
  }
  DUO_LAUNCH_CHECK();
  return DUO_OK;
}

}  // namespace

duo_status gemm_f32(const GemmDesc& d, hipStream_t s) {
  if (d.M <= 0 || d.N <= 0) return DUO_OK;
  if (d.tri != TRI_ALL && d.M != d.N) return DUO_ERR_UNSUPPORTED;
  if (d.dual) {
    if (d.nterms != 2 || d.batch > 1 || d.inplace || !d.C2) return DUO_ERR_UNSUPPORTED;
    // one launch when the fast path takes both (A row-major, B of the first
    // K-contiguous and of the second row-major); otherwise two
    if (d.t[0].a_row && !d.t[0].b_row && d.t[1].a_row && d.t[1].b_row && fast_ok<64>(d))
      return launch<true, false, true, true, true>(d, s);
    GemmDesc p = d;
    p.dual = 0;
    p.nterms = 1;
    if (duo_status st = gemm_f32(p, s); st != DUO_OK) return st;
    p.C = d.C2;
    p.t[0] = d.t[1];
    return gemm_f32(p, s);
  }
  const int c1 = d.t[0].a_row * 2 + d.t[0].b_row;
  if (d.nterms == 1) {
    // one-term products run the two-term kernel with an empty second term
    // (K = 0: it returns before any access).  Compiled on its own, the
    // one-term kernel needs more than 256 VGPRs (one wave per SIMD, or
    // spills at two); in the two-term form it stays near 210.
    GemmDesc e = d;
    e.t[1] = GemmTerm{nullptr, 0, d.t[0].a_row, nullptr, 0, d.t[0].b_row, 0, 0.f, KLO_ZERO, KHI_FULL};
    e.sA[1] = e.sB[1] = 0;
    switch (c1) {
      case 0: return launch<false, false, false, false, true>(e, s);
      case 1: return launch<false, true, false, true, true>(e, s);
      case 2: return launch<true, false, true, false, true>(e, s);
      default: return launch<true, true, true, true, true>(e, s);
    }
  }
  const int c2 = d.t[1].a_row * 2 + d.t[1].b_row;
  if (c1 == 2 && c2 == 3) return launch<true, false, true, true, true>(d, s);
  if (c1 == 2 && c2 == 2) return launch<true, false, true, false, true>(d, s);
  return DUO_ERR_UNSUPPORTED;
}

}  // namespace duo
