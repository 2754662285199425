// Stage 3 column sweep of the DuoGPT layer solver on gfx950 (paper
// Algorithm 1, inner and outer loops; scores from Eq. 7).
//
// Per block of B columns [j0, j0+Bb):
//   select   S = W[:, blk]^2 * fac[blk]; the z lowest by (S, column, row) are
//            pruned.  Every element has the unique key (bits of S,
//            column*n + row).  One launch histograms the top 13 key bits
//            (15 for blocks of 2^20 scores or more) over the block; the next
//            gathers the elements of the bucket that
//            holds the z-th key (normally a few thousand), and a third, one
//            workgroup, finds the exact threshold among them (radix passes
//            in registers down to at most 256, then direct ranking; a bucket
//            too large for the registers is read from the block itself).  Counting
//            uses integer atomics only, so the result is deterministic.
//   in-block one row per 16 lanes (one DPP row), each lane owning the 8 columns
//            c = lane%16 + 16i; L[blk, blk] and D[blk, blk] sit in LDS (an image
//            laid out once per sweep and streamed in per block).  For
//            column j the owner's current value w0 reaches the other 15 lanes
//            by a DPP row broadcast; p = w0 * m_j, e = (w0 - p) / L_jj, and
//            later columns get w -= e L[c][j] - w0 D[j][c].  The 128 steps are
//            unrolled so that every register index is static.  E and W0 are
//            kept for the lazy update.
//   lazy     W[:, rest] += -E L[rest, blk]^T + W0 D[blk, rest] as one two-term
//            fp32 MFMA GEMM (W0 = the columns' values before pruning).
#include <hip/hip_runtime.h>

#include <utility>

#include "internal.h"

namespace duo {

namespace {

enum { MODE_SELECT = 0, MODE_FORCED = 1, MODE_KEEP_ALL = 2, MODE_PRUNE_ALL = 3, MODE_NM = 4 };
// The first launch histograms key bits 31..sh0: sh0 = 19 (8192 bins) for
// blocks of fewer than 2^20 scores, 17 (32768 bins, a quarter of the bucket)
// for larger ones, so that the bucket of the z-th key stays within kSelCap.
constexpr int kShift0 = 17;                 // smallest sh0
constexpr int kBins0 = 1 << (32 - kShift0); // largest bin count (128 KB of LDS)
constexpr int kDigit = 8;                   // radix digit of the W-stream fallback
constexpr int kSelCap = 16384;              // largest bucket gathered (64 candidates per resolving thread)
constexpr int kSelWG = 128;                 // workgroups of a selection launch (at most)
constexpr int kRowU = 16;                   // rows loaded per batch by one thread

struct SelState {
  uint32_t ncand;    // candidates gathered for the current block
  uint32_t key;      // threshold: an element is pruned iff
  uint32_t tie;      //   (key, column*n + row) <= (key, tie)
  uint32_t bin;      // bucket of the z-th key, the rank inside it and its
  uint32_t rank;     //   count, as the gathering launch found them
  uint32_t cnt;
  uint32_t nlo;      // kBins0 - 1 - (lowest occupied bin) and the highest
  uint32_t hi;       //   occupied bin of the block's histogram (atomic max)
};

__global__ void sel_reset_kernel(SelState* st, uint32_t* hist) {
  for (int i = threadIdx.x; i < kBins0; i += blockDim.x) hist[i] = 0;
  if (threadIdx.x < (int)(sizeof(SelState) / 4)) ((uint32_t*)st)[threadIdx.x] = 0;
}

// Inclusive sum over the 256 threads of a workgroup; `tot` gets the total.
__device__ inline uint32_t block_incl_scan(uint32_t v, uint32_t* wsum, uint32_t& tot) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  uint32_t incl = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const uint32_t y = __shfl_up(incl, o);
    if (lane >= o) incl += y;
  }
  __syncthreads();
  if (lane == 63) wsum[wv] = incl;
  __syncthreads();
  uint32_t base = 0;
  tot = 0;
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    if (w < wv) base += wsum[w];
    tot += wsum[w];
  }
  return base + incl;
}

// Bin of a histogram h[0 .. 256*PER) holding the rank-th element (1-based),
// the rank inside that bin and the bin's count.  Called by all 256 threads;
// every thread gets the result.
template <int PER>
__device__ void find_bucket(const uint32_t* h, uint32_t rank, uint32_t* sh, uint32_t& bin, uint32_t& rank_in,
                            uint32_t& cnt) {
  const int b0 = threadIdx.x * PER;
  uint32_t hv[PER];
  uint32_t mine = 0;
#pragma unroll
  for (int q = 0; q < PER; ++q) hv[q] = h[b0 + q];
#pragma unroll
  for (int q = 0; q < PER; ++q) mine += hv[q];
  uint32_t tot;
  const uint32_t incl = block_incl_scan(mine, sh + 4, tot);
  const uint32_t excl = incl - mine;
  if (excl < rank && rank <= incl) {
    uint32_t cum = excl;
#pragma unroll
    for (int q = 0; q < PER; ++q) {
      if (rank > cum && rank <= cum + hv[q]) {
        sh[0] = (uint32_t)(b0 + q);
        sh[1] = rank - cum;
        sh[2] = hv[q];
      }
      cum += hv[q];
    }
  }
  __syncthreads();
  bin = sh[0];
  rank_in = sh[1];
  cnt = sh[2];
  __syncthreads();
}

// find_bucket over the bins [lo, hi] of h (all others are empty): thread t
// sums a contiguous chunk of the range; the thread whose chunk holds the
// rank-th element finds the bin by reading its chunk again.
__device__ void find_bucket_range(const uint32_t* h, int lo, int hi, uint32_t rank, uint32_t* sh, uint32_t& bin,
                                  uint32_t& rank_in, uint32_t& cnt) {
  const int nb = hi >= lo ? hi - lo + 1 : 0;
  const int per = (nb + 255) / 256;
  const int b0 = lo + (int)threadIdx.x * per, b1 = min(hi + 1, b0 + per);
  uint32_t mine = 0;
  for (int b = b0; b < b1; ++b) mine += h[b];
  uint32_t tot;
  const uint32_t incl = block_incl_scan(mine, sh + 4, tot);
  const uint32_t excl = incl - mine;
  if (excl < rank && rank <= incl) {
    uint32_t cum = excl;
    for (int b = b0; b < b1; ++b) {
      const uint32_t hv = h[b];
      if (rank > cum && rank <= cum + hv) {
        sh[0] = (uint32_t)b;
        sh[1] = rank - cum;
        sh[2] = hv;
      }
      cum += hv;
    }
  }
  __syncthreads();
  bin = sh[0];
  rank_in = sh[1];
  cnt = sh[2];
  __syncthreads();
}

// f(row, w) for rows r0+rs, r0+rs+2, ... < r1 of one column.  Loads are
// issued kRowU at a time, unconditionally (clamped to a valid row), so that
// they are all in flight together; the trip count is uniform per wave.
template <class F>
__device__ __forceinline__ void for_rows(const float* Wc, int64_t ldw, int r0, int r1, int rs, bool cv, F&& f) {
  for (int rb = r0 + rs; rb < r1; rb += 2 * kRowU) {
    float v[kRowU];
#pragma unroll
    for (int u = 0; u < kRowU; ++u) {
      const int r = rb + 2 * u < r1 ? rb + 2 * u : rb;
      v[u] = Wc[(int64_t)r * ldw];
    }
#pragma unroll
    for (int u = 0; u < kRowU; ++u)
      if (cv && rb + 2 * u < r1) f(rb + 2 * u, v[u]);
  }
}

// Minimum and maximum over a wave: DPP steps inside each 16-lane row (quad
// swaps, half-row and row mirrors leave the row's result in every lane), then
// the four rows' results read as scalars.
template <bool MAX>
__device__ __forceinline__ uint32_t wave_extreme(uint32_t v) {
  auto pick = [](uint32_t a, uint32_t b) { return MAX ? (a > b ? a : b) : (a < b ? a : b); };
  v = pick(v, (uint32_t)__builtin_amdgcn_update_dpp((int)v, (int)v, 0xB1, 0xF, 0xF, false));   // quad_perm 1,0,3,2
  v = pick(v, (uint32_t)__builtin_amdgcn_update_dpp((int)v, (int)v, 0x4E, 0xF, 0xF, false));   // quad_perm 2,3,0,1
  v = pick(v, (uint32_t)__builtin_amdgcn_update_dpp((int)v, (int)v, 0x141, 0xF, 0xF, false));  // row_half_mirror
  v = pick(v, (uint32_t)__builtin_amdgcn_update_dpp((int)v, (int)v, 0x140, 0xF, 0xF, false));  // row_mirror
  const uint32_t a = pick((uint32_t)__builtin_amdgcn_readlane((int)v, 0), (uint32_t)__builtin_amdgcn_readlane((int)v, 16));
  const uint32_t b = pick((uint32_t)__builtin_amdgcn_readlane((int)v, 32), (uint32_t)__builtin_amdgcn_readlane((int)v, 48));
  return pick(a, b);
}

// Selection of one block in three launches (see the file comment); kernel
// boundaries are the only synchronisation, so no cache-wide fences are needed.
//
// Workgroup b of the first two owns rows [b*rpw, (b+1)*rpw); thread t handles
// column t % 128 (clamped to Bb - 1 and masked) of every second row.

// 1. histogram of key bits 31..17 over the block (optionally writing S).
//    HB: batches of kRowU rows a thread holds in registers (1 or 2), or 0
//    for the streaming form of any height.  Only the bins between the
//    workgroup's smallest and largest key are cleared and flushed, and that
//    range also widens the block's [lo, hi] in the selection state.
template <int HB>
__global__ __launch_bounds__(256) void sel_hist_kernel(const float* __restrict__ W, int64_t ldw, int n, int Bb, int j0,
                                                       const float* __restrict__ fac, uint32_t* hist,
                                                       float* scores_out, int do_hist, SelState* st, int sh0) {
  extern __shared__ __attribute__((aligned(16))) uint32_t lh[];  // [kBins0]
  __shared__ uint32_t rng[8];
  const int tid = threadIdx.x;
  const int rpw = (n + gridDim.x - 1) / gridDim.x;
  const int r0 = blockIdx.x * rpw, r1 = min(n, r0 + rpw);
  const int c = min(tid & 127, Bb - 1), rs = tid >> 7;
  const bool cv = (tid & 127) < Bb;
  const float fc = fac[j0 + c];
  const float* Wc = W + j0 + c;
  uint32_t lo = kBins0, hi = 0;
  if constexpr (HB > 0) {
    if (!do_hist) return;  // (launched with HB > 0 only without scores_out)
    constexpr int NV = HB * kRowU;
    float v[NV];
#pragma unroll
    for (int u = 0; u < NV; ++u) {
      const int r = r0 + rs + 2 * u;
      v[u] = Wc[(int64_t)(r < r1 ? r : min(r0, n - 1)) * ldw];
    }
    uint32_t bk[NV];
#pragma unroll
    for (int u = 0; u < NV; ++u) {
      const bool ok = cv && r0 + rs + 2 * u < r1;
      bk[u] = ok ? orderable(weight_score(v[u], fc)) >> sh0 : (uint32_t)kBins0;  // kBins0: no element
      lo = ok && bk[u] < lo ? bk[u] : lo;
      hi = ok && bk[u] > hi ? bk[u] : hi;
    }
    lo = wave_extreme<false>(lo);
    hi = wave_extreme<true>(hi);
    if ((tid & 63) == 0) {
      rng[tid >> 6] = lo;
      rng[4 + (tid >> 6)] = hi;
    }
    __syncthreads();
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      lo = min(lo, rng[w]);
      hi = max(hi, rng[4 + w]);
    }
    for (int i = (int)lo + tid; i <= (int)hi; i += 256) lh[i] = 0;
    __syncthreads();
#pragma unroll
    for (int u = 0; u < NV; ++u)
      if (bk[u] < (uint32_t)kBins0) atomicAdd(&lh[bk[u]], 1u);
  } else {
    if (do_hist)
      for (int i = tid; i < kBins0 / 4; i += 256) ((u32x4*)lh)[i] = u32x4{0u, 0u, 0u, 0u};
    __syncthreads();
    for_rows(Wc, ldw, r0, r1, rs, cv, [&](int r, float w) {
      const float S = weight_score(w, fc);
      if (scores_out) scores_out[(int64_t)r * ldw + j0 + c] = S;
      if (do_hist) {
        const uint32_t b = orderable(S) >> sh0;
        atomicAdd(&lh[b], 1u);
        lo = b < lo ? b : lo;
        hi = b > hi ? b : hi;
      }
    });
    if (!do_hist) return;
    lo = wave_extreme<false>(lo);
    hi = wave_extreme<true>(hi);
    if ((tid & 63) == 0) {
      rng[tid >> 6] = lo;
      rng[4 + (tid >> 6)] = hi;
    }
    __syncthreads();
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      lo = min(lo, rng[w]);
      hi = max(hi, rng[4 + w]);
    }
  }
  __syncthreads();
  for (int i = (int)lo + tid; i <= (int)hi; i += 256)
    if (lh[i]) atomicAdd(&hist[i], lh[i]);
  if (tid == 0 && lo <= hi) {
    atomicMax(&st->nlo, (uint32_t)(kBins0 - 1) - lo);
    atomicMax(&st->hi, hi);
  }
}

// 2. every workgroup locates the bucket of the z-th key in the histogram
//    (scanning only the block's occupied range [lo, hi]) and appends its
//    elements of that bucket as (low 17 key bits, index) composites; one
//    atomic per workgroup reserves its slots.  HB as for the histogram.
template <int HB>
__global__ __launch_bounds__(256) void sel_gather_kernel(const float* __restrict__ W, int64_t ldw, int n, int Bb, int j0,
                                                         const float* __restrict__ fac, uint32_t z, int idx_bits,
                                                         const uint32_t* hist, SelState* st,
                                                         unsigned long long* cand, int sh0) {
  __shared__ uint32_t sh[16];
  const int tid = threadIdx.x;
  const int rpw = (n + gridDim.x - 1) / gridDim.x;
  const int r0 = blockIdx.x * rpw, r1 = min(n, r0 + rpw);
  const int c = min(tid & 127, Bb - 1), rs = tid >> 7;
  const bool cv = (tid & 127) < Bb;
  const float fc = fac[j0 + c];
  const float* Wc = W + j0 + c;
  // With HB > 0 the thread's rows are loaded before the bucket search (both
  // loads in flight together) and kept for both passes.
  constexpr int NV = HB > 0 ? HB * kRowU : 1;
  uint32_t key1[NV];
  uint32_t vm = 0;  // bit u: row r0 + rs + 2u is in range (and the column is)
  if constexpr (HB > 0) {
#pragma unroll
    for (int u = 0; u < NV; ++u) {
      const int r = r0 + rs + 2 * u;
      key1[u] = orderable(weight_score(Wc[(int64_t)(r < r1 ? r : min(r0, n - 1)) * ldw], fc));
      vm |= (cv && r < r1 ? 1u : 0u) << u;
    }
  }
  uint32_t bin, rank, cnt;
  if (sh0 == kShift0 + 2)  // 8192 bins: all of them, without waiting for the range
    find_bucket<(1 << (30 - kShift0)) / 256>(hist, z, sh, bin, rank, cnt);
  else
    find_bucket_range(hist, (int)(kBins0 - 1 - st->nlo), (int)st->hi, z, sh, bin, rank, cnt);
  if (blockIdx.x == 0 && tid == 0) {  // for the resolving launch
    st->bin = bin;
    st->rank = rank;
    st->cnt = cnt;
  }
  if (cnt > (uint32_t)kSelCap) return;  // the resolving launch reads the block itself
  if constexpr (HB > 0) {
    asm volatile("" : "+v"(vm));  // lane tests where they are used
    uint32_t mine = 0;
#pragma unroll
    for (int u = 0; u < NV; ++u) mine += ((vm >> u) & 1u) && (key1[u] >> sh0) == bin;
    uint32_t tot;
    const uint32_t incl = block_incl_scan(mine, sh + 4, tot);
    if (tid == 0) sh[9] = tot ? atomicAdd(&st->ncand, tot) : 0u;
    __syncthreads();
    uint32_t pos = sh[9] + incl - mine;
    asm volatile("" : "+v"(vm));
#pragma unroll
    for (int u = 0; u < NV; ++u)
      if (((vm >> u) & 1u) && (key1[u] >> sh0) == bin) {
        if (pos < (uint32_t)kSelCap)
          cand[pos] = ((unsigned long long)(key1[u] & ((1u << sh0) - 1u)) << idx_bits) |
                      (unsigned long long)((uint32_t)c * (uint32_t)n + (uint32_t)(r0 + rs + 2 * u));
        ++pos;
      }
    return;
  }
  uint32_t mine = 0;
  for_rows(Wc, ldw, r0, r1, rs, cv, [&](int, float w) { mine += (orderable(weight_score(w, fc)) >> sh0) == bin; });
  uint32_t tot;
  const uint32_t incl = block_incl_scan(mine, sh + 4, tot);
  if (tid == 0) sh[9] = tot ? atomicAdd(&st->ncand, tot) : 0u;
  __syncthreads();
  uint32_t pos = sh[9] + incl - mine;
  for_rows(Wc, ldw, r0, r1, rs, cv, [&](int r, float w) {
    const uint32_t key = orderable(weight_score(w, fc));
    if ((key >> sh0) == bin) {
      if (pos < (uint32_t)kSelCap)
        cand[pos] = ((unsigned long long)(key & ((1u << sh0) - 1u)) << idx_bits) |
                    (unsigned long long)((uint32_t)c * (uint32_t)n + (uint32_t)r);
      ++pos;
    }
  });
}

// 3. one workgroup: the rank-th composite of the bucket (bin, rank and count
//    as the gathering launch left them in the state), then the histogram is
//    cleared for the next block.  Gathered candidates (at most kSelCap) stay
//    in registers, 32 per thread: radix passes of up to kDigitR bits narrow
//    them to the prefix that holds the rank-th composite until at most 256
//    remain, and those are ranked against each other directly (composites
//    are unique, so exactly one has the wanted rank).  A bucket larger than
//    kSelCap is resolved by 8-bit passes straight over the block.
constexpr int kDigitR = 11;
constexpr int kRankMax = 256;
template <int NU>
__global__ __launch_bounds__(256) void sel_resolve_kernel(const float* __restrict__ W, int64_t ldw, int n, int Bb,
                                                          int j0, const float* __restrict__ fac, uint32_t z,
                                                          int idx_bits, uint32_t* hist, SelState* st,
                                                          const unsigned long long* cand, int sh0) {
  extern __shared__ __attribute__((aligned(16))) uint32_t sel_sm[];
  uint32_t* sh = sel_sm;                                                   // [16]
  uint32_t* lh = sel_sm + 16;                                              // [1 << kDigitR]
  unsigned long long* lr = (unsigned long long*)(lh + (1 << kDigitR));     // [kRankMax]
  const int tid = threadIdx.x;
  if (tid == 0) sh[12] = 0;  // compaction counter
  __syncthreads();
  // NU candidates per thread (NU * 256 <= kSelCap slots, all of which exist):
  // they are loaded before the bucket is read, so both loads are in flight
  // together
  static_assert(NU * 256 <= kSelCap, "candidate slots");
  unsigned long long v[NU];
#pragma unroll
  for (int u = 0; u < NU; ++u) v[u] = cand[256 * u + tid];
  const uint32_t bin = st->bin, rank = st->rank, cnt = st->cnt;
  const int tb = sh0 + idx_bits;  // composite bits
  unsigned long long pref = 0;
  if (cnt <= (uint32_t)(NU * 256)) {
    // slots past cnt become all-ones, which matches no prefix (composites
    // are below 2^50)
#pragma unroll
    for (int u = 0; u < NU; ++u) v[u] = (uint32_t)(256 * u + tid) < cnt ? v[u] : ~0ull;
    int s = tb;         // bits [s, tb) of the wanted composite are known (in pref)
    uint32_t rk = rank, cur = cnt;
    while (cur > (uint32_t)kRankMax) {
      const int d = s < kDigitR ? s : kDigitR;
      const int hs = s;
      s -= d;
      for (int i = tid; i < (1 << kDigitR); i += 256) lh[i] = 0;
      __syncthreads();
#pragma unroll
      for (int u = 0; u < NU; ++u)
        if ((v[u] >> hs) == (pref >> hs))
          atomicAdd(&lh[(uint32_t)(v[u] >> s) & ((1u << d) - 1u)], 1u);
      __syncthreads();
      uint32_t dg, rk2, c2;
      find_bucket<(1 << kDigitR) / 256>(lh, rk, sh, dg, rk2, c2);
      pref |= (unsigned long long)dg << s;
      rk = rk2;
      cur = c2;
    }
    // the cur <= kRankMax composites with the known prefix, ranked directly
#pragma unroll
    for (int u = 0; u < NU; ++u)
      if ((v[u] >> s) == (pref >> s)) lr[atomicAdd(&sh[12], 1u)] = v[u];
    __syncthreads();
    if ((uint32_t)tid < cur) {
      const unsigned long long my = lr[tid];
      uint32_t r = 1;
      for (uint32_t j = 0; j < cur; ++j) r += lr[j] < my;
      if (r == rk) {
        sh[13] = (uint32_t)my;
        sh[14] = (uint32_t)(my >> 32);
      }
    }
    __syncthreads();
    pref = (unsigned long long)sh[13] | ((unsigned long long)sh[14] << 32);
  } else {
    // rare: a bucket this large means a long run of nearly equal scores
    const int c = min(tid & 127, Bb - 1), rs = tid >> 7;
    const bool cv = (tid & 127) < Bb;
    const float fc = fac[j0 + c];
    const float* Wc = W + j0 + c;
    const int start = (tb + kDigit - 1) / kDigit * kDigit;
    uint32_t rk = rank;
    for (int s = start - kDigit; s >= 0; s -= kDigit) {
      for (int i = tid; i < (1 << kDigit); i += 256) lh[i] = 0;
      __syncthreads();
      const int hs = s + kDigit;
      for_rows(Wc, ldw, 0, n, rs, cv, [&](int r, float w) {
        const uint32_t key = orderable(weight_score(w, fc));
        if ((key >> sh0) == bin) {
          const unsigned long long v = ((unsigned long long)(key & ((1u << sh0) - 1u)) << idx_bits) |
                                       (unsigned long long)((uint32_t)c * (uint32_t)n + (uint32_t)r);
          if ((v >> hs) == (pref >> hs)) atomicAdd(&lh[(uint32_t)(v >> s) & ((1u << kDigit) - 1u)], 1u);
        }
      });
      __syncthreads();
      uint32_t d, rk2, ct2;
      find_bucket<(1 << kDigit) / 256>(lh, rk, sh, d, rk2, ct2);
      pref |= (unsigned long long)d << s;
      rk = rk2;
    }
  }
  // the histogram is empty outside [lo, hi]: clear that range for the next block
  for (int i = (int)(kBins0 - 1 - st->nlo) + tid; i <= (int)st->hi; i += 256) hist[i] = 0;
  __syncthreads();  // every thread has read the range before it is reset
  if (tid == 0) {
    st->key = (bin << sh0) | (uint32_t)(pref >> idx_bits);
    st->tie = (uint32_t)(pref & ((1ull << idx_bits) - 1ull));
    st->ncand = 0;
    st->nlo = 0;
    st->hi = 0;
  }
}

// ---------------------------------------------------------------------------
// in-block sweep
// ---------------------------------------------------------------------------
constexpr int IB_Q = 16;                  // lanes per row (one DPP row)
constexpr int IB_I = kMaxBlock / IB_Q;    // columns per lane: c = q + 16 i
constexpr int IB_ROWS = 256 / IB_Q;       // rows per workgroup (IB_ROWS2 for row counts past one round)
constexpr int IB_ROWS2 = 512 / IB_Q;
constexpr int IB_QS = IB_I + 1;           // LDS stride between lanes (odd: no bank conflicts)
constexpr int IB_JS = IB_Q * IB_QS;       // LDS floats per column step
// LDS image of one block's operands, [lq | dq | il | lj], padded to whole 4 KB
// rows of a 256-thread copy (16 bytes per thread)
constexpr int IB_IMG_USED = 2 * kMaxBlock * IB_JS + 2 * kMaxBlock;      // floats
constexpr int IB_IMG = (IB_IMG_USED * 4 + 4095) / 4096 * 4096 / 4;      // floats (37888)

// Lane O of every 16-lane row, broadcast to the row.
template <int O>
__device__ __forceinline__ float row_bcast(float v) {
  return __builtin_bit_cast(float,
                            __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x150 + O, 0xF, 0xF, false));
}

struct IbRow {
  float w[IB_I];     // current values of columns q + 16 i
  float y[IB_I];     // Y form only: the block's own part of y = V U for columns q + 16 i
  float e[IB_I];     // E of the columns this lane owns
  float w0[IB_I];    // values before pruning of the columns this lane owns
  uint32_t kb[IB_I]; // keep bits of the row: bit o of kb[g] is column 16 g + o
  float f[IB_I];     // N:M only: score factors of this lane's columns
  float sc[IB_I];    // N:M only: the scores the group selections used
  float qs, qz;      // quantisation only: the row's current grid (step, code of 0)
};

// Options of the sweep that the in-block kernel applies.
struct IbOpts {
  int nm_n;      // N of N:4 (MODE_NM)
  int q_bits;    // quantisation: bits of the grid (QUANT)
  int q_group;   // columns per grid: 16, 32, 64 or 128
  float* q_scale;  // NULL or n x ceil(k / q_group)
  float* q_zero;
};

// LDS operands of one column step: the staged L and D (Y form: U) entries of
// this lane's columns that are still live (i >= g), 1 / L_JJ and L_JJ.
struct IbBuf {
  float l[IB_I], d[IB_I];
  float il, lj;
};

template <int J>
__device__ __forceinline__ void ib_load(IbBuf& b, const float* __restrict__ lq, const float* __restrict__ dq,
                                        const float* __restrict__ il, int q) {
  if constexpr (J < kMaxBlock) {
    constexpr int g = J / IB_Q;
    const float* lr = lq + J * IB_JS + q * IB_QS;
    const float* dr = dq + J * IB_JS + q * IB_QS;
#pragma unroll
    for (int i = g; i < IB_I; ++i) {
      b.l[i] = lr[i];
      b.d[i] = dr[i];
    }
    b.il = il[J];
    b.lj = il[kMaxBlock + J];
  }
}

// Column J = 16 g + o of the block (owner lane o, register g).  The staged L
// column is already divided by L_JJ, so u = w0 - p feeds the update directly
// and e = u / L_JJ is only needed for the owner's record.  Columns past the
// ragged end of the block have zero L, D entries and values: their steps
// change nothing.  Step J issues the LDS reads of step J + 2 (three-slot
// ring); the scheduling barrier keeps the compiler from hoisting more.
template <int O>
__device__ __forceinline__ uint32_t row_bcast_u(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x150 + O, 0xF, 0xF, false);
}

// N:M groups of 4 columns: at the first column of a group every lane of the
// row receives the four columns' current score keys from their owner lanes
// and derives the same keep bits: the nm_n lowest (equal keys in column
// order) are pruned.
// val: this lane's current value of its column in slot G (the Y form adds the
// y terms the column is still owed inside the block, see ib_step).  Only the
// group's own four lanes (q = O .. O + 3) record the score they used.
template <int G, int O>
__device__ __forceinline__ void nm_select(IbRow& s, int nm_n, float val, int q) {
  const float S = weight_score(val, s.f[G]);
  if ((q & ~3) == O) s.sc[G] = S;
  const uint32_t key = orderable(S);
  const uint32_t k0 = row_bcast_u<O>(key), k1 = row_bcast_u<O + 1>(key);
  const uint32_t k2 = row_bcast_u<O + 2>(key), k3 = row_bcast_u<O + 3>(key);
  const int r0 = (k1 < k0) + (k2 < k0) + (k3 < k0);
  const int r1 = (k0 <= k1) + (k2 < k1) + (k3 < k1);
  const int r2 = (k0 <= k2) + (k1 <= k2) + (k3 < k2);
  const int r3 = (k0 <= k3) + (k1 <= k3) + (k2 <= k3);
  const uint32_t keep = (r0 >= nm_n ? 1u : 0u) | (r1 >= nm_n ? 2u : 0u) | (r2 >= nm_n ? 4u : 0u) |
                        (r3 >= nm_n ? 8u : 0u);
  s.kb[G] = (s.kb[G] & ~(0xFu << O)) | (keep << O);
}

// Joint quantisation: at the first column of a group of q_group columns the
// row's grid is fixed from the group's current values (min and max over the
// row's 16 lanes, 0 always inside the range, [-1, 1] for an empty range).
template <int G>
__device__ __forceinline__ void quant_grid(IbRow& s, const IbOpts& opt, int64_t row, bool rv, int q, int gcol,
                                           int ngroups) {
  const int i1 = G + opt.q_group / IB_Q;  // slots G .. i1-1 hold the group's columns
  float mn = 0.f, mx = 0.f;
#pragma unroll
  for (int i = G; i < IB_I; ++i)
    if (i < i1) {
      mn = fminf(mn, s.w[i]);
      mx = fmaxf(mx, s.w[i]);
    }
#pragma unroll
  for (int d = 8; d > 0; d >>= 1) {
    mn = fminf(mn, __shfl_xor(mn, d));
    mx = fmaxf(mx, __shfl_xor(mx, d));
  }
  if (mn == mx) {
    mn = -1.f;
    mx = 1.f;
  }
  s.qs = (mx - mn) / (float)((1 << opt.q_bits) - 1);
  s.qz = rintf(-mn / s.qs);
  if (q == 0 && rv) {
    if (opt.q_scale) opt.q_scale[row * ngroups + gcol] = s.qs;
    if (opt.q_zero) opt.q_zero[row * ngroups + gcol] = s.qz;
  }
}

// YR (the Y form of the sweep, no D): the lane also carries y, the block's
// own part of y = V U for its columns.  Column J's value is w_J + y_J L_JJ;
// after it, every later column c takes w_c += (y_J - e_J) L_cJ and
// y_c += v U_Jc, which is the D-form step w_c += -e_J L_cJ + v D_Jc summed
// over the block (D = U L^T).
template <int J, bool NM, bool QUANT, bool YR>
__device__ __forceinline__ void ib_step(IbRow& s, IbBuf (&buf)[3], const float* __restrict__ lq,
                                        const float* __restrict__ dq, const float* __restrict__ il, int q,
                                        const IbOpts& opt, int64_t row, bool rv, int j0, int Bb, int ngroups) {
  constexpr int g = J / IB_Q, o = J % IB_Q;
  ib_load<J + 2>(buf[(J + 2) % 3], lq, dq, il, q);
  if constexpr (NM && o % 4 == 0) {
    if constexpr (YR) {
      // the group's columns c = J .. J + 3 as they stand now: w_c plus
      // L_ci y_i for i = J .. c with the current y (the y terms the column
      // will still receive inside the block before it is processed); the L
      // entries of steps J, J + 1, J + 2 are in the ring
      const int pos = (q - o) & 3;  // position of this lane's column in the group
      float val = s.w[g] + s.y[g] * il[kMaxBlock + J + pos];
      const float y0 = row_bcast<o>(s.y[g]), y1 = row_bcast<o + 1>(s.y[g]), y2 = row_bcast<o + 2>(s.y[g]);
      const IbBuf &b0 = buf[J % 3], &b1 = buf[(J + 1) % 3], &b2 = buf[(J + 2) % 3];
      if (pos > 0) val = fmaf(b0.l[g] * b0.lj, y0, val);
      if (pos > 1) val = fmaf(b1.l[g] * b1.lj, y1, val);
      if (pos > 2) val = fmaf(b2.l[g] * b2.lj, y2, val);
      nm_select<g, o>(s, opt.nm_n, val, q);
    } else {
      nm_select<g, o>(s, opt.nm_n, s.w[g], q);
    }
  }
  if constexpr (QUANT && o == 0) {
    // groups start inside the block only (a short last block has no more); the
    // Y form is run with one group per block only, fixed at J = 0 where the
    // block's own part of y is still 0 and w holds Algorithm 1's values
    if (J < Bb && J % opt.q_group == 0) quant_grid<g>(s, opt, row, rv, q, (j0 + J) / opt.q_group, ngroups);
  }
  const IbBuf& b = buf[J % 3];
  float t = 0.f;  // YR: y_J L_JJ
  if constexpr (YR) t = row_bcast<o>(s.y[g]) * b.lj;
  const float v = YR ? row_bcast<o>(s.w[g]) + t : row_bcast<o>(s.w[g]);
  const bool kj = (s.kb[g] >> o) & 1u;
  // p: the value the column keeps (its grid value with QUANT), u = v - p the
  // error the later columns compensate
  float p;
  if constexpr (QUANT) {
    const float code = fminf(fmaxf(rintf(v / s.qs) + s.qz, 0.f), (float)((1 << opt.q_bits) - 1));
    p = kj ? s.qs * (code - s.qz) : 0.f;
  } else {
    p = kj ? v : 0.f;
  }
  const float u = v - p;
  if (q == o) {
    s.w[g] = p;
    s.e[g] = u * b.il;
    s.w0[g] = v;
  }
  // materialise the owner's record here: left to itself the compiler keeps
  // every step's u and 1 / L_JJ to the end of the block (about 350 registers,
  // most of them AGPR spill slots)
  asm volatile("" : "+v"(s.e[g]), "+v"(s.w0[g]));
  // columns c = q + 16 i > J; the LDS entries of columns <= J are zero
  if constexpr (YR) {
    const float tu = t - u;  // (y_J - e_J) L_JJ; the staged L column is divided by L_JJ
#pragma unroll
    for (int i = g; i < IB_I; ++i) {
      s.w[i] = fmaf(tu, b.l[i], s.w[i]);
      s.y[i] = fmaf(v, b.d[i], s.y[i]);
    }
  } else {
#pragma unroll
    for (int i = g; i < IB_I; ++i) s.w[i] = fmaf(-u, b.l[i], fmaf(v, b.d[i], s.w[i]));
  }
  __builtin_amdgcn_sched_barrier(0);
}

template <bool NM, bool QUANT, bool YR, int... Js>
__device__ __forceinline__ void ib_steps(IbRow& s, const float* lq, const float* dq, const float* il, int q,
                                         const IbOpts& opt, int64_t row, bool rv, int j0, int Bb, int ngroups,
                                         std::integer_sequence<int, Js...>) {
  IbBuf buf[3];
  ib_load<0>(buf[0], lq, dq, il, q);
  ib_load<1>(buf[1], lq, dq, il, q);
  (ib_step<Js, NM, QUANT, YR>(s, buf, lq, dq, il, q, opt, row, rv, j0, Bb, ngroups), ...);
}

// NM: the N:M variant (mode MODE_NM): the keep bits are chosen inside the
// column loop, and the scores they used go to scores_out when it is set.
// QUANT: joint RTN quantisation of the kept weights (grids per row and group).
// The LDS image of block b (columns j0 = b*B .. j0+Bb) for inblock_kernel:
// the live L and D entries of each lane's columns, 1 / L_jj and L_jj, zeros
// elsewhere (entries of columns <= j, past the ragged end, and the padding
// slot of each lane).  In the Y form D is replaced by U: the entries read
// (column c > j) are the same positions of Q, whose strictly upper part U is.
// One launch covers every block of the sweep.
__global__ __launch_bounds__(256) void ib_image_kernel(const float* __restrict__ L, int64_t ldl,
                                                       const float* __restrict__ D, int64_t ldd, int k, int B,
                                                       float* __restrict__ img) {
  const int b = blockIdx.x, j0 = b * B, Bb = min(B, k - j0);
  float* out = img + (int64_t)b * IB_IMG;
  for (int e = blockIdx.y * 256 + threadIdx.x; e < IB_IMG; e += gridDim.y * 256) {
    float v = 0.f;
    if (e < 2 * kMaxBlock * IB_JS) {
      const bool isd = e >= kMaxBlock * IB_JS;
      const int f = isd ? e - kMaxBlock * IB_JS : e;
      const int j = f / IB_JS, rem = f % IB_JS, q = rem / IB_QS, i = rem % IB_QS;
      const int c = q + IB_Q * i;
      if (i < IB_I && c > j && c < Bb) {
        if (isd)
          v = D[(int64_t)(j0 + j) * ldd + j0 + c];
        else
          v = L[(int64_t)(j0 + c) * ldl + j0 + j] * (1.0f / L[(int64_t)(j0 + j) * ldl + j0 + j]);
      }
    } else if (e < 2 * kMaxBlock * IB_JS + kMaxBlock) {
      const int j = e - 2 * kMaxBlock * IB_JS;
      v = j < Bb ? 1.0f / L[(int64_t)(j0 + j) * ldl + j0 + j] : 1.f;
    } else if (e < IB_IMG_USED) {
      const int j = e - 2 * kMaxBlock * IB_JS - kMaxBlock;
      v = j < Bb ? L[(int64_t)(j0 + j) * ldl + j0 + j] : 0.f;
    }
    out[e] = v;
  }
}

// YR: the Y form (no D; see ib_step).  Yp is the n x k matrix of the earlier
// blocks' part of y; the E slot of EW then receives z = y - e with y the
// whole of it (earlier blocks' part plus the block's own).
// ROWS rows per workgroup (16 lanes each): IB_ROWS, or IB_ROWS2 when the
// rows would otherwise need more than one workgroup per CU (the LDS image
// allows one), so that a block finishes in one round over the CUs.
template <bool NM, bool QUANT, bool YR, int ROWS>
__global__ __launch_bounds__(ROWS * IB_Q) void inblock_kernel(float* __restrict__ Wo, int n, int k, int j0, int Bb, int64_t ew_ld,
                                                      const float* __restrict__ fac, const SelState* st, int mode,
                                                      const uint32_t* __restrict__ mask_in, float* __restrict__ EW,
                                                      uint8_t* __restrict__ bmask, IbOpts opt,
                                                      float* __restrict__ scores_out, const float* __restrict__ img,
                                                      const float* __restrict__ Yp) {
  extern __shared__ __attribute__((aligned(16))) float sm[];
  float* lq = sm;                       // [j][q][i]: L[j0+q+16i][j0+j] / L[j0+j][j0+j] where q+16i > j, else 0
  float* dq = sm + kMaxBlock * IB_JS;   // [j][q][i]: D[j0+j][j0+q+16i] where q+16i > j, else 0
  float* il = dq + kMaxBlock * IB_JS;   // [j]: 1 / L[j0+j][j0+j], then [kMaxBlock + j]: L[j0+j][j0+j]
  const int tid = threadIdx.x;
  // The row's values and score factors are requested first; the block's LDS
  // image (written once per sweep by ib_image_kernel) then streams straight
  // into LDS (global_load_lds, 16 bytes per lane, no register staging), so
  // the two latencies overlap.
  const int q = tid & 15;
  const int row = blockIdx.x * ROWS + (tid >> 4);
  const bool rv = row < n;
  float wv[IB_I], fv[IB_I], yv[IB_I];
#pragma unroll
  for (int i = 0; i < IB_I; ++i) {
    const int c = q + IB_Q * i;
    const bool cv = rv && c < Bb;
    wv[i] = Wo[cv ? (int64_t)row * k + j0 + c : 0];
    fv[i] = fac[c < Bb ? j0 + c : j0];
    if constexpr (YR) yv[i] = cv ? Yp[(int64_t)row * k + j0 + c] : 0.f;
  }
  if (tid < 256) {  // the image in 4 KB rows of 256 x 16 bytes
    const uint8_t* src = (const uint8_t*)img + (tid >> 6) * 1024 + (tid & 63) * 16;
    uint8_t* dst = (uint8_t*)sm + (tid >> 6) * 1024;
#pragma unroll
    for (int t = 0; t < IB_IMG * 4 / 4096; ++t)
      __builtin_amdgcn_global_load_lds((const void*)(src + t * 4096),
                                       (__attribute__((address_space(3))) void*)(dst + t * 4096), 16, 0, 0);
  }
  __syncthreads();  // (waits for every load of the thread, the image's included)

  const int lane = tid & 63;
  uint32_t T = 0, tie = 0;
  if (mode == MODE_SELECT) {
    T = st->key;
    tie = st->tie;
  }
  const int words = (k + 31) / 32;
  IbRow s;
#pragma unroll
  for (int i = 0; i < IB_I; ++i) {
    const int c = q + IB_Q * i;
    const bool cv = rv && c < Bb;
    s.w[i] = cv ? wv[i] : 0.f;
    s.y[i] = 0.f;
    s.e[i] = 0.f;
    s.w0[i] = 0.f;
    if constexpr (NM) {
      s.f[i] = c < Bb ? fv[i] : 0.f;
      s.sc[i] = 0.f;
    }
    bool keep = true;
    if (cv) {
      if (mode == MODE_SELECT) {
        const uint32_t key = orderable(weight_score(s.w[i], fv[i]));
        const uint32_t idx = (uint32_t)c * (uint32_t)n + (uint32_t)row;
        keep = !(key < T || (key == T && idx <= tie));
      } else if (mode == MODE_FORCED) {
        const int gc = j0 + c;
        keep = (mask_in[(int64_t)row * words + gc / 32] >> (gc % 32)) & 1u;
      } else {
        keep = mode == MODE_KEEP_ALL || mode == MODE_NM;  // N:M bits are chosen in the column loop
      }
    }
    const unsigned long long ball = __ballot(keep);
    s.kb[i] = (uint32_t)(ball >> (IB_Q * (lane >> 4))) & 0xFFFFu;
  }
  const int ngroups = QUANT ? (k + opt.q_group - 1) / opt.q_group : 0;
  s.qs = 1.f;
  s.qz = 0.f;
  ib_steps<NM, QUANT, YR>(s, lq, dq, il, q, opt, row, rv, j0, Bb, ngroups, std::make_integer_sequence<int, kMaxBlock>{});
#pragma unroll
  for (int i = 0; i < IB_I; ++i) {
    const int c = q + IB_Q * i;
    if (rv && c < Bb) {
      Wo[(int64_t)row * k + j0 + c] = s.w[i];
      EW[(int64_t)row * ew_ld + c] = YR ? (yv[i] + s.y[i]) - s.e[i] : s.e[i];
      EW[(int64_t)row * ew_ld + (ew_ld >> 1) + c] = s.w0[i];
      bmask[(int64_t)row * k + j0 + c] = (uint8_t)((s.kb[i] >> q) & 1u);
      if (NM && scores_out) scores_out[(int64_t)row * k + j0 + c] = s.sc[i];
    }
  }
}

__global__ void zero_kernel(float* __restrict__ p, int64_t cnt) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < cnt / 4; i += stride)
    ((float4*)p)[i] = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int64_t i = cnt / 4 * 4 + (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < cnt; i += stride) p[i] = 0.f;
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

// 16-byte forms of init_w_kernel and finalize_kernel for k a multiple of 32,
// ldw a multiple of 4 and aligned buffers: one thread per 4 elements (per
// 32 mask bits); the same values as the element kernels.
__global__ void init_w4_kernel(const void* W, int dtype, int64_t ldw, int n, int k, float* Wo) {
  const int64_t id = (int64_t)blockIdx.x * blockDim.x + threadIdx.x, k4 = k / 4;
  if (id >= (int64_t)n * k4) return;
  const int64_t r = id / k4, c = 4 * (id % k4);
  float4 v;
  if (dtype == DUO_BF16) {
    const uint2 b = *(const uint2*)((const uint16_t*)W + r * ldw + c);
    v = make_float4(bf16_bits_to_f32((uint16_t)(b.x & 0xFFFFu)), bf16_bits_to_f32((uint16_t)(b.x >> 16)),
                    bf16_bits_to_f32((uint16_t)(b.y & 0xFFFFu)), bf16_bits_to_f32((uint16_t)(b.y >> 16)));
  } else {
    v = *(const float4*)((const float*)W + r * ldw + c);
  }
  ((float4*)Wo)[id] = v;
}

__global__ void finalize4_kernel(const float* Wo, const uint8_t* bmask, int n, int k, int dtype, void* lowp,
                                 uint32_t* mask_out) {
  const int64_t id = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (mask_out && id < (int64_t)n * (k / 32)) {
    // 32 byte flags (0 or 1) -> 32 bits: each 4-byte group gives a nibble
    // ((v & 0x01010101) * 0x01020408) >> 24 (no carries: at most 15)
    const u32x4* f = (const u32x4*)(bmask + id * 32);
    const u32x4 a = f[0], b = f[1];
    uint32_t bits = 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      bits |= (((a[i] & 0x01010101u) * 0x01020408u) >> 24) << (4 * i);
      bits |= (((b[i] & 0x01010101u) * 0x01020408u) >> 24) << (4 * i + 16);
    }
    mask_out[id] = bits;
  }
  if (lowp && id < (int64_t)n * k / 4) {
    const float4 v = ((const float4*)Wo)[id];
    if (dtype == DUO_BF16)
      ((uint2*)lowp)[id] = make_uint2((uint32_t)f32_to_bf16_bits(v.x) | ((uint32_t)f32_to_bf16_bits(v.y) << 16),
                                      (uint32_t)f32_to_bf16_bits(v.z) | ((uint32_t)f32_to_bf16_bits(v.w) << 16));
    else
      ((float4*)lowp)[id] = v;
  }
}

// Two-level lazy update.  The weight update that a processed block owes the
// columns to its right is linear in that block's (E, W0) pair, so it may be
// applied in pieces: right after block [j0, j1) only the columns up to the
// end of its super-block of kSuper columns are updated (K = block width);
// when a super-block is complete, one product with K = super-block width
// brings every column beyond it up to date.  Each block still sees, before
// its selection, every update owed to it.  EW holds the super-block's pairs,
// row-major with stride 2 S: E of column sb0 + c at c, W0 at S + c.
//
// Y form (U given instead of D; no D = U L^T is formed).  With V the values
// of the processed columns when they were processed (the W0 above), the
// residual terms owed to column c sum to (V D)_c = sum_{i <= c} L_ci y_i,
// y = V U (U strictly upper: y_i depends only on columns before i).  So the
// sweep carries Y, the earlier blocks' part of y, beside W, and a column
// before its block starts holds W_c + sum_{i < block} (y_i - e_i) L_ci.  At
// the start of a block W[:, blk] += Y[:, blk] L[blk, blk]^T adds the terms of
// the block's own columns (L lower), which makes W[:, blk] the values the D
// form has there; the in-block kernel carries the block's own part of y and
// leaves z = y - e in the E slot; the lazy products become
// W[:, rest] += Z L[rest, blk]^T and Y[:, rest] += V U[blk, rest].  Same
// products in count and size as the D form, with the k^3 / 3 of D saved.
// (1024 columns: at the 70B shape the Y form's two passes over C per
// super-block cost 4.5 ms less per layer than with 512; 2048 gained 0.8 ms
// more there and lost at k = 4096 and 11008)
constexpr int kSuper = 1024;

int super_width(int B) { return B * (kSuper / B > 1 ? kSuper / B : 1); }

struct SweepWs {
  SelState* st;
  uint32_t* hist;
  unsigned long long* cand;
  float* EW;
  uint8_t* bmask;
  float* img;  // LDS images of the blocks' L, D operands
  size_t bytes;
};

SweepWs carve(void* ws, int64_t n, int64_t k, int B) {
  Carver c(ws);
  SweepWs w;
  w.st = c.take<SelState>(1);
  w.hist = c.take<uint32_t>(kBins0);
  w.cand = c.take<unsigned long long>(kSelCap);
  w.EW = c.take<float>((size_t)n * 2 * super_width(B));
  w.bmask = c.take<uint8_t>((size_t)n * k);
  w.img = c.take<float>((size_t)cdiv(k, B) * IB_IMG);
  w.bytes = c.off;
  return w;
}

}  // namespace

size_t sweep_ws_bytes(int64_t n, int64_t k, int B) { return carve(nullptr, n, k, B).bytes; }

duo_status sweep_run(const void* W, int32_t w_dtype, int64_t n, int64_t k, int64_t ldw, const float* L, int64_t ldl,
                     const float* D, int64_t ldd, const float* fac, double p_w, const SweepOpts& o, int B,
                     const uint32_t* mask_in, float* W_out, void* W_out_lowp, uint32_t* mask_out, float* scores_out,
                     void* ws, hipStream_t s, const float* U, int64_t ldu, float* Y) {
  const SweepWs w = carve(ws, n, k, B);
  const bool yr = U != nullptr;  // Y form
  // the Y form with quantisation: only grids fixed at a block's first column,
  // where W[:, blk] holds the values of Algorithm 1 after the start product
  if (yr && ((o.q_bits > 0 && o.q_group != B) || !Y)) return DUO_ERR_UNSUPPORTED;
  const int64_t nk = n * k;
  const int64_t S = super_width(B);
  auto al16 = [](const void* q) { return (reinterpret_cast<uintptr_t>(q) & 15) == 0; };
  const bool v4 = k % 32 == 0 && ldw % 4 == 0 && (reinterpret_cast<uintptr_t>(W) & 7) == 0 && al16(W_out) &&
                  (!W_out_lowp || al16(W_out_lowp)) && al16(ws);
  if (v4)
    hipLaunchKernelGGL(init_w4_kernel, dim3((unsigned)cdiv(nk / 4, 256)), dim3(256), 0, s, W, (int)w_dtype, ldw,
                       (int)n, (int)k, W_out);
  else
    hipLaunchKernelGGL(init_w_kernel, dim3((unsigned)cdiv(nk, 256)), dim3(256), 0, s, W, (int)w_dtype, ldw, (int)n,
                       (int)k, W_out);
  DUO_LAUNCH_CHECK();
  hipLaunchKernelGGL(sel_reset_kernel, dim3(1), dim3(256), 0, s, w.st, w.hist);
  DUO_LAUNCH_CHECK();
  const size_t ib_lds = (size_t)IB_IMG * sizeof(float);
  hipLaunchKernelGGL(ib_image_kernel, dim3((unsigned)cdiv(k, B), 16), dim3(256), 0, s, L, ldl, yr ? U : D,
                     yr ? ldu : ldd, (int)k, B, w.img);
  DUO_LAUNCH_CHECK();
  if (yr) {
    hipLaunchKernelGGL(zero_kernel, dim3((unsigned)(cdiv(nk, 1024) < 8192 ? cdiv(nk, 1024) : 8192)), dim3(256), 0, s,
                       Y, nk);
    DUO_LAUNCH_CHECK();
  }
  const bool nm = o.nm_n > 0 && !mask_in;
  const bool qt = o.q_bits > 0;
  const bool wide = !nm && !qt && cdiv(n, IB_ROWS) > 256;  // 32 rows per workgroup
  const int ib_rows = wide ? IB_ROWS2 : IB_ROWS;
  auto ib_kern = yr ? (nm ? (qt ? inblock_kernel<true, true, true, IB_ROWS> : inblock_kernel<true, false, true, IB_ROWS>)
                     : qt ? inblock_kernel<false, true, true, IB_ROWS>
                          : wide ? inblock_kernel<false, false, true, IB_ROWS2> : inblock_kernel<false, false, true, IB_ROWS>)
                 : nm ? (qt ? inblock_kernel<true, true, false, IB_ROWS> : inblock_kernel<true, false, false, IB_ROWS>)
                 : qt ? inblock_kernel<false, true, false, IB_ROWS>
                      : (wide ? inblock_kernel<false, false, false, IB_ROWS2> : inblock_kernel<false, false, false, IB_ROWS>);
  const IbOpts ibo{o.nm_n, o.q_bits, qt ? o.q_group : kMaxBlock, o.q_scale, o.q_zero};
  if (duo_status d = set_max_lds((const void*)ib_kern, ib_lds); d != DUO_OK) return d;
  const size_t sel_lds = (size_t)(16 + (1 << kDigitR)) * sizeof(uint32_t) + (size_t)kRankMax * sizeof(unsigned long long);
  for (const void* f : {(const void*)sel_resolve_kernel<kSelCap / 512>, (const void*)sel_resolve_kernel<kSelCap / 256>})
    if (duo_status d = set_max_lds(f, sel_lds); d != DUO_OK) return d;
  const int P = (int)(cdiv(n, 32) < kSelWG ? cdiv(n, 32) : kSelWG);
  // rows a selection thread holds in registers: one or two batches of kRowU
  // (two threads per column, rpw rows per workgroup), else streamed
  const int64_t rpw = cdiv(n, P);
  const int hb = rpw <= 2 * kRowU ? 1 : (rpw <= 4 * kRowU ? 2 : 0);
  const int sh0 = n * (int64_t)(k < B ? k : B) >= ((int64_t)1 << 20) ? kShift0 : kShift0 + 2;
  // half the candidate registers for the 8192-bin histogram's smaller buckets
  auto resolve_k = sh0 == kShift0 + 2 ? sel_resolve_kernel<kSelCap / 512> : sel_resolve_kernel<kSelCap / 256>;
  auto hist_k = hb == 1 ? sel_hist_kernel<1> : (hb == 2 ? sel_hist_kernel<2> : sel_hist_kernel<0>);
  auto gather_k = hb == 1 ? sel_gather_kernel<1> : (hb == 2 ? sel_gather_kernel<2> : sel_gather_kernel<0>);
  const size_t hist_lds = (size_t)kBins0 * sizeof(uint32_t);
  for (const void* f : {(const void*)sel_hist_kernel<0>, (const void*)sel_hist_kernel<1>, (const void*)sel_hist_kernel<2>})
    if (duo_status d = set_max_lds(f, hist_lds); d != DUO_OK) return d;
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
    else if (nm)
      mode = MODE_NM;
    else if (z <= 0)
      mode = MODE_KEEP_ALL;
    else if (z >= total)
      mode = MODE_PRUNE_ALL;
    int idx_bits = 1;
    while (idx_bits < 31 && ((int64_t)1 << idx_bits) < total) ++idx_bits;
    if (yr && j0 > 0) {
      // Y form: W[:, blk] += Y[:, blk] L[blk, blk]^T (the residual terms of the
      // block's own columns owed by the earlier blocks)
      GemmDesc c{};
      c.M = (int)n;
      c.N = Bb;
      c.C = W_out + j0;
      c.ldc = k;
      c.beta = 1.f;
      c.tri = TRI_ALL;
      c.nterms = 1;
      c.t[0] = GemmTerm{Y + j0, k, 1, L + j0 * ldl + j0, ldl, 0, Bb, 1.f, KLO_ZERO, KHI_FULL};
      prof_begin(DUO_PROF_TRAIL, s);
      duo_status st = gemm_f32(c, s);
      prof_end(DUO_PROF_TRAIL, s);
      if (st != DUO_OK) return st;
    }
    prof_begin(DUO_PROF_SELECT, s);
    if (mode == MODE_SELECT || (scores_out && mode != MODE_NM)) {
      hipLaunchKernelGGL(scores_out ? sel_hist_kernel<0> : hist_k, dim3(P), dim3(256), hist_lds, s,
                         (const float*)W_out, k, (int)n, Bb, (int)j0, fac, w.hist, scores_out,
                         mode == MODE_SELECT ? 1 : 0, w.st, sh0);
      DUO_LAUNCH_CHECK();
    }
    if (mode == MODE_SELECT) {
      hipLaunchKernelGGL(gather_k, dim3(P), dim3(256), 0, s, (const float*)W_out, k, (int)n, Bb, (int)j0, fac,
                         (uint32_t)z, idx_bits, (const uint32_t*)w.hist, w.st, w.cand, sh0);
      DUO_LAUNCH_CHECK();
      hipLaunchKernelGGL(resolve_k, dim3(1), dim3(256), sel_lds, s, (const float*)W_out, k, (int)n, Bb,
                         (int)j0, fac, (uint32_t)z, idx_bits, w.hist, w.st, (const unsigned long long*)w.cand, sh0);
      DUO_LAUNCH_CHECK();
    }
    prof_end(DUO_PROF_SELECT, s);
    prof_begin(DUO_PROF_INBLOCK, s);
    const int64_t sb0 = j0 / S * S, sb1 = sb0 + S < k ? sb0 + S : k;
    hipLaunchKernelGGL(ib_kern, dim3((unsigned)cdiv(n, ib_rows)), dim3(ib_rows * IB_Q), ib_lds, s, W_out, (int)n, (int)k,
                       (int)j0, Bb, (int64_t)2 * S, fac, (const SelState*)w.st, mode, mask_in,
                       w.EW + (j0 - sb0), w.bmask, ibo, scores_out, (const float*)(w.img + (j0 / B) * IB_IMG),
                       (const float*)Y);
    DUO_LAUNCH_CHECK();
    prof_end(DUO_PROF_INBLOCK, s);
    // inside the super-block: columns [j1, sb1) from this block (K = Bb);
    // at its end: columns [sb1, k) from the whole super-block (K = sb1 - sb0)
    const int64_t u0 = j1 < sb1 ? j0 : sb0, c0 = j1, c1 = j1 < sb1 ? sb1 : k;
    if (c0 < c1) {
      const int K = (int)(j1 - u0);
      GemmDesc g{};
      g.M = (int)n;
      g.N = (int)(c1 - c0);
      g.C = W_out + c0;
      g.ldc = k;
      g.beta = 1.f;
      g.tri = TRI_ALL;
      g.nterms = 2;
      if (yr) {
        // W[:, c0:c1] += Z L[c0:c1, u0:j1]^T and Y[:, c0:c1] += V U[u0:j1, c0:c1]:
        // independent, one launch
        g.dual = 1;
        g.C2 = Y + c0;
        g.t[0] = GemmTerm{w.EW + (u0 - sb0), 2 * S, 1, L + c0 * ldl + u0, ldl, 0, K, 1.f, KLO_ZERO, KHI_FULL};
        g.t[1] = GemmTerm{w.EW + S + (u0 - sb0), 2 * S, 1, U + u0 * ldu + c0, ldu, 1, K, 1.f, KLO_ZERO, KHI_FULL};
        prof_begin(DUO_PROF_TRAIL, s);
        duo_status st = gemm_f32(g, s);
        prof_end(DUO_PROF_TRAIL, s);
        if (st != DUO_OK) return st;
      } else {
        g.t[0] = GemmTerm{w.EW + (u0 - sb0), 2 * S, 1, L + c0 * ldl + u0, ldl, 0, K, -1.f, KLO_ZERO, KHI_FULL};
        g.t[1] = GemmTerm{w.EW + S + (u0 - sb0), 2 * S, 1, D + u0 * ldd + c0, ldd, 1, K, 1.f, KLO_ZERO, KHI_FULL};
        prof_begin(DUO_PROF_TRAIL, s);
        duo_status st = gemm_f32(g, s);
        prof_end(DUO_PROF_TRAIL, s);
        if (st != DUO_OK) return st;
      }
    }
  }
  if (mask_out || W_out_lowp) {
    const int64_t words = cdiv(k, 32);
    if (v4) {
      const int64_t cnt = nk / 4 > n * words ? nk / 4 : n * words;
      hipLaunchKernelGGL(finalize4_kernel, dim3((unsigned)cdiv(cnt, 256)), dim3(256), 0, s, (const float*)W_out,
                         (const uint8_t*)w.bmask, (int)n, (int)k, (int)w_dtype, W_out_lowp, mask_out);
    } else {
      const int64_t cnt = nk > n * words ? nk : n * words;
      hipLaunchKernelGGL(finalize_kernel, dim3((unsigned)cdiv(cnt, 256)), dim3(256), 0, s, (const float*)W_out,
                         (const uint8_t*)w.bmask, (int)n, (int)k, (int)w_dtype, W_out_lowp, mask_out);
    }
    DUO_LAUNCH_CHECK();
  }
  return DUO_OK;
}

}  // namespace duo
