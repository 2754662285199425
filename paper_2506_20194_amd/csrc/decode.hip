// Dual-sparse decode GEMV (Preliminaries "Activation Sparsity" and Sec. 4.1):
// y = W (x * m^x) = sum over the channels i whose activation survives of
// W[:, i] x_i.  Only those columns are read, each stored compressed:
//
//   maskT      k x ceil(n/32) uint32, channel-major: bit r % 32 of word r / 32
//              of channel i set when W[r][i] is kept;
//   values     the kept weights of each channel in row order (bf16), channel
//              i at [col_ptr[i], col_ptr[i + 1]);
//   chunk_off  k x ceil(n/256) uint16: kept weights of channel i in rows
//              [0, 256 c), so that row r's value sits at col_ptr[i] +
//              chunk_off[i][r / 256] + (kept rows in [256 (r / 256), r)).
//
// A fetched column costs n/8 + n/128 + 2 nnz bytes (1.13 n at 50 % weight
// sparsity against 2 n dense), and a wave finds its 64 rows' values from two
// mask words and one offset, all wave-uniform (scalar loads).
#include <hip/hip_runtime.h>

#include <cmath>
#include <mutex>

#include "internal.h"

using namespace duo;

namespace {

constexpr int kChunk = 256;     // rows per chunk offset

// magnitude bits (the activation rule's key, as in the Hessian stage) and value
template <typename T>
struct Act;
template <>
struct Act<uint16_t> {
  __device__ static uint32_t mag(uint16_t v) { return v & 0x7fffu; }
  __device__ static float to_f32(uint16_t v) { return bf16_bits_to_f32(v); }
};
template <>
struct Act<float> {
  __device__ static uint32_t mag(float v) { return __float_as_uint(v) & 0x7fffffffu; }
  __device__ static float to_f32(float v) { return v; }
};
constexpr int64_t kMaxDecodeN = 32768;  // rows: 4 mask words per thread

// ---- layout ----

// maskT[i][w] from the sweep's row-major mask (n x ceil(k/32) words).
__global__ __launch_bounds__(256) void dsc_mask_t_kernel(const uint32_t* __restrict__ mrow, int64_t n, int64_t k,
                                                         uint32_t* __restrict__ maskT) {
  const int64_t wn = (n + 31) / 32, wk = (k + 31) / 32;
  const int64_t id = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (id >= k * wn) return;
  const int64_t i = id % k, w = id / k;  // consecutive threads: consecutive channels
  uint32_t bits = 0;
  for (int b = 0; b < 32; ++b) {
    const int64_t r = w * 32 + b;
    if (r >= n) break;
    bits |= ((mrow[r * wk + i / 32] >> (i % 32)) & 1u) << b;
  }
  maskT[i * wn + w] = bits;
}

// Per channel: kept count and the prefix counts at each 256-row chunk.
__global__ __launch_bounds__(256) void dsc_count_kernel(const uint32_t* __restrict__ maskT, int64_t n, int64_t k,
                                                        uint16_t* __restrict__ chunk_off, int64_t* __restrict__ cnt) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= k) return;
  const int64_t wn = (n + 31) / 32, nc = (n + kChunk - 1) / kChunk;
  int64_t c = 0;
  for (int64_t w = 0; w < wn; ++w) {
    if (w % (kChunk / 32) == 0) chunk_off[i * nc + w / (kChunk / 32)] = (uint16_t)c;
    c += __popc(maskT[i * wn + w]);
  }
  cnt[i] = c;
}

// col_ptr = exclusive scan of the counts (one workgroup of 1024 threads).
__global__ __launch_bounds__(1024) void dsc_scan_kernel(const int64_t* __restrict__ cnt, int64_t k,
                                                        int64_t* __restrict__ col_ptr) {
  __shared__ int64_t part[1024];
  const int t = threadIdx.x;
  const int64_t per = (k + 1023) / 1024;
  const int64_t i0 = t * per, i1 = i0 + per < k ? i0 + per : k;
  int64_t s = 0;
  for (int64_t i = i0; i < i1; ++i) s += cnt[i];
  part[t] = s;
  __syncthreads();
  for (int d = 1; d < 1024; d *= 2) {
    const int64_t v = t >= d ? part[t - d] : 0;
    __syncthreads();
    part[t] += v;
    __syncthreads();
  }
  int64_t run = part[t] - s;  // exclusive prefix of this thread's range
  for (int64_t i = i0; i < i1; ++i) {
    col_ptr[i] = run;
    run += cnt[i];
  }
  if (t == 1023) col_ptr[k] = part[1023];
}

// values: one thread per (row, channel) of W (row-major reads).
__global__ __launch_bounds__(256) void dsc_pack_kernel(const void* __restrict__ W, int dtype, int64_t n, int64_t k,
                                                       int64_t ldw, const int64_t* __restrict__ col_ptr,
                                                       const uint32_t* __restrict__ maskT,
                                                       const uint16_t* __restrict__ chunk_off,
                                                       uint16_t* __restrict__ values) {
  const int64_t id = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (id >= n * k) return;
  const int64_t r = id / k, i = id % k;
  const int64_t wn = (n + 31) / 32, nc = (n + kChunk - 1) / kChunk;
  const uint32_t* mw = maskT + i * wn;
  const int64_t w = r / 32;
  if (!((mw[w] >> (r % 32)) & 1u)) return;
  int64_t rank = chunk_off[i * nc + r / kChunk];
  for (int64_t q = (r / kChunk) * (kChunk / 32); q < w; ++q) rank += __popc(mw[q]);
  rank += __popc(mw[w] & ((1u << (r % 32)) - 1u));
  const uint16_t v = dtype == DUO_BF16 ? ((const uint16_t*)W)[r * ldw + i]
                                       : f32_to_bf16_bits(((const float*)W)[r * ldw + i]);
  values[col_ptr[i] + rank] = v;
}

// ---- GEMV ----
//
// One kernel per decode step plus a reduction.  Workgroup (slab sl, share s)
// of ns x S covers output rows [2048 sl, 2048 sl + 2048) (64 mask words, one
// per lane of a wave) and the active channels of rank s, s + S, ... in
// channel order:
//   1. every workgroup selects the active channels itself (the calibration
//      rule over x, a few KB read from L2), so no launch sits between the
//      selection and the GEMV, and keeps its own share in LDS;
//   2. it loads each of its channels' slab window (first value, length) from
//      col_ptr and chunk_off;
//   3. its 16 waves take the share's channels round robin; a wave keeps three
//      channels' loads in flight (mask word, chunk offset and a 16-byte value
//      window per lane, all issued unconditionally at clamped addresses, so
//      the compiler's in-order wait counts let the younger loads stay in
//      flight), stages a channel's values in its own LDS slot and
//      accumulates its 32 rows per lane in registers;
//   4. the 16 waves' sums are added in a fixed order through LDS and the
//      workgroup writes its partial rows; dsc_reduce_kernel adds the S
//      partials of each row in a fixed order.
constexpr int kGemvWaves = 16;
constexpr int kGemvThreads = kGemvWaves * 64;
constexpr int kSlabRows = 2048;               // rows of one slab: 64 words of 32
constexpr int kWindowQ = kSlabRows / 8 + 1;   // 16-byte entries of the largest window (alignment included)
constexpr int kQV = (kWindowQ + 63) / 64;     // 16-byte value loads per lane: a whole window
constexpr int kSlotQ = 64 * kQV;              // a wave's value slot: every lane stores all of its loads
constexpr int kTargetGroups = 256;            // one 1024-thread workgroup per CU

// Exclusive scan over the block's threads in thread order (two barriers).
__device__ inline uint32_t block_excl_scan(uint32_t v, uint32_t* sh, uint32_t& total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  uint32_t incl = v;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const uint32_t o = __shfl_up(incl, d);
    if (lane >= d) incl += o;
  }
  __syncthreads();
  if (lane == 63) sh[wave] = incl;
  __syncthreads();
  uint32_t before = 0;
  total = 0;
#pragma unroll
  for (int w = 0; w < kGemvWaves; ++w) {
    before += w < wave ? sh[w] : 0;
    total += sh[w];
  }
  return before + incl - v;
}

// The magnitudes of channels [c0, c0 + KPT) (all ones past k): 16-byte loads
// where the range is whole and aligned, else clamped element loads; either way
// every load is issued before the first use.
template <typename T, int KPT>
__device__ inline void load_mags(const T* __restrict__ x, int k, int c0, uint32_t (&mag)[KPT]) {
  constexpr int PER = 16 / sizeof(T), NV = KPT / PER;
  if (c0 + KPT <= k && ((uintptr_t)(x + c0) & 15) == 0) {
    u32x4 r[NV];
#pragma unroll
    for (int q = 0; q < NV; ++q) r[q] = ((const u32x4*)(x + c0))[q];
#pragma unroll
    for (int q = 0; q < NV; ++q) {
      const uint32_t wds[4] = {r[q][0], r[q][1], r[q][2], r[q][3]};
#pragma unroll
      for (int h = 0; h < 4; ++h) {
        if constexpr (sizeof(T) == 2) {
          mag[q * PER + 2 * h] = wds[h] & 0x7fffu;
          mag[q * PER + 2 * h + 1] = (wds[h] >> 16) & 0x7fffu;
        } else {
          mag[q * PER + h] = wds[h] & 0x7fffffffu;
        }
      }
    }
  } else {
    T v[KPT];
#pragma unroll
    for (int e = 0; e < KPT; ++e) v[e] = x[c0 + e < k ? c0 + e : k - 1];
#pragma unroll
    for (int e = 0; e < KPT; ++e) mag[e] = c0 + e < k ? Act<T>::mag(v[e]) : 0xffffffffu;
  }
}

// bf16 magnitudes (15 bits): Tm = the z-th smallest (1 <= z < the number of
// valid entries) and the number below it, from one LDS histogram of all 32768
// magnitudes (one atomic per entry; bin b at word b + b / 32, so that thread
// t's 32 bins [32 t, 32 t + 32) sit 33 words from its neighbours' and the
// scan's reads are free of bank conflicts) and a block scan of the bins.
constexpr int kHistWords = 32768 + 32768 / 32;

template <int KPT>
__device__ inline void hist_select(const uint32_t (&mag)[KPT], int z, uint32_t* hist, int* found, uint32_t* sh,
                                   uint32_t& Tm, int& nbelow) {
  const int t = threadIdx.x;
  for (int q = t; q < kHistWords / 4; q += kGemvThreads) ((u32x4*)hist)[q] = u32x4{0u, 0u, 0u, 0u};
  __syncthreads();
#pragma unroll
  for (int e = 0; e < KPT; ++e)
    if (mag[e] < 32768u) atomicAdd(&hist[mag[e] + (mag[e] >> 5)], 1u);
  __syncthreads();
  uint32_t sum = 0;
#pragma unroll
  for (int b = 0; b < 32; ++b) sum += hist[33 * t + b];
  uint32_t tot;
  const uint32_t before = block_excl_scan(sum, sh, tot);
  if ((int)before < z && z <= (int)(before + sum)) {  // one thread: its bins again, all read at once
    uint32_t h[32];
#pragma unroll
    for (int b = 0; b < 32; ++b) h[b] = hist[33 * t + b];
    uint32_t run = before;
    int fb = 0, fr = 0;
#pragma unroll
    for (int b = 0; b < 32; ++b) {
      if ((int)run < z && z <= (int)(run + h[b])) {
        fb = b;
        fr = (int)run;
      }
      run += h[b];
    }
    found[0] = 32 * t + fb;
    found[1] = fr;
  }
  __syncthreads();
  Tm = (uint32_t)found[0];
  nbelow = found[1];
}

// Tm = the z-th smallest magnitude (1 <= z < the number of valid entries) and
// the number of magnitudes below it: a radix select over digits of up to 8
// bits from the top, each digit found from an LDS histogram of the entries
// that match the digits found so far.  Entries past k hold all ones, which
// never match (magnitudes have MB bits).
template <int MB, int KPT>
__device__ inline void radix_select(const uint32_t (&mag)[KPT], int z, uint32_t* hist, int* found, uint32_t& Tm,
                                    int& nbelow) {
  const int t = threadIdx.x;
  uint32_t prefix = 0;
  int need = z, below = 0, top = MB;
  while (top > 0) {
    const int shift = top > 8 ? top - 8 : 0;
    const uint32_t dmask = (1u << (top - shift)) - 1u;
    if (t < 256) hist[t] = 0;
    __syncthreads();
#pragma unroll
    for (int e = 0; e < KPT; ++e)
      if ((mag[e] >> top) == prefix) atomicAdd(&hist[(mag[e] >> shift) & dmask], 1u);
    __syncthreads();
    if (t < 64) {  // one wave: the digit whose bin holds the need-th entry
      uint32_t h[4], local = 0;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        h[q] = hist[4 * t + q];
        local += h[q];
      }
      uint32_t incl = local;
#pragma unroll
      for (int d = 1; d < 64; d <<= 1) {
        const uint32_t o = __shfl_up(incl, d);
        if (t >= d) incl += o;
      }
      int run = (int)(incl - local);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        if (run < need && need <= run + (int)h[q]) {
          found[0] = 4 * t + q;
          found[1] = run;
        }
        run += (int)h[q];
      }
    }
    __syncthreads();
    prefix = (prefix << (top - shift)) | (uint32_t)found[0];
    below += found[1];
    need -= found[1];
    top = shift;
  }
  Tm = prefix;
  nbelow = below;
}

typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2_t;

struct DscSlab {
  uint32_t m;   // the lane's mask word
  uint32_t co;  // kept values of the channel before the word's 256-row chunk
  u32x4 v[kQV];
  // wave-uniform: the channel's first value, its activation (fp32 bits) and
  // the window's aligned start (element offsets into values; the layout has
  // fewer than 2^31 values at the GEMV's size limits)
  uint32_t base, xbits, a0;
};

template <typename T>
__global__ __launch_bounds__(kGemvThreads) void dsc_gemv_kernel(const T* __restrict__ x, int k, int z, int64_t n,
                                                                const int64_t* __restrict__ col_ptr,
                                                                const uint32_t* __restrict__ maskT,
                                                                const uint16_t* __restrict__ chunk_off,
                                                                const uint16_t* __restrict__ values, int S, int cap,
                                                                float* __restrict__ ypart) {
  constexpr int KPT = kMaxK / kGemvThreads;  // channels per thread in the selection: 32
  constexpr int MB = sizeof(T) == 2 ? 15 : 31;  // magnitude bits
  extern __shared__ __attribute__((aligned(16))) uint8_t dyn[];
  __shared__ uint32_t hist[256];
  __shared__ int found[2];
  __shared__ uint32_t scan_sh[kGemvWaves];
  const int t = threadIdx.x, lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);  // uniform: keeps the wave's loop scalar
  const int s = blockIdx.x % S, sl = blockIdx.x / S;
  const int64_t wn = (n + 31) / 32, nc = (n + kChunk - 1) / kChunk;
  int4* lmeta = (int4*)dyn;                         // [cap]: the share's channels
  u32x4* slots = (u32x4*)(dyn + 16 * (size_t)cap);  // [kGemvWaves][1 + kSlotQ]: a guard entry, then the slot

  // 1. selection: the z smallest (|x|, channel) keys are dropped; the
  // workgroup's share is the active channels of rank [lo, hi) in channel order
  const int c0 = t * KPT;
  uint32_t mag[KPT];
  load_mags<T, KPT>(x, k, c0, mag);
  uint32_t Tm = z >= k ? 0xffffffffu : 0u;  // z = 0: everything kept; z >= k: nothing
  int nbelow = 0;
  if (z > 0 && z < k) {
    if constexpr (MB == 15)
      hist_select<KPT>(mag, z, (uint32_t*)dyn, found, scan_sh, Tm, nbelow);
    else
      radix_select<MB, KPT>(mag, z, hist, found, Tm, nbelow);
  }
  const int drop_eq = z > 0 && z < k ? z - nbelow : 0;  // entries equal to Tm dropped, in channel order
  const int nv = min(KPT, max(0, k - c0));                // the thread's valid entries
  uint32_t gt = 0, eq = 0;
#pragma unroll
  for (int e = 0; e < KPT; ++e) {
    gt += e < nv && mag[e] > Tm ? 1u : 0u;
    eq += e < nv && mag[e] == Tm ? 1u : 0u;
  }
  uint32_t tot;  // both counts in one scan: each total is at most 32768
  const uint32_t before = block_excl_scan((gt << 16) | eq, scan_sh, tot);
  const int gt_b = (int)(before >> 16), eq_b = (int)(before & 0xffffu);
  int na = (int)(tot >> 16) + max(0, (int)(tot & 0xffffu) - drop_eq);
  na = __builtin_amdgcn_readfirstlane(na);
  const int j0 = gt_b + max(0, eq_b - drop_eq);  // rank of the thread's first kept channel
  const int kc = (int)gt + max(0, eq_b + (int)eq - max(eq_b, drop_eq));
  const int lo = s * cap, hi = min(na, lo + cap);
  if (kc > 0 && j0 < hi && j0 + kc > lo) {  // the few threads holding the share
    uint32_t gm = 0, em = 0;
#pragma unroll
    for (int e = 0; e < KPT; ++e) {
      gm |= (e < nv && mag[e] > Tm ? 1u : 0u) << e;
      em |= (e < nv && mag[e] == Tm ? 1u : 0u) << e;
    }
    for (int r = drop_eq - eq_b; r > 0 && em; --r) em &= em - 1u;  // the first ties in channel order are dropped
    uint32_t km = gm | em;
    for (int j = j0; km; ++j, km &= km - 1u)
      if (j >= lo && j < hi) lmeta[j - lo] = int4{c0 + (int)__builtin_ctz(km), 0, 0, 0};
  }
  __syncthreads();
  const int mine = max(0, hi - lo);

  // 2. each channel's slab window: values[base + st, base + st + len)
  for (int q = t; q < mine; q += kGemvThreads) {
    const int i = lmeta[q].x;
    const int64_t base = col_ptr[i];
    const int st = sl > 0 ? (int)chunk_off[(int64_t)i * nc + 8 * sl] : 0;
    const int en = 8 * (sl + 1) < nc ? (int)chunk_off[(int64_t)i * nc + 8 * (sl + 1)] : (int)(col_ptr[i + 1] - base);
    lmeta[q] = int4{i, (int)__float_as_uint(Act<T>::to_f32(x[i])), (int)base, st | ((en - st) << 16)};
  }
  __syncthreads();

  // 3. the wave's channels q = wave, wave + 16, ...
  float acc[32];
#pragma unroll
  for (int b = 0; b < 32; ++b) acc[b] = 0.f;
  const int nw = mine > wave ? (mine - wave + kGemvWaves - 1) / kGemvWaves : 0;
  const int64_t w = 64 * (int64_t)sl + lane, wc = w < wn ? w : wn - 1;
  u32x4* slot = slots + wave * (kSlotQ + 1) + 1;
  const uint16_t* slot16 = (const uint16_t*)slot;
  // bf16 activations: each row is one v_dot2 of {w, 0} and {x, 0} (exact
  // bf16 products, fp32 sums); fp32 activations: an fma
  constexpr bool DOT = sizeof(T) == 2;
  auto entry = [&](int q) {  // the wave-uniform entry q
    const int4 e = lmeta[q];
    return int4{__builtin_amdgcn_readfirstlane(e.x), __builtin_amdgcn_readfirstlane(e.y),
                __builtin_amdgcn_readfirstlane(e.z), __builtin_amdgcn_readfirstlane(e.w)};
  };
  const uint32_t wcu = (uint32_t)wc, wnu = (uint32_t)wn, ncu = (uint32_t)nc;
  auto fetch = [&](int jj, DscSlab& c) {
    const int4 e = entry(wave + kGemvWaves * (jj < nw ? jj : nw - 1));
    const uint32_t i = (uint32_t)e.x, st = (uint32_t)e.z + ((uint32_t)e.w & 0xffffu), len = (uint32_t)e.w >> 16;
    const uint32_t a0 = st & ~7u;
    const int nq = (int)((st + len - a0 + 7u) >> 3);
    const int last = nq > 0 ? nq - 1 : 0;
    c.base = (uint32_t)e.z;
    c.xbits = (uint32_t)e.y;
    c.a0 = a0;
    c.m = maskT[i * wnu + wcu];
    c.co = chunk_off[i * ncu + wcu / 8u];
#pragma unroll
    for (int qv = 0; qv < kQV; ++qv) {
      const int idx = lane + 64 * qv < last ? lane + 64 * qv : last;
      c.v[qv] = *(const u32x4*)(values + (a0 + 8u * (uint32_t)idx));
    }
    __builtin_amdgcn_sched_barrier(0);  // issue the loads here, ahead of the consume that follows
  };
  auto consume = [&](const DscSlab& c) {
    const float xv = __uint_as_float(c.xbits);
    const bf16x2_t xb = __builtin_bit_cast(bf16x2_t, c.xbits >> 16);  // {x, 0}: exact for bf16 x
#pragma unroll
    for (int qv = 0; qv < kQV; ++qv) slot[lane + 64 * qv] = c.v[qv];  // past the window: unread
    __builtin_amdgcn_wave_barrier();
    const uint32_t m = w < wn ? c.m : 0u;
    const int p = __popc(m);
    // exclusive prefix of the popcounts over the 8 words of the lane's 256-row chunk (DPP row shifts)
    int incl = p;
    int r = __builtin_amdgcn_update_dpp(0, incl, 0x111, 0xf, 0xf, true);  // row_shr:1
    incl += (lane & 7) >= 1 ? r : 0;
    r = __builtin_amdgcn_update_dpp(0, incl, 0x112, 0xf, 0xf, true);  // row_shr:2
    incl += (lane & 7) >= 2 ? r : 0;
    r = __builtin_amdgcn_update_dpp(0, incl, 0x114, 0xf, 0xf, true);  // row_shr:4
    incl += (lane & 7) >= 4 ? r : 0;
    // branch-free, rows from the top: the pointer sits on the value of the
    // highest kept row not yet passed and steps down past each kept row; a
    // pruned row reads that value (or the guard entry) and masks it to zero
    const uint16_t* ptr = slot16 + ((int)(c.base + c.co + (uint32_t)incl - c.a0) - 1);
#pragma unroll
    for (int g = 24; g >= 0; g -= 8) {
      uint32_t raw[8];
      int mk[8];
#pragma unroll
      for (int b = 7; b >= 0; --b) {
        mk[b] = (int)(m << (31 - g - b)) >> 31;  // all ones where the row is kept
        raw[b] = *ptr;
        ptr += mk[b];
      }
#pragma unroll
      for (int b = 7; b >= 0; --b) {
        if constexpr (DOT)
          acc[g + b] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, raw[b] & (uint32_t)mk[b]), xb,
                                                       acc[g + b], false);
        else
          acc[g + b] = fmaf(__uint_as_float((raw[b] << 16) & (uint32_t)mk[b]), xv, acc[g + b]);
      }
    }
    __builtin_amdgcn_wave_barrier();
  };
  if (nw > 0) {
    // the loop body has no branch, so no later pass can sink a prefetch
    // below the consume it should overlap; fetches past the end re-read the
    // last channel
    DscSlab ca, cb, cc;
    fetch(0, ca);
    fetch(1, cb);
    int jj = 0;
    for (; jj + 3 <= nw; jj += 3) {
      fetch(jj + 2, cc);
      consume(ca);
      fetch(jj + 3, ca);
      consume(cb);
      fetch(jj + 4, cb);
      consume(cc);
    }
    if (jj < nw) consume(ca);
    if (jj + 1 < nw) consume(cb);
  }

  // 4. the waves' sums in a fixed order: (v + v + 8) for v < 8, then in v order
  float* red = (float*)dyn;  // [8][32][65], over the LDS of steps 1-3
  __syncthreads();
  if (wave >= 8)
#pragma unroll
    for (int b = 0; b < 32; ++b) red[((wave - 8) * 32 + b) * 65 + lane] = acc[b];
  __syncthreads();
  if (wave < 8)
#pragma unroll
    for (int b = 0; b < 32; ++b) red[(wave * 32 + b) * 65 + lane] += acc[b];
  __syncthreads();
  for (int rr = t; rr < kSlabRows; rr += kGemvThreads) {
    const int l = rr >> 5, b = rr & 31;
    float y = 0.f;
#pragma unroll
    for (int v = 0; v < 8; ++v) y += red[(v * 32 + b) * 65 + l];
    const int64_t row = (int64_t)kSlabRows * sl + rr;
    if (row < n) ypart[(int64_t)s * n + row] = y;
  }
}

constexpr size_t kRedBytes = 8 * 32 * 65 * sizeof(float);

// y[r] = sum of the S partial rows in a fixed order: 16 strided running sums
// (partials g, g + 16, ...), then the 16 in order; a workgroup of 1024
// threads takes 64 rows, so each thread issues only S / 16 loads at once.
__global__ __launch_bounds__(1024) void dsc_reduce_kernel(const float* __restrict__ ypart, int64_t n, int S,
                                                          float* __restrict__ y) {
  __shared__ float part[16][65];
  const int g = threadIdx.x >> 6, l = threadIdx.x & 63;
  const int64_t r = (int64_t)blockIdx.x * 64 + l;
  float a = 0.f;
  if (r < n) {
#pragma unroll 16
    for (int p = g; p < S; p += 16) a += ypart[(int64_t)p * n + r];
  }
  part[g][l] = a;
  __syncthreads();
  if (g == 0 && r < n) {
    float v = 0.f;
#pragma unroll
    for (int h = 0; h < 16; ++h) v += part[h][l];
    y[r] = v;
  }
}

struct GemvPlan {
  int ns, S, cap;
  size_t lds;
};

GemvPlan gemv_plan(int64_t n, int na) {
  GemvPlan p;
  p.ns = (int)cdiv(n, kSlabRows);
  const int per = kTargetGroups / p.ns > 0 ? kTargetGroups / p.ns : 1;
  p.S = na < per ? (na > 0 ? na : 1) : per;
  p.cap = (na + p.S - 1) / p.S;
  const size_t a = 16 * (size_t)p.cap + (size_t)kGemvWaves * (kSlotQ + 1) * 16;
  p.lds = a > kRedBytes ? a : kRedBytes;
  if (p.lds < kHistWords * sizeof(uint32_t)) p.lds = kHistWords * sizeof(uint32_t);  // the bf16 selection's histogram
  return p;
}

size_t dsc_ws_bytes(int64_t n, int64_t k) {
  const size_t g = align_up((size_t)kTargetGroups * n * sizeof(float));
  const size_t l = align_up((size_t)k * sizeof(int64_t));
  return g > l ? g : l;
}

duo_status gemv_check(const void* x, int32_t x_dtype, int64_t n, int64_t k, duo_act_rule rule,
                      const int64_t* col_ptr, const uint32_t* maskT, const uint16_t* chunk_off,
                      const uint16_t* values, float* y) {
  if (!x || !col_ptr || !maskT || !chunk_off || !values || !y || n < 1 || k < 1) return DUO_ERR_INVALID_ARG;
  if (x_dtype != DUO_F32 && x_dtype != DUO_BF16) return DUO_ERR_INVALID_ARG;
  if (rule.kind != DUO_ACT_NONE &&
      !(rule.kind == DUO_ACT_TOPK_MAG_PER_TOKEN && rule.sparsity >= 0.0 && rule.sparsity <= 1.0))
    return DUO_ERR_INVALID_ARG;
  if (n > kMaxDecodeN || k > kMaxK) return DUO_ERR_UNSUPPORTED;
  if (((uintptr_t)values & 15) != 0) return DUO_ERR_INVALID_ARG;
  return DUO_OK;
}

// The GEMV kernel writes every (share, row) entry of the partial rows before
// the reduction reads them, so the partial buffer needs no clearing.
duo_status gemv_launch(const void* x, int32_t x_dtype, int64_t n, int64_t k, duo_act_rule rule,
                       const int64_t* col_ptr, const uint32_t* maskT, const uint16_t* chunk_off,
                       const uint16_t* values, float* y, float* ypart, hipStream_t s) {
  const int z = rule.kind == DUO_ACT_NONE ? 0 : (int)floor(rule.sparsity * (double)k + 0.5);
  const GemvPlan p = gemv_plan(n, (int)(k - z));  // the rule keeps exactly k - z channels
  const void* kern = x_dtype == DUO_BF16 ? (const void*)dsc_gemv_kernel<uint16_t> : (const void*)dsc_gemv_kernel<float>;
  if (duo_status d = set_max_lds(kern, p.lds); d != DUO_OK) return d;
  prof_begin(DUO_PROF_DECODE, s);
  if (x_dtype == DUO_BF16)
    hipLaunchKernelGGL(dsc_gemv_kernel<uint16_t>, dim3((unsigned)(p.ns * p.S)), dim3(kGemvThreads), p.lds, s,
                       (const uint16_t*)x, (int)k, z, n, col_ptr, maskT, chunk_off, values, p.S, p.cap, ypart);
  else
    hipLaunchKernelGGL(dsc_gemv_kernel<float>, dim3((unsigned)(p.ns * p.S)), dim3(kGemvThreads), p.lds, s,
                       (const float*)x, (int)k, z, n, col_ptr, maskT, chunk_off, values, p.S, p.cap, ypart);
  DUO_LAUNCH_CHECK();
  prof_end(DUO_PROF_DECODE, s);
  hipLaunchKernelGGL(dsc_reduce_kernel, dim3((unsigned)cdiv(n, 64)), dim3(1024), 0, s, (const float*)ypart, n, p.S, y);
  DUO_LAUNCH_CHECK();
  return DUO_OK;
}

// Partial rows of the allocation-free GEMV: at most kTargetGroups shares of
// kSlabRows rows each (gemv_plan gives S * n <= 256 * 2048 for every n),
// 2 MiB per device, held until the process ends.  Host code never passes the
// array's name to a kernel: the device address comes from
// hipGetSymbolAddress, once per device with that device current.
constexpr size_t kScratchFloats = (size_t)kTargetGroups * kSlabRows;

}  // namespace

static __device__ __align__(256) float scratch[kScratchFloats];

namespace {

std::mutex g_scratch_mu;
float* g_scratch_dev[64];  // per device index; set once, then only read

duo_status scratch_address(float** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return DUO_ERR_HIP;
  if (dev < 0 || dev >= 64) return DUO_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_dev[dev]) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return DUO_ERR_HIP;
    g_scratch_dev[dev] = (float*)ptr;
  }
  *out = g_scratch_dev[dev];
  return DUO_OK;
}

}  // namespace

extern "C" {

size_t duo_dsc_workspace_size(int64_t n, int64_t k) {
  if (n < 1 || k < 1 || n > 65535 || k > kMaxK) return 0;
  return dsc_ws_bytes(n, k);
}

duo_status duo_dsc_layout(const uint32_t* mask, int64_t n, int64_t k, int64_t* col_ptr, uint32_t* maskT,
                          uint16_t* chunk_off, void* ws, size_t ws_bytes, void* stream) {
  if (!mask || !col_ptr || !maskT || !chunk_off || n < 1 || k < 1) return DUO_ERR_INVALID_ARG;
  if (n > 65535 || k > kMaxK) return DUO_ERR_UNSUPPORTED;
  if (!ws || ws_bytes < dsc_ws_bytes(n, k) || ((uintptr_t)ws & (kAlign - 1))) return DUO_ERR_WORKSPACE;
  if (duo_status d = device_ok(); d != DUO_OK) return d;
  const hipStream_t s = (hipStream_t)stream;
  const int64_t wn = (n + 31) / 32;
  hipLaunchKernelGGL(dsc_mask_t_kernel, dim3((unsigned)cdiv(k * wn, 256)), dim3(256), 0, s, mask, n, k, maskT);
  DUO_LAUNCH_CHECK();
  int64_t* cnt = (int64_t*)ws;
  hipLaunchKernelGGL(dsc_count_kernel, dim3((unsigned)cdiv(k, 256)), dim3(256), 0, s, (const uint32_t*)maskT, n, k,
                     chunk_off, cnt);
  DUO_LAUNCH_CHECK();
  hipLaunchKernelGGL(dsc_scan_kernel, dim3(1), dim3(1024), 0, s, (const int64_t*)cnt, k, col_ptr);
  DUO_LAUNCH_CHECK();
  return DUO_OK;
}

duo_status duo_dsc_pack(const void* W, int32_t w_dtype, int64_t n, int64_t k, int64_t ldw, const int64_t* col_ptr,
                        const uint32_t* maskT, const uint16_t* chunk_off, uint16_t* values, void* stream) {
  if (!W || !col_ptr || !maskT || !chunk_off || !values || n < 1 || k < 1 || ldw < k) return DUO_ERR_INVALID_ARG;
  if (w_dtype != DUO_F32 && w_dtype != DUO_BF16) return DUO_ERR_INVALID_ARG;
  if (n > 65535 || k > kMaxK) return DUO_ERR_UNSUPPORTED;
  if (duo_status d = device_ok(); d != DUO_OK) return d;
  hipLaunchKernelGGL(dsc_pack_kernel, dim3((unsigned)cdiv(n * k, 256)), dim3(256), 0, (hipStream_t)stream, W,
                     (int)w_dtype, n, k, ldw, col_ptr, maskT, chunk_off, values);
  DUO_LAUNCH_CHECK();
  return DUO_OK;
}

duo_status duo_dsc_gemv(const void* x, int32_t x_dtype, int64_t n, int64_t k, duo_act_rule rule,
                        const int64_t* col_ptr, const uint32_t* maskT, const uint16_t* chunk_off,
                        const uint16_t* values, float* y, void* ws, size_t ws_bytes, void* stream) {
  if (duo_status d = gemv_check(x, x_dtype, n, k, rule, col_ptr, maskT, chunk_off, values, y); d != DUO_OK) return d;
  if (!ws || ws_bytes < dsc_ws_bytes(n, k) || ((uintptr_t)ws & (kAlign - 1))) return DUO_ERR_WORKSPACE;
  if (duo_status d = device_ok(); d != DUO_OK) return d;
  return gemv_launch(x, x_dtype, n, k, rule, col_ptr, maskT, chunk_off, values, y, (float*)ws, (hipStream_t)stream);
}

duo_status duo_dsc_gemv_noalloc(const void* x, int32_t x_dtype, int64_t n, int64_t k, duo_act_rule rule,
                                const int64_t* col_ptr, const uint32_t* maskT, const uint16_t* chunk_off,
                                const uint16_t* values, float* y, void* stream) {
  if (duo_status d = gemv_check(x, x_dtype, n, k, rule, col_ptr, maskT, chunk_off, values, y); d != DUO_OK) return d;
  if (duo_status d = device_ok(); d != DUO_OK) return d;
  const int z = rule.kind == DUO_ACT_NONE ? 0 : (int)floor(rule.sparsity * (double)k + 0.5);
  const GemvPlan p = gemv_plan(n, (int)(k - z));
  if ((size_t)p.S * (size_t)n > kScratchFloats) return DUO_ERR_UNSUPPORTED;
  float* part = nullptr;
  if (duo_status d = scratch_address(&part); d != DUO_OK) return d;
  return gemv_launch(x, x_dtype, n, k, rule, col_ptr, maskT, chunk_off, values, y, part, (hipStream_t)stream);
}

}  // extern "C"
