// act_order (App. B, calibration settings): the channel order by decreasing
// Hessian diagonal, and the row/column gathers that move a layer's operands
// into that order and its outputs back.
#include <hip/hip_runtime.h>

#include "internal.h"

using namespace duo;

namespace {

// Rank of channel p in the order (key descending, index ascending) with key =
// the bit pattern of hdiag[p].  hdiag holds sums of squares (>= +0, or NaN or
// +inf when the input was not finite), whose bit patterns order like their
// values, so the order is a strict total order and the ranks a permutation.
constexpr int kRankTile = 2048;

__global__ __launch_bounds__(256) void act_order_kernel(const double* __restrict__ hdiag, int k,
                                                        int32_t* __restrict__ perm, int32_t* __restrict__ inv) {
  __shared__ unsigned long long key[kRankTile];
  const int p = blockIdx.x * 256 + threadIdx.x;
  const unsigned long long kp = p < k ? (unsigned long long)__double_as_longlong(hdiag[p]) : 0ull;
  int rank = 0;
  for (int q0 = 0; q0 < k; q0 += kRankTile) {
    const int nq = min(kRankTile, k - q0);
    __syncthreads();
    for (int i = threadIdx.x; i < nq; i += 256) key[i] = (unsigned long long)__double_as_longlong(hdiag[q0 + i]);
    __syncthreads();
    for (int i = 0; i < nq; ++i) {
      const unsigned long long kq = key[i];
      rank += (kq > kp || (kq == kp && q0 + i < p)) ? 1 : 0;
    }
  }
  if (p < k) {
    perm[rank] = p;
    if (inv) inv[p] = rank;
  }
}

// dst[i][j] = src[ri][cj] with ri = row_idx ? row_idx[i] : i and cj likewise;
// an index outside the source leaves 0 in dst.
template <typename E>
__global__ __launch_bounds__(256) void permute_kernel(const E* __restrict__ src, int64_t rows, int64_t cols,
                                                      int64_t src_rows, int64_t src_cols, int64_t lds,
                                                      const int32_t* __restrict__ row_idx,
                                                      const int32_t* __restrict__ col_idx, E* __restrict__ dst,
                                                      int64_t ldd) {
  const int64_t j = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t i = blockIdx.y;
  if (j >= cols) return;
  const int64_t ri = row_idx ? (int64_t)row_idx[i] : i;
  const int64_t cj = col_idx ? (int64_t)col_idx[j] : j;
  E v = E(0);
  if (ri >= 0 && ri < src_rows && cj >= 0 && cj < src_cols) v = src[ri * lds + cj];
  dst[i * ldd + j] = v;
}

// Bit-packed masks (rows x ceil(k/32) words): bit j of row r of dst = bit
// col_idx[j] of row r of src (0 for an index outside [0, k)).
__global__ __launch_bounds__(256) void permute_mask_kernel(const uint32_t* __restrict__ src, int64_t n, int64_t k,
                                                           const int32_t* __restrict__ col_idx,
                                                           uint32_t* __restrict__ dst) {
  const int64_t words = (k + 31) / 32;
  const int64_t id = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (id >= n * words) return;
  const int64_t r = id / words, w = id % words;
  uint32_t bits = 0;
  for (int e = 0; e < 32; ++e) {
    const int64_t j = w * 32 + e;
    if (j >= k) break;
    const int64_t c = col_idx[j];
    if (c >= 0 && c < k && ((src[r * words + c / 32] >> (c % 32)) & 1u)) bits |= 1u << e;
  }
  dst[id] = bits;
}

}  // namespace

extern "C" {

duo_status duo_act_order(const double* hdiag, int64_t k, int32_t* perm, int32_t* inv_perm, void* stream) {
  if (!hdiag || !perm || k < 1) return DUO_ERR_INVALID_ARG;
  if (k > kMaxK) return DUO_ERR_UNSUPPORTED;
  if (duo_status d = device_ok(); d != DUO_OK) return d;
  hipLaunchKernelGGL(act_order_kernel, dim3((unsigned)cdiv(k, 256)), dim3(256), 0, (hipStream_t)stream, hdiag,
                     (int)k, perm, inv_perm);
  DUO_LAUNCH_CHECK();
  return DUO_OK;
}

duo_status duo_permute(const void* src, int32_t dtype, int64_t src_rows, int64_t src_cols, int64_t lds,
                       const int32_t* row_idx, const int32_t* col_idx, int64_t rows, int64_t cols, void* dst,
                       int64_t ldd, void* stream) {
  if (dtype != DUO_F32 && dtype != DUO_BF16) return DUO_ERR_INVALID_ARG;
  if (src_rows < 0 || src_cols < 0 || rows < 0 || cols < 0 || lds < src_cols || ldd < cols)
    return DUO_ERR_INVALID_ARG;
  if (!row_idx && rows > src_rows) return DUO_ERR_INVALID_ARG;
  if (!col_idx && cols > src_cols) return DUO_ERR_INVALID_ARG;
  if (rows == 0 || cols == 0) return DUO_OK;
  if (!src || !dst || src == dst) return DUO_ERR_INVALID_ARG;
  if (rows > 65535) return DUO_ERR_UNSUPPORTED;
  if (duo_status d = device_ok(); d != DUO_OK) return d;
  const dim3 grid((unsigned)cdiv(cols, 256), (unsigned)rows);
  if (dtype == DUO_F32)
    hipLaunchKernelGGL(permute_kernel<uint32_t>, grid, dim3(256), 0, (hipStream_t)stream, (const uint32_t*)src, rows,
                       cols, src_rows, src_cols, lds, row_idx, col_idx, (uint32_t*)dst, ldd);
  else
    hipLaunchKernelGGL(permute_kernel<uint16_t>, grid, dim3(256), 0, (hipStream_t)stream, (const uint16_t*)src, rows,
                       cols, src_rows, src_cols, lds, row_idx, col_idx, (uint16_t*)dst, ldd);
  DUO_LAUNCH_CHECK();
  return DUO_OK;
}

duo_status duo_permute_mask(const uint32_t* src, int64_t n, int64_t k, const int32_t* col_idx, uint32_t* dst,
                            void* stream) {
  if (n < 0 || k < 0) return DUO_ERR_INVALID_ARG;
  if (n == 0 || k == 0) return DUO_OK;
  if (!src || !dst || !col_idx || src == dst) return DUO_ERR_INVALID_ARG;
  if (duo_status d = device_ok(); d != DUO_OK) return d;
  const int64_t cnt = n * ((k + 31) / 32);
  hipLaunchKernelGGL(permute_mask_kernel, dim3((unsigned)cdiv(cnt, 256)), dim3(256), 0, (hipStream_t)stream, src, n,
                     k, col_idx, dst);
  DUO_LAUNCH_CHECK();
  return DUO_OK;
}

}  // extern "C"
