// Decoder-block harness: the operations that carry the two activation streams
// of a LLaMA-style decoder block between the solver's groups (the multi-layer
// case of Sec. 4.2: the dense model sees X-tilde, the pruned model sees its
// own, sparsified input).  All activations are bf16 row-major token x feature
// arrays; arithmetic is fp32.
//
//   duo_rmsnorm       y = x / sqrt(mean(x^2) + eps)          (unit gain)
//   duo_act_sparsify  y = x with the per-token (|x|, channel) rule applied
//   duo_linear        Y = X W^T (+ R)                         (rocBLAS, fp32 accumulate)
//   duo_rope          rotary position embedding, rotate-half pairs (i, i + d/2)
//   duo_attention     causal softmax(Q K^T / sqrt(d)) V per sequence and head
//                     (rocBLAS batched products around a causal row softmax;
//                     the probabilities are rounded to bf16 before P V)
//   duo_silu_mul      y = SiLU(g) * u
#include <hip/hip_runtime.h>
#include <rocblas/rocblas.h>

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

__global__ void act_apply_kernel(const uint16_t* __restrict__ X, int64_t ldx, int m, int k,
                                 const int64_t* __restrict__ thr, uint16_t* __restrict__ Y, int64_t ldy) {
  const int64_t id = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (id >= (int64_t)m * k) return;
  const int t = (int)(id / k), c = (int)(id % k);
  const uint16_t x = X[(int64_t)t * ldx + c];
  const int64_t key = ((int64_t)(x & 0x7fffu) << 32) | c;
  Y[(int64_t)t * ldy + c] = key > thr[t] ? x : (uint16_t)0;
}

// Thread (token, head, i) rotates the pair (i, i + d/2) of that head by
// angle pos * theta^(-2i/d), pos = token % seq_len.  Angles in fp64.
__global__ void rope_kernel(uint16_t* __restrict__ X, int64_t ldx, int m, int heads, int hd, int seq_len,
                            double theta) {
  const int half = hd / 2;
  const int64_t id = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (id >= (int64_t)m * heads * half) return;
  const int i = (int)(id % half);
  const int h = (int)((id / half) % heads);
  const int t = (int)(id / ((int64_t)half * heads));
  const double ang = (double)(t % seq_len) * pow(theta, -2.0 * (double)i / (double)hd);
  double sd, cd;
  sincos(ang, &sd, &cd);
  const float s = (float)sd, c = (float)cd;
  uint16_t* p = X + (int64_t)t * ldx + (int64_t)h * hd;
  const float x1 = bf16_bits_to_f32(p[i]), x2 = bf16_bits_to_f32(p[i + half]);
  p[i] = f32_to_bf16_bits(x1 * c - x2 * s);
  p[i + half] = f32_to_bf16_bits(x2 * c + x1 * s);
}

// Causal softmax of one score row: S (fp32, L x L per head, row-major) -> P
// (bf16, same layout); entries above the diagonal become 0.  One 256-thread
// workgroup per (head, row).
__global__ __launch_bounds__(256) void causal_softmax_kernel(const float* __restrict__ S, int L, float scale,
                                                             uint16_t* __restrict__ P) {
  __shared__ float red[8];
  const int row = blockIdx.x % L;
  const int64_t off = (int64_t)blockIdx.x * L;
  const float* s = S + off;
  uint16_t* p = P + off;
  float mx = -INFINITY;
  for (int j = threadIdx.x; j <= row; j += 256) mx = fmaxf(mx, s[j] * scale);
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o));
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = mx;
  __syncthreads();
  mx = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  float sum = 0.f;
  for (int j = threadIdx.x; j <= row; j += 256) sum += expf(s[j] * scale - mx);
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) sum += __shfl_xor(sum, o);
  if ((threadIdx.x & 63) == 0) red[4 + (threadIdx.x >> 6)] = sum;
  __syncthreads();
  const float inv = 1.0f / ((red[4] + red[5]) + (red[6] + red[7]));
  for (int j = threadIdx.x; j < L; j += 256)
    p[j] = j <= row ? f32_to_bf16_bits(expf(s[j] * scale - mx) * inv) : (uint16_t)0;
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
// rocBLAS handles (one per device, created on first use; calls on a handle
// are serialised because the stream and workspace are handle state)
// ---------------------------------------------------------------------------
struct BlasSlot {
  std::mutex mu;
  rocblas_handle h = nullptr;
};
BlasSlot g_blas[64];

constexpr size_t kBlasWs = (size_t)64 << 20;  // rocBLAS workspace carved from the caller's

duo_status blas_status(rocblas_status s) { return s == rocblas_status_success ? DUO_OK : DUO_ERR_HIP; }

struct BlasLock {
  BlasSlot* slot = nullptr;
  std::unique_lock<std::mutex> lk;
  duo_status st = DUO_OK;
  BlasLock(hipStream_t s, void* ws, size_t bytes) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) {
      st = DUO_ERR_NO_DEVICE;
      return;
    }
    slot = &g_blas[dev];
    lk = std::unique_lock<std::mutex>(slot->mu);
    if (!slot->h && rocblas_create_handle(&slot->h) != rocblas_status_success) {
      slot->h = nullptr;
      st = DUO_ERR_HIP;
      return;
    }
    if (rocblas_set_stream(slot->h, s) != rocblas_status_success ||
        rocblas_set_workspace(slot->h, ws, bytes) != rocblas_status_success)
      st = DUO_ERR_HIP;
  }
};

bool aligned(const void* ws) { return (reinterpret_cast<uintptr_t>(ws) % kAlign) == 0; }

int act_zeros(const duo_act_rule& r, int64_t k) {
  if (r.kind == DUO_ACT_NONE) return 0;
  return (int)std::floor(r.sparsity * (double)k + 0.5);
}

}  // namespace

extern "C" {

size_t duo_block_workspace_size(int32_t op, int64_t m, int64_t seq_len, int64_t heads) {
  switch (op) {
    case DUO_BOP_ACT_SPARSIFY: return m < 1 ? 0 : (size_t)rup(m * (int64_t)sizeof(int64_t), kAlign);
    case DUO_BOP_LINEAR: return kBlasWs;
    case DUO_BOP_ATTENTION:
      if (seq_len < 1 || heads < 1) return 0;
      return kBlasWs + (size_t)rup(heads * seq_len * seq_len * (int64_t)sizeof(float), kAlign) +
             (size_t)rup(heads * seq_len * seq_len * (int64_t)sizeof(uint16_t), kAlign);
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
  hipLaunchKernelGGL(act_apply_kernel, dim3((unsigned)cdiv(tot, 256)), dim3(256), 0, s, (const uint16_t*)X, ldx,
                     (int)m, (int)k, (const int64_t*)thr, (uint16_t*)Y, ldy);
  DUO_LAUNCH_CHECK();
  return DUO_OK;
}

duo_status duo_linear(const void* X, int64_t m, int64_t k, int64_t ldx, const void* W, int64_t n, int64_t ldw,
                      const void* R, int64_t ldr, void* Y, int64_t ldy, void* ws, size_t ws_bytes, void* stream) {
  if (m < 0 || k < 1 || n < 1 || ldx < k || ldw < k || ldy < n || (R && ldr < n)) return DUO_ERR_INVALID_ARG;
  if (m > INT32_MAX || n > INT32_MAX || k > INT32_MAX || ldx > INT32_MAX || ldw > INT32_MAX || ldy > INT32_MAX ||
      ldr > INT32_MAX)
    return DUO_ERR_UNSUPPORTED;
  if (m == 0) return DUO_OK;
  if (!X || !W || !Y) return DUO_ERR_INVALID_ARG;
  if (!ws || ws_bytes < kBlasWs || !aligned(ws)) return DUO_ERR_WORKSPACE;
  if (duo_status d = device_ok(); d != DUO_OK) return d;
  BlasLock b((hipStream_t)stream, ws, kBlasWs);
  if (b.st != DUO_OK) return b.st;
  const float alpha = 1.f, beta = R ? 1.f : 0.f;
  // column-major view: Y^T (n x m) = W (n x k, stored as W^T k x n) * X^T (k x m)
  return blas_status(rocblas_gemm_ex(b.slot->h, rocblas_operation_transpose, rocblas_operation_none, (rocblas_int)n,
                                     (rocblas_int)m, (rocblas_int)k, &alpha, W, rocblas_datatype_bf16_r,
                                     (rocblas_int)ldw, X, rocblas_datatype_bf16_r, (rocblas_int)ldx, &beta,
                                     R ? R : Y, rocblas_datatype_bf16_r, (rocblas_int)(R ? ldr : ldy), Y,
                                     rocblas_datatype_bf16_r, (rocblas_int)ldy, rocblas_datatype_f32_r,
                                     rocblas_gemm_algo_standard, 0, 0));
}

duo_status duo_rope(void* X, int64_t m, int64_t heads, int64_t head_dim, int64_t ldx, int64_t seq_len, double theta,
                    void* stream) {
  if (m < 0 || heads < 1 || head_dim < 2 || (head_dim & 1) || ldx < heads * head_dim || seq_len < 1 ||
      !(theta > 0.0) || !std::isfinite(theta))
    return DUO_ERR_INVALID_ARG;
  if (m == 0) return DUO_OK;
  if (!X || m > INT32_MAX) return DUO_ERR_INVALID_ARG;
  if (duo_status d = device_ok(); d != DUO_OK) return d;
  const int64_t tot = m * heads * (head_dim / 2);
  hipLaunchKernelGGL(rope_kernel, dim3((unsigned)cdiv(tot, 256)), dim3(256), 0, (hipStream_t)stream, (uint16_t*)X, ldx,
                     (int)m, (int)heads, (int)head_dim, (int)seq_len, theta);
  DUO_LAUNCH_CHECK();
  return DUO_OK;
}

duo_status duo_attention(const void* Q, const void* K, const void* V, int64_t ld, int64_t nseq, int64_t seq_len,
                         int64_t heads, int64_t head_dim, void* O, int64_t ldo, void* ws, size_t ws_bytes,
                         void* stream) {
  if (nseq < 0 || seq_len < 1 || heads < 1 || head_dim < 1 || ld < heads * head_dim || ldo < heads * head_dim)
    return DUO_ERR_INVALID_ARG;
  if (seq_len > INT32_MAX || ld > INT32_MAX || ldo > INT32_MAX || heads * seq_len > INT32_MAX)
    return DUO_ERR_UNSUPPORTED;
  if (nseq == 0) return DUO_OK;
  if (!Q || !K || !V || !O) return DUO_ERR_INVALID_ARG;
  const size_t need = duo_block_workspace_size(DUO_BOP_ATTENTION, 0, seq_len, heads);
  if (!ws || ws_bytes < need || !aligned(ws)) return DUO_ERR_WORKSPACE;
  if (duo_status d = device_ok(); d != DUO_OK) return d;
  hipStream_t s = (hipStream_t)stream;
  Carver c(ws);
  void* bws = c.take<uint8_t>(kBlasWs);
  float* S = c.take<float>((size_t)(heads * seq_len * seq_len));
  uint16_t* P = c.take<uint16_t>((size_t)(heads * seq_len * seq_len));
  BlasLock b(s, bws, kBlasWs);
  if (b.st != DUO_OK) return b.st;
  const float one = 1.f, zero = 0.f;
  const float scale = 1.0f / std::sqrt((float)head_dim);
  const rocblas_int Li = (rocblas_int)seq_len, hdi = (rocblas_int)head_dim;
  const rocblas_stride sLL = (rocblas_stride)(seq_len * seq_len);
  for (int64_t q = 0; q < nseq; ++q) {
    const int64_t row0 = q * seq_len;
    const uint16_t* Qs = (const uint16_t*)Q + row0 * ld;
    const uint16_t* Ks = (const uint16_t*)K + row0 * ld;
    const uint16_t* Vs = (const uint16_t*)V + row0 * ld;
    uint16_t* Os = (uint16_t*)O + row0 * ldo;
    // S_h[i][j] = q_i . k_j: column-major C = K_h Q_h^T (L x L, ld L) per head
    rocblas_status r = rocblas_gemm_strided_batched_ex(
        b.slot->h, rocblas_operation_transpose, rocblas_operation_none, Li, Li, hdi, &one, Ks, rocblas_datatype_bf16_r,
        (rocblas_int)ld, (rocblas_stride)head_dim, Qs, rocblas_datatype_bf16_r, (rocblas_int)ld,
        (rocblas_stride)head_dim, &zero, S, rocblas_datatype_f32_r, Li, sLL, S, rocblas_datatype_f32_r, Li, sLL,
        (rocblas_int)heads, rocblas_datatype_f32_r, rocblas_gemm_algo_standard, 0, 0);
    if (r != rocblas_status_success) return DUO_ERR_HIP;
    hipLaunchKernelGGL(causal_softmax_kernel, dim3((unsigned)(heads * seq_len)), dim3(256), 0, s, (const float*)S,
                       (int)seq_len, scale, P);
    DUO_LAUNCH_CHECK();
    // O_h = P_h V_h: column-major C (d x L, ldo) = V_h^T (d x L, ld) * P_h^T (L x L, ld L)
    r = rocblas_gemm_strided_batched_ex(b.slot->h, rocblas_operation_none, rocblas_operation_none, hdi, Li, Li, &one,
                                        Vs, rocblas_datatype_bf16_r, (rocblas_int)ld, (rocblas_stride)head_dim, P,
                                        rocblas_datatype_bf16_r, Li, sLL, &zero, Os, rocblas_datatype_bf16_r,
                                        (rocblas_int)ldo, (rocblas_stride)head_dim, Os, rocblas_datatype_bf16_r,
                                        (rocblas_int)ldo, (rocblas_stride)head_dim, (rocblas_int)heads,
                                        rocblas_datatype_f32_r, rocblas_gemm_algo_standard, 0, 0);
    if (r != rocblas_status_success) return DUO_ERR_HIP;
  }
  return DUO_OK;
}

duo_status duo_silu_mul(const void* G, const void* U, int64_t m, int64_t n, int64_t ld, void* Y, int64_t ldy,
                        void* stream) {
  if (m < 0 || n < 1 || ld < n || ldy < n) return DUO_ERR_INVALID_ARG;
  if (m == 0) return DUO_OK;
  if (!G || !U || !Y) return DUO_ERR_INVALID_ARG;
  if (duo_status d = device_ok(); d != DUO_OK) return d;
  const int64_t tot = m * n;
  hipLaunchKernelGGL(silu_mul_kernel, dim3((unsigned)cdiv(tot, 256)), dim3(256), 0, (hipStream_t)stream,
                     (const uint16_t*)G, (const uint16_t*)U, ld, (int)m, (int)n, (uint16_t*)Y, ldy);
  DUO_LAUNCH_CHECK();
  return DUO_OK;
}

}  // extern "C"
