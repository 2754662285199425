// Internal helpers shared by the gfx950 kernels of the DuoGPT layer solver.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "duo.h"

#define DUO_HIP_TRY(expr)                         \
  do {                                            \
    hipError_t duo_e_ = (expr);                   \
    if (duo_e_ != hipSuccess) {                   \
      (void)hipGetLastError(); /* not sticky */   \
      return DUO_ERR_HIP;                         \
    }                                             \
  } while (0)

#define DUO_LAUNCH_CHECK() DUO_HIP_TRY(hipGetLastError())

namespace duo {

constexpr int kWave = 64;
constexpr int kTile = 128;        // square tile edge of every MFMA kernel
constexpr int kTokBlk = 32;       // tokens per packed operand row (one MFMA K step for bf16)
constexpr int kMaxK = 32768;      // per-token selection keeps a token in registers
constexpr int kMaxBlock = 128;    // sweep block width limit
constexpr size_t kAlign = 256;

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) float f4;
typedef __attribute__((ext_vector_type(4))) unsigned int u32x4;

__host__ __device__ inline int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }
__host__ __device__ inline int64_t rup(int64_t a, int64_t b) { return cdiv(a, b) * b; }
inline size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

__device__ inline float bf16_bits_to_f32(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

// round to nearest even; NaN stays NaN
__device__ inline uint16_t f32_to_bf16_bits(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x0040u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

// Index of the lower-triangular pair (i >= j) with linear id p in row-major
// order (0,0),(1,0),(1,1),(2,0)...
__host__ __device__ inline void tri_pair(int64_t p, int* i, int* j) {
  int64_t r = (int64_t)((sqrt(8.0 * (double)p + 1.0) - 1.0) * 0.5);
  while (r * (r + 1) / 2 > p) --r;
  while ((r + 1) * (r + 2) / 2 <= p) ++r;
  *i = (int)r;
  *j = (int)(p - r * (r + 1) / 2);
}

// Score of one weight, S = w^2 * fac, as two rounded products (no fused
// multiply-add) so every kernel that needs it gets the same bits.
__device__ inline float weight_score(float w, float f) { return __fmul_rn(__fmul_rn(w, w), f); }

// Order-preserving map of a float onto uint32 (+0 and -0 are made equal).
__device__ inline uint32_t orderable(float s) {
  if (s == 0.0f) s = 0.0f;
  uint32_t u = __float_as_uint(s);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Workspace carving: successive 256-byte aligned slices.
struct Carver {
  uint8_t* base;
  size_t off;
  explicit Carver(void* b) : base((uint8_t*)b), off(0) {}
  template <typename T>
  T* take(size_t count) {
    T* p = (T*)(base ? base + off : nullptr);
    off = align_up(off + count * sizeof(T));
    return p;
  }
};

}  // namespace duo
