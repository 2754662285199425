// C ABI of the DuoGPT layer solver: argument validation, workspace sizing and
// dispatch to the gfx950 kernels.  Every argument error is reported before
// anything is enqueued.
#include <hip/hip_runtime.h>

#include <atomic>
#include <cmath>
#include <cstring>
#include <mutex>

#include "internal.h"

using namespace duo;

namespace {

bool finite_in(double x, double lo, double hi) { return std::isfinite(x) && x >= lo && x <= hi; }

bool dtype_ok(int32_t t) { return t == DUO_F32 || t == DUO_BF16; }

bool rule_ok(const duo_act_rule& r) {
  if (r.kind == DUO_ACT_NONE) return true;
  return r.kind == DUO_ACT_TOPK_MAG_PER_TOKEN && finite_in(r.sparsity, 0.0, 1.0);
}

int zero_count(const duo_act_rule& r, int64_t k) {
  if (r.kind == DUO_ACT_NONE) return 0;
  return (int)std::floor(r.sparsity * (double)k + 0.5);
}

bool ws_ok(const void* ws, size_t ws_bytes, size_t need) {
  if (need == 0) return true;
  if (!ws || ws_bytes < need) return false;
  return (reinterpret_cast<uintptr_t>(ws) % kAlign) == 0;
}

struct PruneWs {
  float* D;  // D (k x k) in the D form, Y (n x k) in the Y form
  float* fac;
  void* score;
  void* sweep;
  size_t bytes;
};

PruneWs carve_prune(void* ws, int64_t n, int64_t k, int B) {
  Carver c(ws);
  PruneWs w;
  w.D = c.take<float>((size_t)(n > k ? n : k) * k);
  w.fac = c.take<float>((size_t)k);
  w.score = c.take<uint8_t>(score_ws_bytes(k));
  w.sweep = c.take<uint8_t>(sweep_ws_bytes(n, k, B));
  w.bytes = c.off;
  return w;
}

bool k_ok(int64_t k) { return k >= 1 && k <= kMaxK; }

constexpr int64_t kYFormMinK = 6144;  // DUO_FORM_AUTO: the Y form from this k up

}  // namespace

namespace duo {

// 0 unknown, 1 gfx950, 2 something else
static std::atomic<int> g_arch[64];

// The dynamic LDS limit of a kernel is raised once per device (and again only
// when a launch needs more): the attribute call is host work that need not
// sit in front of every launch.
namespace {
struct LdsLimit {
  const void* fn;
  int dev;
  int bytes;
};
std::mutex g_lds_mu;
LdsLimit g_lds[128];
int g_lds_n = 0;
}  // namespace

duo_status set_max_lds(const void* fn, size_t bytes) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return DUO_ERR_NO_DEVICE;
  std::lock_guard<std::mutex> lk(g_lds_mu);
  int slot = -1;
  for (int i = 0; i < g_lds_n; ++i)
    if (g_lds[i].fn == fn && g_lds[i].dev == dev) slot = i;
  if (slot >= 0 && g_lds[slot].bytes >= (int)bytes) return DUO_OK;
  DUO_HIP_TRY(hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes));
  if (slot < 0 && g_lds_n < 128) slot = g_lds_n++;
  if (slot >= 0) g_lds[slot] = LdsLimit{fn, dev, (int)bytes};
  return DUO_OK;
}

duo_status device_ok() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return DUO_ERR_NO_DEVICE;
  if (dev >= 64) return DUO_ERR_UNSUPPORTED;
  int v = g_arch[dev].load(std::memory_order_acquire);
  if (v == 0) {
    hipDeviceProp_t p;
    if (hipGetDeviceProperties(&p, dev) != hipSuccess) return DUO_ERR_NO_DEVICE;
    v = std::strncmp(p.gcnArchName, "gfx950", 6) == 0 ? 1 : 2;
    g_arch[dev].store(v, std::memory_order_release);
  }
  return v == 1 ? DUO_OK : DUO_ERR_NO_DEVICE;
}

}  // namespace duo

extern "C" {

size_t duo_workspace_size(int32_t op, int64_t n, int64_t k, int64_t m, int32_t block) {
  if (k < 1 || k > kMaxK) return 0;
  switch (op) {
    case DUO_OP_HESSIAN: return hessian_ws_bytes(m < 1 ? 1 : m, k);
    case DUO_OP_CHOL_INV: return chol_ws_bytes(k);
    case DUO_OP_SCORE_TERMS: return score_ws_bytes(k);
    case DUO_OP_SWEEP:
      if (n < 1 || block < 1 || block > kMaxBlock) return 0;
      return sweep_ws_bytes(n, k, block);
    case DUO_OP_PRUNE_LAYER:
      if (n < 1 || block < 1 || block > kMaxBlock) return 0;
      return carve_prune(nullptr, n, k, block).bytes;
    default: return 0;
  }
}

const char* duo_status_string(duo_status s) {
  switch (s) {
    case DUO_OK: return "ok";
    case DUO_ERR_INVALID_ARG: return "invalid argument";
    case DUO_ERR_UNSUPPORTED: return "unsupported size or option";
    case DUO_ERR_WORKSPACE: return "workspace missing, too small or not 256-byte aligned";
    case DUO_ERR_NOT_PD: return "damped Hessian is not positive definite";
    case DUO_ERR_NONFINITE: return "non-finite value";
    case DUO_ERR_HIP: return "HIP runtime error";
    case DUO_ERR_NO_DEVICE: return "no gfx950 device is current";
    default: return "unknown status";
  }
}

const char* duo_version(void) { return "duo 0.1.0 gfx950"; }

duo_status duo_act_sparsify_mask(const void* X, int32_t x_dtype, int64_t m, int64_t k, int64_t ldx,
                                 duo_act_rule rule, uint32_t* mask_out, void* ws, size_t ws_bytes, void* stream) {
  if (!dtype_ok(x_dtype) || m < 0 || !rule_ok(rule)) return DUO_ERR_INVALID_ARG;
  if (!k_ok(k)) return k < 1 ? DUO_ERR_INVALID_ARG : DUO_ERR_UNSUPPORTED;
  if (ldx < k) return DUO_ERR_INVALID_ARG;
  if (m == 0) return DUO_OK;
  if (!X || !mask_out) return DUO_ERR_INVALID_ARG;
  if (m > INT32_MAX) return DUO_ERR_UNSUPPORTED;
  if (!ws_ok(ws, ws_bytes, hessian_ws_bytes(m, k))) return DUO_ERR_WORKSPACE;
  duo_status d = device_ok();
  if (d != DUO_OK) return d;
  return act_mask_run(X, x_dtype, m, k, ldx, zero_count(rule, k), mask_out, ws, (hipStream_t)stream);
}

static duo_status hessian_common(const void* X_src, const void* X_dense, int32_t x_dtype, int64_t m, int64_t k,
                                 int64_t ldx, duo_act_rule rule, float* H, int64_t ldh, float* G, int64_t ldg,
                                 int32_t g_part, float* a, double* hdiag, void* ws, size_t ws_bytes, void* stream,
                                 bool want_h) {
  if (!dtype_ok(x_dtype) || m < 0 || !rule_ok(rule)) return DUO_ERR_INVALID_ARG;
  if (g_part != DUO_G_UPPER && g_part != DUO_G_FULL) return DUO_ERR_INVALID_ARG;
  if (!k_ok(k)) return k < 1 ? DUO_ERR_INVALID_ARG : DUO_ERR_UNSUPPORTED;
  if (ldx < k) return DUO_ERR_INVALID_ARG;
  if (want_h && (!H || ldh < k)) return DUO_ERR_INVALID_ARG;
  if ((G == nullptr) != (a == nullptr)) return DUO_ERR_INVALID_ARG;
  if (G && ldg < k) return DUO_ERR_INVALID_ARG;
  if (!want_h && !G) return DUO_ERR_INVALID_ARG;
  if (m == 0) return DUO_OK;
  if (!X_src) return DUO_ERR_INVALID_ARG;
  if (m > INT32_MAX) return DUO_ERR_UNSUPPORTED;
  if (!ws_ok(ws, ws_bytes, hessian_ws_bytes(m, k))) return DUO_ERR_WORKSPACE;
  duo_status d = device_ok();
  if (d != DUO_OK) return d;
  prof_begin(DUO_PROF_HESSIAN, (hipStream_t)stream);
  duo_status r = hessian_run(X_src, X_dense, x_dtype, m, k, ldx, zero_count(rule, k), H, ldh, G, ldg,
                             g_part == DUO_G_FULL ? 1 : 0, a, hdiag, ws, want_h, (hipStream_t)stream);
  prof_end(DUO_PROF_HESSIAN, (hipStream_t)stream);
  return r;
}

duo_status duo_hessian_accum(const void* X_src, const void* X_dense, int32_t x_dtype, int64_t m, int64_t k,
                             int64_t ldx, duo_act_rule rule, float* H, int64_t ldh, float* G, int64_t ldg,
                             int32_t g_part, float* a, double* hdiag, void* ws, size_t ws_bytes, void* stream) {
  return hessian_common(X_src, X_dense, x_dtype, m, k, ldx, rule, H, ldh, G, ldg, g_part, a, hdiag, ws, ws_bytes,
                        stream, true);
}

duo_status duo_residual_term(const void* X_dense, const void* X_src, int32_t x_dtype, int64_t m, int64_t k,
                             int64_t ldx, duo_act_rule rule, float* G, int64_t ldg, int32_t g_part, float* a, void* ws,
                             size_t ws_bytes, void* stream) {
  if (!G || !a) return DUO_ERR_INVALID_ARG;
  if (m > 0 && !X_dense) return DUO_ERR_INVALID_ARG;
  const void* src = X_src ? X_src : X_dense;
  return hessian_common(src, X_dense, x_dtype, m, k, ldx, rule, nullptr, k, G, ldg, g_part, a, nullptr, ws, ws_bytes,
                        stream, false);
}

duo_status duo_hessian_status(const void* ws, size_t ws_bytes, void* stream) {
  if (!ws || ws_bytes < 256 || (reinterpret_cast<uintptr_t>(ws) % kAlign) != 0) return DUO_ERR_INVALID_ARG;
  duo_status d = device_ok();
  if (d != DUO_OK) return d;
  return hessian_status_run(ws, (hipStream_t)stream);
}

duo_status duo_chol_inv(float* H_inout, int64_t k, int64_t ldh, double damp_ratio, duo_chol_info* info, void* ws,
                        size_t ws_bytes, void* stream) {
  if (!H_inout || ldh < k || !std::isfinite(damp_ratio) || damp_ratio < 0.0) return DUO_ERR_INVALID_ARG;
  if (!k_ok(k)) return k < 1 ? DUO_ERR_INVALID_ARG : DUO_ERR_UNSUPPORTED;
  if (!ws_ok(ws, ws_bytes, chol_ws_bytes(k))) return DUO_ERR_WORKSPACE;
  duo_status d = device_ok();
  if (d != DUO_OK) return d;
  CholStatus* st = nullptr;
  const hipStream_t s = (hipStream_t)stream;
  prof_begin(DUO_PROF_CHOL, s);
  duo_status r = chol_run(H_inout, k, ldh, damp_ratio, ws, s, &st);
  prof_end(DUO_PROF_CHOL, s);
  if (r != DUO_OK) return r;
  if (!info) return DUO_OK;
  CholStatus h;
  DUO_HIP_TRY(hipMemcpyAsync(&h, st, sizeof(h), hipMemcpyDeviceToHost, s));
  DUO_HIP_TRY(hipStreamSynchronize(s));
  info->lambda = h.lambda;
  info->fail_index = h.fail;
  info->status = h.status;
  return h.status;
}

duo_status duo_score_terms(const float* L, int64_t ldl, const float* G, int64_t ldg, const float* a, int64_t k,
                           float* D, int64_t ldd, float* fac, void* ws, size_t ws_bytes, void* stream) {
  if (!L || !G || !a || !D || !fac) return DUO_ERR_INVALID_ARG;
  if (!k_ok(k)) return k < 1 ? DUO_ERR_INVALID_ARG : DUO_ERR_UNSUPPORTED;
  if (ldl < k || ldg < k || ldd < k) return DUO_ERR_INVALID_ARG;
  if (!ws_ok(ws, ws_bytes, score_ws_bytes(k))) return DUO_ERR_WORKSPACE;
  duo_status d = device_ok();
  if (d != DUO_OK) return d;
  prof_begin(DUO_PROF_SCORE, (hipStream_t)stream);
  duo_status r = score_run(L, ldl, G, ldg, a, k, D, ldd, fac, ws, (hipStream_t)stream);
  prof_end(DUO_PROF_SCORE, (hipStream_t)stream);
  return r;
}

static duo_status sweep_args(const void* W, int32_t w_dtype, int64_t n, int64_t k, int64_t ldw, double w_sparsity,
                             const duo_sweep_opts* opts, int32_t block, float* W_out, SweepOpts* o) {
  if (!W || !W_out || !dtype_ok(w_dtype)) return DUO_ERR_INVALID_ARG;
  if (n < 1 || ldw < k || !finite_in(w_sparsity, 0.0, 1.0)) return DUO_ERR_INVALID_ARG;
  if (block < 1 || block > kMaxBlock) return DUO_ERR_INVALID_ARG;
  *o = SweepOpts{};
  if (opts) {
    const int nm = opts->nm_n, qb = opts->q_bits, qg = opts->q_group;
    if (nm < 0 || nm > 4 || (nm > 0 && (k % 4 != 0 || block % 4 != 0))) return DUO_ERR_INVALID_ARG;
    if (qb != 0 && (qb < 2 || qb > 8)) return DUO_ERR_INVALID_ARG;
    if (qb > 0 && !((qg == 16 || qg == 32 || qg == 64 || qg == 128) && block % qg == 0)) return DUO_ERR_INVALID_ARG;
    const int form = opts->residual_form;
    if (form != DUO_FORM_AUTO && form != DUO_FORM_D && form != DUO_FORM_Y) return DUO_ERR_INVALID_ARG;
    *o = SweepOpts{nm, qb, qb > 0 ? qg : 0, qb > 0 ? opts->q_scale_out : nullptr, qb > 0 ? opts->q_zero_out : nullptr,
                   form};
  }
  if (!k_ok(k)) return k < 1 ? DUO_ERR_INVALID_ARG : DUO_ERR_UNSUPPORTED;
  if (n > INT32_MAX / 2 || n * k > ((int64_t)1 << 40)) return DUO_ERR_UNSUPPORTED;
  return DUO_OK;
}

duo_status duo_sweep(const void* W, int32_t w_dtype, int64_t n, int64_t k, int64_t ldw, const float* L, int64_t ldl,
                     const float* D, int64_t ldd, const float* fac, double w_sparsity, const duo_sweep_opts* opts,
                     int32_t block, const uint32_t* mask_in, float* W_out, void* W_out_lowp, uint32_t* mask_out,
                     float* block_scores_out, void* ws, size_t ws_bytes, void* stream) {
  SweepOpts o;
  duo_status a = sweep_args(W, w_dtype, n, k, ldw, w_sparsity, opts, block, W_out, &o);
  if (a != DUO_OK) return a;
  if (!L || !D || !fac || ldl < k || ldd < k || o.form == DUO_FORM_Y) return DUO_ERR_INVALID_ARG;
  if (!ws_ok(ws, ws_bytes, sweep_ws_bytes(n, k, block))) return DUO_ERR_WORKSPACE;
  duo_status d = device_ok();
  if (d != DUO_OK) return d;
  prof_begin(DUO_PROF_SWEEP, (hipStream_t)stream);
  duo_status r = sweep_run(W, w_dtype, n, k, ldw, L, ldl, D, ldd, fac, w_sparsity, o, block, mask_in, W_out,
                           W_out_lowp, mask_out, block_scores_out, ws, (hipStream_t)stream);
  prof_end(DUO_PROF_SWEEP, (hipStream_t)stream);
  return r;
}

duo_status duo_prune_layer(const void* W, int32_t w_dtype, int64_t n, int64_t k, int64_t ldw, const float* L,
                           int64_t ldl, const float* G, int64_t ldg, const float* a, double w_sparsity,
                           const duo_sweep_opts* opts, int32_t block, const uint32_t* mask_in, float* W_out,
                           void* W_out_lowp, uint32_t* mask_out, float* block_scores_out, void* ws, size_t ws_bytes,
                           void* stream) {
  SweepOpts o;
  duo_status e = sweep_args(W, w_dtype, n, k, ldw, w_sparsity, opts, block, W_out, &o);
  if (e != DUO_OK) return e;
  if (!L || !G || !a || ldl < k || ldg < k) return DUO_ERR_INVALID_ARG;
  // the Y form takes unstructured and N:4 masks, and quantisation with one
  // grid per row and block (q_group == block: grids fixed at a block's start)
  const bool y_ok = o.q_bits == 0 || o.q_group == block;
  if (o.form == DUO_FORM_Y && !y_ok) return DUO_ERR_UNSUPPORTED;
  const PruneWs pw = carve_prune(nullptr, n, k, block);
  if (!ws_ok(ws, ws_bytes, pw.bytes)) return DUO_ERR_WORKSPACE;
  duo_status d = device_ok();
  if (d != DUO_OK) return d;
  const PruneWs w = carve_prune(ws, n, k, block);
  const hipStream_t s = (hipStream_t)stream;
  // The sweep may run in the Y form (no D = U L^T) unless quantisation
  // groups start inside a block: their grids come from the values of whole
  // groups of columns there, which the Y form would have to rebuild, so those
  // keep D.  Automatic choice: the Y form saves the
  // k^3 / 3 of D but launches two more products per block (measured at
  // n = k = 4096: 0.17 ms slower per layer; k = 11008: 2 ms faster).
  const bool yform = o.form == DUO_FORM_Y || (o.form == DUO_FORM_AUTO && y_ok && k >= kYFormMinK);
  prof_begin(DUO_PROF_SCORE, s);
  duo_status r = score_run(L, ldl, G, ldg, a, k, yform ? nullptr : w.D, k, w.fac, w.score, s);
  prof_end(DUO_PROF_SCORE, s);
  if (r != DUO_OK) return r;
  prof_begin(DUO_PROF_SWEEP, s);
  if (yform)
    r = sweep_run(W, w_dtype, n, k, ldw, L, ldl, nullptr, 0, w.fac, w_sparsity, o, block, mask_in, W_out, W_out_lowp,
                  mask_out, block_scores_out, w.sweep, s, score_u(w.score, k), k, w.D);
  else
    r = sweep_run(W, w_dtype, n, k, ldw, L, ldl, w.D, k, w.fac, w_sparsity, o, block, mask_in, W_out, W_out_lowp,
                  mask_out, block_scores_out, w.sweep, s);
  prof_end(DUO_PROF_SWEEP, s);
  return r;
}

}  // extern "C"
