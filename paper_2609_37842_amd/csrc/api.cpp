// C ABI entry points: argument validation, then enqueue on the caller's stream.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdio>
#include <mutex>
#include <set>
#include <string>
#include <tuple>

#include "common.h"
#include "plan.h"

namespace eogp {
// implemented in the kernel sources
size_t rotate_retain_ws(const eogp_plan* p, int64_t N, int64_t T);
eogp_status rotate_retain(const eogp_plan* p, const void* acts, int64_t ld_acts, const void* grads,
                          int64_t ld_grads, bool bf16_in,
                          const uint8_t* mask, int64_t N, int64_t T, void* Z, bool z16, int64_t ldz,
                          int prec, bool compacted, void* ws, size_t ws_bytes, hipStream_t s);
size_t compact_ws(int64_t N, int64_t T);
eogp_status compact_tokens(const uint8_t* mask, int64_t N, int64_t T, int prec, void* ws,
                           size_t ws_bytes, hipStream_t s);
eogp_status sign_pack(const float* X, int64_t ldx, int64_t N, int64_t k, uint8_t* codes,
                      int64_t cstride, uint16_t* scales, int64_t sstride, hipStream_t s);
size_t pca_ws(int64_t N, int64_t m, int64_t k, eogp_dtype p_dtype);
size_t pca_split_copy_bytes(int64_t m, int64_t k, eogp_dtype p_dtype);
eogp_status pca_project(const void* Z, eogp_dtype z_dtype, int64_t ldz, int64_t N, int64_t m, const void* P,
                        eogp_dtype p_dtype, int64_t ldp, int64_t k, float* X, int64_t ldx,
                        bool accurate, void* ws, size_t ws_bytes, hipStream_t s);
int32_t score_max_topk();
int srht_max_log();
size_t srht_ws(int64_t N, int64_t m);
size_t pca_fit_ws(int64_t n, int64_t m, int64_t k);
eogp_status pca_fit(const float* Z, int64_t ldz, int64_t n, int64_t m, int64_t k, float* Pt,
                    int64_t ldp, float* mu, void* ws, size_t ws_bytes, hipStream_t s);
size_t ekfac_ws(int64_t N, int64_t T, int64_t d_in, int64_t d_out);
eogp_status ekfac_pass(const void* acts, int64_t ld_acts, const void* grads, int64_t ld_grads,
                       bool bf16_in, const uint8_t* mask, int64_t N, int64_t T, int64_t d_in,
                       int64_t d_out, const float* Q_A, const float* Q_S, int prec,
                       int32_t e_acts, int32_t e_grads, float* sq, int accumulate, void* ws,
                       size_t ws_bytes, hipStream_t s);
eogp_status srht_project(const float* Z, int64_t ldz, int64_t N, int64_t m, const int8_t* signs,
                         const int32_t* rows, int64_t k, float* X, int64_t ldx, void* ws,
                         size_t ws_bytes, hipStream_t s);
const char* last_error_cstr();
size_t score_ws(int64_t N, int64_t Q, int32_t U, const int64_t* kmod, int32_t topk);
eogp_status score_topk(const uint8_t* codes, int64_t cstride, const uint16_t* scales, int64_t N,
                       int32_t U, const int64_t* kmod, const float* Y, int64_t ldy, int64_t Q,
                       int32_t topk, int64_t* out_idx, float* out_score, float* full, void* ws,
                       size_t ws_bytes, hipStream_t s);
size_t score_scratch_bytes();
eogp_status score_scratch(void** out);
eogp_status sign_pack_tiled(const float* X, int64_t ldx, int64_t N, int64_t k, int64_t row0,
                            uint8_t* codes, int64_t steps_row, int64_t step0, uint16_t* scales,
                            int64_t sstride, hipStream_t s);
eogp_status score_topk_tiled(const uint8_t* codes, const uint16_t* scales, int64_t N, int32_t U,
                             const int64_t* kmod, const float* Y, int64_t ldy, int64_t Q,
                             int32_t topk, int64_t* out_idx, float* out_score, float* full,
                             void* ws, size_t ws_bytes, hipStream_t s);

namespace {
thread_local std::string g_last_error;
}

void set_error(const std::string& msg) { g_last_error = msg; }

eogp_status fail(eogp_status st, const std::string& msg) {
  g_last_error = msg;
  return st;
}

const char* last_error_cstr() { return g_last_error.c_str(); }

eogp_status check_hip(hipError_t e, const char* what) {
  if (e == hipSuccess) return EOGP_OK;
  g_last_error = std::string(what) + ": " + hipGetErrorString(e);
  return EOGP_ERR_DEVICE;
}

eogp_status ensure_dynamic_lds(const void* fn, int bytes) {
  static std::mutex mu;
  static std::set<std::tuple<const void*, int, int>> done;   // (kernel, device, bytes)
  int dev = 0;
  EOGP_HIP(hipGetDevice(&dev));
  std::lock_guard<std::mutex> g(mu);
  if (done.count({fn, dev, bytes})) return EOGP_OK;
  EOGP_HIP(hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, bytes));
  done.insert({fn, dev, bytes});
  return EOGP_OK;
}

}  // namespace eogp

using namespace eogp;

namespace {
inline hipStream_t S(void* s) { return static_cast<hipStream_t>(s); }
constexpr int64_t kMaxFlat = (int64_t)1 << 31;

eogp_status check_plan_args(const float* eigvals, int64_t d_out, int64_t d_in, double damping,
                            int64_t m, const float* Q_A, const float* Q_S) {
  if (!eigvals || !Q_A || !Q_S) return fail(EOGP_ERR_INVALID, "plan: NULL pointer");
  if (d_out < 1 || d_in < 1) return fail(EOGP_ERR_INVALID, "plan: d_in and d_out must be >= 1");
  if (d_out * d_in >= kMaxFlat) return fail(EOGP_ERR_INVALID, "plan: d_in*d_out must be < 2^31");
  if (m < 1 || m > d_out * d_in) return fail(EOGP_ERR_INVALID, "plan: need 1 <= m <= d_in*d_out");
  if (!(damping > 0.0) || damping != damping) return fail(EOGP_ERR_INVALID, "plan: damping must be > 0");
  return EOGP_OK;
}

eogp_status check_first_stage(const eogp_plan* p, const void* acts, const void* grads,
                              eogp_dtype dt, int64_t N, int64_t T, const void* Z, int64_t ldz,
                              eogp_prec prec) {
  if (!p) return fail(EOGP_ERR_INVALID, "rotate_retain: NULL plan");
  if (N < 0 || T < 0) return fail(EOGP_ERR_INVALID, "rotate_retain: negative size");
  if (N > 0 && T > 0 && (!acts || !grads || !Z)) return fail(EOGP_ERR_INVALID, "rotate_retain: NULL pointer");
  if (N > 0 && !Z) return fail(EOGP_ERR_INVALID, "rotate_retain: NULL Z");
  if (dt != EOGP_F32 && dt != EOGP_BF16)
    return fail(EOGP_ERR_UNSUPPORTED, "rotate_retain: inputs must be fp32 or bf16");
  if (ldz < p->m) return fail(EOGP_ERR_INVALID, "rotate_retain: ldz < m");
  if (prec != EOGP_PREC_FAST && prec != EOGP_PREC_ACCURATE && prec != EOGP_PREC_F16)
    return fail(EOGP_ERR_INVALID, "rotate_retain: unknown precision mode");
  if (N * T + 8 * N + 256 >= kMaxFlat)
    return fail(EOGP_ERR_INVALID, "rotate_retain: N*T + 8N + 256 must be < 2^31");
  return EOGP_OK;
}
eogp_status planned_first_stage(const eogp_plan* plan, const void* acts, int64_t ld_acts,
                                const void* out_grads, int64_t ld_grads, eogp_dtype in_dtype,
                                const uint8_t* token_mask, bool compacted, int64_t N, int64_t T,
                                void* Z, eogp_dtype z_dtype, int64_t ldz, eogp_prec prec, void* ws,
                                size_t ws_bytes, void* stream) {
  eogp_status st = check_first_stage(plan, acts, out_grads, in_dtype, N, T, Z, ldz, prec);
  if (st != EOGP_OK) return st;
  if (z_dtype != EOGP_F32 && z_dtype != EOGP_F16)
    return fail(EOGP_ERR_INVALID, "rotate_retain: Z must be fp32 or fp16");
  if (ld_acts == 0) ld_acts = plan->d_in;
  if (ld_grads == 0) ld_grads = plan->d_out;
  if (ld_acts < plan->d_in || ld_grads < plan->d_out)
    return fail(EOGP_ERR_INVALID, "rotate_retain: token stride smaller than the width");
  if (in_dtype == EOGP_BF16 &&
      (ld_acts % 8 || ld_grads % 8 || (uintptr_t)acts % 16 || (uintptr_t)out_grads % 16))
    return fail(EOGP_ERR_UNSUPPORTED,
                "rotate_retain: bf16 token rows must start on 16-byte boundaries");
  if (N * T * std::max(ld_acts, ld_grads) >= ((int64_t)1 << 62))
    return fail(EOGP_ERR_INVALID, "rotate_retain: inputs too large");
  if (N == 0) return EOGP_OK;
  if (ws_bytes < rotate_retain_ws(plan, N, T) || !ws)
    return fail(EOGP_ERR_WORKSPACE, "rotate_retain: workspace too small");
  int dev = -1;
  if (hipGetDevice(&dev) == hipSuccess && dev != plan->device)
    return fail(EOGP_ERR_INVALID, "rotate_retain: plan belongs to another device");
  return rotate_retain(plan, acts, ld_acts, out_grads, ld_grads, in_dtype == EOGP_BF16,
                       token_mask, N, T, Z, z_dtype == EOGP_F16, ldz, (int)prec, compacted, ws,
                       ws_bytes, S(stream));
}
}  // namespace

extern "C" {

const char* eogp_status_string(eogp_status st) {
  switch (st) {
    case EOGP_OK: return "ok";
    case EOGP_ERR_INVALID: return "invalid argument";
    case EOGP_ERR_UNSUPPORTED: return "unsupported";
    case EOGP_ERR_DEVICE: return "device error";
    case EOGP_ERR_WORKSPACE: return "workspace too small";
    default: return "unknown status";
  }
}

const char* eogp_last_error(void) { return last_error_cstr(); }

int32_t eogp_version(void) { return 100; }

eogp_status eogp_plan_create(const float* eigvals, int64_t d_out, int64_t d_in, double damping,
                             int64_t m, const float* Q_A, const float* Q_S, void* stream,
                             eogp_plan** out) {
  if (!out) return fail(EOGP_ERR_INVALID, "plan: NULL output handle");
  *out = nullptr;
  eogp_status st = check_plan_args(eigvals, d_out, d_in, damping, m, Q_A, Q_S);
  if (st != EOGP_OK) return st;
  return build_plan(eigvals, d_out, d_in, damping, m, Q_A, Q_S, S(stream), out);
}

void eogp_plan_destroy(eogp_plan* plan) { free_plan(plan); }

eogp_status eogp_plan_get_info(const eogp_plan* p, eogp_plan_info* info) {
  if (!p || !info) return fail(EOGP_ERR_INVALID, "plan_get_info: NULL pointer");
  info->d_out = p->d_out;
  info->d_in = p->d_in;
  info->m = p->m;
  info->damping = p->damping;
  info->n_rows = p->n_rows;
  info->n_cols = p->n_cols;
  info->n_tiles = p->n_tiles;
  info->retained_flat = p->ret_flat;
  info->retained_weight = p->ret_w;
  return EOGP_OK;
}

eogp_status eogp_plan_copy_retained(const eogp_plan* p, int32_t* flat_out, float* weight_out,
                                    void* stream) {
  if (!p) return fail(EOGP_ERR_INVALID, "plan_copy_retained: NULL plan");
  if (flat_out)
    EOGP_HIP(hipMemcpyAsync(flat_out, p->ret_flat, p->m * 4, hipMemcpyDeviceToDevice, S(stream)));
  if (weight_out)
    EOGP_HIP(hipMemcpyAsync(weight_out, p->ret_w, p->m * 4, hipMemcpyDeviceToDevice, S(stream)));
  return EOGP_OK;
}

eogp_status eogp_plan_set_input_exponents(eogp_plan* p, int32_t e_acts, int32_t e_grads) {
  if (!p) return fail(EOGP_ERR_INVALID, "plan_set_input_exponents: NULL plan");
  if (e_acts < -60 || e_acts > 60 || e_grads < -60 || e_grads > 60)
    return fail(EOGP_ERR_INVALID, "plan_set_input_exponents: exponents must lie in [-60, 60]");
  p->e_acts = e_acts;
  p->e_grads = e_grads;
  return EOGP_OK;
}

size_t eogp_rotate_retain_workspace_size(const eogp_plan* plan, int64_t N, int64_t T) {
  if (!plan || N < 0 || T < 0) return 0;
  return rotate_retain_ws(plan, N, T);
}


eogp_status eogp_rotate_retain_planned(const eogp_plan* plan, const void* acts,
                                       int64_t ld_acts, const void* out_grads, int64_t ld_grads,
                                       eogp_dtype in_dtype, const uint8_t* token_mask, int64_t N,
                                       int64_t T, void* Z, eogp_dtype z_dtype, int64_t ldz,
                                       eogp_prec prec, void* ws, size_t ws_bytes, void* stream) {
  return planned_first_stage(plan, acts, ld_acts, out_grads, ld_grads, in_dtype, token_mask, false,
                             N, T, Z, z_dtype, ldz, prec, ws, ws_bytes, stream);
}

size_t eogp_compact_tokens_workspace_size(int64_t N, int64_t T) {
  if (N < 0 || T < 0 || N * T + 8 * N + 256 >= kMaxFlat) return 0;
  return compact_ws(N, T);
}

eogp_status eogp_compact_tokens(const uint8_t* token_mask, int64_t N, int64_t T, eogp_prec prec,
                                void* ws, size_t ws_bytes, void* stream) {
  if (N < 0 || T < 0) return fail(EOGP_ERR_INVALID, "compact_tokens: negative size");
  if (N * T + 8 * N + 256 >= kMaxFlat)
    return fail(EOGP_ERR_INVALID, "compact_tokens: N*T + 8N + 256 must be < 2^31");
  if (prec != EOGP_PREC_ACCURATE && prec != EOGP_PREC_FAST && prec != EOGP_PREC_F16)
    return fail(EOGP_ERR_INVALID, "compact_tokens: unknown precision");
  if (N == 0) return EOGP_OK;
  if (!ws || ws_bytes < compact_ws(N, T))
    return fail(EOGP_ERR_WORKSPACE, "compact_tokens: workspace too small");
  return compact_tokens(token_mask, N, T, (int)prec, ws, ws_bytes, S(stream));
}

eogp_status eogp_rotate_retain_compacted(const eogp_plan* plan, const void* acts, int64_t ld_acts,
                                         const void* out_grads, int64_t ld_grads,
                                         eogp_dtype in_dtype, int64_t N, int64_t T, void* Z,
                                         eogp_dtype z_dtype, int64_t ldz, eogp_prec prec,
                                         void* ws, size_t ws_bytes, void* stream) {
  return planned_first_stage(plan, acts, ld_acts, out_grads, ld_grads, in_dtype, nullptr, true, N,
                             T, Z, z_dtype, ldz, prec, ws, ws_bytes, stream);
}

size_t eogp_rotate_retain_oneshot_workspace_size(int64_t N, int64_t T, int64_t d_in,
                                                 int64_t d_out, int64_t m) {
  if (N < 0 || T < 0 || d_in < 1 || d_out < 1 || m < 1) return 0;
  eogp_plan probe;
  probe.rows_pad = round_up(d_out, kPanelTile);
  probe.cols_pad = round_up(d_in, kPanelTile);
  probe.m = m;
  return rotate_retain_ws(&probe, N, T);
}

eogp_status eogp_rotate_retain(const void* acts, int64_t ld_acts, const void* out_grads,
                               int64_t ld_grads, eogp_dtype in_dtype,
                               const uint8_t* token_mask, int64_t N, int64_t T, int64_t d_in,
                               int64_t d_out, const float* Q_A, const float* Q_S,
                               const float* eigvals, double damping, int64_t m, float* Z,
                               int64_t ldz, eogp_prec prec, void* ws, size_t ws_bytes,
                               void* stream) {
  eogp_status st = check_plan_args(eigvals, d_out, d_in, damping, m, Q_A, Q_S);
  if (st != EOGP_OK) return st;
  if (ldz < m) return fail(EOGP_ERR_INVALID, "rotate_retain: ldz < m");
  if (ws_bytes < eogp_rotate_retain_oneshot_workspace_size(N, T, d_in, d_out, m) || (!ws && N > 0))
    return fail(EOGP_ERR_WORKSPACE, "rotate_retain: workspace too small");
  eogp_plan* plan = nullptr;
  st = build_plan(eigvals, d_out, d_in, damping, m, Q_A, Q_S, S(stream), &plan);
  if (st != EOGP_OK) return st;
  st = eogp_rotate_retain_planned(plan, acts, ld_acts, out_grads, ld_grads, in_dtype, token_mask,
                                  N, T, Z, EOGP_F32, ldz, prec, ws, ws_bytes, stream);
  hipError_t e = hipStreamSynchronize(S(stream));
  free_plan(plan);
  if (st == EOGP_OK && e != hipSuccess) return check_hip(e, "rotate_retain");
  return st;
}

size_t eogp_pca_project_workspace_size(int64_t N, int64_t m, int64_t k, eogp_dtype p_dtype,
                                       eogp_prec prec) {
  (void)prec;
  if (N < 0 || m < 1 || k < 1) return 0;
  return pca_ws(N, m, k, p_dtype);
}

eogp_status eogp_pca_project(const void* Z, eogp_dtype z_dtype, int64_t ldz, int64_t N, int64_t m,
                             const void* P, eogp_dtype p_dtype, int64_t ldp, int64_t k, float* X,
                             int64_t ldx, eogp_prec prec, void* ws, size_t ws_bytes, void* stream) {
  if (N < 0 || m < 1 || k < 1) return fail(EOGP_ERR_INVALID, "pca_project: bad sizes");
  if (k > m) return fail(EOGP_ERR_INVALID, "pca_project: need k <= m");
  if (prec != EOGP_PREC_FAST && prec != EOGP_PREC_ACCURATE)
    return fail(EOGP_ERR_INVALID, "pca_project: precision must be FAST or ACCURATE");
  if (N > 0 && (!Z || !P || !X)) return fail(EOGP_ERR_INVALID, "pca_project: NULL pointer");
  if (ldz < m || ldp < m || ldx < k) return fail(EOGP_ERR_INVALID, "pca_project: leading dimension too small");
  if (p_dtype != EOGP_F32 && p_dtype != EOGP_BF16 && p_dtype != EOGP_F16)
    return fail(EOGP_ERR_INVALID, "pca_project: bad P dtype");
  if (z_dtype != EOGP_F32 && z_dtype != EOGP_F16 && z_dtype != EOGP_BF16)
    return fail(EOGP_ERR_INVALID, "pca_project: bad Z dtype");
  if (z_dtype != EOGP_F32 && z_dtype != p_dtype)
    return fail(EOGP_ERR_UNSUPPORTED, "pca_project: 16-bit Z needs P of the same type");
  if (z_dtype != EOGP_F32 && N > 0 && (ldz % 8 || (uintptr_t)Z % 16))
    return fail(EOGP_ERR_UNSUPPORTED, "pca_project: 16-bit Z rows must start on 16-byte boundaries");
  if (ws_bytes < pca_split_copy_bytes(m, k, p_dtype) || (p_dtype == EOGP_F32 && !ws))
    return fail(EOGP_ERR_WORKSPACE, "pca_project: workspace too small for fp32 P");
  return pca_project(Z, z_dtype, ldz, N, m, P, p_dtype, ldp, k, X, ldx,
                     prec == EOGP_PREC_ACCURATE, ws, ws_bytes, S(stream));
}

eogp_status eogp_sign_pack(const float* X, int64_t ldx, int64_t N, int64_t k, uint8_t* codes,
                           int64_t code_row_stride, uint16_t* scales, int64_t scale_stride,
                           void* stream) {
  if (N < 0 || k < 1) return fail(EOGP_ERR_INVALID, "sign_pack: bad sizes");
  if (N >= kMaxFlat) return fail(EOGP_ERR_INVALID, "sign_pack: N must be < 2^31");
  if (N > 0 && (!X || !codes || !scales)) return fail(EOGP_ERR_INVALID, "sign_pack: NULL pointer");
  if (ldx < k) return fail(EOGP_ERR_INVALID, "sign_pack: ldx < k");
  if (code_row_stride < (k + 7) / 8) return fail(EOGP_ERR_INVALID, "sign_pack: code row stride too small");
  if (scale_stride < 1) return fail(EOGP_ERR_INVALID, "sign_pack: scale stride must be >= 1");
  return sign_pack(X, ldx, N, k, codes, code_row_stride, scales, scale_stride, S(stream));
}

eogp_status eogp_sign_pack_tiled(const float* X, int64_t ldx, int64_t N, int64_t k, int64_t row0,
                                 uint8_t* codes, int64_t steps_per_row, int64_t step0,
                                 uint16_t* scales, int64_t scale_stride, void* stream) {
  if (N < 0 || k < 512 || k % 512 != 0)
    return fail(EOGP_ERR_INVALID, "sign_pack_tiled: k must be a positive multiple of 512");
  if (row0 < 0 || N >= kMaxFlat || row0 >= ((int64_t)1 << 40))
    return fail(EOGP_ERR_INVALID, "sign_pack_tiled: bad row range");
  if (step0 < 0 || step0 + k / 512 > steps_per_row)
    return fail(EOGP_ERR_INVALID, "sign_pack_tiled: the module's steps must lie inside the row");
  if (N > 0 && (!X || !codes || !scales)) return fail(EOGP_ERR_INVALID, "sign_pack_tiled: NULL pointer");
  if ((uintptr_t)codes % 16 != 0) return fail(EOGP_ERR_INVALID, "sign_pack_tiled: codes must be 16-byte aligned");
  if (ldx < k) return fail(EOGP_ERR_INVALID, "sign_pack_tiled: ldx < k");
  if (scale_stride < 1) return fail(EOGP_ERR_INVALID, "sign_pack_tiled: scale stride must be >= 1");
  return sign_pack_tiled(X, ldx, N, k, row0, codes, steps_per_row, step0, scales, scale_stride,
                         S(stream));
}

size_t eogp_ekfac_workspace_size(int64_t N, int64_t T, int64_t d_in, int64_t d_out) {
  if (N < 0 || T < 0 || d_in < 1 || d_out < 1) return 0;
  return ekfac_ws(N, T, d_in, d_out);
}

eogp_status eogp_ekfac_eigenvalues(const void* acts, int64_t ld_acts, const void* out_grads,
                                   int64_t ld_grads, eogp_dtype in_dtype,
                                   const uint8_t* token_mask, int64_t N, int64_t T,
                                   int64_t d_in, int64_t d_out, const float* Q_A,
                                   const float* Q_S, eogp_prec prec, int32_t e_acts,
                                   int32_t e_grads, float* sq_sum, int32_t accumulate, void* ws,
                                   size_t ws_bytes, void* stream) {
  if (N < 0 || T < 0 || d_in < 1 || d_out < 1) return fail(EOGP_ERR_INVALID, "ekfac: bad sizes");
  if (d_out * d_in >= kMaxFlat) return fail(EOGP_ERR_INVALID, "ekfac: d_in*d_out must be < 2^31");
  if (N * T + 8 * N + 256 >= kMaxFlat)
    return fail(EOGP_ERR_INVALID, "ekfac: N*T + 8N + 256 must be < 2^31");
  if (e_acts < -60 || e_acts > 60 || e_grads < -60 || e_grads > 60)
    return fail(EOGP_ERR_INVALID, "ekfac: input exponents must lie in [-60, 60]");
  if (!Q_A || !Q_S || !sq_sum) return fail(EOGP_ERR_INVALID, "ekfac: NULL pointer");
  if (N > 0 && T > 0 && (!acts || !out_grads)) return fail(EOGP_ERR_INVALID, "ekfac: NULL pointer");
  if (in_dtype != EOGP_F32 && in_dtype != EOGP_BF16)
    return fail(EOGP_ERR_UNSUPPORTED, "ekfac: inputs must be fp32 or bf16");
  if (prec != EOGP_PREC_FAST && prec != EOGP_PREC_ACCURATE && prec != EOGP_PREC_F16)
    return fail(EOGP_ERR_INVALID, "ekfac: unknown precision mode");
  if (ld_acts == 0) ld_acts = d_in;
  if (ld_grads == 0) ld_grads = d_out;
  if (ld_acts < d_in || ld_grads < d_out)
    return fail(EOGP_ERR_INVALID, "ekfac: token stride smaller than the width");
  if (in_dtype == EOGP_BF16 &&
      (ld_acts % 8 || ld_grads % 8 || (uintptr_t)acts % 16 || (uintptr_t)out_grads % 16))
    return fail(EOGP_ERR_UNSUPPORTED, "ekfac: bf16 token rows must start on 16-byte boundaries");
  if (ws_bytes < ekfac_ws(N, T, d_in, d_out) || !ws)
    return fail(EOGP_ERR_WORKSPACE, "ekfac: workspace too small");
  return ekfac_pass(acts, ld_acts, out_grads, ld_grads, in_dtype == EOGP_BF16, token_mask, N, T,
                    d_in, d_out, Q_A, Q_S, (int)prec, e_acts, e_grads, sq_sum, accumulate, ws,
                    ws_bytes, S(stream));
}

size_t eogp_srht_project_workspace_size(int64_t N, int64_t m) {
  if (N < 0 || m < 1 || m > ((int64_t)1 << srht_max_log())) return 0;
  return srht_ws(N, m);
}

eogp_status eogp_srht_project(const float* Z, int64_t ldz, int64_t N, int64_t m,
                              const int8_t* signs, const int32_t* rows, int64_t k, float* X,
                              int64_t ldx, void* ws, size_t ws_bytes, void* stream) {
  if (N < 0 || m < 1 || k < 1) return fail(EOGP_ERR_INVALID, "srht_project: bad sizes");
  if (N >= kMaxFlat) return fail(EOGP_ERR_INVALID, "srht_project: N must be < 2^31");
  if (m > ((int64_t)1 << srht_max_log()))
    return fail(EOGP_ERR_UNSUPPORTED, "srht_project: m > 2^20 is not supported");
  int64_t p = 1;
  while (p < m) p <<= 1;
  if (k > p) return fail(EOGP_ERR_INVALID, "srht_project: need k <= p = 2^ceil(log2 m)");
  if (ldz < m || ldx < k) return fail(EOGP_ERR_INVALID, "srht_project: leading dimension too small");
  if (N > 0 && (!Z || !signs || !rows || !X)) return fail(EOGP_ERR_INVALID, "srht_project: NULL pointer");
  if (ws_bytes < srht_ws(N, m) || (srht_ws(N, m) > 0 && !ws))
    return fail(EOGP_ERR_WORKSPACE, "srht_project: workspace too small");
  return srht_project(Z, ldz, N, m, signs, rows, k, X, ldx, ws, ws_bytes, S(stream));
}

size_t eogp_pca_fit_workspace_size(int64_t n, int64_t m, int64_t k) {
  if (n < 1 || m < 1 || k < 1 || k > std::min(n, m) || n >= kMaxFlat) {
    (void)fail(EOGP_ERR_INVALID, "pca_fit: need 1 <= k <= min(n, m) and n < 2^31");
    return 0;
  }
  return pca_fit_ws(n, m, k);
}

eogp_status eogp_pca_fit(const float* Z, int64_t ldz, int64_t n, int64_t m, int64_t k, float* Pt,
                         int64_t ldp, float* mu, void* ws, size_t ws_bytes, void* stream) {
  if (n < 1 || m < 1 || k < 1) return fail(EOGP_ERR_INVALID, "pca_fit: bad sizes");
  if (k > std::min(n, m)) return fail(EOGP_ERR_INVALID, "pca_fit: need k <= min(n, m)");
  if (n >= kMaxFlat) return fail(EOGP_ERR_INVALID, "pca_fit: n must be < 2^31");
  if (ldz < m || ldp < m) return fail(EOGP_ERR_INVALID, "pca_fit: leading dimension too small");
  if (!Z || !Pt || !mu || !ws) return fail(EOGP_ERR_INVALID, "pca_fit: NULL pointer");
  return pca_fit(Z, ldz, n, m, k, Pt, ldp, mu, ws, ws_bytes, S(stream));
}

size_t eogp_score_topk_workspace_size(int64_t N, int64_t Q, int32_t U, const int64_t* k_per_module,
                                      int32_t topk) {
  if (N < 0 || Q < 0 || U < 1 || !k_per_module || topk < 1) return 0;
  return score_ws(N, Q, U, k_per_module, topk);
}

namespace {
eogp_status check_score_args(const uint8_t* codes, int64_t code_row_stride,
                             const uint16_t* scales, int64_t N, int32_t U,
                             const int64_t* k_per_module, const float* Y, int64_t ldy, int64_t Q,
                             int32_t topk, int64_t* out_idx, float* out_score) {
  if (N < 0 || Q < 0 || U < 1 || !k_per_module) return fail(EOGP_ERR_INVALID, "score_topk: bad sizes");
  if (topk < 1 || topk > score_max_topk()) return fail(EOGP_ERR_INVALID, "score_topk: topk out of range");
  if (N >= ((int64_t)1 << 32) - 1) return fail(EOGP_ERR_INVALID, "score_topk: N too large");
  int64_t ksum = 0;
  for (int u = 0; u < U; ++u) {
    if (k_per_module[u] < 64 || k_per_module[u] % 64 != 0)
      return fail(EOGP_ERR_INVALID, "score_topk: every k_u must be a positive multiple of 64");
    if (k_per_module[u] > ((int64_t)1 << 22))
      return fail(EOGP_ERR_INVALID, "score_topk: k_u must be at most 2^22");
    ksum += k_per_module[u];
  }
  if (ksum >= kMaxFlat) return fail(EOGP_ERR_INVALID, "score_topk: sum of k_u too large");
  if (code_row_stride < ksum / 8) return fail(EOGP_ERR_INVALID, "score_topk: code row stride too small");
  if (code_row_stride % 8 != 0 || (uintptr_t)codes % 8 != 0)
    return fail(EOGP_ERR_INVALID, "score_topk: codes rows must be 8-byte aligned");
  if (ldy < ksum) return fail(EOGP_ERR_INVALID, "score_topk: ldy too small");
  if (Q > 0 && (!Y || !out_idx || !out_score)) return fail(EOGP_ERR_INVALID, "score_topk: NULL pointer");
  if (N > 0 && (!codes || !scales)) return fail(EOGP_ERR_INVALID, "score_topk: NULL pointer");
  if (Q > 65535) return fail(EOGP_ERR_INVALID, "score_topk: Q too large for one call");
  return EOGP_OK;
}
}  // namespace

eogp_status eogp_score_topk(const uint8_t* codes, int64_t code_row_stride, const uint16_t* scales,
                            int64_t N, int32_t U, const int64_t* k_per_module, const float* Y,
                            int64_t ldy, int64_t Q, int32_t topk, int64_t* out_idx,
                            float* out_score, float* full_scores, void* ws, size_t ws_bytes,
                            void* stream) {
  const eogp_status st = check_score_args(codes, code_row_stride, scales, N, U, k_per_module, Y,
                                          ldy, Q, topk, out_idx, out_score);
  if (st != EOGP_OK) return st;
  if (ws_bytes < score_ws(N, Q, U, k_per_module, topk) || !ws)
    return fail(EOGP_ERR_WORKSPACE, "score_topk: workspace too small");
  return score_topk(codes, code_row_stride, scales, N, U, k_per_module, Y, ldy, Q, topk, out_idx,
                    out_score, full_scores, ws, ws_bytes, S(stream));
}

eogp_status eogp_score_topk_tiled(const uint8_t* codes, const uint16_t* scales, int64_t N,
                                  int32_t U, const int64_t* k_per_module, const float* Y,
                                  int64_t ldy, int64_t Q, int32_t topk, int64_t* out_idx,
                                  float* out_score, float* full_scores, void* ws, size_t ws_bytes,
                                  void* stream) {
  if (U < 1 || !k_per_module) return fail(EOGP_ERR_INVALID, "score_topk_tiled: bad sizes");
  int64_t ksum = 0;
  for (int u = 0; u < U; ++u) {
    if (k_per_module[u] < 512 || k_per_module[u] % 512 != 0)
      return fail(EOGP_ERR_INVALID, "score_topk_tiled: every k_u must be a positive multiple of 512");
    ksum += k_per_module[u];
  }
  // a tiled store row holds ksum / 8 bytes (a multiple of 64); the other checks as for
  // the row-major layout
  const eogp_status st = check_score_args(codes, ksum / 8, scales, N, U, k_per_module, Y, ldy, Q,
                                          topk, out_idx, out_score);
  if (st != EOGP_OK) return st;
  if ((uintptr_t)codes % 16 != 0) return fail(EOGP_ERR_INVALID, "score_topk_tiled: codes must be 16-byte aligned");
  if (ws_bytes < score_ws(N, Q, U, k_per_module, topk) || !ws)
    return fail(EOGP_ERR_WORKSPACE, "score_topk_tiled: workspace too small");
  return score_topk_tiled(codes, scales, N, U, k_per_module, Y, ldy, Q, topk, out_idx, out_score,
                          full_scores, ws, ws_bytes, S(stream));
}

eogp_status eogp_score_topk_noalloc(const uint8_t* codes, int64_t code_row_stride,
                                    const uint16_t* scales, int64_t N, int32_t U,
                                    const int64_t* k_per_module, const float* Y, int64_t ldy,
                                    int64_t Q, int32_t topk, int64_t* out_idx, float* out_score,
                                    float* full_scores, void* stream) {
  eogp_status st = check_score_args(codes, code_row_stride, scales, N, U, k_per_module, Y, ldy, Q,
                                    topk, out_idx, out_score);
  if (st != EOGP_OK) return st;
  const size_t need = score_ws(N, Q, U, k_per_module, topk);
  if (need > score_scratch_bytes())
    return fail(EOGP_ERR_INVALID, "score_topk_noalloc: this call needs " + std::to_string(need) +
                                      " bytes of scratch, more than the " +
                                      std::to_string(score_scratch_bytes()) +
                                      " bytes the entry point holds per GPU (use eogp_score_topk "
                                      "with a workspace, or fewer queries per call)");
  void* scratch = nullptr;
  st = score_scratch(&scratch);
  if (st != EOGP_OK) return st;
  return score_topk(codes, code_row_stride, scales, N, U, k_per_module, Y, ldy, Q, topk, out_idx,
                    out_score, full_scores, scratch, score_scratch_bytes(), S(stream));
}

}  // extern "C"
