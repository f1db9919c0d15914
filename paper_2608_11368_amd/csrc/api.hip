// C entry points of libpair.  Every argument a host can check is checked
// here, before anything is enqueued; the kernels only see validated sizes
// and re-check device-resident offsets themselves.
#include <hip/hip_runtime.h>

#include <atomic>

#include "../../include/pair.h"
#include "launch.hpp"

namespace pair {

int device_cu_count() {
  static std::atomic<int> cached[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return 256;
  if (dev < 64) {
    int v = cached[dev].load(std::memory_order_relaxed);
    if (v > 0) return v;
  }
  int cus = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      cus <= 0)
    cus = 256;
  if (dev < 64) cached[dev].store(cus, std::memory_order_relaxed);
  return cus;
}

}  // namespace pair

namespace {

constexpr int64_t kMaxCount = (int64_t)1 << 40;

bool aligned16(const void* ptr) { return (reinterpret_cast<uintptr_t>(ptr) & 15u) == 0; }

int check_groups(int64_t B, int64_t nv, int32_t gmax, const int64_t* offsets) {
  if (offsets == nullptr) return PAIR_EINVAL;
  if (B < 1 || B > 0x7fffffffLL || nv < 2 || nv > kMaxCount) return PAIR_EINVAL;
  if (gmax < 2 || gmax > PAIR_GMAX_LIMIT) return PAIR_ERANGE;
  return PAIR_OK;
}

int check_scores(const void* scores, int32_t dtype, int64_t D, int64_t ld) {
  if (scores == nullptr) return PAIR_EINVAL;
  if (dtype != PAIR_F32 && dtype != PAIR_BF16) return PAIR_EDTYPE;
  if (D < 1 || ld < D || D > kMaxCount || ld > kMaxCount) return PAIR_ERANGE;
  const int64_t elt = dtype == PAIR_BF16 ? 2 : 4;
  if (!aligned16(scores) || (ld * elt) % 16 != 0) return PAIR_EALIGN;
  return PAIR_OK;
}

hipStream_t as_stream(void* s) { return static_cast<hipStream_t>(s); }

}  // namespace

extern "C" {

int pair_design_inclusion(int64_t B, int64_t nv, int32_t gmax, const int64_t* offsets,
                          const float* p, uint64_t seed, int64_t rep0, int64_t R, uint8_t* mask,
                          float* pi, int32_t* edge_count, int32_t* completed, int32_t* d_status,
                          void* stream) {
  int st = check_groups(B, nv, gmax, offsets);
  if (st) return st;
  if (p == nullptr) return PAIR_EINVAL;
  if (R < 1 || rep0 < 0 || R > kMaxCount || rep0 > kMaxCount) return PAIR_ERANGE;
  if (mask == nullptr && pi == nullptr && edge_count == nullptr && completed == nullptr)
    return PAIR_EINVAL;
  if (mask != nullptr && R > kMaxCount / nv) return PAIR_ERANGE;
  if ((edge_count != nullptr || completed != nullptr) && R > kMaxCount / B) return PAIR_ERANGE;
  return pair::launch_design(B, nv, gmax, offsets, p, seed, rep0, R, mask, pi, edge_count,
                             completed, d_status, as_stream(stream));
}

static int check_rule(int32_t rule, float wmax) {
  if (rule < PAIR_RULE_HT || rule > PAIR_RULE_MARGINAL) return PAIR_EINVAL;
  if (rule == PAIR_RULE_CLIPPED && !(wmax > 0.0f && wmax <= 3.4e38f)) return PAIR_EINVAL;
  return PAIR_OK;
}

int pair_edge_coeffs_rule(int64_t B, int64_t nv, int32_t gmax, const int64_t* offsets,
                          const float* rewards, const uint8_t* mask, const float* pi,
                          int32_t rule, float wmax, float* coeff, int32_t* edge_count, float* ess,
                          float* max_weight, int32_t* d_status, void* stream) {
  int st = check_groups(B, nv, gmax, offsets);
  if (st) return st;
  st = check_rule(rule, wmax);
  if (st) return st;
  if (rewards == nullptr || coeff == nullptr) return PAIR_EINVAL;
  return pair::launch_coeffs(B, nv, gmax, offsets, rewards, mask, pi, rule, wmax, coeff,
                             edge_count, ess, max_weight, d_status, as_stream(stream));
}

int pair_design_coeffs(int64_t B, int64_t nv, int32_t gmax, const int64_t* offsets,
                       const float* p, const float* rewards, uint64_t seed, int64_t rep,
                       uint8_t* mask, float* pi, float* coeff, int32_t* edge_count,
                       int32_t* completed, int32_t* d_status, void* stream) {
  int st = check_groups(B, nv, gmax, offsets);
  if (st) return st;
  if (p == nullptr || rewards == nullptr || coeff == nullptr) return PAIR_EINVAL;
  if (rep < 0 || rep > kMaxCount) return PAIR_ERANGE;
  return pair::launch_design_coeffs(B, nv, gmax, offsets, p, rewards, seed, rep, mask, pi, coeff,
                                    edge_count, completed, d_status, as_stream(stream));
}

int pair_edge_coeffs(int64_t B, int64_t nv, int32_t gmax, const int64_t* offsets,
                     const float* rewards, const uint8_t* mask, const float* pi, float* coeff,
                     int32_t* edge_count, int32_t* d_status, void* stream) {
  return pair_edge_coeffs_rule(B, nv, gmax, offsets, rewards, mask, pi, PAIR_RULE_HT, 0.0f, coeff,
                               edge_count, nullptr, nullptr, d_status, stream);
}

int pair_weighted_grad(int64_t B, int64_t nv, const int64_t* offsets, int64_t D,
                       const void* scores, int32_t dtype, int64_t ld, const float* coeff,
                       float* out, int32_t reduce, int32_t* d_status, void* stream) {
  if (offsets == nullptr || coeff == nullptr || out == nullptr) return PAIR_EINVAL;
  if (reduce != 0 && reduce != 1) return PAIR_EINVAL;
  if (B < 1 || B > 0x7fffffffLL || nv < 0 || nv > kMaxCount) return PAIR_EINVAL;
  int st = check_scores(scores, dtype, D, ld);
  if (st) return st;
  if (B > kMaxCount / D) return PAIR_ERANGE;
  return pair::launch_wgrad(B, nv, offsets, D, scores, dtype, ld, coeff, out, reduce, d_status,
                            as_stream(stream));
}

size_t pair_audit_workspace_bytes(int64_t B, int32_t gmax, int64_t D, int64_t R) {
  if (B < 1 || gmax < 2 || gmax > PAIR_GMAX_LIMIT || D < 1 || R < 1 || R > kMaxCount ||
      B > kMaxCount / (R + 1))
    return 0;
  return pair::audit_workspace_bytes(B, gmax, D, R);
}

int pair_audit_rule(int64_t B, int64_t nv, int32_t gmax, const int64_t* offsets, int64_t D,
                    const void* scores, int32_t dtype, int64_t ld, const float* rewards,
                    const float* p, const float* pi_w, int32_t rule, float wmax, uint64_t seed,
                    int64_t rep0, int64_t R, double* mse, double* bias_norm, float* rep_sqerr,
                    int32_t* edge_count, void* workspace, size_t ws_bytes, int32_t* d_status,
                    void* stream) {
  int st = check_groups(B, nv, gmax, offsets);
  if (st) return st;
  st = check_rule(rule, wmax);
  if (st) return st;
  if (dtype != PAIR_BF16) return PAIR_EDTYPE;
  st = check_scores(scores, dtype, D, ld);
  if (st) return st;
  if (rewards == nullptr || p == nullptr || mse == nullptr || bias_norm == nullptr)
    return PAIR_EINVAL;
  if (R < 1 || rep0 < 0 || R > kMaxCount || rep0 > kMaxCount) return PAIR_ERANGE;
  const size_t need = pair_audit_workspace_bytes(B, gmax, D, R);
  if (need == 0) return PAIR_ERANGE;
  if (workspace == nullptr || (reinterpret_cast<uintptr_t>(workspace) & 255u) != 0 ||
      ws_bytes < need)
    return PAIR_EWORKSPACE;
  return pair::launch_audit(B, nv, gmax, offsets, D, scores, ld, rewards, p, pi_w, rule, wmax,
                            seed, rep0, 0, R,
                            mse, bias_norm, rep_sqerr, edge_count, workspace, d_status,
                            as_stream(stream));
}

size_t pair_audit_direction_workspace_bytes(int64_t B, int32_t gmax, int64_t D, int64_t R) {
  if (B < 1 || gmax < 2 || gmax > PAIR_GMAX_LIMIT || D < 1 || D > kMaxCount || R < 1 ||
      R > kMaxCount || B > kMaxCount / (R + 1))
    return 0;
  return pair::direction_workspace_bytes(B, gmax, D, R);
}

int pair_audit_direction(int64_t B, int64_t nv, int32_t gmax, const int64_t* offsets, int64_t D,
                         const void* scores, int32_t dtype, int64_t ld, const float* rewards,
                         const float* p, const float* pi_w, int32_t rule, float wmax,
                         uint64_t seed, int64_t rep0, int64_t R, double* cosine,
                         double* target_norm, void* workspace, size_t ws_bytes,
                         int32_t* d_status, void* stream) {
  int st = check_groups(B, nv, gmax, offsets);
  if (st) return st;
  st = check_rule(rule, wmax);
  if (st) return st;
  if (dtype != PAIR_BF16) return PAIR_EDTYPE;
  st = check_scores(scores, dtype, D, ld);
  if (st) return st;
  if (rewards == nullptr || p == nullptr || cosine == nullptr || target_norm == nullptr)
    return PAIR_EINVAL;
  if (R < 1 || rep0 < 0 || R > kMaxCount || rep0 > kMaxCount) return PAIR_ERANGE;
  const size_t need = pair_audit_direction_workspace_bytes(B, gmax, D, R);
  if (need == 0) return PAIR_ERANGE;
  if (workspace == nullptr || (reinterpret_cast<uintptr_t>(workspace) & 255u) != 0 ||
      ws_bytes < need)
    return PAIR_EWORKSPACE;
  return pair::launch_audit_direction(B, nv, gmax, offsets, D, scores, ld, rewards, p, pi_w, rule,
                                      wmax, seed, rep0, R, cosine, target_norm, workspace,
                                      d_status, as_stream(stream));
}

int pair_design_alloc_ex(int64_t B, int64_t nv, int32_t gmax, const int64_t* offsets,
                         const float* p_hat, const float* c_hat, const float* m_hat,
                         const float* budget, float pi_min, int32_t design, const float* pi_prev,
                         int32_t max_sweeps, float* pi, double* objective, int32_t* iters,
                         double* residual, int32_t* d_status, void* stream) {
  if (offsets == nullptr || p_hat == nullptr || c_hat == nullptr || budget == nullptr ||
      pi == nullptr)
    return PAIR_EINVAL;
  if (B < 1 || B > 0x7fffffffLL || nv < 0 || nv > kMaxCount) return PAIR_EINVAL;
  if (gmax < 1 || gmax > PAIR_GMAX_LIMIT) return PAIR_ERANGE;
  if (design < PAIR_DESIGN_PAIR || design > PAIR_DESIGN_UNIFORM) return PAIR_EINVAL;
  if (!(pi_min > 0.0f && pi_min <= 1.0f)) return PAIR_ERANGE;
  if (max_sweeps < 0) return PAIR_ERANGE;
  return pair::launch_alloc(B, nv, gmax, offsets, p_hat, c_hat, m_hat, budget, pi_min, design,
                            pi_prev, max_sweeps, pi, objective, iters, residual, d_status,
                            as_stream(stream));
}

int pair_design_alloc(int64_t B, int64_t nv, int32_t gmax, const int64_t* offsets,
                      const float* p_hat, const float* c_hat, const float* m_hat,
                      const float* budget, float pi_min, int32_t design, float* pi,
                      double* objective, int32_t* iters, int32_t* d_status, void* stream) {
  return pair_design_alloc_ex(B, nv, gmax, offsets, p_hat, c_hat, m_hat, budget, pi_min, design,
                              nullptr, 0, pi, objective, iters, nullptr, d_status, stream);
}

int pair_cps_fit(int64_t B, int64_t nv, int32_t gmax, const int64_t* offsets,
                 const float* pi_target, double* w, int32_t* n_out, float* pi_joint,
                 int32_t* iters, int32_t* d_status, void* stream) {
  int st = check_groups(B, nv, gmax, offsets);
  if (st) return st;
  if (pi_target == nullptr || w == nullptr) return PAIR_EINVAL;
  return pair::launch_cps_fit(B, nv, gmax, offsets, pi_target, w, n_out, pi_joint, iters,
                              d_status, as_stream(stream));
}

int pair_cps_draw(int64_t B, int64_t nv, int32_t gmax, const int64_t* offsets, const double* w,
                  const int32_t* n, uint64_t seed, int64_t rep0, int64_t R, uint8_t* mask,
                  int32_t* edge_count, int32_t* d_status, void* stream) {
  if (offsets == nullptr || w == nullptr || n == nullptr || mask == nullptr) return PAIR_EINVAL;
  if (B < 1 || B > 0x7fffffffLL || nv < 0 || nv > kMaxCount) return PAIR_EINVAL;
  if (gmax < 1 || gmax > PAIR_GMAX_LIMIT) return PAIR_ERANGE;
  if (R < 1 || rep0 < 0 || R > kMaxCount || rep0 > kMaxCount || R > kMaxCount / (nv > 0 ? nv : 1))
    return PAIR_ERANGE;
  return pair::launch_cps_draw(B, nv, gmax, offsets, w, n, seed, rep0, R, mask, edge_count,
                               d_status, as_stream(stream));
}

size_t pair_audit_exact_workspace_bytes(int64_t B, int32_t gmax, int64_t D) {
  if (B < 1 || gmax < 2 || gmax > PAIR_GMAX_LIMIT || D < 1 || D > kMaxCount) return 0;
  return pair::exact_workspace_bytes(B, gmax, D);
}

int pair_audit_exact(int64_t B, int64_t nv, int32_t gmax, const int64_t* offsets, int64_t D,
                     const void* scores, int32_t dtype, int64_t ld, const float* rewards,
                     const float* p, const float* pi_w, int32_t rule, float wmax, double* mse,
                     double* bias_norm, double* gram, void* workspace, size_t ws_bytes,
                     int32_t* d_status, void* stream) {
  int st = check_groups(B, nv, gmax, offsets);
  if (st) return st;
  st = check_rule(rule, wmax);
  if (st) return st;
  if (rule == PAIR_RULE_RATIO_KE || rule == PAIR_RULE_SELFNORM) return PAIR_EINVAL;
  if (dtype != PAIR_BF16) return PAIR_EDTYPE;
  st = check_scores(scores, dtype, D, ld);
  if (st) return st;
  if (rewards == nullptr || p == nullptr || mse == nullptr || bias_norm == nullptr)
    return PAIR_EINVAL;
  const size_t need = pair_audit_exact_workspace_bytes(B, gmax, D);
  if (need == 0) return PAIR_ERANGE;
  if (workspace == nullptr || (reinterpret_cast<uintptr_t>(workspace) & 255u) != 0 ||
      ws_bytes < need)
    return PAIR_EWORKSPACE;
  return pair::launch_audit_exact(B, nv, gmax, offsets, D, scores, ld, rewards, p, pi_w, rule,
                                  wmax, mse, bias_norm, gram, workspace, d_status,
                                  as_stream(stream));
}

int pair_audit(int64_t B, int64_t nv, int32_t gmax, const int64_t* offsets, int64_t D,
               const void* scores, int32_t dtype, int64_t ld, const float* rewards,
               const float* p, const float* pi_w, uint64_t seed, int64_t rep0, int64_t R,
               double* mse, double* bias_norm, float* rep_sqerr, int32_t* edge_count,
               void* workspace, size_t ws_bytes, int32_t* d_status, void* stream) {
  return pair_audit_rule(B, nv, gmax, offsets, D, scores, dtype, ld, rewards, p, pi_w,
                         PAIR_RULE_HT, 0.0f, seed, rep0, R, mse, bias_norm, rep_sqerr, edge_count,
                         workspace, ws_bytes, d_status, stream);
}

int pair_audit_noalloc(int64_t B, int64_t nv, int32_t gmax, const int64_t* offsets, int64_t D,
                       const void* scores, int32_t dtype, int64_t ld, const float* rewards,
                       const float* p, const float* pi_w, uint64_t seed, int64_t rep0, int64_t R,
                       double* mse, double* bias_norm, float* rep_sqerr, int32_t* edge_count,
                       int32_t* d_status, void* stream) {
  int st = check_groups(B, nv, gmax, offsets);
  if (st) return st;
  if (dtype != PAIR_BF16) return PAIR_EDTYPE;
  st = check_scores(scores, dtype, D, ld);
  if (st) return st;
  if (rewards == nullptr || p == nullptr || mse == nullptr || bias_norm == nullptr)
    return PAIR_EINVAL;
  if (R < 1 || rep0 < 0 || R > kMaxCount || rep0 > kMaxCount) return PAIR_ERANGE;
  if (pair_audit_workspace_bytes(B, gmax, D, R) == 0) return PAIR_ERANGE;
  return pair::launch_audit_noalloc(B, nv, gmax, offsets, D, scores, ld, rewards, p, pi_w, seed,
                                    rep0, R, mse, bias_norm, rep_sqerr, edge_count, d_status,
                                    as_stream(stream));
}

const char* pair_strerror(int code) {
  switch (code) {
    case PAIR_OK: return "ok";
    case PAIR_EINVAL: return "invalid argument (null pointer or malformed size)";
    case PAIR_EDTYPE: return "unsupported score dtype";
    case PAIR_ERANGE: return "size out of the supported range";
    case PAIR_EALIGN: return "scores base pointer or row stride not 16-byte aligned";
    case PAIR_EHIP: return "HIP launch or runtime error";
    case PAIR_EWORKSPACE: return "workspace missing, misaligned or too small";
    case PAIR_ESCRATCH:
      return "one prompt's audit workspace exceeds the no-alloc entry point's static scratch";
    default: return "unknown error code";
  }
}

int pair_version(void) { return 300; }   // 0.3.0: pair_audit_noalloc added

}  // extern "C"
