// Internal host-side launchers (C++ linkage, not exported).  Arguments are
// validated by the C entry points in api.hip before any of these run.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace pair {

// Compute units of the current device (cached per device).
int device_cu_count();

int launch_design(int64_t B, int64_t nv, int32_t gmax, const int64_t* offsets, const float* p,
                  uint64_t seed, int64_t rep0, int64_t R, uint8_t* mask, float* pi,
                  int32_t* edge_count, int32_t* completed, int32_t* d_status, hipStream_t stream);

int launch_coeffs(int64_t B, int64_t nv, int32_t gmax, const int64_t* offsets,
                  const float* rewards, const uint8_t* mask, const float* pi, int32_t rule,
                  float wmax, float* coeff, int32_t* edge_count, float* ess, float* max_weight,
                  int32_t* d_status, hipStream_t stream);

int launch_design_coeffs(int64_t B, int64_t nv, int32_t gmax, const int64_t* offsets,
                         const float* p, const float* rewards, uint64_t seed, int64_t rep,
                         uint8_t* mask, float* pi, float* coeff, int32_t* edge_count,
                         int32_t* completed, int32_t* d_status, hipStream_t stream);

int launch_wgrad(int64_t B, int64_t nv, const int64_t* offsets, int64_t D, const void* scores,
                 int32_t dtype, int64_t ld, const float* coeff, float* out, int32_t reduce,
                 int32_t* d_status, hipStream_t stream);

size_t audit_workspace_bytes(int64_t B, int32_t gmax, int64_t D, int64_t R);

// Prompt b of the call is prompt pbase + b of the generator's counter (its
// design draws are those of that prompt index); 0 for a whole batch.
int launch_audit(int64_t B, int64_t nv, int32_t gmax, const int64_t* offsets, int64_t D,
                 const void* scores, int64_t ld, const float* rewards, const float* p,
                 const float* pi_w, int32_t rule, float wmax, uint64_t seed, int64_t rep0,
                 int64_t pbase, int64_t R, double* mse, double* bias_norm, float* rep_sqerr,
                 int32_t* edge_count, void* workspace, int32_t* d_status, hipStream_t stream);

// pair_audit with the library's static scratch as the workspace, the prompts
// in chunks that fit it (PAIR_ESCRATCH if one prompt does not).
int64_t audit_noalloc_chunk(int64_t B, int32_t gmax, int64_t D, int64_t R);
int launch_audit_noalloc(int64_t B, int64_t nv, int32_t gmax, const int64_t* offsets, int64_t D,
                         const void* scores, int64_t ld, const float* rewards, const float* p,
                         const float* pi_w, uint64_t seed, int64_t rep0, int64_t R, double* mse,
                         double* bias_norm, float* rep_sqerr, int32_t* edge_count,
                         int32_t* d_status, hipStream_t stream);

// max_sweeps <= 0: the library's default cap on a prompt's coordinate sweeps.
int launch_alloc(int64_t B, int64_t nv, int32_t gmax, const int64_t* offsets, const float* p_hat,
                 const float* c_hat, const float* m_hat, const float* budget, float pi_min,
                 int32_t design, const float* pi_prev, int32_t max_sweeps, float* pi,
                 double* objective, int32_t* iters, double* residual, int32_t* d_status,
                 hipStream_t stream);

int launch_cps_fit(int64_t B, int64_t nv, int32_t gmax, const int64_t* offsets,
                   const float* pi_target, double* w, int32_t* n_out, float* pi_joint,
                   int32_t* iters, int32_t* d_status, hipStream_t stream);

int launch_cps_draw(int64_t B, int64_t nv, int32_t gmax, const int64_t* offsets, const double* w,
                    const int32_t* n, uint64_t seed, int64_t rep0, int64_t R, uint8_t* mask,
                    int32_t* edge_count, int32_t* d_status, hipStream_t stream);

size_t exact_workspace_bytes(int64_t B, int32_t gmax, int64_t D);

int launch_audit_exact(int64_t B, int64_t nv, int32_t gmax, const int64_t* offsets, int64_t D,
                       const void* scores, int64_t ld, const float* rewards, const float* p,
                       const float* pi_w, int32_t rule, float wmax, double* mse,
                       double* bias_norm, double* gram, void* workspace, int32_t* d_status,
                       hipStream_t stream);

// Gram matrices K_b = S_b S_b^T in fp64 ([B][gmax][gmax], entries beyond G_b
// not written); the workspace is exact_workspace_bytes(B, gmax, D).
int launch_gram(int64_t B, int64_t nv, int32_t gmax, const int64_t* offsets, int64_t D,
                const void* scores, int64_t ld, double* gram, void* workspace, int32_t* d_status,
                hipStream_t stream);

size_t direction_workspace_bytes(int64_t B, int32_t gmax, int64_t D, int64_t R);

int launch_audit_direction(int64_t B, int64_t nv, int32_t gmax, const int64_t* offsets, int64_t D,
                           const void* scores, int64_t ld, const float* rewards, const float* p,
                           const float* pi_w, int32_t rule, float wmax, uint64_t seed,
                           int64_t rep0, int64_t R, double* cosine, double* target_norm,
                           void* workspace, int32_t* d_status, hipStream_t stream);

}  // namespace pair
