// Edge-coefficient fold: pair-corrected sequence advantages, paper Eq.
// (pair-advantage), accumulated over the induced edges as in Algorithm 1 and
// finished as App. C describes (fp32 accumulation, centred over the observed
// endpoints).
//
// The same fold serves the estimator variants of the audit and ablation
// tables (edge-weight rules: unweighted, observed-edge mean, clipped,
// self-normalised, marginal-only); it also reports the weights' effective
// sample size (sum w)^2 / sum w^2 and the largest weight (App. D metrics).
//
// One 64-lane wavefront per prompt, lane i = vertex i.  The prompt's rho
// block is staged in LDS (row stride gmax + 1 so that a column walk is
// conflict-free); lane i then walks j = 0..G-1 in order and adds
// (r_i - r_j) / rho_ij for every observed edge, dividing only when both
// endpoints completed (rho may be 0 on edges that were never observable).
#include "common.hpp"
#include "launch.hpp"

namespace pair {

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int m = 1; m < kWave; m <<= 1) v = fmaxf(v, __shfl_xor(v, m, kWave));
  return v;
}

__global__ __launch_bounds__(64) void edge_coeffs_kernel(
    int64_t B, int64_t nv, int32_t gmax, const int64_t* __restrict__ offsets,
    const float* __restrict__ rewards, const uint8_t* __restrict__ mask,
    const float* __restrict__ pi, int32_t rule, float wmax, float* __restrict__ coeff,
    int32_t* __restrict__ edge_count, float* __restrict__ ess, float* __restrict__ max_weight,
    int32_t* d_status) {
  extern __shared__ float rho_lds[];  // [gmax][gmax + 1]
  const int64_t b = blockIdx.x;
  const int lane = threadIdx.x;
  int64_t o0, g;
  if (!prompt_bounds(offsets, b, nv, 2, gmax, &o0, &g, d_status, lane == 0)) return;
  const int stride = gmax + 1;

  if (pi != nullptr) {
    const float* blk = pi + b * (int64_t)gmax * gmax;
    for (int64_t idx = lane; idx < g * g; idx += kWave) {
      const int64_t i = idx / g, j = idx - i * g;
      rho_lds[i * stride + j] = blk[i * gmax + j];
    }
  }
  __syncthreads();

  const bool vert = lane < g;
  const bool m_i = vert && (mask == nullptr || mask[o0 + lane] != 0);
  const float r_i = vert ? rewards[o0 + lane] : 0.0f;
  const uint64_t obs = __ballot(m_i);
  const int k = __popcll(obs);
  const float pii = (pi != nullptr && vert) ? rho_lds[lane * stride + lane] : 1.0f;

  float c = 0.0f, nsn = 0.0f, sw = 0.0f, sw2 = 0.0f, wmx = 0.0f;
  bool bad_rho = false;
  for (int j = 0; j < g; ++j) {
    const float r_j = lane_value(r_i, j);
    if (!((obs >> j) & 1ull) || !m_i || j == lane) continue;
    float rho = 1.0f, pij = 1.0f;
    if (pi != nullptr) {
      const int lo = lane < j ? lane : j, hi = lane < j ? j : lane;
      rho = rho_lds[lo * stride + hi];
      pij = rho_lds[j * stride + j];
    }
    float term, we, ir;
    if (!rule_term(rule, wmax, r_i - r_j, rho, pii, pij, &term, &we, &ir)) {
      bad_rho = true;
      continue;
    }
    c += term;
    nsn += ir;
    sw += we;
    sw2 += we * we;
    wmx = fmaxf(wmx, we);
  }
  if (bad_rho) raise_status(d_status, PAIR_ST_RHO_RANGE);

  // A~_i = c_i / (2N): 2N = G (G - 1) for HT, unweighted, clipped and
  // marginal-only; k (k - 1) for the observed-edge mean; sum over both
  // endpoints of 1/rho for the self-normalised rule.  Centre over the
  // completed vertices except for the marginal-only rule, whose fold is not
  // antisymmetric.
  float den = (float)(g * (g - 1));
  if (rule == PAIR_RULE_RATIO_KE) den = (float)(k * (k - 1));
  if (rule == PAIR_RULE_SELFNORM) den = wave_sum(nsn);
  float a = 0.0f;
  if (m_i && k >= 2) a = c / den;
  if (rule != PAIR_RULE_MARGINAL) {
    const float total = wave_sum(a);
    if (k >= 2 && m_i) a = a - total / (float)k;
  }
  if (!(k >= 2 && m_i)) a = 0.0f;
  if (vert) coeff[o0 + lane] = a;
  // Every edge was visited from both endpoints: (S/2)^2 / (S2/2) = S^2 / (2 S2).
  const float s1 = wave_sum(sw), s2 = wave_sum(sw2), mx = wave_max(wmx);
  if (lane == 0) {
    if (edge_count != nullptr) edge_count[b] = k * (k - 1) / 2;
    if (ess != nullptr) ess[b] = k >= 2 ? s1 * s1 / (2.0f * s2) : 0.0f;
    if (max_weight != nullptr) max_weight[b] = k >= 2 ? mx : 0.0f;
  }
}

// Design draw and HT coefficient fold of one replicate in one launch: one
// wavefront per prompt, lane i = vertex i.  The indicators are drawn exactly
// as design_draw_kernel draws them, the logged rho_ij = fl32(p_i p_j) is
// formed on the fly (the value the design writes to its pi block), and the
// fold adds (r_i - r_j) / rho_ij over observed partners in ascending order,
// then centres -- the same arithmetic as edge_coeffs_kernel on the logged
// block, so the coefficients are bitwise those of the two-call path.
// The kernel is one latency chain, so each lane reads its p_i and r_i once;
// partners' values move between lanes (scalar lane reads in the fold,
// shuffles for the rho block), and the rho block is written last.
__global__ __launch_bounds__(64) void design_coeffs_kernel(
    int64_t B, int64_t nv, int32_t gmax, const int64_t* __restrict__ offsets,
    const float* __restrict__ p, const float* __restrict__ rewards, uint64_t seed, int64_t rep,
    uint8_t* __restrict__ mask, float* __restrict__ pi, float* __restrict__ coeff,
    int32_t* __restrict__ edge_count, int32_t* __restrict__ completed, int32_t* d_status) {
  const int64_t b = blockIdx.x;
  const int lane = threadIdx.x;
  int64_t o0, g;
  const bool ok = prompt_bounds(offsets, b, nv, 2, gmax, &o0, &g, d_status, lane == 0);
  if (!ok) {
    if (pi != nullptr) {   // a malformed prompt logs an all-zero block
      float* blk = pi + b * (int64_t)gmax * gmax;
      for (int idx = lane; idx < gmax * gmax; idx += kWave) blk[idx] = 0.0f;
    }
    return;
  }
  const bool vert = lane < g;
  const float p_i = vert ? p[o0 + lane] : 1.0f;
  const float r_i = vert ? rewards[o0 + lane] : 0.0f;
  int J = 0;
  if (vert) {
    const Philox4x64 x = philox4x64_10((uint64_t)rep, (uint64_t)b, (uint64_t)(lane >> 2), 0ull,
                                       seed, 0ull);
    const uint64_t u32 = philox_word(x, lane & 3) >> 32;
    if (p_in_range(p_i)) {
      J = u32 < inclusion_threshold(p_i) ? 1 : 0;
    } else {
      raise_status(d_status, PAIR_ST_P_RANGE);
    }
    if (mask != nullptr) mask[o0 + lane] = (uint8_t)J;
  }
  const uint64_t obs = __ballot(J != 0);
  const int k = __popcll(obs);
  const bool m_i = J != 0;
  float c = 0.0f;
  bool bad_rho = false;
  for (int j = 0; j < g; ++j) {
    const float r_j = lane_value(r_i, j);
    const float p_j = lane_value(p_i, j);
    if (!((obs >> j) & 1ull) || !m_i || j == lane) continue;
    const float rho = lane < j ? p_i * p_j : p_j * p_i;
    if (!(rho > 0.0f && rho <= 1.0f)) {
      bad_rho = true;
      continue;
    }
    c += (r_i - r_j) / rho;
  }
  if (bad_rho) raise_status(d_status, PAIR_ST_RHO_RANGE);
  float a = 0.0f;
  if (m_i && k >= 2) a = c / (float)(g * (g - 1));
  const float total = wave_sum(a);
  if (k >= 2 && m_i) {
    a = a - total / (float)k;
  } else {
    a = 0.0f;
  }
  if (vert) coeff[o0 + lane] = a;
  if (lane == 0) {
    if (edge_count != nullptr) edge_count[b] = k * (k - 1) / 2;
    if (completed != nullptr) completed[b] = k;
  }
  if (pi != nullptr) {
    // Logged rho block: fl32(p_i p_j) off the diagonal, p_i on it, zero
    // outside the G_b x G_b corner.
    float* blk = pi + b * (int64_t)gmax * gmax;
    // Whole-wave iterations: every lane takes part in the shuffles (a
    // shuffle from an inactive lane is not defined), only the store is
    // guarded.
    for (int base = 0; base < gmax * gmax; base += kWave) {
      const int idx = base + lane;
      const int i = idx / gmax, j = idx - i * gmax;
      const float pa = __shfl(p_i, i < kWave ? i : 0, kWave);
      const float pb = __shfl(p_i, j, kWave);
      float v = 0.0f;
      if (i < g && j < g) v = (i == j) ? pa : pa * pb;
      if (idx < gmax * gmax) blk[idx] = v;
    }
  }
}

int launch_design_coeffs(int64_t B, int64_t nv, int32_t gmax, const int64_t* offsets,
                         const float* p, const float* rewards, uint64_t seed, int64_t rep,
                         uint8_t* mask, float* pi, float* coeff, int32_t* edge_count,
                         int32_t* completed, int32_t* d_status, hipStream_t stream) {
  hipLaunchKernelGGL(design_coeffs_kernel, dim3((unsigned)B), dim3(64), 0, stream, B, nv, gmax,
                     offsets, p, rewards, seed, rep, mask, pi, coeff, edge_count, completed,
                     d_status);
  return hipGetLastError() == hipSuccess ? PAIR_OK : PAIR_EHIP;
}

int launch_coeffs(int64_t B, int64_t nv, int32_t gmax, const int64_t* offsets,
                  const float* rewards, const uint8_t* mask, const float* pi, int32_t rule,
                  float wmax, float* coeff, int32_t* edge_count, float* ess, float* max_weight,
                  int32_t* d_status, hipStream_t stream) {
  const size_t lds = pi != nullptr ? (size_t)gmax * (gmax + 1) * sizeof(float) : 0;
  hipLaunchKernelGGL(edge_coeffs_kernel, dim3((unsigned)B), dim3(64), lds, stream, B, nv, gmax,
                     offsets, rewards, mask, pi, rule, wmax, coeff, edge_count, ess, max_weight,
                     d_status);
  return hipGetLastError() == hipSuccess ? PAIR_OK : PAIR_EHIP;
}

}  // namespace pair
