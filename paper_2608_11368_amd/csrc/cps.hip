// Conditional Poisson (fixed-size) design: paper App. B "Fixed-size and
// exact-cost designs" (Hajek 1964 rejective sampling): exactly n of the G
// candidates continue, with first-order probabilities prescribed by the
// allocation and joint probabilities that do not factorise and are computed
// exactly from the design.
//
// With odds w, P(S) = prod_{i in S} w_i / e_n(w) over |S| = n, where e_k is
// the elementary symmetric polynomial, and
//     pi_i  = w_i e_{n-1}(w without i) / e_n(w),
//     pi_ij = w_i w_j e_{n-2}(w without i, j) / e_n(w)
//           = (w_j pi_i - w_i pi_j) / (w_j - w_i)          (w_i != w_j).
//
//  cps_fit_kernel   one wavefront per prompt, fp64.  Each iteration builds the
//                   prefix polynomials e_k(w_0..w_{m-1}) and the suffix
//                   polynomials e_k(w_{m+1}..w_{G-1}) for all m (lane k holds
//                   coefficient k; adding a unit is one whole-wave DPP shift
//                   and one multiply-add), and lane i gets the leave-one-out
//                   coefficient e_{n-1}(w without i) as the convolution
//                   sum_k prefix_i[k] suffix_i[n-1-k] (all terms positive);
//                   the log-odds then take a Newton step whose Hessian is
//                   the design covariance pi_ij - pi_i pi_j (solved by
//                   Gaussian elimination in LDS, lane = row), halved until
//                   the concave objective rises, until every pi_i is within
//                   1e-12 of its target (3-8 evaluations where a plain
//                   fixed point w_i <- w_i pi_target_i / pi_i takes
//                   100-500).  The joint block uses the difference formula
//                   when the two odds differ by more than 1e-5 relative and
//                   the direct leave-two-out polynomial otherwise.
//  cps_draw_kernel  lane = replicate.  The workgroup builds the suffix table
//                   E[i][k] = e_k(w_i .. w_{G-1}) in LDS (lane k, units from
//                   the last); each lane then walks the units in order and
//                   selects unit i with probability
//                   w_i E[i+1][k-1] / E[i][k], k the units still to select,
//                   comparing the top 32 bits of Philox4x64-10 word (i & 3) at
//                   counter (replicate, prompt, i >> 2, 0) with that
//                   probability times 2^32.  The table and the thresholds use
//                   unfused fp64 operations in a fixed order, so each draw is
//                   a deterministic function of (seed, replicate, prompt, w).
#include "common.hpp"
#include "launch.hpp"

namespace pair {

namespace {

constexpr int kMaxFitIter = 200;   // evaluations of pi(w), rejected steps included

// e_0..e_{KP-1} (only k <= n meaningful) of the units 0..g-1 excluding skip1
// and skip2, the units' odds taken from the wave (lane m holds w_m).
template <int KP>
__device__ __forceinline__ void esp_excl(double w, int g, int n, int skip1, int skip2,
                                         double (&e)[KP]) {
  e[0] = 1.0;
#pragma unroll
  for (int k = 1; k < KP; ++k) e[k] = 0.0;
  for (int m = 0; m < g; ++m) {
    const double wm0 = readlane_d(w, m);
    const double wm = (m == skip1 || m == skip2) ? 0.0 : wm0;
#pragma unroll
    for (int k = KP - 1; k >= 1; --k)
      if (k <= n) e[k] = __dadd_rn(e[k], __dmul_rn(wm, e[k - 1]));
  }
}

// e[k] for a run-time k, by an unrolled select (keeps e in registers).
template <int KP>
__device__ __forceinline__ double pick(const double (&e)[KP], int k) {
  double v = 0.0;
#pragma unroll
  for (int q = 0; q < KP; ++q) v = q == k ? e[q] : v;
  return v;
}

// Prefix rows Pf[m][k] = e_k(w_0 .. w_{m-1}), m = 0..g, and suffix rows
// Sf[m][k] = e_k(w_{m+1} .. w_{g-1}), m = 0..g-1, for k <= n, written to LDS
// with row stride kS.  Lane k carries coefficient k; adding unit m is
// e_k <- e_k + w_m e_{k-1}, where e_{k-1} arrives from lane k - 1 by a
// whole-wave DPP shift (lane 0 receives 0).
constexpr int kS = 65;

template <int KP>
__device__ __forceinline__ void esp_tables(double w, int g, int n, int lane, double* Pf,
                                           double* Sf) {
  double col = lane == 0 ? 1.0 : 0.0;
  if (lane <= n) Pf[lane] = col;
  for (int m = 0; m < g; ++m) {
    const double wm = readlane_d(w, m);
    col = __dadd_rn(col, __dmul_rn(wm, dpp_d<0x138>(col)));   // wave_shr:1
    if (lane <= n) Pf[(m + 1) * kS + lane] = col;
  }
  col = lane == 0 ? 1.0 : 0.0;
  if (lane <= n) Sf[(g - 1) * kS + lane] = col;
  for (int m = g - 1; m >= 1; --m) {
    const double wm = readlane_d(w, m);
    col = __dadd_rn(col, __dmul_rn(wm, dpp_d<0x138>(col)));
    if (lane <= n) Sf[(m - 1) * kS + lane] = col;
  }
  __syncthreads();
}

template <int KP>
__global__ __launch_bounds__(kWave) void cps_fit_kernel(
    int64_t B, int64_t nv, int32_t gmax, const int64_t* __restrict__ offsets,
    const float* __restrict__ pi_target, double* __restrict__ w_out, int32_t* __restrict__ n_out,
    float* __restrict__ pi_joint, int32_t* __restrict__ iters, int32_t* d_status) {
  __shared__ double Pf[(KP + 1) * kS];
  __shared__ double Sf[KP * kS];
  const int64_t b = blockIdx.x;
  const int lane = threadIdx.x;
  int64_t o0, g64;
  if (!prompt_bounds(offsets, b, nv, 2, gmax, &o0, &g64, d_status, lane == 0)) return;
  const int g = (int)g64;
  const bool unit = lane < g;
  double t = unit ? (double)pi_target[o0 + lane] : 0.0;
  const double sum = wave_sum_d(t);
  const int n = (int)rint(sum);
  bool bad = unit && !(t > 0.0 && t < 1.0);
  bad = __ballot(bad) != 0ull || n < 1 || n >= g || fabs(sum - (double)n) > 1e-4 * (double)n;
  if (!bad) {
    t = unit ? t * ((double)n / sum) : 0.0;
    bad = __ballot(unit && !(t < 1.0)) != 0ull;
  }
  if (bad) {
    if (lane == 0) {
      raise_status(d_status, PAIR_ST_P_RANGE);
      if (n_out != nullptr) n_out[b] = 0;
      if (iters != nullptr) iters[b] = 0;
    }
    if (unit) w_out[o0 + lane] = 0.0;
    return;
  }

  // Newton's method on the log-odds theta (mean zero, so the geometric mean
  // of the odds is 1).  The fitted odds maximise the concave
  //     F(theta) = sum_i t_i theta_i - log e_n(exp(theta)),
  // whose gradient is t - pi(theta) and whose negative Hessian is the
  // design's covariance H_ij = pi_ij - pi_i pi_j (H_ii = pi_i (1 - pi_i)).
  // H 1 = 0 (the odds are defined up to scale), so the step solves
  // (H + 1 1^T / g) d = t - pi, whose solution is orthogonal to 1.  A step
  // is kept when F rises by at least 1e-4 of the predicted amount or the
  // largest relative error falls; otherwise it is halved.
  // Wave reductions and lane reads run in uniform control flow: every lane
  // takes part, and lanes beyond the group contribute 0.
  double th = unit ? log(t / (1.0 - t)) : 0.0;
  const double mean0 = wave_sum_d(th) / (double)g;
  th = unit ? th - mean0 : 0.0;
  double w = 0.0, pi = 0.0, en_last = 1.0;
  double th0 = 0.0, d = 0.0, f0 = 0.0, err0 = 0.0, slope = 0.0, step = 1.0;
  bool have_base = false;
  int it = 0;
  bool converged = false;
  for (; it < kMaxFitIter; ++it) {
    w = unit ? exp(th) : 0.0;
    // pi_i(w) for every unit from the prefix and suffix polynomial tables.
    esp_tables<KP>(w, g, n, lane, Pf, Sf);
    const double en = Pf[g * kS + n];
    en_last = en;
    pi = 0.0;
    if (unit) {
      double e1 = 0.0;   // e_{n-1}(w without i) = sum_k Pf[i][k] Sf[i][n-1-k]
      for (int k = 0; k < n; ++k)
        e1 = __dadd_rn(e1, __dmul_rn(Pf[lane * kS + k], Sf[lane * kS + (n - 1 - k)]));
      pi = w * e1 / en;
    }
    const double f = wave_sum_d(unit ? t * th : 0.0) - log(en);
    const double err = wave_max_d(unit ? fabs(pi / t - 1.0) : 0.0);
    __syncthreads();   // every lane has read the tables before the Newton system overwrites them
    if (have_base) {
      const bool ok = isfinite(f) && isfinite(err) &&
                      (f >= f0 + 1e-4 * step * slope || err < err0);
      if (!ok && step > 1e-9) {
        step *= 0.5;
        th = unit ? th0 + step * d : 0.0;
        continue;
      }
    }
    if (err <= 1e-12) {
      converged = true;
      break;
    }
    th0 = th;
    f0 = f;
    err0 = err;
    have_base = true;

    // Row `lane` of H + 1 1^T / g, in registers (entry j in a[j], zero
    // beyond the group).  Off the diagonal pi_ij comes from the difference
    // formula; where two odds agree to 1e-6 it is numerically unreliable, and
    // those entries share what the row identity
    // sum_{j != i} pi_ij = (n - 1) pi_i leaves (exact for equal odds).
    const double inv_g = 1.0 / (double)g;
    double a[KP];
    double known = 0.0;
    int nclose = 0;
#pragma unroll
    for (int j = 0; j < KP; ++j) {
      const double wj = readlane_d(w, j), pj = readlane_d(pi, j);
      const bool off = unit && j < g && j != lane;
      const bool sep = fabs(wj - w) > 1e-6 * fmax(wj, w);
      const double pij = (off && sep) ? (wj * pi - w * pj) / (wj - w) : 0.0;
      known += pij;
      nclose += (off && !sep) ? 1 : 0;
      a[j] = (off && sep) ? pij - pi * pj + inv_g
                          : ((unit && j == lane) ? pi * (1.0 - pi) + inv_g : 0.0);
    }
    if (__ballot(nclose > 0) != 0ull) {
      const double share = nclose > 0 ? ((double)(n - 1) * pi - known) / (double)nclose : 0.0;
#pragma unroll
      for (int j = 0; j < KP; ++j) {
        const double wj = readlane_d(w, j), pj = readlane_d(pi, j);
        const bool close = unit && j < g && j != lane && !(fabs(wj - w) > 1e-6 * fmax(wj, w));
        if (close) a[j] = share - pi * pj + inv_g;
      }
    }
    // Gaussian elimination without pivoting (the matrix is symmetric
    // positive definite).  Lane i owns row i and right-hand side entry x_i.
    // At step k every row is shifted left by k, so the pivot column is
    // always a[0] and all register indices are compile-time constants; the
    // pivot row (row k, shifted) and its right-hand side are kept in LDS
    // (U, xs) for the back substitution.  Rows at or above the pivot compute
    // values that are never used.
    double x = unit ? t - pi : 0.0;
    double* U = Pf;          // U[k][j] = row k's entry k + j after step k
    double* xs = Sf;         // right-hand side of pivot row k
    for (int k = 0; k < g; ++k) {
      if (lane == k) {
#pragma unroll
        for (int j = 0; j < KP; ++j) U[k * KP + j] = a[j];
        xs[k] = x;
      }
      __syncthreads();
      const double xk = readlane_d(x, k);
      const double m = a[0] / U[k * KP];
#pragma unroll
      for (int j = 1; j < KP; ++j) a[j - 1] = a[j] - m * U[k * KP + j];
      a[KP - 1] = 0.0;
      x -= m * xk;
    }
    // Back substitution, one column of U per step: lane i keeps the still
    // unresolved part y_i of its equation and ends holding x_i.
    double y = unit ? xs[lane] : 0.0;
    for (int k = g - 1; k >= 0; --k) {
      const double xk = readlane_d(y, k) / U[k * KP];
      if (lane == k) y = xk;
      if (lane < k) y -= U[lane * KP + (k - lane)] * xk;
    }
    x = y;
    d = unit ? x : 0.0;
    slope = wave_sum_d(unit ? (t - pi) * d : 0.0);
    step = 1.0;
    th = unit ? th0 + d : 0.0;
    const double mean = wave_sum_d(th) / (double)g;
    th = unit ? th - mean : 0.0;
    __syncthreads();   // the tables are rebuilt by the next iteration
  }
  if (!converged && lane == 0) raise_status(d_status, PAIR_ST_P_RANGE);
  if (unit) w_out[o0 + lane] = w;
  if (lane == 0) {
    if (n_out != nullptr) n_out[b] = n;
    if (iters != nullptr) iters[b] = converged ? it : -it;
  }

  if (pi_joint != nullptr) {
    // Row i of the joint block by lane i, from the last evaluation's pi and
    // e_n(w).  The difference formula loses about eps / gap of relative
    // accuracy, so it is used where the two odds differ by more than 1e-5
    // (error below 1e-8, under the fp32 output's rounding); closer pairs
    // take the leave-two-out polynomial.
    float* row = pi_joint + (b * (int64_t)gmax + lane) * gmax;
    for (int j = 0; j < gmax; ++j) {
      const double wj = readlane_d(w, j < g ? j : 0), pj = readlane_d(pi, j < g ? j : 0);
      const bool pair_ij = unit && j < g && j != lane;
      const bool sep = fabs(wj - w) > 1e-5 * fmax(wj, w);
      double v = 0.0;
      if (unit && j == lane) v = pi;
      if (pair_ij && sep) v = (wj * pi - w * pj) / (wj - w);
      const bool direct = pair_ij && !sep && n >= 2;
      if (__ballot(direct) != 0ull) {
        double e2[KP];
        esp_excl<KP>(w, g, n - 2, lane, j, e2);   // w of lane j is excluded too
        if (direct) v = w * wj * pick<KP>(e2, n - 2) / en_last;
      }
      if (lane < gmax) row[j] = (float)v;
    }
  }
}

template <int KP>
__global__ __launch_bounds__(kWave) void cps_draw_kernel(
    int64_t B, int64_t nv, int32_t gmax, const int64_t* __restrict__ offsets,
    const double* __restrict__ w, const int32_t* __restrict__ n_in, uint64_t seed, int64_t rep0,
    int64_t R, int64_t nwg, uint8_t* __restrict__ mask, int32_t* __restrict__ edge_count,
    int32_t* d_status) {
  __shared__ double E[(KP + 1) * (KP + 1)];   // E[i][k], row stride KP + 1
  __shared__ double wl[KP];
  const int64_t b = blockIdx.x / nwg;
  const int64_t chunk = blockIdx.x - b * nwg;
  const int lane = threadIdx.x;
  int64_t o0, g64;
  if (!prompt_bounds(offsets, b, nv, 1, gmax, &o0, &g64, d_status, chunk == 0 && lane == 0))
    return;
  const int g = (int)g64;
  const int n = n_in[b];
  bool bad = n < 0 || n > g;
  if (!bad && lane < g) {
    const double wv = w[o0 + lane];
    bad = !(wv > 0.0 && wv < 1e300);
    wl[lane] = wv;
  }
  if (__ballot(bad) != 0ull) {
    if (chunk == 0 && lane == 0) raise_status(d_status, PAIR_ST_P_RANGE);
    return;
  }
  constexpr int S = KP + 1;
  const bool all_or_none = n == 0 || n == g;   // no randomness: the table is not needed
  if (!all_or_none) {
    if (lane <= n) E[g * S + lane] = lane == 0 ? 1.0 : 0.0;
  }
  __syncthreads();
  for (int i = all_or_none ? -1 : g - 1; i >= 0; --i) {
    if (lane <= n) {
      double v = 1.0;
      if (lane >= 1) {
        const double tmul = __dmul_rn(wl[i], E[(i + 1) * S + lane - 1]);
        v = __dadd_rn(E[(i + 1) * S + lane], tmul);
      }
      E[i * S + lane] = v;
    }
    __syncthreads();
  }

  const int64_t r = chunk * kWave + lane;
  if (r >= R) return;
  const uint64_t rg = (uint64_t)(rep0 + r);
  uint8_t* mrow = mask + r * nv + o0;
  int k = n;
  Philox4x64 x;
  for (int i = 0; i < g; ++i) {
    if (all_or_none) {
      mrow[i] = (uint8_t)(n == g ? 1 : 0);
      continue;
    }
    if ((i & 3) == 0) x = philox4x64_10(rg, (uint64_t)b, (uint64_t)(i >> 2), 0ull, seed, 0ull);
    const double u = (double)(philox_word(x, i & 3) >> 32);
    int take = 0;
    if (k > 0) {
      const double num = __dmul_rn(wl[i], E[(i + 1) * S + k - 1]);
      const double prob = __ddiv_rn(num, E[i * S + k]);
      take = u < __dmul_rn(prob, 4294967296.0) ? 1 : 0;
    }
    mrow[i] = (uint8_t)take;
    k -= take;
  }
  if (edge_count != nullptr) edge_count[r * B + b] = n * (n - 1) / 2;
}

}  // namespace

int launch_cps_fit(int64_t B, int64_t nv, int32_t gmax, const int64_t* offsets,
                   const float* pi_target, double* w, int32_t* n_out, float* pi_joint,
                   int32_t* iters, int32_t* d_status, hipStream_t stream) {
  const int ks = (gmax + 15) / 16;
#define PAIR_CPS_FIT(KP_)                                                                        \
  hipLaunchKernelGGL(cps_fit_kernel<KP_>, dim3((unsigned)B), dim3(kWave), 0, stream, B, nv, gmax, \
                     offsets, pi_target, w, n_out, pi_joint, iters, d_status)
  switch (ks) {
    case 1: PAIR_CPS_FIT(16); break;
    case 2: PAIR_CPS_FIT(32); break;
    case 3: PAIR_CPS_FIT(48); break;
    default: PAIR_CPS_FIT(64); break;
  }
#undef PAIR_CPS_FIT
  return hipGetLastError() == hipSuccess ? PAIR_OK : PAIR_EHIP;
}

int launch_cps_draw(int64_t B, int64_t nv, int32_t gmax, const int64_t* offsets, const double* w,
                    const int32_t* n, uint64_t seed, int64_t rep0, int64_t R, uint8_t* mask,
                    int32_t* edge_count, int32_t* d_status, hipStream_t stream) {
  const int ks = (gmax + 15) / 16;
  const int64_t nwg = (R + kWave - 1) / kWave;
  const int64_t grid = B * nwg;
  if (grid > 0x7fffffffLL) return PAIR_ERANGE;
#define PAIR_CPS_DRAW(KP_)                                                                     \
  hipLaunchKernelGGL(cps_draw_kernel<KP_>, dim3((unsigned)grid), dim3(kWave), 0, stream, B, nv, \
                     gmax, offsets, w, n, seed, rep0, R, nwg, mask, edge_count, d_status)
  switch (ks) {
    case 1: PAIR_CPS_DRAW(16); break;
    case 2: PAIR_CPS_DRAW(32); break;
    case 3: PAIR_CPS_DRAW(48); break;
    default: PAIR_CPS_DRAW(64); break;
  }
#undef PAIR_CPS_DRAW
  return hipGetLastError() == hipSuccess ? PAIR_OK : PAIR_EHIP;
}

}  // namespace pair
