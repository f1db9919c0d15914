// Graph-coupled probability design (paper Sec. 4.3-4.4): continuation
// probabilities from the prefix statistics, batched over prompts.
//
//   d_ij = p_i (1 - p_j) + (1 - p_i) p_j                 Eq. (disagreement)
//   a_ij = d_ij, or d_ij (m_i + m_j)^2 / 4               Eq. (edge-proxy)
//   b_i  = (sum_{j != i} sqrt(a_ij))^2 - sum_{j != i} a_ij
//   min  Phi = sum_{i<j} a_ij / (pi_i pi_j) + sum_i b_i / pi_i
//   s.t. sum_i c_i pi_i <= budget,  pi_min <= pi_i <= 1
// which is Eqs. (convex-objective)-(budget) in pi = e^{-x}.
//
// One 64-lane wavefront per prompt, lane i = vertex i, all arithmetic in
// fp64.  With A_i = sum_{j != i} a_ij / pi_j + b_i, the Lagrangian
// Phi + lam (c^T pi - budget) restricted to coordinate i is A_i / pi_i +
// lam c_i pi_i + const, minimised over the box exactly at
//     pi_i = clip( sqrt(A_i / (lam c_i)), pi_min, 1 ).
// For a fixed multiplier lam, cyclic coordinate descent with these exact
// updates converges to the minimiser of the (convex) Lagrangian; the spent
// budget c^T pi(lam) does not increase with lam, so lam is found by a
// safeguarded false-position search (Illinois) in log space between a
// multiplier that puts every vertex at pi_min and one that puts every vertex
// with positive A at 1, each inner solve warm-started from the previous one.  A_i for one coordinate is a
// wave reduction in which lane j contributes a_ji / pi_j, with a_ji formed on
// the fly from p_j and the wave-uniform p_i, so nothing G x G is stored.
//
// The pointwise comparison design is the same program with a = 0 and
// b_i = p_i (1 - p_i); the uniform design spends the budget with one
// probability.  Vertices whose A is identically zero (no contrast with any
// other vertex) take pi_min.
#include "common.hpp"
#include "launch.hpp"

namespace pair {

namespace {

constexpr int kMaxSweeps = 400;     // inner coordinate-descent sweeps per multiplier
constexpr int kMaxBisect = 200;     // multiplier search steps

__device__ __forceinline__ double wave_min_d(double v) {
#pragma unroll
  for (int m = 1; m < kWave; m <<= 1) v = fmin(v, __shfl_xor(v, m, kWave));
  return v;
}

// Edge proxy a_ij seen from lane j (vertex j) for a wave-uniform vertex i.
__device__ __forceinline__ double proxy(double pi_hat, double pj_hat, double mi, double mj,
                                        bool scaled) {
  double d = pi_hat * (1.0 - pj_hat) + (1.0 - pi_hat) * pj_hat;
  if (scaled) d *= 0.25 * (mi + mj) * (mi + mj);
  return d;
}

__global__ __launch_bounds__(kWave) void alloc_kernel(
    int64_t B, int64_t nv, int32_t gmax, const int64_t* __restrict__ offsets,
    const float* __restrict__ p_hat, const float* __restrict__ c_hat,
    const float* __restrict__ m_hat, const float* __restrict__ budget, float pi_min_f,
    int32_t design, float* __restrict__ pi_out, double* __restrict__ objective,
    int32_t* __restrict__ iters, int32_t* d_status) {
  const int64_t b = blockIdx.x;
  const int lane = threadIdx.x;
  int64_t o0, g;
  if (!prompt_bounds(offsets, b, nv, 1, gmax, &o0, &g, d_status, lane == 0)) return;
  const int gi = (int)g;
  const bool vert = lane < gi;
  const bool scaled = m_hat != nullptr;
  const double pmin = (double)pi_min_f;
  const double p = vert ? (double)p_hat[o0 + lane] : 0.0;
  const double c = vert ? (double)c_hat[o0 + lane] : 0.0;
  const double m = (vert && scaled) ? (double)m_hat[o0 + lane] : 0.0;
  const double bud = (double)budget[b];
  const bool bad_in = vert && !(p >= 0.0 && p <= 1.0 && c > 0.0 && c < 1e300 &&
                                (!scaled || (m >= 0.0 && m < 1e300)));
  if (__ballot(bad_in) != 0ull || !(bud > 0.0) || !(pmin > 0.0 && pmin <= 1.0)) {
    if (lane == 0) raise_status(d_status, PAIR_ST_BUDGET);
    if (vert) pi_out[o0 + lane] = pi_min_f;
    return;
  }

  // Vertex term b_i (pointwise design: p (1 - p)); A_i's range over the box.
  double bv = 0.0, arow = 0.0;
  for (int i = 0; i < gi; ++i) {
    const double p_i = readlane_d(p, i), m_i = readlane_d(m, i);
    const double a = (vert && lane != i && design == PAIR_DESIGN_PAIR)
                         ? proxy(p_i, p, m_i, m, scaled) : 0.0;
    const double s1 = wave_sum_d(sqrt(a)), s2 = wave_sum_d(a);
    if (lane == i) {
      bv = design == PAIR_DESIGN_PAIR ? s1 * s1 - s2 : p * (1.0 - p);
      if (bv < 0.0) bv = 0.0;   // rounding: the exact value is >= 0 (Cauchy-Schwarz)
      arow = s2;
    }
  }

  const double csum = wave_sum_d(c);
  double pi = 1.0;
  int it = 0;
  if (csum <= bud) {
    pi = 1.0;
  } else if (bud < pmin * csum * (1.0 - 1e-12)) {
    if (lane == 0) raise_status(d_status, PAIR_ST_BUDGET);
    pi = pmin;
  } else if (bud <= pmin * csum) {
    pi = pmin;
  } else if (design == PAIR_DESIGN_UNIFORM) {
    pi = fmin(fmax(bud / csum, pmin), 1.0);
  } else {
    // Multiplier bracket: at lam_hi every vertex sits at pi_min; at lam_lo
    // every vertex with A > 0 sits at 1.
    const double a_hi = arow / pmin + bv, a_lo = arow + bv;
    const double lam_hi = 2.0 * wave_max_d(vert ? a_hi / (c * pmin * pmin) : 0.0);
    const double lam_lo =
        0.5 * wave_min_d((vert && a_lo > 0.0) ? a_lo / c : 1e308);
    if (!(lam_hi > 0.0)) {
      pi = pmin;   // no contrast anywhere: the cheapest feasible design
    } else {
      // Root of f(t) = log(c^T pi(e^t)) - log(budget), nonincreasing in t,
      // by Illinois false position on [tlo, thi]: f(tlo) >= 0 >= f(thi);
      // when the same end is replaced twice in a row, the other end's value
      // is halved.  Each evaluation is an inner coordinate descent at
      // lam = e^t, warm-started from the previous iterate.
      double spent = 0.0;
      auto solve_at = [&](double t) -> double {
        const double lam = exp(t);
        for (int sw = 0; sw < kMaxSweeps; ++sw) {
          double change = 0.0;
          for (int i = 0; i < gi; ++i) {
            const double p_i = readlane_d(p, i), m_i = readlane_d(m, i);
            const double a = (vert && lane != i && design == PAIR_DESIGN_PAIR)
                                 ? proxy(p_i, p, m_i, m, scaled) : 0.0;
            const double Ai = wave_sum_d(a / pi);
            if (lane == i) {
              const double A = Ai + bv;
              double nw = A > 0.0 ? sqrt(A / (lam * c)) : pmin;
              nw = fmin(fmax(nw, pmin), 1.0);
              change = fabs(nw - pi) / pi;
              pi = nw;
            }
          }
          ++it;
          if (wave_max_d(change) <= 1e-13) break;
        }
        spent = wave_sum_d(vert ? c * pi : 0.0);
        return log(spent) - log(bud);
      };
      double tlo = log(fmin(lam_lo, lam_hi * 0.5)), thi = log(lam_hi);
      pi = 1.0;
      double flo = solve_at(tlo);
      if (flo > 0.0 && fabs(spent - bud) > 1e-13 * bud) {   // otherwise the budget does not bind
        pi = pmin;
        double fhi = solve_at(thi);
        int side = 0;
        for (int k = 0; k < kMaxBisect && fhi < 0.0 && fabs(spent - bud) > 1e-13 * bud; ++k) {
          double t = (tlo * fhi - thi * flo) / (fhi - flo);
          if (!(t > tlo && t < thi)) t = 0.5 * (tlo + thi);
          const double ft = solve_at(t);
          if (fabs(spent - bud) <= 1e-13 * bud) break;
          if (ft > 0.0) {
            tlo = t;
            flo = ft;
            if (side == 1) fhi *= 0.5;
            side = 1;
          } else {
            thi = t;
            fhi = ft;
            if (side == -1) flo *= 0.5;
            side = -1;
          }
          if (thi - tlo <= 1e-15) break;
        }
      }
      // The last multiplier may leave the budget overspent by a rounding
      // amount: keep the iterate of the feasible side.
      spent = wave_sum_d(vert ? c * pi : 0.0);
      if (spent > bud) pi = fmax(pmin, pi * (bud / spent));
    }
  }

  if (vert) pi_out[o0 + lane] = (float)pi;
  if (objective != nullptr || iters != nullptr) {
    // Phi at the returned probabilities (the PAIR proxy for every design).
    double phi = 0.0;
    for (int i = 0; i < gi; ++i) {
      const double p_i = readlane_d(p, i), m_i = readlane_d(m, i);
      const double pi_i = readlane_d(pi, i);
      const double a = (vert && lane > i) ? proxy(p_i, p, m_i, m, scaled) : 0.0;
      phi += a / (pi_i * pi);
    }
    // b of the PAIR proxy (for the non-PAIR designs bv holds their own term).
    double bp = 0.0;
    for (int i = 0; i < gi; ++i) {
      const double p_i = readlane_d(p, i), m_i = readlane_d(m, i);
      const double a = (vert && lane != i) ? proxy(p_i, p, m_i, m, scaled) : 0.0;
      const double s1 = wave_sum_d(sqrt(a)), s2 = wave_sum_d(a);
      if (lane == i) bp = fmax(s1 * s1 - s2, 0.0);
    }
    phi += vert ? bp / pi : 0.0;
    phi = wave_sum_d(phi);
    if (lane == 0) {
      if (objective != nullptr) objective[b] = phi;
      if (iters != nullptr) iters[b] = it;
    }
  }
}

}  // namespace

int launch_alloc(int64_t B, int64_t nv, int32_t gmax, const int64_t* offsets, const float* p_hat,
                 const float* c_hat, const float* m_hat, const float* budget, float pi_min,
                 int32_t design, float* pi, double* objective, int32_t* iters, int32_t* d_status,
                 hipStream_t stream) {
  hipLaunchKernelGGL(alloc_kernel, dim3((unsigned)B), dim3(kWave), 0, stream, B, nv, gmax, offsets,
                     p_hat, c_hat, m_hat, budget, pi_min, design, pi, objective, iters, d_status);
  return hipGetLastError() == hipSuccess ? PAIR_OK : PAIR_EHIP;
}

}  // namespace pair
