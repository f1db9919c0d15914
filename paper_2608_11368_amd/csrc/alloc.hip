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

constexpr int kMaxSweeps = 400;       // inner coordinate-descent sweeps per multiplier
constexpr int kMaxBisect = 200;       // multiplier search steps
constexpr int kDefaultCap = 10000;    // total sweeps of one prompt unless the caller caps them

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

// Median of v over the lanes with `in` set (the mean of the two middle values
// for an even count), the same in every lane; 0 if no lane is set.  Ranks
// are counted per lane, ties broken by lane index.
__device__ double wave_median_d(double v, bool in, int g, int lane) {
  const uint64_t mask = __ballot(in);
  const int n = __popcll(mask);
  if (n == 0) return 0.0;
  int rank = 0;
  for (int j = 0; j < g; ++j) {
    const double vj = readlane_d(v, j);
    if (((mask >> j) & 1ull) && (vj < v || (vj == v && j < lane))) ++rank;
  }
  const int r1 = (n - 1) / 2, r2 = n / 2;
  const double lo = wave_sum_d((in && rank == r1) ? v : 0.0);
  const double hi = wave_sum_d((in && rank == r2) ? v : 0.0);
  return r1 == r2 ? lo : 0.5 * (lo + hi);
}

__global__ __launch_bounds__(kWave) void alloc_kernel(
    int64_t B, int64_t nv, int32_t gmax, const int64_t* __restrict__ offsets,
    const float* __restrict__ p_hat, const float* __restrict__ c_hat,
    const float* __restrict__ m_hat, const float* __restrict__ budget, float pi_min_f,
    int32_t design, const float* __restrict__ pi_prev, int32_t cap,
    float* __restrict__ pi_out, double* __restrict__ objective, int32_t* __restrict__ iters,
    double* __restrict__ residual, int32_t* d_status) {
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
  // The program's edge weights: the proxy for the PAIR design (and for the
  // residual of the uniform design), none for the pointwise design.
  const bool edges = design != PAIR_DESIGN_POINTWISE;

  // Vertex term b_i (pointwise design: p (1 - p)); A_i's range over the box.
  double bv = 0.0, arow = 0.0;
  for (int i = 0; i < gi; ++i) {
    const double p_i = readlane_d(p, i), m_i = readlane_d(m, i);
    const double a = (vert && lane != i && edges) ? proxy(p_i, p, m_i, m, scaled) : 0.0;
    const double s1 = wave_sum_d(sqrt(a)), s2 = wave_sum_d(a);
    if (lane == i) {
      bv = edges ? s1 * s1 - s2 : p * (1.0 - p);
      if (bv < 0.0) bv = 0.0;   // rounding: the exact value is >= 0 (Cauchy-Schwarz)
      arow = s2;
    }
  }
  // A_i = sum_{j != i} a_ij / x_j + b_i of the program at probabilities x,
  // in lane i (one wave reduction per vertex).
  auto a_vec = [&](double x) -> double {
    double out = 0.0;
    for (int i = 0; i < gi; ++i) {
      const double p_i = readlane_d(p, i), m_i = readlane_d(m, i);
      const double a = (vert && lane != i && edges) ? proxy(p_i, p, m_i, m, scaled) : 0.0;
      const double Ai = wave_sum_d(a / x);
      if (lane == i) out = Ai + bv;
    }
    return out;
  };

  const double csum = wave_sum_d(c);
  const double uni = fmin(fmax(bud / csum, pmin), 1.0);   // the uniform design's probability
  double pi = 1.0;
  int it = 0;
  bool failed = false;
  if (csum <= bud) {
    pi = 1.0;
  } else if (bud < pmin * csum * (1.0 - 1e-12)) {
    if (lane == 0) raise_status(d_status, PAIR_ST_BUDGET);
    pi = pmin;
  } else if (bud <= pmin * csum) {
    pi = pmin;
  } else if (design == PAIR_DESIGN_UNIFORM) {
    pi = uni;
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
      // by Illinois false position on a bracket [tlo, thi] with
      // f(tlo) >= 0 >= f(thi); when the same end is replaced twice in a row,
      // the other end's value is halved.  Each evaluation is an inner
      // coordinate descent at lam = e^t, warm-started from the previous
      // iterate; `inner_ok` records whether the last one converged.  Every
      // sweep counts against the prompt's cap.
      double spent = 0.0;
      bool inner_ok = false;
      auto solve_at = [&](double t) -> double {
        const double lam = exp(t);
        inner_ok = false;
        for (int sw = 0; sw < kMaxSweeps && it < cap; ++sw) {
          double change = 0.0;
          for (int i = 0; i < gi; ++i) {
            const double p_i = readlane_d(p, i), m_i = readlane_d(m, i);
            const double a = (vert && lane != i && edges) ? proxy(p_i, p, m_i, m, scaled) : 0.0;
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
          if (wave_max_d(change) <= 1e-13) {
            inner_ok = true;
            break;
          }
        }
        spent = wave_sum_d(vert ? c * pi : 0.0);
        return log(spent) - log(bud);
      };
      auto met = [&]() { return fabs(spent - bud) <= 1e-13 * bud; };
      const double tmin = log(fmin(lam_lo, lam_hi * 0.5)), tmax = log(lam_hi);
      double tlo = tmin, thi = tmax, flo = 0.0, fhi = 0.0;
      bool bracketed = false, done = false;
      double t0 = 0.0;
      bool warm = false;
      if (pi_prev != nullptr) {
        // Warm start: the previous probabilities (clipped to the box; NaN
        // reads as pi_min) and the multiplier their KKT conditions imply,
        // the median over interior vertices of A_i / (c_i pi_i^2).
        pi = vert ? fmin(fmax((double)pi_prev[o0 + lane], pmin), 1.0) : 1.0;
        const double A = a_vec(pi);
        const bool interior = vert && pi > pmin * (1.0 + 1e-7) && pi < 1.0 - 1e-7;
        const double lam0 = wave_median_d(interior ? A / (c * pi * pi) : 0.0, interior, gi, lane);
        if (lam0 > 0.0) {
          warm = true;
          t0 = fmin(fmax(log(lam0), tmin), tmax);
        }
      }
      if (warm) {
        // Bracket the root by steps growing fourfold from t0, each solve
        // warm-started from the last.  d f / d t lies in [-1/2, 0] (an
        // interior pi_i moves as lam^(-1/2)), so the root is at least 2 |f0|
        // away and the first step is 4 |f0|.
        const double f0 = solve_at(t0);
        const double step0 = fmax(4.0 * fabs(f0), 1e-12);
        if (met()) {
          done = true;
        } else if (f0 > 0.0) {
          tlo = t0;
          flo = f0;
          for (double step = step0; it < cap; step *= 4.0) {
            const double t = fmin(tlo + step, tmax);
            const double ft = solve_at(t);
            if (met()) {
              done = true;
              break;
            }
            if (ft <= 0.0) {
              thi = t;
              fhi = ft;
              bracketed = true;
              break;
            }
            tlo = t;
            flo = ft;
            if (t >= tmax) break;
          }
        } else {
          thi = t0;
          fhi = f0;
          for (double step = step0; it < cap; step *= 4.0) {
            const double t = fmax(thi - step, tmin);
            const double ft = solve_at(t);
            if (met()) {
              done = true;
              break;
            }
            if (ft > 0.0) {
              tlo = t;
              flo = ft;
              bracketed = true;
              break;
            }
            thi = t;
            fhi = ft;
            if (t <= tmin) {   // every vertex with contrast at 1: the budget does not bind
              done = true;
              break;
            }
          }
        }
      } else {
        pi = 1.0;
        flo = solve_at(tlo);
        if (flo > 0.0 && !met()) {   // otherwise the budget does not bind
          pi = pmin;
          fhi = solve_at(thi);
          bracketed = fhi < 0.0 && !met();
          done = !bracketed;
        } else {
          done = true;
        }
      }
      if (bracketed) {
        int side = 0;
        for (int k = 0; k < kMaxBisect && it < cap; ++k) {
          double t = (tlo * fhi - thi * flo) / (fhi - flo);
          if (!(t > tlo && t < thi)) t = 0.5 * (tlo + thi);
          const double ft = solve_at(t);
          if (met()) {
            done = true;
            break;
          }
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
          if (thi - tlo <= 1e-15) {   // the multiplier is fixed to rounding
            done = true;
            break;
          }
        }
      }
      // Solver failure (App. C): the cap or a search limit reached before the
      // budget was met, or a last inner solve that did not converge.  The
      // prompt then gets the uniform design with the same expected cost.
      failed = !done || !inner_ok || !isfinite(pi);
      failed = __ballot(failed) != 0ull;
      if (failed) {
        pi = uni;
      } else {
        // The last multiplier may leave the budget overspent by a rounding
        // amount: keep the iterate of the feasible side.
        spent = wave_sum_d(vert ? c * pi : 0.0);
        if (spent > bud) pi = fmax(pmin, pi * (bud / spent));
      }
    }
  }
  if (failed && lane == 0) raise_status(d_status, PAIR_ST_SOLVER);

  if (vert) pi_out[o0 + lane] = (float)pi;
  if (objective != nullptr || iters != nullptr || residual != nullptr) {
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
    // KKT residual of the design's program at the returned (fp32) probabilities
    // x, with the negative gradient g_i = A_i / x_i^2 and one budget
    // multiplier lam: interior vertices need g_i / c_i = lam, vertices at 1
    // need g_i / c_i >= lam, vertices at pi_min need g_i / c_i <= lam, and a
    // positive lam needs the budget spent.  lam is the median of g_i / c_i
    // over the interior vertices; with none, 0 if the budget is slack, else
    // the largest g_i / c_i at pi_min.  Violations are relative to the largest
    // g_i / c_i, the budget's to the budget.
    double res = 0.0;
    if (residual != nullptr) {
      const double x = vert ? (double)(float)pi : 1.0;
      const double ax = a_vec(x);   // wave reductions: every lane takes part
      const double gc = vert ? ax / (x * x) / c : 0.0;
      const double tol = 1e-7;
      const bool interior = vert && x > pmin * (1.0 + tol) && x < 1.0 - tol;
      const bool top = vert && x >= 1.0 - tol;
      const bool bot = vert && x <= pmin * (1.0 + tol);
      const double spent_x = wave_sum_d(vert ? c * x : 0.0);
      double lam;
      if (__ballot(interior) != 0ull)
        lam = wave_median_d(gc, interior, gi, lane);
      else if (spent_x < bud * (1.0 - 1e-9))
        lam = 0.0;
      else
        lam = fmax(wave_max_d(bot ? gc : 0.0), 0.0);
      const double scale = fmax(wave_max_d(vert ? gc : -1e308), 1e-300);
      double r = 0.0;
      if (interior) r = fabs(gc - lam) / scale;
      if (top) r = fmax(r, fmax(lam - gc, 0.0) / scale);
      if (bot) r = fmax(r, fmax(gc - lam, 0.0) / scale);
      res = wave_max_d(r);
      if (lam > 0.0) res = fmax(res, fabs(spent_x - bud) / bud);
      res = fmax(res, fmax(spent_x - bud, 0.0) / bud);
    }
    if (lane == 0) {
      if (objective != nullptr) objective[b] = phi;
      if (iters != nullptr) iters[b] = failed ? -it : it;
      if (residual != nullptr) residual[b] = res;
    }
  }
}

}  // namespace

int launch_alloc(int64_t B, int64_t nv, int32_t gmax, const int64_t* offsets, const float* p_hat,
                 const float* c_hat, const float* m_hat, const float* budget, float pi_min,
                 int32_t design, const float* pi_prev, int32_t max_sweeps, float* pi,
                 double* objective, int32_t* iters, double* residual, int32_t* d_status,
                 hipStream_t stream) {
  const int32_t cap = max_sweeps > 0 ? max_sweeps : kDefaultCap;
  hipLaunchKernelGGL(alloc_kernel, dim3((unsigned)B), dim3(kWave), 0, stream, B, nv, gmax, offsets,
                     p_hat, c_hat, m_hat, budget, pi_min, design, pi_prev, cap, pi, objective,
                     iters, residual, d_status);
  return hipGetLastError() == hipSuccess ? PAIR_OK : PAIR_EHIP;
}

}  // namespace pair
