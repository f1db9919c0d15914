/* Address-sanitizer driver for the C oracle (test infrastructure).
 *
 * Built together with oracle/pair_oracle.c under -fsanitize=address,undefined
 * and run as its own program, so that the sanitizer runtime is the first
 * library loaded.  Every buffer is allocated with exactly the size the
 * oracle's contract gives it (no slack), so any read or write past an end,
 * use of freed memory or leak aborts the run.  The inputs are small ragged
 * batches drawn from a fixed-seed generator: group sizes in [2, 19], score
 * widths off any power of two, padded row strides, fp32 and bf16 scores,
 * every edge-weight rule, and fixed-size designs.  Results are only checked
 * for being finite; the pins check their values.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

int orc_design_inclusion(int64_t, const int64_t*, int32_t, const float*, uint64_t, int64_t,
                         int64_t, const int64_t*, uint8_t*, float*, int32_t*, int32_t*);
int orc_pair_grad(int64_t, const int64_t*, int32_t, int64_t, const void*, int, int64_t,
                  const float*, const uint8_t*, const float*, double*, int32_t*);
int orc_pair_grad_rule(int64_t, const int64_t*, int32_t, int64_t, const void*, int, int64_t,
                       const float*, const uint8_t*, const float*, int, double, double*,
                       int32_t*, double*, double*);
int orc_pair_coeffs(int64_t, const int64_t*, int32_t, const float*, const uint8_t*,
                    const float*, double*, int32_t*);
int orc_pair_coeffs_rule(int64_t, const int64_t*, int32_t, const float*, const uint8_t*,
                         const float*, int, double, double*, int32_t*, double*, double*);
int orc_audit(int64_t, const int64_t*, int32_t, int64_t, const void*, int, int64_t,
              const float*, const float*, const float*, uint64_t, int64_t, int64_t,
              const int64_t*, double*, double*, double*, int32_t*);
int orc_audit_rule(int64_t, const int64_t*, int32_t, int64_t, const void*, int, int64_t,
                   const float*, const float*, const float*, int, double, uint64_t, int64_t,
                   int64_t, const int64_t*, double*, double*, double*, int32_t*, double*,
                   double*);
int orc_audit_exact(int64_t, const int64_t*, int32_t, int64_t, const void*, int, int64_t,
                    const float*, const float*, const float*, int, double, double*, double*);
int orc_cps_inclusion(const double*, int64_t, int64_t, double*, double*);
int orc_cps_fit(const double*, int64_t, int64_t, double, int64_t, double*, int64_t*);
int orc_cps_draw(int64_t, const int64_t*, const double*, const int32_t*, uint64_t, int64_t,
                 int64_t, uint8_t*);

static uint64_t rng_state = 0x9E3779B97F4A7C15ull;
static uint64_t next_u64(void) { /* splitmix64 */
  uint64_t z = (rng_state += 0x9E3779B97F4A7C15ull);
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}
static double unif(void) { return (double)(next_u64() >> 11) * 0x1.0p-53; }
static int64_t irange(int64_t lo, int64_t hi) { return lo + (int64_t)(next_u64() % (uint64_t)(hi - lo + 1)); }

static void* xmalloc(size_t n) {
  void* q = malloc(n ? n : 1);
  if (!q) { fprintf(stderr, "out of memory\n"); exit(2); }
  return q;
}

static int failures = 0;
static void expect(int ok, const char* what, int64_t c) {
  if (!ok) { fprintf(stderr, "FAIL %s (case %lld)\n", what, (long long)c); failures++; }
}
static int all_finite(const double* x, int64_t n) {
  for (int64_t i = 0; i < n; ++i) if (!isfinite(x[i])) return 0;
  return 1;
}

static uint16_t to_bf16(float f) {
  uint32_t u; memcpy(&u, &f, 4);
  return (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}

static void run_case(int64_t c) {
  const int64_t B = irange(1, 6);
  int64_t* off = xmalloc((size_t)(B + 1) * sizeof(int64_t));
  off[0] = 0;
  int32_t gmax = 0;
  for (int64_t b = 0; b < B; ++b) {
    int64_t g = irange(2, 19);
    off[b + 1] = off[b] + g;
    if (g > gmax) gmax = (int32_t)g;
  }
  const int64_t nv = off[B];
  const int64_t D = irange(1, 45);
  const int64_t ld = D + irange(0, 5);
  const int bf16 = (int)(c & 1);
  const int64_t R = irange(1, 9);
  const uint64_t seed = next_u64();
  const int64_t rep0 = irange(0, 1000);

  float* rewards = xmalloc((size_t)nv * sizeof(float));
  float* p = xmalloc((size_t)nv * sizeof(float));
  for (int64_t i = 0; i < nv; ++i) {
    rewards[i] = (c % 3 == 0) ? (float)(next_u64() & 1) : (float)unif();
    p[i] = (i % 5 == 0) ? 1.0f : (float)(0.05 + 0.95 * unif());
  }
  /* Scores: nv rows of ld entries; the padding holds NaN (fp32) or a bf16 NaN. */
  void* scores;
  if (bf16) {
    uint16_t* s = xmalloc((size_t)(nv * ld) * sizeof(uint16_t));
    for (int64_t i = 0; i < nv * ld; ++i)
      s[i] = (i % ld < D) ? to_bf16((float)(2.0 * unif() - 1.0)) : (uint16_t)0x7FC0;
    scores = s;
  } else {
    float* s = xmalloc((size_t)(nv * ld) * sizeof(float));
    for (int64_t i = 0; i < nv * ld; ++i) s[i] = (i % ld < D) ? (float)(2.0 * unif() - 1.0) : NAN;
    scores = s;
  }
  int64_t* pid = xmalloc((size_t)B * sizeof(int64_t));
  for (int64_t b = 0; b < B; ++b) pid[b] = irange(0, 100000);

  /* Design draw. */
  uint8_t* mask = xmalloc((size_t)(R * nv));
  float* pi = xmalloc((size_t)(B * gmax * gmax) * sizeof(float));
  int32_t* ec = xmalloc((size_t)(R * B) * sizeof(int32_t));
  int32_t* comp = xmalloc((size_t)(R * B) * sizeof(int32_t));
  expect(orc_design_inclusion(B, off, gmax, p, seed, rep0, R, (c & 2) ? pid : NULL, mask, pi,
                              ec, comp) == 0, "design_inclusion", c);

  /* Estimator and fold on the first replicate's mask. */
  double* out = xmalloc((size_t)(B * D) * sizeof(double));
  double* coeff = xmalloc((size_t)nv * sizeof(double));
  int32_t* ecb = xmalloc((size_t)B * sizeof(int32_t));
  double* ess = xmalloc((size_t)B * sizeof(double));
  double* mw = xmalloc((size_t)B * sizeof(double));
  expect(orc_pair_grad(B, off, gmax, D, scores, bf16, ld, rewards, mask, pi, out, ecb) == 0,
         "pair_grad", c);
  expect(all_finite(out, B * D), "pair_grad finite", c);
  expect(orc_pair_coeffs(B, off, gmax, rewards, mask, pi, coeff, ecb) == 0, "pair_coeffs", c);
  expect(all_finite(coeff, nv), "pair_coeffs finite", c);
  expect(orc_pair_grad(B, off, gmax, D, scores, bf16, ld, rewards, NULL, NULL, out, ecb) == 0,
         "pair_grad complete", c);
  for (int rule = 0; rule <= 5; ++rule) {
    const double wmax = 1.0 + 4.0 * unif();
    expect(orc_pair_grad_rule(B, off, gmax, D, scores, bf16, ld, rewards, mask, pi, rule, wmax,
                              out, ecb, ess, mw) == 0, "pair_grad_rule", c);
    expect(all_finite(out, B * D), "pair_grad_rule finite", c);
    expect(orc_pair_coeffs_rule(B, off, gmax, rewards, mask, pi, rule, wmax, coeff, ecb, ess,
                                mw) == 0, "pair_coeffs_rule", c);
  }

  /* Monte-Carlo audit (with and without the per-replicate outputs) and the exact audit. */
  double* mse = xmalloc((size_t)B * sizeof(double));
  double* bias = xmalloc((size_t)B * sizeof(double));
  double* reps = xmalloc((size_t)(B * R) * sizeof(double));
  int32_t* rec = xmalloc((size_t)(B * R) * sizeof(int32_t));
  const float* pi_w = (c & 4) ? pi : NULL;
  expect(orc_audit(B, off, gmax, D, scores, bf16, ld, rewards, p, pi_w, seed, rep0, R,
                   (c & 2) ? pid : NULL, mse, bias, reps, rec) == 0, "audit", c);
  expect(all_finite(mse, B) && all_finite(bias, B) && all_finite(reps, B * R), "audit finite", c);
  for (int rule = 0; rule <= 5; ++rule) {
    double* cosv = xmalloc((size_t)B * sizeof(double));
    double* tnorm = xmalloc((size_t)B * sizeof(double));
    int rc = orc_audit_rule(B, off, gmax, D, scores, bf16, ld, rewards, p, pi_w, rule, 2.0, seed,
                            rep0, R, NULL, mse, bias, NULL, NULL, cosv, tnorm);
    if (rc == 0) {
      expect(all_finite(cosv, B) && all_finite(tnorm, B), "audit cosine finite", c);
      for (int64_t b = 0; b < B; ++b) expect(fabs(cosv[b]) <= 1.0 + 1e-12, "cosine in [-1, 1]", c);
    }
    free(cosv);
    free(tnorm);
    expect(rc == 0, "audit_rule", c);
    rc = orc_audit_exact(B, off, gmax, D, scores, bf16, ld, rewards, p, pi_w, rule, 2.0, mse, bias);
    expect(rc == 0 || rc == -1, "audit_exact", c);
    if (rc == 0) expect(all_finite(mse, B) && all_finite(bias, B), "audit_exact finite", c);
  }

  /* Fixed-size (conditional Poisson) design on each prompt's group. */
  double* w = xmalloc((size_t)nv * sizeof(double));
  int32_t* n = xmalloc((size_t)B * sizeof(int32_t));
  for (int64_t b = 0; b < B; ++b) {
    const int64_t g = off[b + 1] - off[b];
    const int64_t nb = irange(1, g - 1);
    n[b] = (int32_t)nb;
    double* target = xmalloc((size_t)g * sizeof(double));
    double* pib = xmalloc((size_t)g * sizeof(double));
    double* pij = xmalloc((size_t)(g * g) * sizeof(double));
    double tsum = 0.0;
    for (int64_t i = 0; i < g; ++i) { target[i] = 0.5 + unif(); tsum += target[i]; }
    for (int64_t i = 0; i < g; ++i) target[i] *= (double)nb / tsum;
    int ok = 1;
    for (int64_t i = 0; i < g; ++i) ok &= target[i] < 1.0;
    int64_t iters = 0;
    if (ok) {
      expect(orc_cps_fit(target, g, nb, 1e-10, 10000, w + off[b], &iters) == 0, "cps_fit", c);
    } else {
      for (int64_t i = 0; i < g; ++i) w[off[b] + i] = 0.5 + unif();
    }
    expect(orc_cps_inclusion(w + off[b], g, nb, pib, pij) == 0, "cps_inclusion", c);
    expect(all_finite(pib, g) && all_finite(pij, g * g), "cps_inclusion finite", c);
    free(target); free(pib); free(pij);
  }
  expect(orc_cps_draw(B, off, w, n, seed, rep0, R, mask) == 0, "cps_draw", c);

  free(w); free(n); free(mse); free(bias); free(reps); free(rec);
  free(out); free(coeff); free(ecb); free(ess); free(mw);
  free(mask); free(pi); free(ec); free(comp); free(pid);
  free(scores); free(rewards); free(p); free(off);
}

int main(int argc, char** argv) {
  const int64_t cases = argc > 1 ? atoll(argv[1]) : 40;
  for (int64_t c = 0; c < cases; ++c) run_case(c);
  if (failures) { fprintf(stderr, "%d failures\n", failures); return 1; }
  printf("oracle sanitizer driver: %lld cases clean\n", (long long)cases);
  return 0;
}
