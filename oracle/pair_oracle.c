/*
 * pair_oracle.c -- plain, slow, obviously correct CPU reference for the PAIR
 * pair-inclusion-weighted gradient estimator and its frozen-population audit.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path may call, link or
 * load this file; only the test-suite, the smoke check and the bench's CPU
 * baseline leg use it.  It shares no code, header, table or constant with the
 * HIP library: everything below is written from the paper's definitions.
 *
 * Arithmetic is IEEE fp64, built with -ffp-contract=off and without fast-math.
 * Inputs are the exact fp32 / bf16 values the GPU sees, widened exactly.
 *
 * Paper sections followed:
 *   - Sec. 3.1, Eq. (loo)            leave-one-out gradient (used only by pins)
 *   - Sec. 3.2, Eq. (pair-kernel)    h_ij = 1/2 (r_i - r_j)(s_i - s_j)
 *   - Sec. 3.2, Eq. (pair-average)   complete-pair average, M = C(G,2)
 *   - Sec. 3.3                       adaptive continuation: J_i, I_ij = J_i J_j,
 *                                    rho_ij = P(J_i J_j = 1), independent
 *                                    Bernoulli => rho_ij = pi_i pi_j, logged
 *   - Sec. 4.5, Eq. (pair-ht)        induced-edge Horvitz-Thompson estimator
 *   - Sec. 4.5, Eq. (pair-advantage) sequence advantages A~_i
 *   - Algorithm 1 (pair-corrected update): every observed edge adds its
 *                                    1/rho-weighted term to both endpoints
 *   - App. B "At least two completed vertices": a draw with fewer than two
 *                                    completed vertices contributes zero
 *   - Sec. 6.2 frozen-policy audit and App. D metrics: MSE = E||g^ - g_full||^2,
 *                                    bias = || mean_r g^_r - g_full ||,
 *                                    ESS = (sum_e w_e)^2 / sum_e w_e^2
 *   - App. A "Naive selection bias" and App. B "Estimated and stabilized
 *     propensities": the estimator variants of Tables 4 and 5 (edge-weight
 *     rules, below)
 *   - Prop. 1 and App. A "Design covariance": the exact design bias and
 *     covariance trace of a linear rule (orc_audit_exact)
 *   - App. B "Fixed-size and exact-cost designs": conditional Poisson
 *     sampling of a fixed number of endpoints (Hajek 1964) with its exact,
 *     non-factorising joint inclusion probabilities (orc_cps_*)
 *
 * Random design draws.  The paper only requires fresh randomisation for the
 * continuation indicators.  This oracle fixes one counter-based generator, the
 * published Philox4x64 with 10 rounds (Salmon, Moraes, Dror, Shaw, "Parallel
 * random numbers: as easy as 1, 2, 3", SC'11), and the reading:
 *   key     = (seed, 0)
 *   counter = (replicate r, prompt id b, i >> 2, 0)
 *   u_i     = top 32 bits of output word (i & 3)
 *   J_i     = [ u_i < floor(p_i * 2^32) ]     (p_i >= 1 always includes)
 * so that P(J_i = 1) = floor(p_i 2^32) / 2^32, which equals p_i exactly for
 * every fp32 p_i >= 2^-9.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORC_OK 0
#define ORC_EINVAL (-1)   /* malformed sizes / offsets / pointers            */
#define ORC_EDTYPE (-2)   /* unknown score dtype                              */
#define ORC_ERHO (-3)     /* observed edge with rho outside (0, 1]            */
#define ORC_EP (-4)       /* continuation probability outside (0, 1]          */
#define ORC_EGROUP (-5)   /* a prompt with fewer than two candidates          */

#define ORC_F32 0
#define ORC_BF16 1

/* Edge-weight rules.  Every rule estimates
 *     g = (1/N) sum_{i<j observed} 1/2 (r_i - r_j) (w_i s_i - w_j s_j)
 * with the weights (w_i, w_j) on the two halves of the edge term h_ij and the
 * normaliser N:
 *   HT          w_i = w_j = 1/rho_ij,              N = M = C(G, 2)   Eq. (pair-ht)
 *   UNWEIGHTED  w_i = w_j = 1,                     N = M             (naive, g~_0)
 *   RATIO_KE    w_i = w_j = 1,                     N = K_E           (observed-edge mean)
 *   CLIPPED     w_i = w_j = min(1/rho_ij, w_max),  N = M
 *   SELFNORM    w_i = w_j = 1/rho_ij,              N = sum_e I_e / rho_e   (Hajek)
 *   MARGINAL    w_i = 1/pi_i, w_j = 1/pi_j,        N = M   (per-rollout propensity only;
 *               pi_i is the diagonal of the logged block)
 * A draw with no observed edge gives the zero vector under every rule.  The
 * edge weight entering ESS and the maximum weight is w_i = w_j for the
 * symmetric rules and (w_i + w_j) / 2 for MARGINAL. */
#define ORC_RULE_HT 0
#define ORC_RULE_UNWEIGHTED 1
#define ORC_RULE_RATIO_KE 2
#define ORC_RULE_CLIPPED 3
#define ORC_RULE_SELFNORM 4
#define ORC_RULE_MARGINAL 5

/* ------------------------------------------------------------------------ */
/* Philox4x64-10, written from the SC'11 description: each round multiplies  */
/* words 0 and 2 by the two round multipliers, takes the 128-bit products'   */
/* high and low halves, and xors the high halves with the other two words    */
/* and the key; the key is bumped by the two Weyl constants between rounds.  */
/* ------------------------------------------------------------------------ */
static void mul64_full(uint64_t a, uint64_t b, uint64_t* hi, uint64_t* lo) {
    unsigned __int128 prod = (unsigned __int128)a * (unsigned __int128)b;
    *hi = (uint64_t)(prod >> 64);
    *lo = (uint64_t)prod;
}

void orc_philox4x64_10(const uint64_t ctr_in[4], const uint64_t key_in[2], uint64_t out[4]) {
    const uint64_t mult0 = 0xD2E7470EE14C6C93ULL, mult1 = 0xCA5A826395121157ULL;
    const uint64_t weyl0 = 0x9E3779B97F4A7C15ULL, weyl1 = 0xBB67AE8584CAA73BULL;
    uint64_t x0 = ctr_in[0], x1 = ctr_in[1], x2 = ctr_in[2], x3 = ctr_in[3];
    uint64_t k0 = key_in[0], k1 = key_in[1];
    for (int round = 0; round < 10; ++round) {
        if (round > 0) {
            k0 += weyl0;
            k1 += weyl1;
        }
        uint64_t hi0, lo0, hi1, lo1;
        mul64_full(mult0, x0, &hi0, &lo0);
        mul64_full(mult1, x2, &hi1, &lo1);
        uint64_t y0 = hi1 ^ x1 ^ k0;
        uint64_t y1 = lo1;
        uint64_t y2 = hi0 ^ x3 ^ k1;
        uint64_t y3 = lo0;
        x0 = y0; x1 = y1; x2 = y2; x3 = y3;
    }
    out[0] = x0; out[1] = x1; out[2] = x2; out[3] = x3;
}

/* Continuation indicator J_i for vertex i of prompt id b in replicate r. */
int orc_draw_indicator(uint64_t seed, int64_t r, int64_t b, int64_t i, float p) {
    uint64_t ctr[4] = {(uint64_t)r, (uint64_t)b, (uint64_t)(i >> 2), 0};
    uint64_t key[2] = {seed, 0};
    uint64_t w[4];
    orc_philox4x64_10(ctr, key, w);
    uint64_t u = w[i & 3] >> 32;
    if (p >= 1.0f) return 1;
    uint64_t thr = (uint64_t)ldexp((double)p, 32); /* exact: p*2^32 < 2^32 */
    return u < thr ? 1 : 0;
}

/* Score element s[v][d] widened exactly to fp64. */
static double score_at(const void* scores, int dtype, int64_t ld, int64_t v, int64_t d) {
    if (dtype == ORC_F32) {
        return (double)((const float*)scores)[v * ld + d];
    }
    uint16_t h = ((const uint16_t*)scores)[v * ld + d];
    uint32_t bits = ((uint32_t)h) << 16; /* bf16 is the top half of an fp32 */
    float f;
    memcpy(&f, &bits, sizeof f);
    return (double)f;
}

static int check_offsets(int64_t B, const int64_t* offsets, int32_t gmax) {
    if (B < 1 || offsets == NULL || offsets[0] != 0) return ORC_EINVAL;
    for (int64_t b = 0; b < B; ++b) {
        int64_t g = offsets[b + 1] - offsets[b];
        if (g < 2) return ORC_EGROUP;
        if (gmax > 0 && g > gmax) return ORC_EINVAL;
    }
    return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* Design draw (Sec. 3.3): independent Bernoulli continuation with logged    */
/* joint inclusion probabilities rho_ij = pi_i pi_j.                         */
/*   mask[r][v]        J for vertex v in replicate rep0 + r                  */
/*   pi[b][i][j]       fp32 rho_ij (i != j), pi_i on the diagonal, 0 beyond  */
/*                     G_b; rounded once from the exact fp64 product         */
/*   edge_count[r][b]  K_E = number of i < j with J_i = J_j = 1 (brute force) */
/*   completed[r][b]   number of completed vertices                          */
/* prompt_id: RNG prompt index of each prompt (NULL => 0..B-1).              */
/* ------------------------------------------------------------------------ */
int orc_design_inclusion(int64_t B, const int64_t* offsets, int32_t gmax, const float* p,
                         uint64_t seed, int64_t rep0, int64_t R, const int64_t* prompt_id,
                         uint8_t* mask, float* pi, int32_t* edge_count, int32_t* completed) {
    int st = check_offsets(B, offsets, gmax);
    if (st) return st;
    if (R < 0 || p == NULL) return ORC_EINVAL;
    int64_t nv = offsets[B];
    for (int64_t v = 0; v < nv; ++v)
        if (!(p[v] > 0.0f && p[v] <= 1.0f)) return ORC_EP;

    if (pi != NULL) {
        for (int64_t b = 0; b < B; ++b) {
            int64_t o = offsets[b], g = offsets[b + 1] - offsets[b];
            float* blk = pi + b * (int64_t)gmax * gmax;
            for (int64_t i = 0; i < gmax; ++i)
                for (int64_t j = 0; j < gmax; ++j) {
                    float val = 0.0f;
                    if (i < g && j < g) {
                        if (i == j)
                            val = p[o + i];
                        else
                            val = (float)((double)p[o + i] * (double)p[o + j]);
                    }
                    blk[i * gmax + j] = val;
                }
        }
    }
    int64_t gcap = 0;
    for (int64_t b = 0; b < B; ++b)
        if (offsets[b + 1] - offsets[b] > gcap) gcap = offsets[b + 1] - offsets[b];
    int* J = (int*)malloc((size_t)gcap * sizeof(int));
    if (J == NULL) return ORC_EINVAL;
    for (int64_t r = 0; r < R; ++r) {
        for (int64_t b = 0; b < B; ++b) {
            int64_t o = offsets[b], g = offsets[b + 1] - offsets[b];
            int64_t bid = prompt_id ? prompt_id[b] : b;
            int32_t k = 0, ke = 0;
            for (int64_t i = 0; i < g; ++i) {
                J[i] = orc_draw_indicator(seed, rep0 + r, bid, i, p[o + i]);
                if (mask) mask[r * nv + o + i] = (uint8_t)J[i];
                k += J[i];
            }
            for (int64_t i = 0; i < g; ++i) /* brute-force count of induced edges */
                for (int64_t j = i + 1; j < g; ++j)
                    if (J[i] && J[j]) ++ke;
            if (edge_count) edge_count[r * B + b] = ke;
            if (completed) completed[r * B + b] = k;
        }
    }
    free(J);
    return ORC_OK;
}

/* rho_ij read from the upper triangle of one prompt's dense gmax x gmax block. */
static double rho_of(const float* blk, int32_t gmax, int64_t i, int64_t j) {
    int64_t lo = i < j ? i : j, hi = i < j ? j : i;
    return (double)blk[lo * gmax + hi];
}

/* Weights of the two halves of observed edge (i, j) under `rule` (see the
 * rule table above), and the edge's share 1/rho_ij of the self-normalised
 * denominator.  blk == NULL means rho == pi == 1. */
static int edge_weights(int rule, double wmax, const float* blk, int32_t gmax, int64_t i,
                        int64_t j, double* wi, double* wj, double* inv_rho) {
    double rho = blk ? rho_of(blk, gmax, i, j) : 1.0;
    *inv_rho = 0.0;
    if (rule == ORC_RULE_HT || rule == ORC_RULE_CLIPPED || rule == ORC_RULE_SELFNORM) {
        if (!(rho > 0.0 && rho <= 1.0)) return ORC_ERHO;
        double w = 1.0 / rho;
        if (rule == ORC_RULE_CLIPPED && w > wmax) w = wmax;
        *wi = *wj = w;
        *inv_rho = 1.0 / rho;
    } else if (rule == ORC_RULE_MARGINAL) {
        double pii = blk ? (double)blk[i * gmax + i] : 1.0;
        double pjj = blk ? (double)blk[j * gmax + j] : 1.0;
        if (!(pii > 0.0 && pii <= 1.0 && pjj > 0.0 && pjj <= 1.0)) return ORC_ERHO;
        *wi = 1.0 / pii;
        *wj = 1.0 / pjj;
    } else if (rule == ORC_RULE_UNWEIGHTED || rule == ORC_RULE_RATIO_KE) {
        *wi = *wj = 1.0;
    } else {
        return ORC_EINVAL;
    }
    return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* One prompt's estimate under `rule`, columns [0, D), by explicit edges:    */
/*   g = (1/N) sum_{i<j, J_i J_j = 1} 1/2 (r_i - r_j)(w_i s_i - w_j s_j);     */
/* for the HT rule this is Eq. (pair-ht) with the edge kernel h_ij of        */
/* Eq. (pair-kernel).  mask == NULL means every vertex completed; blk ==     */
/* NULL means rho == 1 (with both: the complete-pair average, Eq.            */
/* (pair-average)).  Optional: K_E, ESS and the largest edge weight.         */
/* ------------------------------------------------------------------------ */
static int rule_estimate_one(int64_t o, int64_t g, int64_t D, const void* scores, int dtype,
                             int64_t ld, const float* rewards, const uint8_t* mask,
                             const float* blk, int32_t gmax, int rule, double wmax, double* out,
                             int32_t* edges, double* ess, double* maxw) {
    const double M = (double)g * (double)(g - 1) / 2.0;
    int32_t ke = 0;
    double nsn = 0.0, sw = 0.0, sw2 = 0.0, wmx = 0.0;
    for (int64_t d = 0; d < D; ++d) out[d] = 0.0;
    for (int64_t i = 0; i < g; ++i) {
        for (int64_t j = i + 1; j < g; ++j) {
            int Ji = mask ? mask[o + i] != 0 : 1;
            int Jj = mask ? mask[o + j] != 0 : 1;
            if (!(Ji && Jj)) continue; /* I_ij = 0: the edge is not observed */
            ++ke;
            double wi, wj, ir;
            int st = edge_weights(rule, wmax, blk, gmax, i, j, &wi, &wj, &ir);
            if (st) return st;
            nsn += ir;
            double we = 0.5 * (wi + wj);
            sw += we;
            sw2 += we * we;
            if (we > wmx) wmx = we;
            double ri = (double)rewards[o + i], rj = (double)rewards[o + j];
            for (int64_t d = 0; d < D; ++d) {
                double si = score_at(scores, dtype, ld, o + i, d);
                double sj = score_at(scores, dtype, ld, o + j, d);
                out[d] += 0.5 * (ri - rj) * (wi * si - wj * sj);
            }
        }
    }
    double N = M;
    if (rule == ORC_RULE_RATIO_KE) N = (double)ke;
    if (rule == ORC_RULE_SELFNORM) N = nsn;
    for (int64_t d = 0; d < D; ++d) out[d] = ke > 0 ? out[d] / N : 0.0;
    if (edges) *edges = ke;
    if (ess) *ess = ke > 0 ? sw * sw / sw2 : 0.0;
    if (maxw) *maxw = wmx;
    return ORC_OK;
}

static int ht_estimate_one(int64_t o, int64_t g, int64_t D, const void* scores, int dtype,
                           int64_t ld, const float* rewards, const uint8_t* mask,
                           const float* rho_blk, int32_t gmax, double* out, int32_t* edges) {
    return rule_estimate_one(o, g, D, scores, dtype, ld, rewards, mask, rho_blk, gmax,
                             ORC_RULE_HT, 0.0, out, edges, NULL, NULL);
}

static int check_rule(int rule, double wmax) {
    if (rule < ORC_RULE_HT || rule > ORC_RULE_MARGINAL) return ORC_EINVAL;
    if (rule == ORC_RULE_CLIPPED && !(wmax > 0.0 && wmax < INFINITY)) return ORC_EINVAL;
    return ORC_OK;
}

/* Batched estimate under `rule`: out[b][d] for every prompt; optional
 * edge_count[b] = K_E, ess[b], max_weight[b]. */
int orc_pair_grad_rule(int64_t B, const int64_t* offsets, int32_t gmax, int64_t D,
                       const void* scores, int dtype, int64_t ld, const float* rewards,
                       const uint8_t* mask, const float* pi, int rule, double wmax, double* out,
                       int32_t* edge_count, double* ess, double* max_weight) {
    int st = check_offsets(B, offsets, gmax);
    if (st) return st;
    st = check_rule(rule, wmax);
    if (st) return st;
    if (dtype != ORC_F32 && dtype != ORC_BF16) return ORC_EDTYPE;
    if (D < 0 || ld < D || scores == NULL || rewards == NULL || out == NULL) return ORC_EINVAL;
    int err = ORC_OK;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t b = 0; b < B; ++b) {
        int64_t o = offsets[b], g = offsets[b + 1] - offsets[b];
        const float* blk = pi ? pi + b * (int64_t)gmax * gmax : NULL;
        int s = rule_estimate_one(o, g, D, scores, dtype, ld, rewards, mask, blk, gmax, rule, wmax,
                                  out + b * D, edge_count ? edge_count + b : NULL,
                                  ess ? ess + b : NULL, max_weight ? max_weight + b : NULL);
        if (s) {
#pragma omp critical
            err = s;
        }
    }
    return err;
}

/* Batched Eq. (pair-ht): out[b][d] for every prompt; edge_count[b] = K_E. */
int orc_pair_grad(int64_t B, const int64_t* offsets, int32_t gmax, int64_t D, const void* scores,
                  int dtype, int64_t ld, const float* rewards, const uint8_t* mask, const float* pi,
                  double* out, int32_t* edge_count) {
    return orc_pair_grad_rule(B, offsets, gmax, D, scores, dtype, ld, rewards, mask, pi,
                              ORC_RULE_HT, 0.0, out, edge_count, NULL, NULL);
}

/* ------------------------------------------------------------------------ */
/* Sequence advantages, Eq. (pair-advantage), in the order of Algorithm 1:   */
/* for every observed edge (i, j), i < j, the edge term puts                 */
/* w_i (r_i - r_j) / 2 on s_i and -w_j (r_i - r_j) / 2 on s_j; divide by N.  */
/* For the HT rule w = 1/rho and N = M.  No centring: in exact arithmetic    */
/* the symmetric rules sum to zero already.                                  */
/* ------------------------------------------------------------------------ */
int orc_pair_coeffs_rule(int64_t B, const int64_t* offsets, int32_t gmax, const float* rewards,
                         const uint8_t* mask, const float* pi, int rule, double wmax,
                         double* coeff, int32_t* edge_count, double* ess, double* max_weight) {
    int st = check_offsets(B, offsets, gmax);
    if (st) return st;
    st = check_rule(rule, wmax);
    if (st) return st;
    if (rewards == NULL || coeff == NULL) return ORC_EINVAL;
    for (int64_t b = 0; b < B; ++b) {
        int64_t o = offsets[b], g = offsets[b + 1] - offsets[b];
        const float* blk = pi ? pi + b * (int64_t)gmax * gmax : NULL;
        double M = (double)g * (double)(g - 1) / 2.0;
        int32_t ke = 0;
        double nsn = 0.0, sw = 0.0, sw2 = 0.0, wmx = 0.0;
        for (int64_t i = 0; i < g; ++i) coeff[o + i] = 0.0;
        for (int64_t i = 0; i < g; ++i) {
            for (int64_t j = i + 1; j < g; ++j) {
                int Ji = mask ? mask[o + i] != 0 : 1;
                int Jj = mask ? mask[o + j] != 0 : 1;
                if (!(Ji && Jj)) continue;
                ++ke;
                double wi, wj, ir;
                st = edge_weights(rule, wmax, blk, gmax, i, j, &wi, &wj, &ir);
                if (st) return st;
                nsn += ir;
                double we = 0.5 * (wi + wj);
                sw += we;
                sw2 += we * we;
                if (we > wmx) wmx = we;
                double dr = (double)rewards[o + i] - (double)rewards[o + j];
                coeff[o + i] += 0.5 * dr * wi;
                coeff[o + j] -= 0.5 * dr * wj;
            }
        }
        double N = M;
        if (rule == ORC_RULE_RATIO_KE) N = (double)ke;
        if (rule == ORC_RULE_SELFNORM) N = nsn;
        for (int64_t i = 0; i < g; ++i) coeff[o + i] = ke > 0 ? coeff[o + i] / N : 0.0;
        if (edge_count) edge_count[b] = ke;
        if (ess) ess[b] = ke > 0 ? sw * sw / sw2 : 0.0;
        if (max_weight) max_weight[b] = wmx;
    }
    return ORC_OK;
}

int orc_pair_coeffs(int64_t B, const int64_t* offsets, int32_t gmax, const float* rewards,
                    const uint8_t* mask, const float* pi, double* coeff, int32_t* edge_count) {
    return orc_pair_coeffs_rule(B, offsets, gmax, rewards, mask, pi, ORC_RULE_HT, 0.0, coeff,
                                edge_count, NULL, NULL);
}

/* ------------------------------------------------------------------------ */
/* Frozen-population audit (Sec. 6.2, App. D).  For each prompt:             */
/*   target  t   = complete-pair average, Eq. (pair-average)                 */
/*   for r in [rep0, rep0 + R): draw J^(r) as orc_design_inclusion does,     */
/*       g_r = the estimate under `rule` (Eq. (pair-ht) for the HT rule),    */
/*       rho = pi_w[b][i][j] when pi_w is given, otherwise the logged        */
/*       fl32(p_i p_j) with p_i on the diagonal;                             */
/*       e_r = || g_r - t ||^2                                               */
/*   mse  = (1/R) sum_r e_r ;  bias = || (1/R) sum_r g_r - t ||              */
/* rep_sqerr[b][R] and edge_count[b][R] are optional per-replicate outputs. */
/* Update direction (Sec. 6.2 and the audit matrix of App. E: the cosine    */
/* between an estimate and the target): cos_r = <g_r, t> / (|g_r| |t|),     */
/* taken as 0 when either vector is zero (a draw with no observed edge, or  */
/* a prompt whose target vanishes); cosine[b] = (1/R) sum_r cos_r and       */
/* target_norm[b] = |t| are optional outputs.                               */
/* ------------------------------------------------------------------------ */
int orc_audit_rule(int64_t B, const int64_t* offsets, int32_t gmax, int64_t D,
                   const void* scores, int dtype, int64_t ld, const float* rewards,
                   const float* p, const float* pi_w, int rule, double wmax, uint64_t seed,
                   int64_t rep0, int64_t R, const int64_t* prompt_id, double* mse,
                   double* bias_norm, double* rep_sqerr, int32_t* edge_count, double* cosine,
                   double* target_norm) {
    int st = check_offsets(B, offsets, gmax);
    if (st) return st;
    st = check_rule(rule, wmax);
    if (st) return st;
    if (dtype != ORC_F32 && dtype != ORC_BF16) return ORC_EDTYPE;
    if (D < 1 || ld < D || R < 1 || scores == NULL || rewards == NULL || p == NULL) return ORC_EINVAL;
    int64_t nv = offsets[B];
    for (int64_t v = 0; v < nv; ++v)
        if (!(p[v] > 0.0f && p[v] <= 1.0f)) return ORC_EP;
    int err = ORC_OK;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t b = 0; b < B; ++b) {
        int64_t o = offsets[b], g = offsets[b + 1] - offsets[b];
        int64_t bid = prompt_id ? prompt_id[b] : b;
        double* t = (double*)calloc((size_t)D, sizeof(double));
        double* gr = (double*)calloc((size_t)D, sizeof(double));
        double* gsum = (double*)calloc((size_t)D, sizeof(double));
        uint8_t* m = (uint8_t*)calloc((size_t)nv, 1);
        float* own = (float*)calloc((size_t)gmax * gmax, sizeof(float));
        int s = ORC_OK;
        if (!t || !gr || !gsum || !m || !own) s = ORC_EINVAL;
        /* weights' rho: the caller's block, or the logged fl32(p_i p_j) */
        const float* blk = own;
        if (pi_w) {
            blk = pi_w + b * (int64_t)gmax * gmax;
        } else {
            for (int64_t i = 0; s == ORC_OK && i < g; ++i)
                for (int64_t j = 0; j < g; ++j)
                    own[i * gmax + j] =
                        i != j ? (float)((double)p[o + i] * (double)p[o + j]) : p[o + i];
        }
        if (s == ORC_OK)
            s = ht_estimate_one(o, g, D, scores, dtype, ld, rewards, NULL, NULL, gmax, t, NULL);
        double tt = 0.0;
        for (int64_t d = 0; s == ORC_OK && d < D; ++d) tt += t[d] * t[d];
        double esum = 0.0, csum = 0.0;
        for (int64_t r = 0; s == ORC_OK && r < R; ++r) {
            for (int64_t i = 0; i < g; ++i)
                m[o + i] = (uint8_t)orc_draw_indicator(seed, rep0 + r, bid, i, p[o + i]);
            int32_t ke = 0;
            s = rule_estimate_one(o, g, D, scores, dtype, ld, rewards, m, blk, gmax, rule, wmax, gr,
                                  &ke, NULL, NULL);
            if (s) break;
            double e = 0.0, gt = 0.0, gg = 0.0;
            for (int64_t d = 0; d < D; ++d) {
                double dev = gr[d] - t[d];
                e += dev * dev;
                gsum[d] += gr[d];
                gt += gr[d] * t[d];
                gg += gr[d] * gr[d];
            }
            esum += e;
            if (gg > 0.0 && tt > 0.0) csum += gt / (sqrt(gg) * sqrt(tt));
            if (rep_sqerr) rep_sqerr[b * R + r] = e;
            if (edge_count) edge_count[b * R + r] = ke;
        }
        if (s == ORC_OK) {
            double bb = 0.0;
            for (int64_t d = 0; d < D; ++d) {
                double dev = gsum[d] / (double)R - t[d];
                bb += dev * dev;
            }
            if (mse) mse[b] = esum / (double)R;
            if (bias_norm) bias_norm[b] = sqrt(bb);
            if (cosine) cosine[b] = csum / (double)R;
            if (target_norm) target_norm[b] = sqrt(tt);
        } else {
#pragma omp critical
            err = s;
        }
        free(t); free(gr); free(gsum); free(m); free(own);
    }
    return err;
}

int orc_audit(int64_t B, const int64_t* offsets, int32_t gmax, int64_t D, const void* scores,
              int dtype, int64_t ld, const float* rewards, const float* p, const float* pi_w,
              uint64_t seed, int64_t rep0, int64_t R, const int64_t* prompt_id, double* mse,
              double* bias_norm, double* rep_sqerr, int32_t* edge_count) {
    return orc_audit_rule(B, offsets, gmax, D, scores, dtype, ld, rewards, p, pi_w, ORC_RULE_HT,
                          0.0, seed, rep0, R, prompt_id, mse, bias_norm, rep_sqerr, edge_count,
                          NULL, NULL);
}

/* ------------------------------------------------------------------------ */
/* Exact design audit (Prop. 1 and App. A "Design covariance"), no draws.    */
/* For a rule that is linear in the edge indicators (HT, UNWEIGHTED,         */
/* CLIPPED, MARGINAL), g^ = (1/M) sum_e I_e v_e with the edge vectors        */
/*     v_ij = 1/2 (r_i - r_j) (w_i s_i - w_j s_j)                            */
/* (weights from the logged rho: pi_w when given, else fl32(p_i p_j), p_i    */
/* on the diagonal).  Under the true design, independent Bernoulli(p_i)      */
/* vertices with rho_e = p_i p_j (exact fp64 products):                      */
/*     E g^ = (1/M) sum_e rho_e v_e,   bias = || E g^ - t ||,                */
/*     tr Cov g^ = (1/M^2) [ sum_e rho_e (1 - rho_e) ||v_e||^2               */
/*        + sum_i sum_{j != k, both != i} p_i p_j p_k (1 - p_i) <v_ij, v_ik> ]*/
/* (the shared-vertex covariance of I_ij and I_ik, over ordered pairs), and  */
/*     mse = bias^2 + tr Cov = E || g^ - t ||^2,                             */
/* with t the complete-pair average.  Every vector is formed explicitly.     */
/* ------------------------------------------------------------------------ */
int orc_audit_exact(int64_t B, const int64_t* offsets, int32_t gmax, int64_t D,
                    const void* scores, int dtype, int64_t ld, const float* rewards,
                    const float* p, const float* pi_w, int rule, double wmax, double* mse,
                    double* bias_norm) {
    int st = check_offsets(B, offsets, gmax);
    if (st) return st;
    st = check_rule(rule, wmax);
    if (st) return st;
    if (rule == ORC_RULE_RATIO_KE || rule == ORC_RULE_SELFNORM) return ORC_EINVAL;
    if (dtype != ORC_F32 && dtype != ORC_BF16) return ORC_EDTYPE;
    if (D < 1 || ld < D || scores == NULL || rewards == NULL || p == NULL) return ORC_EINVAL;
    if (gmax < 2) return ORC_EINVAL;
    int64_t nv = offsets[B];
    for (int64_t v = 0; v < nv; ++v)
        if (!(p[v] > 0.0f && p[v] <= 1.0f)) return ORC_EP;
    int err = ORC_OK;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t b = 0; b < B; ++b) {
        int64_t o = offsets[b], g = offsets[b + 1] - offsets[b];
        double M = (double)g * (double)(g - 1) / 2.0;
        double* v = (double*)calloc((size_t)(g * g * D), sizeof(double)); /* v[(i*g+j)*D] */
        double* t = (double*)calloc((size_t)D, sizeof(double));
        double* mu = (double*)calloc((size_t)D, sizeof(double));
        float* own = (float*)calloc((size_t)gmax * gmax, sizeof(float));
        int s = (v && t && mu && own) ? ORC_OK : ORC_EINVAL;
        const float* blk = own;
        if (pi_w) {
            blk = pi_w + b * (int64_t)gmax * gmax;
        } else {
            for (int64_t i = 0; i < g; ++i)
                for (int64_t j = 0; j < g; ++j)
                    own[i * gmax + j] =
                        i != j ? (float)((double)p[o + i] * (double)p[o + j]) : p[o + i];
        }
        /* edge vectors, both orientations (v_ij = v_ji), and the target */
        for (int64_t i = 0; s == ORC_OK && i < g; ++i) {
            for (int64_t j = i + 1; j < g; ++j) {
                double wi, wj, ir;
                s = edge_weights(rule, wmax, blk, gmax, i, j, &wi, &wj, &ir);
                if (s) break;
                double dr = (double)rewards[o + i] - (double)rewards[o + j];
                double* vij = v + (i * g + j) * D;
                double* vji = v + (j * g + i) * D;
                for (int64_t d = 0; d < D; ++d) {
                    double si = score_at(scores, dtype, ld, o + i, d);
                    double sj = score_at(scores, dtype, ld, o + j, d);
                    vij[d] = 0.5 * dr * (wi * si - wj * sj);
                    vji[d] = vij[d];
                    t[d] += 0.5 * dr * (si - sj) / M;
                }
            }
        }
        double tr = 0.0, bb = 0.0;
        if (s == ORC_OK) {
            for (int64_t i = 0; i < g; ++i) {
                double pi_ = (double)p[o + i];
                for (int64_t j = 0; j < g; ++j) {
                    if (j == i) continue;
                    double pj = (double)p[o + j];
                    const double* vij = v + (i * g + j) * D;
                    if (j > i) {
                        double rho = pi_ * pj, nn = 0.0;
                        for (int64_t d = 0; d < D; ++d) {
                            mu[d] += rho * vij[d] / M;
                            nn += vij[d] * vij[d];
                        }
                        tr += rho * (1.0 - rho) * nn;
                    }
                    for (int64_t k = 0; k < g; ++k) {
                        if (k == i || k == j) continue;
                        double pk = (double)p[o + k];
                        const double* vik = v + (i * g + k) * D;
                        double ip = 0.0;
                        for (int64_t d = 0; d < D; ++d) ip += vij[d] * vik[d];
                        tr += pi_ * pj * pk * (1.0 - pi_) * ip;
                    }
                }
            }
            tr /= M * M;
            for (int64_t d = 0; d < D; ++d) {
                double e = mu[d] - t[d];
                bb += e * e;
            }
            mse[b] = bb + tr;
            bias_norm[b] = sqrt(bb);
        } else {
#pragma omp critical
            err = s;
        }
        free(v); free(t); free(mu); free(own);
    }
    return err;
}

/* ------------------------------------------------------------------------ */
/* Conditional Poisson sampling (App. B; Hajek 1964; Chen, Dempster and Liu  */
/* 1994): a sample S of exactly n of the G units with                        */
/*     P(S) = prod_{i in S} w_i / e_n(w),                                    */
/* e_k the elementary symmetric polynomial of the odds w.  Then              */
/*     pi_i  = w_i e_{n-1}(w without i) / e_n(w),                            */
/*     pi_ij = w_i w_j e_{n-2}(w without i, j) / e_n(w).                     */
/* Every polynomial is built by the textbook recursion over units,           */
/* e_k(w_1..w_m) = e_k(w_1..w_{m-1}) + w_m e_{k-1}(w_1..w_{m-1}), all terms  */
/* positive.                                                                 */
/* ------------------------------------------------------------------------ */
/* e_0..e_n of the units 0..g-1 except skip1 and skip2 (-1: none). */
static void esp_excluding(const double* w, int64_t g, int64_t n, int64_t skip1, int64_t skip2,
                          double* e) {
    e[0] = 1.0;
    for (int64_t k = 1; k <= n; ++k) e[k] = 0.0;
    for (int64_t m = 0; m < g; ++m) {
        if (m == skip1 || m == skip2) continue;
        for (int64_t k = n; k >= 1; --k) e[k] = e[k] + w[m] * e[k - 1];
    }
}

/* First- and second-order inclusion probabilities of one prompt's design:
 * pi[i], pij[i * g + j] (pij[i * g + i] = pi[i]).  0 < n < g. */
int orc_cps_inclusion(const double* w, int64_t g, int64_t n, double* pi, double* pij) {
    if (g < 1 || n < 0 || n > g || w == NULL || pi == NULL) return ORC_EINVAL;
    for (int64_t i = 0; i < g; ++i)
        if (!(w[i] > 0.0 && w[i] < INFINITY)) return ORC_EINVAL;
    double* e = (double*)malloc((size_t)(n + 1) * sizeof(double));
    if (!e) return ORC_EINVAL;
    esp_excluding(w, g, n, -1, -1, e);
    const double en = e[n];
    for (int64_t i = 0; i < g; ++i) {
        if (n == 0) {
            pi[i] = 0.0;
            continue;
        }
        esp_excluding(w, g, n - 1, i, -1, e);
        pi[i] = w[i] * e[n - 1] / en;
    }
    if (pij) {
        for (int64_t i = 0; i < g; ++i) {
            pij[i * g + i] = pi[i];
            for (int64_t j = i + 1; j < g; ++j) {
                double v = 0.0;
                if (n >= 2) {
                    esp_excluding(w, g, n - 2, i, j, e);
                    v = w[i] * w[j] * e[n - 2] / en;
                }
                pij[i * g + j] = v;
                pij[j * g + i] = v;
            }
        }
    }
    free(e);
    return ORC_OK;
}

/* Odds w whose design has first-order probabilities pi_target (each in
 * (0, 1), summing to the integer n within 1e-4 n; the target is first scaled
 * by n / sum so that it sums to n): the fixed-point iteration
 * w_i <- w_i pi_target_i / pi_i(w), rescaled to a geometric mean of 1 (the
 * design does not change when every odds is multiplied by one constant),
 * until max_i |pi_i(w) / pi_target_i - 1| <= tol or max_iter iterations.
 * Returns the number of iterations in *iters (negative: not converged). */
int orc_cps_fit(const double* pi_target, int64_t g, int64_t n, double tol, int64_t max_iter,
                double* w, int64_t* iters) {
    if (g < 1 || n < 1 || n >= g || pi_target == NULL || w == NULL) return ORC_EINVAL;
    double sum = 0.0;
    for (int64_t i = 0; i < g; ++i) {
        if (!(pi_target[i] > 0.0 && pi_target[i] < 1.0)) return ORC_EP;
        sum += pi_target[i];
    }
    if (fabs(sum - (double)n) > 1e-4 * (double)n) return ORC_EP;
    double* pi = (double*)malloc((size_t)g * 2 * sizeof(double));
    if (!pi) return ORC_EINVAL;
    double* tg = pi + g;
    for (int64_t i = 0; i < g; ++i) {
        tg[i] = pi_target[i] * ((double)n / sum);
        if (!(tg[i] < 1.0)) {
            free(pi);
            return ORC_EP;
        }
        w[i] = tg[i] / (1.0 - tg[i]);
    }
    {   /* start at a geometric mean of 1 too, so the output always has it */
        double lg0 = 0.0;
        for (int64_t i = 0; i < g; ++i) lg0 += log(w[i]);
        lg0 = exp(-lg0 / (double)g);
        for (int64_t i = 0; i < g; ++i) w[i] *= lg0;
    }
    int64_t it = 0;
    int ok = 0;
    for (; it < max_iter; ++it) {
        orc_cps_inclusion(w, g, n, pi, NULL);
        double err = 0.0, lg = 0.0;
        for (int64_t i = 0; i < g; ++i) {
            double r = fabs(pi[i] / tg[i] - 1.0);
            if (r > err) err = r;
        }
        if (err <= tol) {
            ok = 1;
            break;
        }
        for (int64_t i = 0; i < g; ++i) {
            w[i] *= tg[i] / pi[i];
            lg += log(w[i]);
        }
        lg = exp(-lg / (double)g);
        for (int64_t i = 0; i < g; ++i) w[i] *= lg;
    }
    free(pi);
    if (iters) *iters = ok ? it : -it;
    return ORC_OK;
}

/* Sequential conditional Poisson draw of one prompt for replicate r: units in
 * order i = 0..g-1, with k units still to select, unit i is selected with
 * probability w_i e_{k-1}(w_{i+1..g-1}) / e_k(w_{i..g-1}) (so the sample has
 * exactly n units and probability prod w / e_n).  The uniform of unit i is
 * the top 32 bits of Philox4x64-10 word (i & 3) at counter
 * (r, prompt id, i >> 2, 0), key (seed, 0) -- the same reading as the
 * Bernoulli draw -- and the unit is selected iff u_i < P * 2^32, all in fp64
 * with unfused operations in the order written. */
int orc_cps_draw_one(const double* w, int64_t g, int64_t n, uint64_t seed, int64_t r, int64_t bid,
                     uint8_t* mask) {
    if (g < 1 || n < 0 || n > g) return ORC_EINVAL;
    /* suffix table E[i][k] = e_k(w_i .. w_{g-1}), i = g..0 */
    double* E = (double*)calloc((size_t)(g + 1) * (size_t)(n + 1), sizeof(double));
    if (!E) return ORC_EINVAL;
    E[g * (n + 1) + 0] = 1.0;
    for (int64_t i = g - 1; i >= 0; --i) {
        E[i * (n + 1) + 0] = 1.0;
        for (int64_t k = 1; k <= n; ++k) {
            double t = w[i] * E[(i + 1) * (n + 1) + k - 1];
            E[i * (n + 1) + k] = E[(i + 1) * (n + 1) + k] + t;
        }
    }
    int64_t k = n;
    uint64_t key[2] = {seed, 0};
    for (int64_t i = 0; i < g; ++i) {
        uint64_t ctr[4] = {(uint64_t)r, (uint64_t)bid, (uint64_t)(i >> 2), 0};
        uint64_t out[4];
        orc_philox4x64_10(ctr, key, out);
        double u = (double)(out[i & 3] >> 32);
        int take = 0;
        if (k > 0) {
            double num = w[i] * E[(i + 1) * (n + 1) + k - 1];
            double prob = num / E[i * (n + 1) + k];
            take = u < prob * 4294967296.0;
        }
        mask[i] = (uint8_t)take;
        k -= take;
    }
    free(E);
    return k == 0 ? ORC_OK : ORC_EINVAL;
}

/* Batched draw: mask[r][v] for replicates rep0..rep0+R-1 of every prompt,
 * with per-prompt sizes n[b] and odds w[v]; prompt ids 0..B-1. */
int orc_cps_draw(int64_t B, const int64_t* offsets, const double* w, const int32_t* n,
                 uint64_t seed, int64_t rep0, int64_t R, uint8_t* mask) {
    if (B < 1 || offsets == NULL || w == NULL || n == NULL || mask == NULL || R < 0)
        return ORC_EINVAL;
    int64_t nv = offsets[B];
    int err = ORC_OK;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t r = 0; r < R; ++r) {
        for (int64_t b = 0; b < B; ++b) {
            int64_t o = offsets[b], g = offsets[b + 1] - offsets[b];
            int s = orc_cps_draw_one(w + o, g, n[b], seed, rep0 + r, b, mask + r * nv + o);
            if (s) {
#pragma omp critical
                err = s;
            }
        }
    }
    return err;
}

/* Number of OpenMP threads the parallel loops above will use. */
int orc_num_threads(void) {
#ifdef _OPENMP
    extern int omp_get_max_threads(void);
    return omp_get_max_threads();
#else
    return 1;
#endif
}
