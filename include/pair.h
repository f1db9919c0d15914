/*
 * pair.h -- C ABI of libpair: the data-parallel hot path of PAIR
 * (Pairwise-Aware Inclusion Reweighting) on AMD Instinct MI355X (gfx950).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Every array argument is a DEVICE pointer owned by the caller.  The library
 *    never allocates, frees or retains caller memory; scratch space is passed
 *    in explicitly (the audits' workspaces).
 *  - `stream` is a hipStream_t passed as void* (NULL = the default stream).
 *    All work is enqueued asynchronously on it; nothing blocks the host.
 *  - Host-detectable argument errors return a negative PAIR_E* code and
 *    enqueue nothing.  A failed launch returns PAIR_EHIP.
 *  - Data-dependent errors found on the device are OR-ed into *d_status
 *    (device int32, optional: NULL disables reporting) as PAIR_ST_* bits; the
 *    outputs of the affected prompt are then unspecified.  Callers that pass
 *    d_status clear it before the call.
 *  - Prompts are packed ragged: `offsets` is int64 [B+1] with offsets[0] = 0,
 *    offsets[B] = nv; prompt b owns packed vertices (rollouts)
 *    offsets[b] .. offsets[b+1]-1, and G_b = offsets[b+1] - offsets[b].
 *  - Joint inclusion probabilities are a dense fp32 block per prompt,
 *    pi[B][gmax][gmax]; entry (i, j) with i < j defines rho_ij = rho_ji (the
 *    upper triangle is the only part read); the diagonal and the entries
 *    beyond G_b are ignored on input.
 *  - Scores are row-major [nv][ld] (ld >= D elements) in fp32 or bf16; the
 *    base pointer and every row must be 16-byte aligned.
 *  - Calls are deterministic: the same inputs give bitwise-identical outputs
 *    (no floating-point atomics).  Concurrent calls on different streams
 *    share no library state.
 *
 * Notation follows the paper: G candidate rollouts per prompt, rewards r_i,
 * continuation indicators J_i, joint inclusion probabilities rho_ij, pair
 * kernel h_ij = 1/2 (r_i - r_j)(s_i - s_j), M = C(G, 2).
 */
#ifndef PAIR_H
#define PAIR_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Return codes. */
#define PAIR_OK 0
#define PAIR_EINVAL (-1)     /* null pointer or malformed size                 */
#define PAIR_EDTYPE (-2)     /* unknown score dtype                             */
#define PAIR_ERANGE (-3)     /* gmax outside [2, 64], D < 1, R < 1, ld < D ...  */
#define PAIR_EALIGN (-4)     /* scores base or row stride not 16-byte aligned   */
#define PAIR_EHIP (-5)       /* a HIP launch or runtime call failed             */
#define PAIR_EWORKSPACE (-6) /* workspace missing, misaligned or too small      */
#define PAIR_ESCRATCH (-7)   /* one prompt's audit needs more than the static
                                scratch of pair_audit_noalloc                  */

/* Score dtypes. */
#define PAIR_F32 0
#define PAIR_BF16 1

/* Device status bits (OR-ed into *d_status). */
#define PAIR_ST_BAD_GROUP 1  /* G_b < 2, G_b > gmax or offsets not monotone    */
#define PAIR_ST_RHO_RANGE 2  /* an OBSERVED edge has rho outside (0, 1]        */
#define PAIR_ST_P_RANGE 4    /* a continuation probability outside (0, 1]      */
#define PAIR_ST_NONFINITE 8  /* a non-finite score in an audited score block    */
#define PAIR_ST_BUDGET 16    /* design: budget below pi_min * sum(c), or an
                                invalid prefix statistic (p outside [0, 1],
                                c or m not positive and finite)               */
#define PAIR_ST_SOLVER 32    /* design: the solver reached its sweep cap or a
                                search limit before converging; the prompt
                                fell back to the uniform design               */

/* Edge-weight rules: the estimator variants compared in the paper's audit and
 * ablation tables (Sec. 6, Tables 2, 4, 5; App. A "Naive selection bias" and
 * App. B "Estimated and stabilized propensities").  Each rule estimates
 *     g = (1/N) sum_{i<j observed} 1/2 (r_i - r_j) (w_i s_i - w_j s_j):
 *   HT          w = 1/rho_ij,              N = M = C(G, 2)  exact PAIR, Eq. (pair-ht)
 *   UNWEIGHTED  w = 1,                     N = M            naive selection
 *   RATIO_KE    w = 1,                     N = K_E          mean over observed edges
 *   CLIPPED     w = min(1/rho_ij, wmax),   N = M            stabilised weights
 *   SELFNORM    w = 1/rho_ij,              N = sum over observed edges of 1/rho_ij
 *   MARGINAL    w_i = 1/pi_i, w_j = 1/pi_j, N = M           per-rollout propensity only;
 *               pi_i is the diagonal of the pi block (the paper names this
 *               variant without a formula; this is the library's reading)
 * HT, UNWEIGHTED and CLIPPED/SELFNORM coefficients are centred over the
 * completed vertices (a rounding-level step: their folds sum to zero); the
 * MARGINAL fold does not sum to zero and is not centred.  A prompt with fewer
 * than two completed vertices gets exact zeros under every rule. */
#define PAIR_RULE_HT 0
#define PAIR_RULE_UNWEIGHTED 1
#define PAIR_RULE_RATIO_KE 2
#define PAIR_RULE_CLIPPED 3
#define PAIR_RULE_SELFNORM 4
#define PAIR_RULE_MARGINAL 5

/* Probability designs for pair_design_alloc. */
#define PAIR_DESIGN_PAIR 0       /* graph-coupled convex design, Sec. 4.4        */
#define PAIR_DESIGN_POINTWISE 1  /* pointwise p (1 - p) allocation               */
#define PAIR_DESIGN_UNIFORM 2    /* one probability, the same expected cost      */

/* Largest group size supported by the design draw, the coefficient fold and
 * the audit (one 64-lane wavefront holds one prompt's vertices). */
#define PAIR_GMAX_LIMIT 64

/*
 * pair_design_inclusion -- randomized continuation design (paper Sec. 3.3;
 * the design draw of Algorithm 1, a new independent draw per step; Theorem
 * 2's requirement that rho_ij is logged before rewards are seen).
 *
 * Independent Bernoulli vertices: J_i ~ Bernoulli(p_i), I_ij = J_i J_j,
 * rho_ij = p_i p_j.  The indicators come from the counter-based generator
 * Philox4x64-10 (Salmon et al., SC'11):
 *     key = (seed, 0), counter = (rep0 + r, b, i >> 2, 0),
 *     u   = top 32 bits of output word (i & 3),
 *     J_i = [u < floor(p_i * 2^32)]    (p_i = 1 always includes),
 * so P(J_i = 1) = p_i exactly for every fp32 p_i >= 2^-9, and any range of
 * replicates can be regenerated independently (resumable, shardable).
 *
 *   B, nv, gmax   prompts, packed vertices, dense block size (2 <= gmax <= 64)
 *   offsets       int64 [B+1]
 *   p             fp32 [nv] continuation probabilities in (0, 1]
 *   seed, rep0, R generator key, first replicate index, replicate count (R >= 1)
 *   mask          uint8 [R][nv] out: J for replicate rep0 + r       (or NULL)
 *   pi            fp32 [B][gmax][gmax] out: logged rho_ij = fl32(p_i p_j) for
 *                 i != j, p_i on the diagonal, 0 beyond G_b        (or NULL)
 *   edge_count    int32 [R][B] out: observed edges K_E = C(k, 2)    (or NULL)
 *   completed     int32 [R][B] out: completed vertices k            (or NULL)
 * Device status: PAIR_ST_BAD_GROUP, PAIR_ST_P_RANGE.
 */
int pair_design_inclusion(int64_t B, int64_t nv, int32_t gmax, const int64_t* offsets,
                          const float* p, uint64_t seed, int64_t rep0, int64_t R,
                          uint8_t* mask, float* pi, int32_t* edge_count, int32_t* completed,
                          int32_t* d_status, void* stream);

/*
 * pair_design_alloc -- graph-coupled probability design (paper Sec. 4.3 and
 * Sec. 4.4, Eqs. (disagreement), (edge-proxy), (convex-objective), (budget)):
 * continuation probabilities for every prompt from its prefix statistics.
 *     d_ij = p_i (1 - p_j) + (1 - p_i) p_j,  a_ij = d_ij [ (m_i + m_j)^2 / 4 ]
 *     b_i  = (sum_{j != i} sqrt(a_ij))^2 - sum_{j != i} a_ij
 *     pi = argmin sum_{i<j} a_ij / (pi_i pi_j) + sum_i b_i / pi_i
 *          s.t. sum_i c_i pi_i <= budget_b,  pi_min <= pi_i <= 1
 * (the paper's program in pi_i = e^{-x_i}), solved to the optimum in fp64:
 * exact cyclic coordinate minimisation of the Lagrangian for a multiplier
 * found by a bracketed false-position search (each coordinate sweep to a
 * relative change of 1e-13, the budget to 1e-13 relative; the defaults of
 * pair_design_alloc_ex below).  The budget is spent exactly unless sum_i c_i <=
 * budget_b (then pi = 1).  Vertices with no contrast to any other vertex
 * (all a_ij = 0 and b_i = 0) take pi_min.  The PAIR_DESIGN_POINTWISE design
 * is the same program with a = 0 and b_i = p_i (1 - p_i); PAIR_DESIGN_UNIFORM
 * is pi_i = clip(budget_b / sum_i c_i, pi_min, 1).  The output feeds
 * pair_design_inclusion as p.
 *
 *   p_hat          fp32 [nv] predicted success probabilities in [0, 1]
 *   c_hat          fp32 [nv] predicted remaining costs (> 0)
 *   m_hat          fp32 [nv] score-norm predictions (>= 0) for the scaled
 *                  proxy, or NULL for the parameter-free a = d
 *   budget         fp32 [B] expected-cost budget of each prompt (> 0)
 *   pi_min         probability floor in (0, 1] (the paper's default: 0.08)
 *   design         PAIR_DESIGN_*
 *   pi             fp32 [nv] out: continuation probabilities
 *   objective      fp64 [B] out: the PAIR proxy Phi at pi (every design)  (or NULL)
 *   iters          int32 [B] out: coordinate sweeps used (negative: the
 *                  solver failed and the prompt got the uniform design)   (or NULL)
 * Group sizes 1 <= G_b <= gmax <= 64.  Device status: PAIR_ST_BAD_GROUP;
 * PAIR_ST_BUDGET (budget_b < pi_min sum c: that prompt gets pi = pi_min;
 * invalid statistics: pi = pi_min); PAIR_ST_SOLVER (see
 * pair_design_alloc_ex).
 */
int pair_design_alloc(int64_t B, int64_t nv, int32_t gmax, const int64_t* offsets,
                      const float* p_hat, const float* c_hat, const float* m_hat,
                      const float* budget, float pi_min, int32_t design, float* pi,
                      double* objective, int32_t* iters, int32_t* d_status, void* stream);

/*
 * pair_design_alloc_ex -- pair_design_alloc with the solver settings of the
 * paper's implementation (App. C "Probability optimization"): a warm start
 * from the previous step's probabilities, an iteration cap with a fallback to
 * uniform probabilities of the same expected cost when the solver fails, and
 * the solver residual per prompt.  pair_design_alloc is this call with
 * pi_prev = NULL, max_sweeps = 0 and residual = NULL.
 *
 *   pi_prev        fp32 [nv] previous probabilities (or NULL: a cold start).
 *                  They are clipped to [pi_min, 1] (NaN reads as pi_min); the
 *                  multiplier search starts at the multiplier their KKT
 *                  conditions imply (the median of A_i / (c_i pi_i^2) over the
 *                  interior vertices) and brackets the root from there; a
 *                  start with no interior vertex is a cold start.
 *   max_sweeps     cap on a prompt's coordinate sweeps over all multipliers
 *                  (>= 0; 0: 10000).  A prompt that reaches it, or a search
 *                  limit (400 sweeps per multiplier, 200 multipliers), before
 *                  converging gets the uniform design clip(budget_b / sum c,
 *                  pi_min, 1), its iters is minus the sweeps used, and
 *                  PAIR_ST_SOLVER is set.
 *   residual       fp64 [B] out: KKT residual of the design's program at the
 *                  returned fp32 probabilities x (for PAIR_DESIGN_UNIFORM, of
 *                  the PAIR program).  With g_i = A_i / x_i^2, A_i =
 *                  sum_{j != i} a_ij / x_j + b_i, and lam the median of
 *                  g_i / c_i over interior vertices (with none: 0 if the
 *                  budget is slack, else the largest g_i / c_i at pi_min), it
 *                  is the largest of |g_i / c_i - lam| (interior), lam - g_i /
 *                  c_i (at 1), g_i / c_i - lam (at pi_min), all over
 *                  max_i g_i / c_i, and of |c^T x - budget_b| / budget_b
 *                  (lam > 0) and the relative overspend.  A vertex is at a
 *                  bound within 1e-7 relative.                          (or NULL)
 * Other arguments and device status as pair_design_alloc, plus
 * PAIR_ST_SOLVER; max_sweeps < 0 returns PAIR_ERANGE.
 */
int pair_design_alloc_ex(int64_t B, int64_t nv, int32_t gmax, const int64_t* offsets,
                         const float* p_hat, const float* c_hat, const float* m_hat,
                         const float* budget, float pi_min, int32_t design, const float* pi_prev,
                         int32_t max_sweeps, float* pi, double* objective, int32_t* iters,
                         double* residual, int32_t* d_status, void* stream);

/*
 * pair_cps_fit -- fixed-size continuation design (paper App. B "Fixed-size
 * and exact-cost designs": conditional Poisson sampling, Hajek 1964): exactly
 * n_b = round(sum_i pi_target_i) of the G_b candidates continue, each with
 * first-order probability pi_target_i (the target is scaled by n_b / sum to
 * sum to n_b exactly).  Samples S of size n_b have probability
 * prod_{i in S} w_i / e_n(w) with odds w fitted here in fp64 (Newton's
 * method on the log-odds, the Hessian being the design's own covariance
 * pi_ij - pi_i pi_j, with step halving; to 1e-12 relative on every pi_i), and
 * the
 * exact joint probabilities
 *     pi_ij = w_i w_j e_{n-2}(w without i, j) / e_n(w)
 * do not factorise; they are what the estimator must weight with.
 *
 *   pi_target      fp32 [nv] in (0, 1), each prompt's sum within 1e-4 of an
 *                  integer n_b with 1 <= n_b < G_b
 *   w              fp64 [nv] out: the odds (geometric mean 1 per prompt)
 *   n_out          int32 [B] out: n_b                                  (or NULL)
 *   pi_joint       fp32 [B][gmax][gmax] out: pi_ij for i != j < G_b, pi_i on the
 *                  diagonal, 0 beyond G_b -- the pi block that
 *                  pair_edge_coeffs and pair_audit_rule take       (or NULL)
 *   iters          int32 [B] out: evaluations of pi(w), halved steps
 *                  included (negative: not converged in 200)        (or NULL)
 * Device status: PAIR_ST_BAD_GROUP; PAIR_ST_P_RANGE (a target outside (0, 1)
 * or a sum not within 1e-4 of an admissible integer: that prompt's w is 0,
 * n_b = 0 and iters 0; no convergence: the last odds are written and iters
 * is negative).
 */
int pair_cps_fit(int64_t B, int64_t nv, int32_t gmax, const int64_t* offsets,
                 const float* pi_target, double* w, int32_t* n_out, float* pi_joint,
                 int32_t* iters, int32_t* d_status, void* stream);

/*
 * pair_cps_draw -- fixed-size draws of the conditional Poisson design for
 * replicates rep0 .. rep0+R-1: units are visited in order and unit i is
 * selected with probability w_i e_{k-1}(w_{i+1..}) / e_k(w_{i..}), k the
 * units still to select, so every draw has exactly n_b units and sample
 * probability prod w / e_n.  The uniform for unit i is the top 32 bits of
 * Philox4x64-10 word (i & 3) at counter (rep0 + r, b, i >> 2, 0), key
 * (seed, 0), as in pair_design_inclusion; the threshold is computed in fp64
 * with unfused operations in a fixed order.
 *
 *   w, n           from pair_cps_fit (w > 0 finite; 0 <= n_b <= G_b)
 *   mask           uint8 [R][nv] out
 *   edge_count     int32 [R][B] out: n_b (n_b - 1) / 2                  (or NULL)
 * Device status: PAIR_ST_BAD_GROUP, PAIR_ST_P_RANGE (invalid w or n_b: that
 * prompt's masks are not written).
 */
int pair_cps_draw(int64_t B, int64_t nv, int32_t gmax, const int64_t* offsets, const double* w,
                  const int32_t* n, uint64_t seed, int64_t rep0, int64_t R, uint8_t* mask,
                  int32_t* edge_count, int32_t* d_status, void* stream);

/*
 * pair_edge_coeffs -- pair-corrected sequence advantages, paper Eq.
 * (pair-advantage), each observed edge's weighted term added to both of its
 * endpoints as in Algorithm 1's pair-corrected update, with App. C's numerics
 * (fp32 accumulation, centred across the observed endpoints):
 *     A~_i = J_i / (2M) * sum_{j != i} J_j (r_i - r_j) / rho_ij,
 * then A~_i -= mean of A~ over completed vertices.  Unobserved vertices get
 * exactly 0, and so does every vertex of a prompt with fewer than two
 * completed vertices (App. B) or with equal observed rewards.  M = C(G_b, 2)
 * counts the candidate pool, not the observed edges.
 *
 *   rewards       fp32 [nv]
 *   mask          uint8 [nv] completion indicators J (NULL: all completed)
 *   pi            fp32 [B][gmax][gmax] logged rho (NULL: rho = 1, i.e. the
 *                 unweighted estimator / the complete-pair coefficients)
 *   coeff         fp32 [nv] out: A~
 *   edge_count    int32 [B] out: observed edges K_E                 (or NULL)
 * Device status: PAIR_ST_BAD_GROUP, PAIR_ST_RHO_RANGE.
 */
int pair_edge_coeffs(int64_t B, int64_t nv, int32_t gmax, const int64_t* offsets,
                     const float* rewards, const uint8_t* mask, const float* pi, float* coeff,
                     int32_t* edge_count, int32_t* d_status, void* stream);

/*
 * pair_design_coeffs -- the design draw of one replicate and the HT
 * coefficient fold in a single launch (paper Sec. 3.3 and Eq.
 * (pair-advantage), as pair_design_inclusion followed by pair_edge_coeffs on
 * its logged block).  The indicators, the logged rho_ij = fl32(p_i p_j) and
 * the coefficients are bitwise those of the two calls with R = 1 and
 * rep0 = rep; the mask and pi block are written only if asked for.
 *
 *   p, rewards     fp32 [nv]
 *   seed, rep      generator key and the replicate index
 *   mask           uint8 [nv] out                                    (or NULL)
 *   pi             fp32 [B][gmax][gmax] out, as pair_design_inclusion (or NULL)
 *   coeff          fp32 [nv] out: A~
 *   edge_count, completed  int32 [B] out                             (or NULL)
 * Device status: PAIR_ST_BAD_GROUP, PAIR_ST_P_RANGE, PAIR_ST_RHO_RANGE.
 */
int pair_design_coeffs(int64_t B, int64_t nv, int32_t gmax, const int64_t* offsets,
                       const float* p, const float* rewards, uint64_t seed, int64_t rep,
                       uint8_t* mask, float* pi, float* coeff, int32_t* edge_count,
                       int32_t* completed, int32_t* d_status, void* stream);

/*
 * pair_edge_coeffs_rule -- pair_edge_coeffs under any edge-weight rule
 * (PAIR_RULE_*), plus the per-prompt weight diagnostics the paper logs
 * (App. C "Probability optimization"; App. D metrics):
 *     ess[b]        = (sum_e w_e)^2 / sum_e w_e^2 over the observed edges
 *     max_weight[b] = max_e w_e
 * with w_e the rule's edge weight ((w_i + w_j)/2 for MARGINAL); both are 0
 * when fewer than two vertices completed.  pair_edge_coeffs is this call
 * with PAIR_RULE_HT and no diagnostics.
 *
 *   rule           PAIR_RULE_* (anything else: PAIR_EINVAL)
 *   wmax           weight cap for PAIR_RULE_CLIPPED (> 0, finite: else
 *                  PAIR_EINVAL); ignored by the other rules
 *   ess, max_weight  fp32 [B] out                                    (or NULL)
 * Device status: as pair_edge_coeffs; PAIR_ST_RHO_RANGE also flags a
 * marginal pi_i outside (0, 1] under PAIR_RULE_MARGINAL.  UNWEIGHTED and
 * RATIO_KE read no rho.
 */
int pair_edge_coeffs_rule(int64_t B, int64_t nv, int32_t gmax, const int64_t* offsets,
                          const float* rewards, const uint8_t* mask, const float* pi,
                          int32_t rule, float wmax, float* coeff, int32_t* edge_count, float* ess,
                          float* max_weight, int32_t* d_status, void* stream);

/*
 * pair_weighted_grad -- the induced-edge HT gradient, paper Eq. (pair-ht)
 * written as sum_i A~_i s_i (Sec. 4.5), batched over prompts:
 *     reduce = 0:  out[b][d] = sum_{i < G_b} coeff[offsets[b] + i] * s[offsets[b] + i][d]
 *     reduce = 1:  out[d]    = (1/B) sum_b (the same per-prompt sum),
 * i.e. the batch mean of the per-prompt estimates, summed flat over the packed
 * rows offsets[0] .. offsets[B]-1.  fp32 accumulation in a fixed order.  Rows
 * whose coefficient is exactly zero (unobserved rollouts, saturated prompts)
 * are neither read nor summed: an uncompleted rollout has no score, so its
 * row may hold anything.
 *
 *   D, scores, dtype, ld   score block (PAIR_F32 or PAIR_BF16), row stride ld
 *   coeff          fp32 [nv] (from pair_edge_coeffs)
 *   out            fp32 [B][D] (reduce = 0, rows packed with stride D) or
 *                  fp32 [D] (reduce = 1) out
 *   reduce         0 or 1 (anything else: PAIR_EINVAL)
 * Any G_b >= 0 is accepted here.  Device status: PAIR_ST_BAD_GROUP (offsets
 * not monotone or beyond nv: with reduce = 0 that prompt's row is not
 * written; with reduce = 1 the output is unspecified).
 */
int pair_weighted_grad(int64_t B, int64_t nv, const int64_t* offsets, int64_t D,
                       const void* scores, int32_t dtype, int64_t ld, const float* coeff,
                       float* out, int32_t reduce, int32_t* d_status, void* stream);

/*
 * pair_audit_workspace_bytes -- device workspace that pair_audit needs for
 * B prompts of at most gmax vertices, D score columns and R replicates.
 */
size_t pair_audit_workspace_bytes(int64_t B, int32_t gmax, int64_t D, int64_t R);

/*
 * pair_audit -- frozen-population estimator audit (paper Sec. 6.2, Table 2,
 * App. D metrics).  For each prompt the complete candidate population is
 * fixed; R design replicates rep0 .. rep0+R-1 are drawn exactly as
 * pair_design_inclusion draws them (same seed => same masks), each one gives
 * the HT estimate g_r = sum_i A~^(r)_i s_i, and against the complete-pair
 * target t = sum_i a_i s_i, a_i = A~ with every vertex completed and rho = 1
 * (= (r_i - mean r)/(G - 1), Theorem 1):
 *     e_r  = || g_r - t ||^2 = || (A~^(r) - a) S_b ||^2
 *     mse  = (1/R) sum_r e_r
 *     bias = || (1/R) sum_r g_r - t ||
 * The R x D estimates are never materialised: (A~^(r) - a) times S_b runs on
 * the matrix cores with the squared norm reduced in the epilogue.  Operands
 * are fp16 after power-of-two rescaling: each score row by its largest
 * magnitude within a column slice, then rounded to nearest fp16, which is
 * exact for entries within 2^17 of that maximum and off by at most 2^-25 of
 * it below; each replicate row of A~^(r) - a by its largest entry, then one
 * fp16 rounding (2^-11 relative).  With delta_r = A~^(r) - a, y_r =
 * delta_r S_b, z_r = S_b y_r^T (so e_r = delta_r . z_r) and u = 2^-11, that
 * rounding has the same relative error in every score column, so to first
 * order |Delta e_r| <= 2 u sum_i |delta_ri z_ri|, plus terms of 2^-25 of
 * the row maxima M_i for fp16 subnormals: at most 2u e_r when the terms
 * delta_ri z_ri share a sign (near-orthogonal score rows), more only when
 * they cancel, as with a single score column.  The bias row
 * (1/R) sum_r (A~^(r) - a) is applied in fp32 on the vector units, without
 * that rounding.  A replicate's e_r does not depend on R or rep0: calls over
 * consecutive replicate ranges return bitwise the rep_sqerr of one call over
 * their union.  Weights use rho = pi_w when given (e.g. all ones replays the
 * unweighted estimator of Prop. 1), else the logged fl32(p_i p_j).
 *
 *   scores, dtype  PAIR_BF16 only, finite values
 *   rewards, p     fp32 [nv]
 *   pi_w           fp32 [B][gmax][gmax] rho used in the weights      (or NULL)
 *   mse, bias_norm fp64 [B] out
 *   rep_sqerr      fp32 [B][R] out: e_r                              (or NULL)
 *   edge_count     int32 [B][R] out: observed edges per replicate    (or NULL)
 *   workspace      device scratch of ws_bytes >= pair_audit_workspace_bytes,
 *                  256-byte aligned; contents on entry do not matter
 * A prompt whose rewards are all equal has A~^(r) - a = 0 in every replicate
 * (every edge term carries r_i - r_j): its e_r, mse and bias are exact zeros,
 * its draws and edge counts are still made, and its score rows are not read.
 * Device status: PAIR_ST_BAD_GROUP, PAIR_ST_P_RANGE, PAIR_ST_RHO_RANGE,
 * PAIR_ST_NONFINITE (a non-finite score of a prompt that is swept).
 */
int pair_audit(int64_t B, int64_t nv, int32_t gmax, const int64_t* offsets, int64_t D,
               const void* scores, int32_t dtype, int64_t ld, const float* rewards,
               const float* p, const float* pi_w, uint64_t seed, int64_t rep0, int64_t R,
               double* mse, double* bias_norm, float* rep_sqerr, int32_t* edge_count,
               void* workspace, size_t ws_bytes, int32_t* d_status, void* stream);

/*
 * pair_audit_noalloc -- pair_audit for callers that cannot allocate device
 * memory: code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc.  The arguments are pair_audit's without the workspace.
 * Its workspace is instead a static device array of the library,
 * PAIR_AUDIT_SCRATCH_BYTES (64 MiB), which each GPU the library runs on holds
 * until the process ends (it is part of the library's device code, whether
 * or not this entry point is called).  The prompts are audited in
 * consecutive chunks whose pair_audit_workspace_bytes fits that array, so the
 * outputs are bitwise those of pair_audit with the same arguments (the audit
 * workload's shape, G = 16, D = 65536, R = 4096, takes about 80 prompts per
 * chunk).  If a single prompt needs more than the array it returns
 * PAIR_ESCRATCH and enqueues nothing.  The call allocates nothing and calls no
 * allocating routine.  Every call on one GPU uses that GPU's one array, which
 * keeps the last call's contents: calls ordered on one stream are safe, but
 * calls that overlap on one GPU (other streams, other host threads) race and
 * their outputs are undefined.
 */
#define PAIR_AUDIT_SCRATCH_BYTES ((size_t)64 << 20)
int pair_audit_noalloc(int64_t B, int64_t nv, int32_t gmax, const int64_t* offsets, int64_t D,
                       const void* scores, int32_t dtype, int64_t ld, const float* rewards,
                       const float* p, const float* pi_w, uint64_t seed, int64_t rep0, int64_t R,
                       double* mse, double* bias_norm, float* rep_sqerr, int32_t* edge_count,
                       int32_t* d_status, void* stream);

/*
 * pair_audit_rule -- pair_audit replaying the estimator under an edge-weight
 * rule (PAIR_RULE_*, wmax as in pair_edge_coeffs_rule) against the same
 * complete-pair target: the audit matrix of the paper's Tables 2, 4 and 5
 * (bias norm and MSE of each variant on a frozen population).  The marginal
 * pi_i is the diagonal of pi_w when given, else p_i.  pair_audit is this call
 * with PAIR_RULE_HT.
 */
int pair_audit_rule(int64_t B, int64_t nv, int32_t gmax, const int64_t* offsets, int64_t D,
                    const void* scores, int32_t dtype, int64_t ld, const float* rewards,
                    const float* p, const float* pi_w, int32_t rule, float wmax, uint64_t seed,
                    int64_t rep0, int64_t R, double* mse, double* bias_norm, float* rep_sqerr,
                    int32_t* edge_count, void* workspace, size_t ws_bytes, int32_t* d_status,
                    void* stream);

/*
 * pair_audit_direction_workspace_bytes -- device workspace that
 * pair_audit_direction needs for B prompts of at most gmax vertices, D score
 * columns and R replicates (0 when a size is out of range).
 */
size_t pair_audit_direction_workspace_bytes(int64_t B, int32_t gmax, int64_t D, int64_t R);

/*
 * pair_audit_direction -- the update-direction column of the frozen-policy
 * audit (paper Sec. 6.2 lists the cosine among the audit metrics; the audit
 * matrix of App. E reports it per design): for the replicates rep0 ..
 * rep0+R-1, drawn and folded exactly as pair_audit_rule draws and folds them,
 *     cos_r     = <g_r, t> / (|g_r| |t|)    (0 when g_r = 0 or t = 0)
 *     cosine[b] = (1/R) sum_r cos_r,   target_norm[b] = |t|,
 * with g_r the replicate's estimate under `rule` and t the complete-pair
 * target.  It is evaluated through the prompt's Gram matrix K = S_b S_b^T
 * (fp64 from fp32 matrix-core partial sums): with u_r the replicate's
 * coefficients and a the target's, cos_r = u_r K a / sqrt(u_r K u_r a K a).
 * A prompt whose target is zero (equal rewards) reports cosine 0 and
 * target_norm 0.
 *
 *   arguments      as pair_audit_rule (PAIR_BF16 scores only)
 *   cosine, target_norm  fp64 [B] out
 *   workspace      device scratch of ws_bytes >=
 *                  pair_audit_direction_workspace_bytes, 256-byte aligned;
 *                  contents on entry do not matter
 * Device status: PAIR_ST_BAD_GROUP, PAIR_ST_P_RANGE, PAIR_ST_RHO_RANGE,
 * PAIR_ST_NONFINITE.
 */
int pair_audit_direction(int64_t B, int64_t nv, int32_t gmax, const int64_t* offsets, int64_t D,
                         const void* scores, int32_t dtype, int64_t ld, const float* rewards,
                         const float* p, const float* pi_w, int32_t rule, float wmax,
                         uint64_t seed, int64_t rep0, int64_t R, double* cosine,
                         double* target_norm, void* workspace, size_t ws_bytes,
                         int32_t* d_status, void* stream);

/*
 * pair_audit_exact_workspace_bytes -- device workspace that pair_audit_exact
 * needs for B prompts of at most gmax vertices and D score columns.
 */
size_t pair_audit_exact_workspace_bytes(int64_t B, int32_t gmax, int64_t D);

/*
 * pair_audit_exact -- the exact design audit, with no replicate draws (paper
 * Prop. 1 and App. A "Design covariance"): for an estimator that is linear in
 * the edge indicators, g^ = (1/M) sum_e I_e v_e with
 * v_ij = 1/2 (r_i - r_j)(w_i s_i - w_j s_j), under independent Bernoulli(p_i)
 * vertices (rho_ij = p_i p_j),
 *     bias = || E g^ - t ||,
 *     mse  = bias^2 + tr Cov g^
 *          = bias^2 + (1/M^2) [ sum_{i<j} rho_ij (1 - rho_ij) ||v_ij||^2
 *            + sum_i sum_{j != k; j, k != i} p_i p_j p_k (1 - p_i) <v_ij, v_ik> ]
 * with t the complete-pair average, i.e. mse = E || g^ - t ||^2 exactly (the
 * limit of pair_audit's Monte-Carlo mse as R grows; for the HT rule bias = 0,
 * Theorem 2).  Every inner product is taken from the prompt's Gram matrix
 * K = S_b S_b^T, formed on the matrix cores (bf16 products, fp32 partial sums
 * per column slice, fp64 across slices); the closed form is evaluated in fp64.
 *
 *   rule, wmax     PAIR_RULE_HT, _UNWEIGHTED, _CLIPPED or _MARGINAL (the rules
 *                  linear in the indicators; others: PAIR_EINVAL); the
 *                  weights use pi_w when given, else the logged fl32(p_i p_j)
 *                  with p_i as the marginal; the design itself is p
 *   scores, dtype  PAIR_BF16 only
 *   mse, bias_norm fp64 [B] out
 *   gram           fp64 [B][gmax][gmax] out: K_ij for i, j < G_b (other
 *                  entries untouched)                             (or NULL)
 *   workspace      device scratch of ws_bytes >=
 *                  pair_audit_exact_workspace_bytes, 256-byte aligned
 * Device status: PAIR_ST_BAD_GROUP, PAIR_ST_P_RANGE, PAIR_ST_RHO_RANGE,
 * PAIR_ST_NONFINITE (a non-finite Gram entry).
 */
int pair_audit_exact(int64_t B, int64_t nv, int32_t gmax, const int64_t* offsets, int64_t D,
                     const void* scores, int32_t dtype, int64_t ld, const float* rewards,
                     const float* p, const float* pi_w, int32_t rule, float wmax, double* mse,
                     double* bias_norm, double* gram, void* workspace, size_t ws_bytes,
                     int32_t* d_status, void* stream);

/* Human-readable text for a return code. */
const char* pair_strerror(int code);

/* Library ABI version (major * 10000 + minor * 100 + patch). */
int pair_version(void);

#ifdef __cplusplus
}
#endif

#endif /* PAIR_H */
