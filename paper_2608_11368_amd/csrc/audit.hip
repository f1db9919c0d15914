// Frozen-population estimator audit (paper Sec. 6.2, Table 2; App. D
// metrics MSE = E||g^ - g_full||^2 and the bias norm).
//
// The complete-pair target of a prompt is itself a combination of its score
// rows, t = a S_b with a = (r_i - mean r)/(G - 1) (Theorem 1), and each
// replicate's HT estimate is g_r = A~^(r) S_b (Eq. pair-advantage).  So the
// deviation is a single contraction,
//     g_r - t = (A~^(r) - a) S_b = delta_r S_b,
// and the audit needs e_r = ||delta_r S_b||^2 for every replicate r plus
// ||delta_bar S_b|| for the bias (delta_bar = mean_r delta_r).
//
// Pipeline (all on the caller's stream):
//  1. audit_coeffs  one workgroup per (prompt, 256 replicates), one lane per
//                   replicate: Philox draw of J^(r) (same counter reading as
//                   the design draw), the coefficient fold over a per-prompt
//                   table W_ij = (r_i - r_j)/rho_ij in LDS, centring over the
//                   completed vertices, delta_r stored in fp32, and a
//                   fixed-order partial sum of delta over the 256 lanes.
//  2. audit_prep    replicate rows padded with zero rows to a whole number
//                   of tile pairs (R rounded up to 64), delta_bar stored
//                   in the row after them.  One extra workgroup lists the
//                   live prompts in ascending order: those whose rewards are
//                   not all equal.  A prompt with equal rewards has
//                   W = 0 and a = 0, so every delta_r is exactly zero and so
//                   are its e_r, MSE and bias; the matrix-core grid covers
//                   the live prompts only.
//  3. audit_mfma    the contraction on v_mfma_f32_32x32x16_f16.  Each score
//                   row of a column slice is rescaled by 2^-e_i, with e_i
//                   the exponent of the row's largest magnitude within the
//                   slice, and rounded to fp16 (to nearest), which is exact
//                   for every entry within 2^17 of that maximum and off by
//                   at most 2^-25 of it below (8 significant bits fit in
//                   11, down to fp16's subnormals); each
//                   replicate row of delta is rescaled by 2^(e_i - f_r), with
//                   f_r chosen so its largest entry lies in [1, 2), and rounded
//                   once to fp16 (2^-11 relative).  The products are
//                   rescalings of delta_r S_b by 2^-f_r, so e_r = 4^f_r * sum
//                   of squares.
//                   A workgroup owns one prompt and one slice of score
//                   columns: the slice is converted once into LDS and every
//                   replicate row sweeps over it, so S_b is read from HBM
//                   once; the squares of every output tile are summed in the
//                   epilogue and the rows x D product is never written.
//                   The live (prompt, slice) pairs are split evenly over the
//                   8 XCDs, each XCD taking a contiguous range, so the
//                   workgroups of a prompt share that XCD's L2 for its delta
//                   rows.  The
//                   delta_bar row is one fp32 dot product per score column
//                   on the vector units against the same LDS slice.
//  4. audit_sqerr   e_r = per-slice partial sums reduced in fixed order, one
//                   thread per (prompt, replicate), exactly 0 for a prompt
//                   that is not live; fp64 partial sums of e_r
//     audit_final   per prompt: MSE = fp64 mean of e_r, bias = sqrt(e of the
//                   delta_bar row).
#include "common.hpp"
#include "launch.hpp"

namespace pair {

namespace {

typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int kCoefThreads = 256;    // replicates per audit_coeffs workgroup
constexpr int kSqThreads = 256;      // replicates per audit_sqerr workgroup
constexpr int kMfmaThreads = 512;    // 8 waves per workgroup
constexpr int kMfmaWaves = kMfmaThreads / kWave;
constexpr int kTile = 32;            // replicate rows (and score columns) per matrix instruction
constexpr int kPair = 2;             // replicate tiles a wave carries at once

// Score columns per workgroup slice: the slice of S_b (16 * ks rows, fp16,
// plus one skew row per 8) stays resident in LDS while all replicate rows
// sweep over it.
constexpr int slice_cols(int ks) { return ks == 1 ? 2048 : (ks == 2 ? 1024 : 512); }

inline int64_t round_up(int64_t x, int64_t m) { return (x + m - 1) / m * m; }

struct AuditLayout {
  int ks;            // 16-wide K steps (ceil(gmax / 16))
  int kp;            // 16 * ks: padded K extent
  int64_t rbar;      // the delta_bar row: R rounded up to whole pairs of tiles
  int64_t ntiles;    // 32-row tiles per prompt: rbar / 32 replicate tiles + the delta_bar tile
  int64_t rrows;     // ntiles * 32
  int64_t nslices;   // score-column slices per prompt
  int64_t nwg;       // audit_coeffs workgroups per prompt
  int64_t nsq;       // audit_sqerr workgroups per prompt
  size_t delta_off, epart_off, dsum_off, rpart_off, ebar_off, live_off, total;
};

AuditLayout audit_layout(int64_t B, int32_t gmax, int64_t D, int64_t R) {
  AuditLayout L;
  L.ks = (gmax + 15) / 16;
  L.kp = 16 * L.ks;
  L.rbar = round_up(R, (int64_t)kPair * kTile);
  L.ntiles = L.rbar / kTile + 1;
  L.rrows = L.ntiles * kTile;
  L.nslices = (D + slice_cols(L.ks) - 1) / slice_cols(L.ks);
  L.nwg = (R + kCoefThreads - 1) / kCoefThreads;
  L.nsq = (R + 1 + kSqThreads - 1) / kSqThreads;
  size_t off = 0;
  L.delta_off = off;
  off += (size_t)round_up(B * L.rrows * L.kp * 4, 256);            // fp32 delta rows
  L.epart_off = off;
  off += (size_t)round_up(B * L.nslices * L.rrows * 4, 256);       // per-slice squared errors
  L.dsum_off = off;
  off += (size_t)round_up(B * L.nwg * gmax * 4, 256);               // partial delta sums
  L.rpart_off = off;
  off += (size_t)round_up(B * L.nsq * 8, 256);                      // fp64 partial sums of e_r
  L.ebar_off = off;
  off += (size_t)round_up(B * 4, 256);                              // e of the delta_bar row
  L.live_off = off;
  off += (size_t)round_up((2 * B + 1) * 4, 256);                    // live count, list, flags
  L.total = off;
  return L;
}

// Complete-pair coefficient a_i of vertex `lane` (0 beyond the group): the
// fold with every vertex completed and rho = 1, centred over all G vertices
// (Theorem 1: (r_i - mean r) / (G - 1) in exact arithmetic).  The whole wave
// calls it; lane i holds r_i.
__device__ __forceinline__ float complete_pair_coeff(float r_i, int lane, int g) {
  const bool vert = lane < g;
  float cf = 0.0f;
  for (int j = 0; j < g; ++j) {
    const float r_j = lane_value(r_i, j);
    if (vert && j != lane) cf += r_i - r_j;
  }
  float a_full = vert ? cf / (float)(g * (g - 1)) : 0.0f;
  const float tot = wave_sum(a_full);
  return vert ? a_full - tot / (float)g : 0.0f;
}

// ---------------------------------------------------------------------------
// 1. Replicate coefficients.  A workgroup owns one prompt and 256 replicates
//    (one per lane).  The edge table W, the probabilities and the
//    complete-pair coefficients are built once per workgroup in LDS; each lane
//    then draws its indicators, folds c_i = sum_j J_j W_ij with W read by
//    broadcast (W_ii = 0, so no j != i test is needed, and a zero indicator
//    adds exactly nothing), centres, and keeps its KP deviations in registers.
// ---------------------------------------------------------------------------
template <int KP>
__global__ __launch_bounds__(kCoefThreads) void audit_coeffs_kernel(
    int64_t B, int64_t nv, int32_t gmax, const int64_t* __restrict__ offsets,
    const float* __restrict__ rewards, const float* __restrict__ p,
    const float* __restrict__ pi_w, int32_t rule, float wmax, uint64_t seed, int64_t rep0,
    int64_t pbase, int64_t R, int64_t nwg, int64_t rrows, float* __restrict__ delta,
    float* __restrict__ dsum, int32_t* __restrict__ edge_count, int32_t* d_status) {
  constexpr int kWaves = kCoefThreads / kWave;
  __shared__ __align__(16) float W[KP * KP];     // rule weight x (r_i - r_j), zero on and past G
  __shared__ __align__(16) float V[KP * KP];     // 1/rho_ij (self-normalised denominator)
  __shared__ float pl[KP], rl[KP], af[KP];
  __shared__ float wsum[kWaves][KP];
  const int64_t b = blockIdx.x / nwg;
  const int64_t chunk = blockIdx.x - b * nwg;
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = tid / kWave;
  int64_t o0, g;
  if (!prompt_bounds(offsets, b, nv, 2, gmax, &o0, &g, d_status, chunk == 0 && tid == 0)) return;

  if (wave == 0) {
    const bool vert = lane < g;
    const float r_i = vert ? rewards[o0 + lane] : 0.0f;
    const float p_i = vert ? p[o0 + lane] : 1.0f;
    if (lane < KP) {
      pl[lane] = p_i;
      rl[lane] = r_i;
    }
    if (vert && !p_in_range(p_i) && chunk == 0) raise_status(d_status, PAIR_ST_P_RANGE);
    const float a_full = complete_pair_coeff(r_i, lane, (int)g);
    if (lane < KP) af[lane] = a_full;
  }
  __syncthreads();

  bool bad_rho = false;
  for (int idx = tid; idx < KP * KP; idx += kCoefThreads) {
    const int i = idx / KP, j = idx - i * KP;
    float w = 0.0f, v = 0.0f;
    if (i != j && i < g && j < g) {
      float rho, pii = pl[i], pij = pl[j];
      if (pi_w != nullptr) {
        const float* blk = pi_w + b * (int64_t)gmax * gmax;
        const int lo = i < j ? i : j, hi = i < j ? j : i;
        rho = blk[lo * gmax + hi];
        pii = blk[i * gmax + i];
        pij = blk[j * gmax + j];
      } else {
        rho = pl[i] * pl[j];
      }
      float we;
      if (!rule_term(rule, wmax, rl[i] - rl[j], rho, pii, pij, &w, &we, &v)) {
        w = 0.0f;
        v = 0.0f;
        bad_rho = true;
      }
    }
    W[idx] = w;
    V[idx] = v;
  }
  if (bad_rho && chunk == 0) raise_status(d_status, PAIR_ST_RHO_RANGE);
  __syncthreads();

  // Indicators of this lane's replicate.
  const int64_t rloc = chunk * kCoefThreads + tid;
  const bool valid = rloc < R;
  uint64_t bits = 0;
  if (valid) {
    const uint64_t rg = (uint64_t)(rep0 + rloc);
    for (int blk = 0; blk * 4 < g; ++blk) {
      const Philox4x64 x =
          philox4x64_10(rg, (uint64_t)(pbase + b), (uint64_t)blk, 0ull, seed, 0ull);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int i = blk * 4 + q;
        if (i < g) {
          const float pv = pl[i];
          const uint64_t u = x.w[q] >> 32;
          if (p_in_range(pv) && u < inclusion_threshold(pv)) bits |= 1ull << i;
        }
      }
    }
  }
  const int k = __popcll(bits);
  if (valid && edge_count != nullptr) edge_count[b * R + rloc] = k * (k - 1) / 2;
  if (k < 2) bits = 0;   // fewer than two completed vertices: A~ = 0

  // Fold: A~_i = J_i (1/(2N)) sum_j J_j W_ij, in ascending j; then centre over
  // the completed vertices (not for the marginal-only rule, whose fold is not
  // antisymmetric).  2N = G (G - 1), or k (k - 1) for the observed-edge mean,
  // or sum_{i, j observed} 1/rho_ij for the self-normalised rule.
  float m[KP], d[KP];
#pragma unroll
  for (int j = 0; j < KP; ++j) m[j] = ((bits >> j) & 1ull) ? 1.0f : 0.0f;
  float den = (float)(g * (g - 1));
  if (rule == PAIR_RULE_RATIO_KE) den = (float)(k * (k - 1));
  if (rule == PAIR_RULE_SELFNORM) {
    float n2 = 0.0f;
#pragma unroll
    for (int i = 0; i < KP; ++i) {
      float c = 0.0f;
#pragma unroll
      for (int j0 = 0; j0 < KP; j0 += 4) {
        const float4 v4 = *reinterpret_cast<const float4*>(&V[i * KP + j0]);
        c = __builtin_fmaf(m[j0], v4.x, c);
        c = __builtin_fmaf(m[j0 + 1], v4.y, c);
        c = __builtin_fmaf(m[j0 + 2], v4.z, c);
        c = __builtin_fmaf(m[j0 + 3], v4.w, c);
      }
      n2 = __builtin_fmaf(m[i], c, n2);
    }
    den = n2;
  }
  float sum_obs = 0.0f;
#pragma unroll
  for (int i = 0; i < KP; ++i) {
    float c = 0.0f;
#pragma unroll
    for (int j0 = 0; j0 < KP; j0 += 4) {
      const float4 w4 = *reinterpret_cast<const float4*>(&W[i * KP + j0]);
      c = __builtin_fmaf(m[j0], w4.x, c);
      c = __builtin_fmaf(m[j0 + 1], w4.y, c);
      c = __builtin_fmaf(m[j0 + 2], w4.z, c);
      c = __builtin_fmaf(m[j0 + 3], w4.w, c);
    }
    const float ai = m[i] != 0.0f ? c / den : 0.0f;
    sum_obs += ai;
    d[i] = ai;
  }
  const float mean = (k >= 2 && rule != PAIR_RULE_MARGINAL) ? sum_obs / (float)k : 0.0f;
#pragma unroll
  for (int i = 0; i < KP; ++i) d[i] = valid ? (m[i] != 0.0f ? d[i] - mean : 0.0f) - af[i] : 0.0f;

  if (valid) {
    float* drow = delta + (b * rrows + rloc) * KP;
#pragma unroll
    for (int i0 = 0; i0 < KP; i0 += 4)
      *reinterpret_cast<float4*>(drow + i0) = make_float4(d[i0], d[i0 + 1], d[i0 + 2], d[i0 + 3]);
  }

  // Fixed-order column sums: a wave sum (DPP steps within rows of 16 lanes,
  // then the four rows in order) in each wave, then the waves in order.
#pragma unroll
  for (int i = 0; i < KP; ++i) {
    const float sw = wave_sum(d[i]);
    if (lane == 0) wsum[wave][i] = sw;
  }
  __syncthreads();
  if (tid < g) {
    float sc = 0.0f;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) sc += wsum[w][tid];
    dsum[(b * nwg + chunk) * gmax + tid] = sc;
  }
}

// ---------------------------------------------------------------------------
// 2. delta_bar row and zero padding.
// ---------------------------------------------------------------------------
constexpr int kPrepThreads = 256;

// Live prompts: live[0] = their count, live[1 ..] = their indices in
// ascending order, live[1 + B + b] = 1 if prompt b is live, else 0.  A prompt
// is live when its group is valid and some reward differs from the first (a
// NaN reward counts as different).  One workgroup, chunks of 256 prompts, a
// ballot prefix count within each wave and the waves in order.
__device__ void list_live_prompts(int64_t B, int64_t nv, int32_t gmax,
                                  const int64_t* __restrict__ offsets,
                                  const float* __restrict__ rewards, int32_t* __restrict__ live) {
  constexpr int kWaves = kPrepThreads / kWave;
  __shared__ int32_t wcount[kWaves];
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = tid / kWave;
  int32_t base = 0;
  for (int64_t c0 = 0; c0 < B; c0 += kPrepThreads) {
    const int64_t b = c0 + tid;
    bool lv = false;
    if (b < B) {
      int64_t o0, g;
      if (prompt_bounds(offsets, b, nv, 2, gmax, &o0, &g, nullptr, false)) {
        const float r0 = rewards[o0];
        for (int64_t i = 1; i < g; ++i) lv = lv || !(rewards[o0 + i] == r0);
      }
      live[1 + B + b] = lv ? 1 : 0;
    }
    const uint64_t m = __ballot(lv);
    const int before = __popcll(m & ((1ull << lane) - 1ull));
    if (lane == 0) wcount[wave] = __popcll(m);
    __syncthreads();
    int32_t off = base, tot = 0;
    for (int w = 0; w < kWaves; ++w) {
      if (w < wave) off += wcount[w];
      tot += wcount[w];
    }
    if (lv) live[1 + off + before] = (int32_t)b;
    base += tot;
    __syncthreads();
  }
  if (tid == 0) live[0] = base;
}

__global__ __launch_bounds__(kPrepThreads) void audit_prep_kernel(
    int64_t B, int64_t nv, int32_t gmax, int kp, const int64_t* __restrict__ offsets,
    const float* __restrict__ rewards, int64_t R, int64_t rbar, int64_t nwg, int64_t rrows,
    const float* __restrict__ dsum, float* __restrict__ delta, int32_t* __restrict__ live) {
  const int64_t b = blockIdx.x;
  if (b == B) {
    list_live_prompts(B, nv, gmax, offsets, rewards, live);
    return;
  }
  int64_t o0, g;
  if (!prompt_bounds(offsets, b, nv, 2, gmax, &o0, &g, nullptr, false)) return;
  const int tid = threadIdx.x;
  if (tid < kp) {
    float v = 0.0f;
    if (tid < g) {
      float s = 0.0f;
      for (int64_t c = 0; c < nwg; ++c) s += dsum[(b * nwg + c) * gmax + tid];
      v = s / (float)R;
    }
    delta[(b * rrows + rbar) * kp + tid] = v;
  }
  // Zero rows: R .. rbar-1 (padding of the replicate tiles) and the rest of
  // the delta_bar tile.
  const int64_t pad1 = (rbar - R) * kp;
  float* dst1 = delta + (b * rrows + R) * kp;
  for (int64_t idx = tid; idx < pad1; idx += blockDim.x) dst1[idx] = 0.0f;
  const int64_t pad2 = (rrows - rbar - 1) * kp;
  float* dst2 = delta + (b * rrows + rbar + 1) * kp;
  for (int64_t idx = tid; idx < pad2; idx += blockDim.x) dst2[idx] = 0.0f;
}

// ---------------------------------------------------------------------------
// 3. Matrix-core contraction with the squared-norm epilogue.
//
// A workgroup owns one prompt and one slice of score columns.  It converts
// the slice to rescaled fp16 once, keeps it in LDS ([d][i], transposed, one
// skew row per 8), and then every replicate row of the prompt sweeps over it.
//
// v_mfma_f32_32x32x16_f16 (wave64): lane l holds row l % 32 of A and column
// l % 32 of B, K elements 8*(l/32) .. 8*(l/32)+7 of each 16-wide K step; the
// 16 accumulators of lane l hold column l % 32 and rows 8*(v/4) + 4*(l/32) +
// (v%4).  Here A = the S_b slice transposed (rows = score columns d) and
// B = delta^T (columns = replicates r), so all 16 accumulators of a lane
// belong to ONE replicate (l % 32): the squared norm is summed inside the
// lane, and lanes l and l + 32 (the two halves of the d rows) are combined
// once per tile.  Two accumulator sets alternate between 32-column steps so
// the matrix instruction of step s issues next to the FMAs squaring step s-1.
// ---------------------------------------------------------------------------
template <int KS>
__global__ __launch_bounds__(kMfmaThreads) __attribute__((amdgpu_waves_per_eu(KS == 1 ? 4 : 2))) void audit_mfma_kernel(
    int64_t B, int64_t nv, int32_t gmax, const int64_t* __restrict__ offsets, int64_t D,
    const uint16_t* __restrict__ scores, int64_t ld, int64_t rrows, int64_t ntiles,
    int64_t nslices, const float* __restrict__ delta, const int32_t* __restrict__ live,
    float* __restrict__ epart, int32_t* d_status) {
  constexpr int KP = 16 * KS;
  constexpr int SW = slice_cols(KS);
  constexpr int kSteps = SW / kTile;
  constexpr int kRowsLds = SW + SW / 8;
  constexpr int kPieces = KP * (SW / 8);    // 16-byte pieces of the slice
  constexpr int kPerThread = (kPieces + kMfmaThreads - 1) / kMfmaThreads;
  __shared__ __align__(16) uint16_t S_lds[kRowsLds * KP];
  __shared__ float bar_part[kMfmaWaves];
  __shared__ float wbar[KP];
  __shared__ int fbar;
  __shared__ uint32_t row_max[KP];
  __shared__ int32_t ex[KP];
  static_assert(kSteps % 2 == 0 && kSteps >= 4 && SW % kMfmaThreads == 0 && KP <= kWave,
                "slice shape");

  // XCD-aware placement: hardware round-robins workgroup ids over 8 XCDs.
  // The grid has room for every prompt; the n live (prompt, slice) pairs are
  // split into 8 contiguous ranges of ceil(n / 8), one per XCD, so the
  // workgroups of a prompt share that XCD's L2 for the delta rows and the
  // XCDs get equal work.  Workgroups beyond the live work exit at once.
  const int64_t n_live = (int64_t)live[0] * nslices;
  const int64_t per_xcd = (n_live + 7) / 8;
  const int64_t j = blockIdx.x / 8;
  if (j >= per_xcd) return;
  const int64_t L = (int64_t)(blockIdx.x % 8) * per_xcd + j;
  if (L >= n_live) return;
  const int64_t b = live[1 + L / nslices];
  const int64_t sl = L - (L / nslices) * nslices;
  int64_t o0, g;
  if (!prompt_bounds(offsets, b, nv, 2, gmax, &o0, &g, nullptr, false)) return;

  const int tid = threadIdx.x;
  const int wave = tid / kWave;
  const int lane = tid & (kWave - 1);
  const int64_t col0 = sl * (int64_t)SW;
  if (tid < KP) row_max[tid] = 0u;
  __syncthreads();

  // Stage the slice in two passes.  Pass 1 loads the 16-byte pieces
  // (piece p -> row i = p % KP, columns d0 .. d0 + 7 with d0 = 8 (p / KP);
  // columns past D and rows past G read as zero) and finds each row's largest
  // magnitude within the slice as bf16 bits (integer order = magnitude
  // order).  Pass 2 rescales row i by 2^-e_i, 2^e_i <= max |s_i| < 2^(e_i+1),
  // and converts to fp16 with round-to-nearest-even: exact for every value
  // within 2^17 of that maximum (8 significant bits fit in fp16's normal
  // range and its subnormals down to 2^-17); smaller values land on fp16's
  // subnormal grid of 2^-24, an absolute error of at most 2^-25 of the row's
  // slice maximum.
  uint4 pv[kPerThread];
  {
    const uint16_t* sb = scores + o0 * ld;
    int cur = -1;
    uint32_t m = 0;
#pragma unroll
    for (int t = 0; t < kPerThread; ++t) {
      const int pidx = tid + t * kMfmaThreads;
      uint4 v = make_uint4(0u, 0u, 0u, 0u);
      if (pidx < kPieces) {
        const int i = pidx % KP;
        const int64_t col = col0 + 8 * (pidx / KP);
        if (i < g) {
          const uint16_t* src = sb + (int64_t)i * ld + col;
          if (col + 8 <= D) {
            v = load_nt16(src);
          } else if (col < D) {
            uint16_t h[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) h[e] = (col + e < D) ? src[e] : (uint16_t)0;
            v.x = (uint32_t)h[0] | ((uint32_t)h[1] << 16);
            v.y = (uint32_t)h[2] | ((uint32_t)h[3] << 16);
            v.z = (uint32_t)h[4] | ((uint32_t)h[5] << 16);
            v.w = (uint32_t)h[6] | ((uint32_t)h[7] << 16);
          }
        }
        const uint32_t w4[4] = {v.x, v.y, v.z, v.w};
        uint32_t mp = 0;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const uint32_t lo = w4[k] & 0x7fffu, hi = (w4[k] >> 16) & 0x7fffu;
          mp = lo > mp ? lo : mp;
          mp = hi > mp ? hi : mp;
        }
        if (i != cur) {
          if (cur >= 0 && m != 0u) atomicMax(&row_max[cur], m);
          cur = i;
          m = 0;
        }
        m = mp > m ? mp : m;
      }
      pv[t] = v;
    }
    if (cur >= 0 && m != 0u) atomicMax(&row_max[cur], m);
  }
  __syncthreads();
  // Per-row exponents, and the delta_bar row rescaled like a replicate row:
  // w_i = delta_bar_i 2^(e_i - f) with f putting the largest entry in [1, 2).
  // The first wave holds all KP rows; its shuffles run on every lane.
  const float* dbar = delta + (b * rrows + (ntiles - 1) * kTile) * KP;
  if (wave == 0) {
    float y = 0.0f;
    if (lane < KP) {
      const uint32_t mm = row_max[lane];
      int32_t e = 0;
      if (mm >= 0x7f80u) {               // inf or NaN in the row
        raise_status(d_status, PAIR_ST_NONFINITE);
      } else if (mm != 0u) {
        e = (int32_t)(mm >> 7) - 127;    // -127 for a row of subnormals
      }
      ex[lane] = e;
      y = ldexpf(dbar[lane], e);
    }
    float m = fabsf(y);
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) m = fmaxf(m, __shfl_xor(m, o, kWave));
    const int f = m > 0.0f ? ilogbf(m) : 0;
    if (lane < KP) wbar[lane] = ldexpf(y, -f);
    if (lane == 0) fbar = f;
  }
  __syncthreads();
#pragma unroll
  for (int t = 0; t < kPerThread; ++t) {
    const int pidx = tid + t * kMfmaThreads;
    if (pidx < kPieces) {
      const int i = pidx % KP;
      const int d0 = 8 * (pidx / KP);
      const int ne = -ex[i];
      const uint32_t w4[4] = {pv[t].x, pv[t].y, pv[t].z, pv[t].w};
      uint16_t* dst = &S_lds[(d0 + d0 / 8) * KP + i];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const float lo = ldexpf(bf16lo_to_f32(w4[k]), ne), hi = ldexpf(bf16hi_to_f32(w4[k]), ne);
        dst[(2 * k) * KP] = __builtin_bit_cast(uint16_t, (_Float16)lo);
        dst[(2 * k + 1) * KP] = __builtin_bit_cast(uint16_t, (_Float16)hi);
      }
    }
  }
  __syncthreads();

  // A fragment (score columns) of step s: lane l reads column 32 s + l % 32 and
  // the 8 rows 8 (l / 32) .. +7 of every 16-row K step.
  const int dl = lane & 31;
  const int aoff = (dl + dl / 8) * KP + 8 * (lane >> 5);
  auto read_a = [&](int step, f16x8_t (&Af)[KS]) {
    const uint16_t* src = &S_lds[step * (kTile + kTile / 8) * KP + aoff];
#pragma unroll
    for (int s = 0; s < KS; ++s)
      Af[s] = __builtin_bit_cast(f16x8_t, *reinterpret_cast<const uint4*>(src + 16 * s));
  };
  // B fragment (replicate rows) of tile t: lane l holds replicate row
  // 32 t + l % 32, K entries 16 s + 8 (l / 32) + j, rescaled by 2^(e_i - f_r)
  // with f_r putting the row's largest entry in [1, 2).
  auto load_b = [&](int64_t t, f16x8_t (&Bf)[KS], int& f) {
    const int kh = 8 * (lane >> 5);
    const float* src = delta + (b * rrows + t * kTile + dl) * KP + kh;
    float y[KS][8];
    float m = 0.0f;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const float4 u0 = *reinterpret_cast<const float4*>(src + 16 * s);
      const float4 u1 = *reinterpret_cast<const float4*>(src + 16 * s + 4);
      const float x[8] = {u0.x, u0.y, u0.z, u0.w, u1.x, u1.y, u1.z, u1.w};
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        y[s][j] = ldexpf(x[j], ex[16 * s + kh + j]);
        m = fmaxf(m, fabsf(y[s][j]));
      }
    }
    m = fmaxf(m, __shfl_xor(m, 32, kWave));   // the row's other K half
    f = m > 0.0f ? ilogbf(m) : 0;
#pragma unroll
    for (int s = 0; s < KS; ++s)
#pragma unroll
      for (int j = 0; j < 8; ++j) Bf[s][j] = (_Float16)ldexpf(y[s][j], -f);
  };

  // Sweep a pair of tiles over all steps of the slice; returns each tile's
  // sum of squares for replicate row l % 32 (lanes l and l + 32 combined).
  auto sweep = [&](const f16x8_t (&Bt)[kPair][KS], float (&out)[kPair]) {
    f32x16_t accA[kPair], accB[kPair];
    float sq[kPair][4];
#pragma unroll
    for (int q = 0; q < kPair; ++q)
#pragma unroll
      for (int k = 0; k < 4; ++k) sq[q][k] = 0.0f;
    auto first = [&](const f16x8_t (&Af)[KS], f32x16_t (&acc)[kPair]) {
#pragma unroll
      for (int q = 0; q < kPair; ++q) {
        f32x16_t a;
#pragma unroll
        for (int v = 0; v < 16; ++v) a[v] = 0.0f;
#pragma unroll
        for (int s = 0; s < KS; ++s)
          a = __builtin_amdgcn_mfma_f32_32x32x16_f16(Af[s], Bt[q][s], a, 0, 0, 0);
        acc[q] = a;
      }
    };
    auto step = [&](const f16x8_t (&Af)[KS], f32x16_t (&acc)[kPair], const f32x16_t (&prev)[kPair]) {
#pragma unroll
      for (int q = 0; q < kPair; ++q) {
        f32x16_t a;
#pragma unroll
        for (int v = 0; v < 16; ++v) a[v] = 0.0f;
#pragma unroll
        for (int s = 0; s < KS; ++s)
          a = __builtin_amdgcn_mfma_f32_32x32x16_f16(Af[s], Bt[q][s], a, 0, 0, 0);
        acc[q] = a;
#pragma unroll
        for (int v = 0; v < 16; ++v)
          sq[q][v & 3] = __builtin_fmaf(prev[q][v], prev[q][v], sq[q][v & 3]);
        __builtin_amdgcn_sched_group_barrier(0x008, KS, 0);
        __builtin_amdgcn_sched_group_barrier(0x002, 16, 0);
      }
      __builtin_amdgcn_sched_barrier(0);
    };
    // Step 0 has no previous step to square; steps 1 .. kSteps-1 each square
    // the one before, and the last is squared after the loop.
    f16x8_t A0[KS], A1[KS];
    read_a(0, A0);
    read_a(1, A1);
    first(A0, accA);
    read_a(2, A0);
    step(A1, accB, accA);
    for (int st = 2; st < kSteps; st += 2) {
      read_a(st + 1, A1);
      step(A0, accA, accB);
      if (st + 2 < kSteps) read_a(st + 2, A0);
      step(A1, accB, accA);
    }
#pragma unroll
    for (int q = 0; q < kPair; ++q) {
#pragma unroll
      for (int v = 0; v < 16; ++v) sq[q][v & 3] = __builtin_fmaf(accB[q][v], accB[q][v], sq[q][v & 3]);
      float tot = (sq[q][0] + sq[q][1]) + (sq[q][2] + sq[q][3]);
      tot += __shfl_xor(tot, 32, kWave);
      out[q] = tot;
    }
  };

  // The delta_bar row on the vector units: one dot product per score column
  // of the slice (KP FMAs against the fp16 slice in LDS), squares summed per
  // thread, then over the wave and the waves in a fixed order.  It is one row
  // against the slice's 2 x (R rounded up to 64) replicate-row sweeps.
  {
    float bsq = 0.0f;
    for (int c = tid; c < SW; c += kMfmaThreads) {
      const int cl = c % kTile;
      const uint16_t* src = &S_lds[(c / kTile) * (kTile + kTile / 8) * KP + (cl + cl / 8) * KP];
      float y = 0.0f;
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        const uint4 h0 = *reinterpret_cast<const uint4*>(src + 16 * s);
        const uint4 h1 = *reinterpret_cast<const uint4*>(src + 16 * s + 8);
        const uint32_t hw[8] = {h0.x, h0.y, h0.z, h0.w, h1.x, h1.y, h1.z, h1.w};
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const float lo = (float)__builtin_bit_cast(_Float16, (uint16_t)(hw[j] & 0xffffu));
          const float hi = (float)__builtin_bit_cast(_Float16, (uint16_t)(hw[j] >> 16));
          y = __builtin_fmaf(wbar[16 * s + 2 * j], lo, y);
          y = __builtin_fmaf(wbar[16 * s + 2 * j + 1], hi, y);
        }
      }
      bsq = __builtin_fmaf(y, y, bsq);
    }
#pragma unroll
    for (int o = kWave / 2; o >= 1; o >>= 1) bsq += __shfl_xor(bsq, o, kWave);
    if (lane == 0) bar_part[wave] = bsq;
  }

  float* eo = epart + (b * nslices + sl) * rrows;
  // Replicate tiles (an even count) in pairs, round-robin over the waves, so
  // every replicate's partial is formed the same way whatever R and the first
  // replicate index.
  const int64_t per_round = (int64_t)kPair * kMfmaWaves;
  const int64_t nmain = ntiles - 1;
  for (int64_t t0 = (int64_t)wave * kPair; t0 < nmain; t0 += per_round) {
    f16x8_t Bt[kPair][KS];
    int fr[kPair];
#pragma unroll
    for (int q = 0; q < kPair; ++q) load_b(t0 + q, Bt[q], fr[q]);
    float out[kPair];
    sweep(Bt, out);
    if (lane < kTile) {
#pragma unroll
      for (int q = 0; q < kPair; ++q) eo[(t0 + q) * kTile + lane] = ldexpf(out[q], 2 * fr[q]);
    }
  }
  __syncthreads();
  if (tid == 0) {
    float tot = 0.0f;
    for (int w = 0; w < kMfmaWaves; ++w) tot += bar_part[w];
    eo[nmain * kTile] = ldexpf(tot, 2 * fbar);
  }
}

// ---------------------------------------------------------------------------
// 4. Fixed-order reductions.  audit_sqerr: one thread per (prompt, replicate
//    row) sums the per-slice partials in slice order (fp32) into e_r, and
//    each workgroup writes the fp64 sum of its e_r; audit_final: per prompt,
//    MSE = (sum of those partials in order) / R and bias = sqrt(e of delta_bar).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kSqThreads) void audit_sqerr_kernel(
    int64_t B, int64_t nv, int32_t gmax, const int64_t* __restrict__ offsets, int64_t R,
    int64_t rbar, int64_t rrows, int64_t nslices, int64_t nsq, const float* __restrict__ epart,
    const int32_t* __restrict__ live, double* __restrict__ rpart, float* __restrict__ ebar,
    float* __restrict__ rep_sqerr) {
  __shared__ double part[kSqThreads / kWave];
  const int64_t b = blockIdx.x / nsq;
  const int64_t c = blockIdx.x - b * nsq;
  int64_t o0, g;
  if (!prompt_bounds(offsets, b, nv, 2, gmax, &o0, &g, nullptr, false)) return;
  const int64_t r = c * kSqThreads + threadIdx.x;
  const bool is_live = live[1 + B + b] != 0;   // not live: every delta_r is 0, so e_r = 0
  float e = 0.0f;
  if (r <= R && is_live) {
    const float* eb = epart + b * nslices * rrows + (r < R ? r : rbar);
    int64_t k = 0;
    for (; k + 8 <= nslices; k += 8) {
      float v[8];
#pragma unroll
      for (int q = 0; q < 8; ++q) v[q] = eb[(k + q) * rrows];
#pragma unroll
      for (int q = 0; q < 8; ++q) e += v[q];
    }
    for (; k < nslices; ++k) e += eb[k * rrows];
  }
  if (r < R && rep_sqerr != nullptr) rep_sqerr[b * R + r] = e;
  if (r == R) ebar[b] = e;
  double s = r < R ? (double)e : 0.0;
#pragma unroll
  for (int m = 1; m < kWave; m <<= 1) s += __shfl_xor(s, m, kWave);
  const int wave = threadIdx.x / kWave;
  if ((threadIdx.x & (kWave - 1)) == 0) part[wave] = s;
  __syncthreads();
  if (threadIdx.x == 0) {
    double t = 0.0;
    for (int w = 0; w < kSqThreads / kWave; ++w) t += part[w];
    rpart[b * nsq + c] = t;
  }
}

__global__ __launch_bounds__(256) void audit_final_kernel(
    int64_t B, int64_t nv, int32_t gmax, const int64_t* __restrict__ offsets, int64_t R,
    int64_t nsq, const double* __restrict__ rpart, const float* __restrict__ ebar,
    double* __restrict__ mse, double* __restrict__ bias_norm) {
  const int64_t b = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= B) return;
  int64_t o0, g;
  if (!prompt_bounds(offsets, b, nv, 2, gmax, &o0, &g, nullptr, false)) return;
  double t = 0.0;
  for (int64_t c = 0; c < nsq; ++c) t += rpart[b * nsq + c];
  mse[b] = t / (double)R;
  bias_norm[b] = sqrt((double)ebar[b]);
}

// ---------------------------------------------------------------------------
// Update direction (Sec. 6.2 audit metrics; the Cosine column of the audit
// matrix, App. E).  Replicate r's estimate is g_r = u_r S_b with
// u_r = delta_r + a (its fold's coefficients) and the target is t = a S_b, so
// with the fp64 Gram matrix K = S_b S_b^T
//     cos_r = u_r K a / sqrt(u_r K u_r * a K a),
// taken as 0 when either quadratic form is not positive (a draw with no
// observed edge has u_r = 0 exactly; a prompt with equal rewards has a = 0).
// A workgroup owns one prompt and 256 replicates (one per thread) and writes
// the fixed-order sum of its cosines; a second kernel adds the chunks in
// order.  a is recomputed exactly as audit_coeffs_kernel computes it, so
// delta_r + a restores the fold's coefficients to within one fp32 rounding.
// ---------------------------------------------------------------------------
constexpr int kCosThreads = 256;

template <int KP>
__global__ __launch_bounds__(kCosThreads) void audit_cosine_kernel(
    int64_t B, int64_t nv, int32_t gmax, const int64_t* __restrict__ offsets,
    const float* __restrict__ rewards, int64_t R, int64_t nwg, int64_t rrows,
    const float* __restrict__ delta, const double* __restrict__ gram, double* __restrict__ cpart,
    double* __restrict__ target_norm) {
  constexpr int kWaves = kCosThreads / kWave;
  __shared__ double K[KP * KP];
  __shared__ double ka[KP];
  __shared__ float af[KP];
  __shared__ double red[kWaves];
  __shared__ double tt_s;
  const int64_t b = blockIdx.x / nwg;
  const int64_t chunk = blockIdx.x - b * nwg;
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = tid / kWave;
  int64_t o0, g64;
  if (!prompt_bounds(offsets, b, nv, 2, gmax, &o0, &g64, nullptr, false)) return;
  const int g = (int)g64;

  if (wave == 0) {
    const float r_i = lane < g ? rewards[o0 + lane] : 0.0f;
    const float a_full = complete_pair_coeff(r_i, lane, g);
    if (lane < KP) af[lane] = a_full;
  }
  for (int idx = tid; idx < KP * KP; idx += kCosThreads) {
    const int i = idx / KP, j = idx - i * KP;
    K[idx] = (i < g && j < g) ? gram[(b * gmax + i) * (int64_t)gmax + j] : 0.0;
  }
  __syncthreads();
  if (tid < KP) {
    double v = 0.0;
    for (int j = 0; j < g; ++j) v += K[tid * KP + j] * (double)af[j];
    ka[tid] = v;
  }
  __syncthreads();
  if (tid == 0) {
    double t2 = 0.0;
    for (int i = 0; i < g; ++i) t2 += (double)af[i] * ka[i];
    tt_s = t2;
    if (chunk == 0) target_norm[b] = t2 > 0.0 ? sqrt(t2) : 0.0;
  }
  __syncthreads();
  const double tt = tt_s;

  const int64_t rloc = chunk * kCosThreads + tid;
  double cosv = 0.0;
  if (rloc < R && tt > 0.0) {
    const float* drow = delta + (b * rrows + rloc) * KP;
    double u[KP];
#pragma unroll
    for (int i0 = 0; i0 < KP; i0 += 4) {
      const float4 v4 = *reinterpret_cast<const float4*>(drow + i0);
      u[i0] = (double)(v4.x + af[i0]);
      u[i0 + 1] = (double)(v4.y + af[i0 + 1]);
      u[i0 + 2] = (double)(v4.z + af[i0 + 2]);
      u[i0 + 3] = (double)(v4.w + af[i0 + 3]);
    }
    double uka = 0.0, uku = 0.0;
    for (int i = 0; i < g; ++i) {
      double ki = 0.0;
#pragma unroll
      for (int j = 0; j < KP; ++j) ki += K[i * KP + j] * u[j];
      double ui = 0.0;
#pragma unroll
      for (int q = 0; q < KP; ++q) ui = q == i ? u[q] : ui;
      uku += ui * ki;
      uka += ui * ka[i];
    }
    if (uku > 0.0) cosv = uka / sqrt(uku * tt);
  }
  // Fixed-order sum: butterfly within each wave, then the waves in order.
#pragma unroll
  for (int m = 1; m < kWave; m <<= 1) cosv += __shfl_xor(cosv, m, kWave);
  if (lane == 0) red[wave] = cosv;
  __syncthreads();
  if (tid == 0) {
    double sum = 0.0;
    for (int w = 0; w < kWaves; ++w) sum += red[w];
    cpart[b * nwg + chunk] = sum;
  }
}

__global__ __launch_bounds__(256) void audit_cosine_final_kernel(
    int64_t B, int64_t nv, int32_t gmax, const int64_t* __restrict__ offsets, int64_t R,
    int64_t nwg, const double* __restrict__ cpart, double* __restrict__ cosine) {
  const int64_t b = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= B) return;
  int64_t o0, g;
  if (!prompt_bounds(offsets, b, nv, 2, gmax, &o0, &g, nullptr, false)) return;
  double sum = 0.0;
  for (int64_t c = 0; c < nwg; ++c) sum += cpart[b * nwg + c];
  cosine[b] = sum / (double)R;
}

}  // namespace

size_t audit_workspace_bytes(int64_t B, int32_t gmax, int64_t D, int64_t R) {
  return audit_layout(B, gmax, D, R).total;
}

// Workspace of launch_audit_direction: the Gram slice partials, the fp64
// Gram matrices, the replicate deviations and their partial sums (as in the
// audit), and the per-chunk cosine sums.
struct DirectionLayout {
  size_t gram_part_off, gram_off, delta_off, dsum_off, cpart_off, total;
};

DirectionLayout direction_layout(int64_t B, int32_t gmax, int64_t D, int64_t R) {
  const AuditLayout A = audit_layout(B, gmax, D, R);
  DirectionLayout L;
  size_t off = 0;
  L.gram_part_off = off;
  off += (size_t)round_up((int64_t)exact_workspace_bytes(B, gmax, D), 256);
  L.gram_off = off;
  off += (size_t)round_up(B * (int64_t)gmax * gmax * 8, 256);
  L.delta_off = off;
  off += (size_t)round_up(B * A.rrows * A.kp * 4, 256);
  L.dsum_off = off;
  off += (size_t)round_up(B * A.nwg * gmax * 4, 256);
  L.cpart_off = off;
  off += (size_t)round_up(B * A.nwg * 8, 256);
  L.total = off;
  return L;
}

size_t direction_workspace_bytes(int64_t B, int32_t gmax, int64_t D, int64_t R) {
  return direction_layout(B, gmax, D, R).total;
}

int launch_audit_direction(int64_t B, int64_t nv, int32_t gmax, const int64_t* offsets, int64_t D,
                           const void* scores, int64_t ld, const float* rewards, const float* p,
                           const float* pi_w, int32_t rule, float wmax, uint64_t seed,
                           int64_t rep0, int64_t R, double* cosine, double* target_norm,
                           void* workspace, int32_t* d_status, hipStream_t stream) {
  const AuditLayout A = audit_layout(B, gmax, D, R);
  const DirectionLayout L = direction_layout(B, gmax, D, R);
  unsigned char* ws = static_cast<unsigned char*>(workspace);
  double* gram = reinterpret_cast<double*>(ws + L.gram_off);
  float* delta = reinterpret_cast<float*>(ws + L.delta_off);
  float* dsum = reinterpret_cast<float*>(ws + L.dsum_off);
  double* cpart = reinterpret_cast<double*>(ws + L.cpart_off);

  int st = launch_gram(B, nv, gmax, offsets, D, scores, ld, gram, ws + L.gram_part_off, d_status,
                       stream);
  if (st != PAIR_OK) return st;
  const int64_t grid = B * A.nwg;
  if (grid > 0x7fffffffLL) return PAIR_ERANGE;
#define PAIR_DIR(KP_)                                                                           \
  hipLaunchKernelGGL(audit_coeffs_kernel<KP_>, dim3((unsigned)grid), dim3(kCoefThreads), 0,      \
                     stream, B, nv, gmax, offsets, rewards, p, pi_w, rule, wmax, seed, rep0, 0,  \
                     R, A.nwg, A.rrows, delta, dsum, nullptr, d_status);                        \
  if (hipGetLastError() != hipSuccess) return PAIR_EHIP;                                        \
  hipLaunchKernelGGL(audit_cosine_kernel<KP_>, dim3((unsigned)grid), dim3(kCosThreads), 0,       \
                     stream, B, nv, gmax, offsets, rewards, R, A.nwg, A.rrows, delta, gram,       \
                     cpart, target_norm)
  switch (A.ks) {
    case 1: PAIR_DIR(16); break;
    case 2: PAIR_DIR(32); break;
    case 3: PAIR_DIR(48); break;
    default: PAIR_DIR(64); break;
  }
#undef PAIR_DIR
  if (hipGetLastError() != hipSuccess) return PAIR_EHIP;
  hipLaunchKernelGGL(audit_cosine_final_kernel, dim3((unsigned)((B + 255) / 256)), dim3(256), 0,
                     stream, B, nv, gmax, offsets, R, A.nwg, cpart, cosine);
  return hipGetLastError() == hipSuccess ? PAIR_OK : PAIR_EHIP;
}

int launch_audit(int64_t B, int64_t nv, int32_t gmax, const int64_t* offsets, int64_t D,
                 const void* scores, int64_t ld, const float* rewards, const float* p,
                 const float* pi_w, int32_t rule, float wmax, uint64_t seed, int64_t rep0,
                 int64_t pbase, int64_t R, double* mse, double* bias_norm, float* rep_sqerr,
                 int32_t* edge_count, void* workspace, int32_t* d_status, hipStream_t stream) {
  const AuditLayout L = audit_layout(B, gmax, D, R);
  unsigned char* ws = static_cast<unsigned char*>(workspace);
  float* delta = reinterpret_cast<float*>(ws + L.delta_off);
  float* epart = reinterpret_cast<float*>(ws + L.epart_off);
  float* dsum = reinterpret_cast<float*>(ws + L.dsum_off);
  double* rpart = reinterpret_cast<double*>(ws + L.rpart_off);
  float* ebar = reinterpret_cast<float*>(ws + L.ebar_off);
  int32_t* live = reinterpret_cast<int32_t*>(ws + L.live_off);
  const uint16_t* s = static_cast<const uint16_t*>(scores);

  // Every grid size is checked before the first launch.
  const int64_t coef_grid = B * L.nwg;
  const int64_t grid = round_up(B * L.nslices, 8);
  const int64_t sq_grid = B * L.nsq;
  if (coef_grid > 0x7fffffffLL || B + 1 > 0x7fffffffLL || grid > 0x7fffffffLL ||
      sq_grid > 0x7fffffffLL)
    return PAIR_ERANGE;
#define PAIR_AUDIT_COEFFS(KP_)                                                                  \
  hipLaunchKernelGGL(audit_coeffs_kernel<KP_>, dim3((unsigned)coef_grid), dim3(kCoefThreads), 0, \
                     stream, B, nv, gmax, offsets, rewards, p, pi_w, rule, wmax, seed, rep0,     \
                     pbase, R, L.nwg, L.rrows, delta, dsum, edge_count, d_status)
  switch (L.ks) {
    case 1: PAIR_AUDIT_COEFFS(16); break;
    case 2: PAIR_AUDIT_COEFFS(32); break;
    case 3: PAIR_AUDIT_COEFFS(48); break;
    default: PAIR_AUDIT_COEFFS(64); break;
  }
#undef PAIR_AUDIT_COEFFS
  if (hipGetLastError() != hipSuccess) return PAIR_EHIP;

  hipLaunchKernelGGL(audit_prep_kernel, dim3((unsigned)(B + 1)), dim3(kPrepThreads), 0, stream, B,
                     nv, gmax, L.kp, offsets, rewards, R, L.rbar, L.nwg, L.rrows, dsum, delta,
                     live);
  if (hipGetLastError() != hipSuccess) return PAIR_EHIP;

#define PAIR_AUDIT_MFMA(KS_)                                                                   \
  hipLaunchKernelGGL(audit_mfma_kernel<KS_>, dim3((unsigned)grid), dim3(kMfmaThreads), 0, stream, \
                     B, nv, gmax, offsets, D, s, ld, L.rrows, L.ntiles, L.nslices, delta, live,   \
                     epart, d_status)
  switch (L.ks) {
    case 1: PAIR_AUDIT_MFMA(1); break;
    case 2: PAIR_AUDIT_MFMA(2); break;
    case 3: PAIR_AUDIT_MFMA(3); break;
    default: PAIR_AUDIT_MFMA(4); break;
  }
#undef PAIR_AUDIT_MFMA
  if (hipGetLastError() != hipSuccess) return PAIR_EHIP;

  hipLaunchKernelGGL(audit_sqerr_kernel, dim3((unsigned)sq_grid), dim3(kSqThreads), 0, stream, B,
                     nv, gmax, offsets, R, L.rbar, L.rrows, L.nslices, L.nsq, epart, live, rpart,
                     ebar, rep_sqerr);
  if (hipGetLastError() != hipSuccess) return PAIR_EHIP;
  hipLaunchKernelGGL(audit_final_kernel, dim3((unsigned)((B + 255) / 256)), dim3(256), 0, stream,
                     B, nv, gmax, offsets, R, L.nsq, rpart, ebar, mse, bias_norm);
  return hipGetLastError() == hipSuccess ? PAIR_OK : PAIR_EHIP;
}

}  // namespace pair
