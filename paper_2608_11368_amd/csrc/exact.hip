// Exact design audit (paper Prop. 1; App. A "Design covariance"): the design
// bias and MSE of an estimator that is linear in the edge indicators, with no
// replicate draws.
//
// Such an estimator is g^ = (1/M) sum_e I_e v_e with edge vectors
//     v_ij = A_ij s_i + C_ij s_j,  A_ij = 1/2 (r_i - r_j) w_i,
//                                  C_ij = -1/2 (r_i - r_j) w_j
// (w from the edge-weight rule and the logged rho).  Under independent
// Bernoulli(p_i) vertices,
//     E g^ - t = sum_i beta_i s_i,
//         beta_i = (1/M) sum_{j != i} (p_i p_j A_ij - 1/2 (r_i - r_j)),
//     tr Cov g^ = (1/M^2) [ sum_{i<j} rho (1 - rho) <v_ij, v_ij>
//                 + sum_i sum_{j != k; j, k != i} p_i p_j p_k (1 - p_i) <v_ij, v_ik> ],
// and every inner product is a combination of entries of the Gram matrix
// K = S_b S_b^T.  So the audit is one G x G x D contraction per prompt on the
// matrix cores plus O(G^3) fp64 work:
//
//  1. gram_kernel    workgroup = (prompt, column slice), 4 waves.  With
//                    v_mfma_f32_16x16x32_bf16 the A fragment (rows of S) and
//                    the B fragment (columns of S^T) of a lane are the same
//                    registers, so K_partial = sum_k S[m][k] S[n][k] needs one
//                    16-byte fragment per row block per lane and step; only
//                    the upper triangle of row blocks is multiplied.  The
//                    slice is streamed in chunks of 512 columns: every wave
//                    loads whole 1 KB runs of its rows (coalesced), the chunk
//                    is staged in LDS (two buffers, rows skewed by 16 bytes),
//                    and lane l then reads the fragment of row 16 q + l % 16,
//                    columns 128 w + 32 t + 8 (l / 16) .. + 7 of wave w's
//                    part, step t = 0..3.  The loads of the next chunks (two
//                    ahead for G <= 16, one ahead above) are in flight while
//                    a chunk is multiplied.  The four waves are added in
//                    fixed order in LDS and the slice's fp32 partial Gram is
//                    written out.
//  2. exact_final_kernel  workgroup per prompt: K in fp64 (slices summed in
//                    order), the rule's coefficients, beta^T K beta and the
//                    covariance trace with a fixed-order reduction.
#include "common.hpp"
#include "launch.hpp"

namespace pair {

namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

constexpr int kGramThreads = 256;
constexpr int kGramWaves = kGramThreads / kWave;
constexpr int kStepCols = 128;                       // columns per wave step (4 matrix instructions)
constexpr int kChunkCols = kGramWaves * kStepCols;   // columns staged per chunk
constexpr int kChunkStride = kChunkCols + 8;         // LDS row stride (bf16), 16-byte skew
constexpr int kFinalThreads = 256;

__host__ __device__ inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

struct ExactLayout {
  int ks, kp;
  int64_t nsl;     // column slices per prompt
  int64_t slice;   // columns per slice (multiple of kChunkCols)
  size_t total;
};

ExactLayout exact_layout(int64_t B, int32_t gmax, int64_t D) {
  ExactLayout L;
  L.ks = (gmax + 15) / 16;
  L.kp = 16 * L.ks;
  // About 8192 workgroups over the batch, slices of at least one chunk.
  int64_t nsl = ceil_div(8192, B);
  const int64_t max_sl = ceil_div(D, kChunkCols);
  if (nsl > max_sl) nsl = max_sl;
  if (nsl < 1) nsl = 1;
  L.slice = ceil_div(ceil_div(D, nsl), kChunkCols) * kChunkCols;
  L.nsl = ceil_div(D, L.slice);
  L.total = (size_t)B * L.nsl * L.kp * L.kp * sizeof(float);
  return L;
}

template <int KS>
__global__ __launch_bounds__(kGramThreads) void gram_kernel(
    int64_t B, int64_t nv, int32_t gmax, const int64_t* __restrict__ offsets, int64_t D,
    const uint16_t* __restrict__ scores, int64_t ld, int64_t nsl, int64_t slice,
    float* __restrict__ part) {
  constexpr int KP = 16 * KS;
  constexpr int kAhead = KS == 1 ? 2 : 1;        // chunks whose loads are in flight
  constexpr int kRows = KP / kGramWaves;          // rows each wave loads per chunk
  constexpr int kBufElems = KP * kChunkStride;    // one staged chunk
  static_assert(2 * kBufElems * 2 >= KP * KP * 4, "the reduction reuses the staging buffers");
  __shared__ __align__(16) uint16_t stage[2 * kBufElems];
  float* red = reinterpret_cast<float*>(stage);   // wave sums, after the last chunk
  const int64_t b = blockIdx.x / nsl;
  const int64_t sl = blockIdx.x - b * nsl;
  int64_t o0, g;
  if (!prompt_bounds(offsets, b, nv, 2, gmax, &o0, &g, nullptr, false)) return;
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = tid / kWave;
  const int rsub = lane & 15;
  const int kgrp = lane >> 4;

  const int64_t c_lo = sl * slice;
  const int64_t c_hi = c_lo + slice < D ? c_lo + slice : D;
  const int nchunks = (int)ceil_div(c_hi - c_lo, kChunkCols);

  // Chunk k, row wave + 4 i, columns c_lo + 512 k + 8 lane .. + 7 (zero past
  // the slice or the prompt's rows).
  auto gload = [&](int k, uint4 (&r)[kRows]) {
#pragma unroll
    for (int i = 0; i < kRows; ++i) {
      const int row = wave + kGramWaves * i;
      const int64_t col = c_lo + (int64_t)k * kChunkCols + 8 * lane;
      uint4 v = make_uint4(0u, 0u, 0u, 0u);
      if (row < g) {
        const uint16_t* src = scores + (o0 + row) * ld + col;
        if (col + 8 <= c_hi) {
          v = load_nt16(src);
        } else if (col < c_hi) {
          uint16_t h[8];
#pragma unroll
          for (int e = 0; e < 8; ++e) h[e] = (col + e < c_hi) ? src[e] : (uint16_t)0;
          v.x = (uint32_t)h[0] | ((uint32_t)h[1] << 16);
          v.y = (uint32_t)h[2] | ((uint32_t)h[3] << 16);
          v.z = (uint32_t)h[4] | ((uint32_t)h[5] << 16);
          v.w = (uint32_t)h[6] | ((uint32_t)h[7] << 16);
        }
      }
      r[i] = v;
    }
  };
  auto lstore = [&](int k, const uint4 (&r)[kRows]) {
    uint16_t* dst = stage + (k & 1) * kBufElems;
#pragma unroll
    for (int i = 0; i < kRows; ++i)
      *reinterpret_cast<uint4*>(dst + (wave + kGramWaves * i) * kChunkStride + 8 * lane) = r[i];
  };

  f32x4_t acc[KS][KS];
#pragma unroll
  for (int a = 0; a < KS; ++a)
#pragma unroll
    for (int c = 0; c < KS; ++c) acc[a][c] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};

  // Register slot u % kAhead holds chunk u until it is staged in LDS.
  uint4 st[kAhead][kRows];
#pragma unroll
  for (int u = 0; u < kAhead; ++u)
    if (u < nchunks) gload(u, st[u]);
  lstore(0, st[0]);
  __syncthreads();
  for (int k0 = 0; k0 < nchunks; k0 += kAhead) {
#pragma unroll
    for (int u = 0; u < kAhead; ++u) {
      const int k = k0 + u;
      if (k < nchunks) {
        // slot u held chunk k, already staged: refill it with chunk k + kAhead
        if (k + kAhead < nchunks) gload(k + kAhead, st[u]);
        const uint16_t* cur = stage + (k & 1) * kBufElems;
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          bf16x8_t fr[KS];
#pragma unroll
          for (int q = 0; q < KS; ++q)
            fr[q] = __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const uint4*>(
                cur + (16 * q + rsub) * kChunkStride + kStepCols * wave + 32 * t + 8 * kgrp));
#pragma unroll
          for (int a = 0; a < KS; ++a)
#pragma unroll
            for (int c2 = a; c2 < KS; ++c2)
              acc[a][c2] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fr[a], fr[c2], acc[a][c2],
                                                                    0, 0, 0);
        }
        if (k + 1 < nchunks) lstore(k + 1, st[(u + 1) % kAhead]);
        __syncthreads();
      }
    }
  }

  // Accumulator v of tile (a, c2): row 16 a + 4 (l / 16) + v, column
  // 16 c2 + l % 16.  Waves are added in order 0, 1, 2, 3.
  for (int w = 0; w < kGramWaves; ++w) {
    if (wave == w) {
#pragma unroll
      for (int a = 0; a < KS; ++a)
#pragma unroll
        for (int c2 = a; c2 < KS; ++c2)
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            const int idx = (16 * a + 4 * kgrp + v) * KP + 16 * c2 + rsub;
            red[idx] = (w == 0 ? 0.0f : red[idx]) + acc[a][c2][v];
          }
    }
    __syncthreads();
  }
  float* dst = part + (b * nsl + sl) * (int64_t)KP * KP;
  for (int idx = tid; idx < KP * KP; idx += kGramThreads) {
    const int i = idx / KP, j = idx - i * KP;
    // Only row blocks a <= c2 were multiplied: read the upper triangle.
    dst[idx] = (i / 16 <= j / 16) ? red[idx] : red[j * KP + i];
  }
}

__device__ __forceinline__ double block_sum(double v, double* sh) {
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
#pragma unroll
  for (int m = 1; m < kWave; m <<= 1) v += __shfl_xor(v, m, kWave);
  __syncthreads();
  if (lane == 0) sh[wave] = v;
  __syncthreads();
  double t = 0.0;
  for (int w = 0; w < kFinalThreads / kWave; ++w) t += sh[w];
  return t;
}

template <int KP>
__global__ __launch_bounds__(kFinalThreads) void exact_final_kernel(
    int64_t B, int64_t nv, int32_t gmax, const int64_t* __restrict__ offsets,
    const float* __restrict__ rewards, const float* __restrict__ p,
    const float* __restrict__ pi_w, int32_t rule, float wmax, int64_t nsl,
    const float* __restrict__ part, double* __restrict__ mse, double* __restrict__ bias_norm,
    double* __restrict__ gram, int32_t* d_status) {
  __shared__ double K[KP * KP];
  __shared__ double Ac[KP * KP];   // A_ij: coefficient of s_i in v_ij; C_ij = A_ji
  __shared__ double beta[KP], pd[KP], rd[KP];
  __shared__ double sh[kFinalThreads / kWave];
  const int64_t b = blockIdx.x;
  int64_t o0, g;
  if (!prompt_bounds(offsets, b, nv, 2, gmax, &o0, &g, d_status, threadIdx.x == 0)) return;
  const int tid = threadIdx.x;
  const int gi = (int)g;

  if (tid < KP) {
    pd[tid] = tid < gi ? (double)p[o0 + tid] : 1.0;
    rd[tid] = tid < gi ? (double)rewards[o0 + tid] : 0.0;
    if (tid < gi && !p_in_range(p[o0 + tid])) raise_status(d_status, PAIR_ST_P_RANGE);
  }
  bool nonfinite = false;
  for (int idx = tid; idx < KP * KP; idx += kFinalThreads) {
    double k = 0.0;
    const int i = idx / KP, j = idx - i * KP;
    if (i < gi && j < gi) {
      // slice partials added in slice order; loaded eight at a time
      const float* src = part + b * nsl * (int64_t)KP * KP + idx;
      int64_t s = 0;
      for (; s + 8 <= nsl; s += 8) {
        float v[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) v[q] = src[(s + q) * (int64_t)KP * KP];
#pragma unroll
        for (int q = 0; q < 8; ++q) k += (double)v[q];
      }
      for (; s < nsl; ++s) k += (double)src[s * (int64_t)KP * KP];
      if (!isfinite(k)) nonfinite = true;
      if (gram != nullptr) gram[(b * gmax + i) * (int64_t)gmax + j] = k;
    }
    K[idx] = k;
  }
  if (nonfinite) raise_status(d_status, PAIR_ST_NONFINITE);
  __syncthreads();

  // Rule coefficients of every ordered pair, weights from the logged rho.
  bool bad = false;
  for (int idx = tid; idx < KP * KP; idx += kFinalThreads) {
    const int i = idx / KP, j = idx - i * KP;
    double a = 0.0;
    if (i != j && i < gi && j < gi) {
      double rho = pd[i] * pd[j], pii = pd[i], pij = pd[j];
      if (pi_w != nullptr) {
        const float* blk = pi_w + b * (int64_t)gmax * gmax;
        const int lo = i < j ? i : j, hi = i < j ? j : i;
        rho = (double)blk[lo * gmax + hi];
        pii = (double)blk[i * gmax + i];
        pij = (double)blk[j * gmax + j];
      } else {
        rho = (double)(float)(pd[i] * pd[j]);   // the logged fl32(p_i p_j)
      }
      double wi = 1.0;
      if (rule == PAIR_RULE_MARGINAL) {
        if (!(pii > 0.0 && pii <= 1.0 && pij > 0.0 && pij <= 1.0)) bad = true;
        wi = 1.0 / pii;
      } else if (rule != PAIR_RULE_UNWEIGHTED) {
        if (!(rho > 0.0 && rho <= 1.0)) bad = true;
        wi = 1.0 / rho;
        if (rule == PAIR_RULE_CLIPPED && wi > (double)wmax) wi = (double)wmax;
      }
      a = 0.5 * (rd[i] - rd[j]) * wi;
    }
    Ac[idx] = a;
  }
  if (bad) raise_status(d_status, PAIR_ST_RHO_RANGE);
  __syncthreads();

  const double M = 0.5 * (double)gi * (double)(gi - 1);
  if (tid < KP) {
    double be = 0.0;
    if (tid < gi)
      for (int j = 0; j < gi; ++j)
        if (j != tid) be += pd[tid] * pd[j] * Ac[tid * KP + j] - 0.5 * (rd[tid] - rd[j]);
    beta[tid] = be / M;
  }
  __syncthreads();

  // beta^T K beta and the covariance trace; thread per ordered pair (i, j).
  double bk = 0.0, tr = 0.0;
  for (int idx = tid; idx < gi * gi; idx += kFinalThreads) {
    const int i = idx / gi, j = idx - i * gi;
    bk += beta[i] * beta[j] * K[i * KP + j];
    if (i == j) continue;
    const double aij = Ac[i * KP + j], cij = Ac[j * KP + i];
    if (j > i) {
      const double rho = pd[i] * pd[j];
      const double nn = aij * aij * K[i * KP + i] + 2.0 * aij * cij * K[i * KP + j] +
                        cij * cij * K[j * KP + j];
      tr += rho * (1.0 - rho) * nn;
    }
    const double wpre = pd[i] * pd[j] * (1.0 - pd[i]);
    for (int k = 0; k < gi; ++k) {
      if (k == i || k == j) continue;
      const double aik = Ac[i * KP + k], cik = Ac[k * KP + i];
      const double ip = aij * aik * K[i * KP + i] + aij * cik * K[i * KP + k] +
                        cij * aik * K[j * KP + i] + cij * cik * K[j * KP + k];
      tr += wpre * pd[k] * ip;
    }
  }
  const double bb = block_sum(bk, sh);
  const double tt = block_sum(tr, sh);
  if (tid == 0) {
    const double b2 = bb > 0.0 ? bb : 0.0;
    mse[b] = b2 + tt / (M * M);
    bias_norm[b] = sqrt(b2);
  }
}

// K = S_b S_b^T of every prompt in fp64 (the slice partials added in slice
// order, as exact_final_kernel adds them), for callers that only need the
// Gram matrices.  gram[b][i][j] for i, j < G_b; entries beyond are not
// written.
template <int KP>
__global__ __launch_bounds__(kFinalThreads) void gram_sum_kernel(
    int64_t B, int64_t nv, int32_t gmax, const int64_t* __restrict__ offsets, int64_t nsl,
    const float* __restrict__ part, double* __restrict__ gram, int32_t* d_status) {
  const int64_t b = blockIdx.x;
  int64_t o0, g;
  if (!prompt_bounds(offsets, b, nv, 2, gmax, &o0, &g, d_status, threadIdx.x == 0)) return;
  const int gi = (int)g;
  bool nonfinite = false;
  for (int idx = threadIdx.x; idx < KP * KP; idx += kFinalThreads) {
    const int i = idx / KP, j = idx - i * KP;
    if (i >= gi || j >= gi) continue;
    const float* src = part + b * nsl * (int64_t)KP * KP + idx;
    double k = 0.0;
    for (int64_t s = 0; s < nsl; ++s) k += (double)src[s * (int64_t)KP * KP];
    if (!isfinite(k)) nonfinite = true;
    gram[(b * gmax + i) * (int64_t)gmax + j] = k;
  }
  if (nonfinite) raise_status(d_status, PAIR_ST_NONFINITE);
}

}  // namespace

size_t exact_workspace_bytes(int64_t B, int32_t gmax, int64_t D) {
  return exact_layout(B, gmax, D).total;
}

int launch_gram(int64_t B, int64_t nv, int32_t gmax, const int64_t* offsets, int64_t D,
                const void* scores, int64_t ld, double* gram, void* workspace, int32_t* d_status,
                hipStream_t stream) {
  const ExactLayout L = exact_layout(B, gmax, D);
  float* part = static_cast<float*>(workspace);
  const uint16_t* s = static_cast<const uint16_t*>(scores);
  const int64_t grid = B * L.nsl;
  if (grid > 0x7fffffffLL) return PAIR_ERANGE;
#define PAIR_GRAM(KS_)                                                                         \
  hipLaunchKernelGGL(gram_kernel<KS_>, dim3((unsigned)grid), dim3(kGramThreads), 0, stream, B, \
                     nv, gmax, offsets, D, s, ld, L.nsl, L.slice, part)
#define PAIR_GSUM(KP_)                                                                        \
  hipLaunchKernelGGL(gram_sum_kernel<KP_>, dim3((unsigned)B), dim3(kFinalThreads), 0, stream, \
                     B, nv, gmax, offsets, L.nsl, part, gram, d_status)
  switch (L.ks) {
    case 1: PAIR_GRAM(1); break;
    case 2: PAIR_GRAM(2); break;
    case 3: PAIR_GRAM(3); break;
    default: PAIR_GRAM(4); break;
  }
  if (hipGetLastError() != hipSuccess) return PAIR_EHIP;
  switch (L.ks) {
    case 1: PAIR_GSUM(16); break;
    case 2: PAIR_GSUM(32); break;
    case 3: PAIR_GSUM(48); break;
    default: PAIR_GSUM(64); break;
  }
#undef PAIR_GRAM
#undef PAIR_GSUM
  return hipGetLastError() == hipSuccess ? PAIR_OK : PAIR_EHIP;
}

int launch_audit_exact(int64_t B, int64_t nv, int32_t gmax, const int64_t* offsets, int64_t D,
                       const void* scores, int64_t ld, const float* rewards, const float* p,
                       const float* pi_w, int32_t rule, float wmax, double* mse,
                       double* bias_norm, double* gram, void* workspace, int32_t* d_status,
                       hipStream_t stream) {
  const ExactLayout L = exact_layout(B, gmax, D);
  float* part = static_cast<float*>(workspace);
  const uint16_t* s = static_cast<const uint16_t*>(scores);
  const int64_t grid = B * L.nsl;
  if (grid > 0x7fffffffLL) return PAIR_ERANGE;
#define PAIR_GRAM(KS_)                                                                         \
  hipLaunchKernelGGL(gram_kernel<KS_>, dim3((unsigned)grid), dim3(kGramThreads), 0, stream, B, \
                     nv, gmax, offsets, D, s, ld, L.nsl, L.slice, part)
#define PAIR_FINAL(KP_)                                                                     \
  hipLaunchKernelGGL(exact_final_kernel<KP_>, dim3((unsigned)B), dim3(kFinalThreads), 0,    \
                     stream, B, nv, gmax, offsets, rewards, p, pi_w, rule, wmax, L.nsl, part, \
                     mse, bias_norm, gram, d_status)
  switch (L.ks) {
    case 1: PAIR_GRAM(1); break;
    case 2: PAIR_GRAM(2); break;
    case 3: PAIR_GRAM(3); break;
    default: PAIR_GRAM(4); break;
  }
  if (hipGetLastError() != hipSuccess) return PAIR_EHIP;
  switch (L.ks) {
    case 1: PAIR_FINAL(16); break;
    case 2: PAIR_FINAL(32); break;
    case 3: PAIR_FINAL(48); break;
    default: PAIR_FINAL(64); break;
  }
#undef PAIR_GRAM
#undef PAIR_FINAL
  return hipGetLastError() == hipSuccess ? PAIR_OK : PAIR_EHIP;
}

}  // namespace pair
