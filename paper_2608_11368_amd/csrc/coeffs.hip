// Edge-coefficient fold: pair-corrected sequence advantages, paper Eq.
// (pair-advantage), accumulated over the induced edges as in Algorithm 1 and
// finished as App. C describes (fp32 accumulation, centred over the observed
// endpoints).
//
// One 64-lane wavefront per prompt, lane i = vertex i.  The prompt's rho
// block is staged in LDS (row stride gmax + 1 so that a column walk is
// conflict-free); lane i then walks j = 0..G-1 in order and adds
// (r_i - r_j) / rho_ij for every observed edge, dividing only when both
// endpoints completed (rho may be 0 on edges that were never observable).
#include "common.hpp"
#include "launch.hpp"

namespace pair {

__global__ __launch_bounds__(64) void edge_coeffs_kernel(
    int64_t B, int64_t nv, int32_t gmax, const int64_t* __restrict__ offsets,
    const float* __restrict__ rewards, const uint8_t* __restrict__ mask,
    const float* __restrict__ pi, float* __restrict__ coeff, int32_t* __restrict__ edge_count,
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

  float c = 0.0f;
  bool bad_rho = false;
  for (int j = 0; j < g; ++j) {
    const float r_j = __shfl(r_i, j, kWave);
    if (!((obs >> j) & 1ull) || !m_i || j == lane) continue;
    float rho = 1.0f;
    if (pi != nullptr) {
      const int lo = lane < j ? lane : j, hi = lane < j ? j : lane;
      rho = rho_lds[lo * stride + hi];
    }
    if (!(rho > 0.0f && rho <= 1.0f)) {
      bad_rho = true;
      continue;
    }
    c += (r_i - r_j) / rho;
  }
  if (bad_rho) raise_status(d_status, PAIR_ST_RHO_RANGE);

  // A~_i = c_i / (2M), 2M = G (G - 1); centre over the completed vertices.
  float a = 0.0f;
  if (m_i && k >= 2) a = c / (float)(g * (g - 1));
  const float total = wave_sum(a);
  if (k >= 2 && m_i) {
    a = a - total / (float)k;
  } else {
    a = 0.0f;
  }
  if (vert) coeff[o0 + lane] = a;
  if (lane == 0 && edge_count != nullptr) edge_count[b] = k * (k - 1) / 2;
}

int launch_coeffs(int64_t B, int64_t nv, int32_t gmax, const int64_t* offsets,
                  const float* rewards, const uint8_t* mask, const float* pi, float* coeff,
                  int32_t* edge_count, int32_t* d_status, hipStream_t stream) {
  const size_t lds = pi != nullptr ? (size_t)gmax * (gmax + 1) * sizeof(float) : 0;
  hipLaunchKernelGGL(edge_coeffs_kernel, dim3((unsigned)B), dim3(64), lds, stream, B, nv, gmax,
                     offsets, rewards, mask, pi, coeff, edge_count, d_status);
  return hipGetLastError() == hipSuccess ? PAIR_OK : PAIR_EHIP;
}

}  // namespace pair
