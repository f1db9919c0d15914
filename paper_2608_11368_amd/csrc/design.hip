// Design draw: independent Bernoulli continuation indicators and the logged
// joint inclusion probabilities (paper Sec. 3.3; the design draw of Algorithm
// 1, new for every step; rho_ij must be logged before rewards, Theorem 2).
//
// One 64-lane wavefront per (replicate, prompt) unit, lane i = vertex i.  Each
// lane evaluates Philox4x64-10 at counter (r, b, i >> 2, 0) and keeps word
// i & 3 (lanes of one group of four compute the same block in lockstep, so
// this costs one generator evaluation per unit).  Completed-vertex and edge
// counts come from a ballot + popcount.  The waves of replicate 0 also write
// their prompt's logged rho block, so one launch serves both outputs.
#include "common.hpp"
#include "launch.hpp"

namespace pair {

__global__ __launch_bounds__(256) void design_draw_kernel(
    int64_t B, int64_t nv, int32_t gmax, const int64_t* __restrict__ offsets,
    const float* __restrict__ p, uint64_t seed, int64_t rep0, int64_t R, uint8_t* __restrict__ mask,
    float* __restrict__ pi, int32_t* __restrict__ edge_count, int32_t* __restrict__ completed,
    int32_t* d_status) {
  const int lane = threadIdx.x & (kWave - 1);
  const int64_t units = B * R;
  const int64_t waves_total = (int64_t)gridDim.x * (blockDim.x / kWave);
  const bool draws = mask != nullptr || edge_count != nullptr || completed != nullptr;
  for (int64_t u = (int64_t)blockIdx.x * (blockDim.x / kWave) + threadIdx.x / kWave; u < units;
       u += waves_total) {
    const int64_t r = u / B;  // replicate-major: consecutive waves share r
    const int64_t b = u - r * B;
    int64_t o0, g;
    const bool ok = prompt_bounds(offsets, b, nv, 2, gmax, &o0, &g, d_status, r == 0);
    const bool active = ok && lane < g;
    const float pv = active ? p[o0 + lane] : 1.0f;
    if (r == 0 && pi != nullptr) {
      // Logged rho block: fl32(p_i p_j) off the diagonal, p_i on it, zero
      // outside the G_b x G_b corner (all zero for a malformed prompt).
      // Whole-wave iterations so that every lane takes part in the shuffles
      // of p; only the store is guarded.
      float* blk = pi + b * (int64_t)gmax * gmax;
      for (int base = 0; base < gmax * gmax; base += kWave) {
        const int idx = base + lane;
        const int i = idx / gmax, j = idx - i * gmax;
        const float pa = __shfl(pv, i < kWave ? i : 0, kWave);
        const float pb = __shfl(pv, j, kWave);
        float v = 0.0f;
        if (ok && i < g && j < g) v = (i == j) ? pa : pa * pb;
        if (idx < gmax * gmax) blk[idx] = v;
      }
    }
    if (!ok || !draws) continue;
    int J = 0;
    if (active) {
      const Philox4x64 x = philox4x64_10((uint64_t)(rep0 + r), (uint64_t)b, (uint64_t)(lane >> 2),
                                         0ull, seed, 0ull);
      const uint64_t u32 = philox_word(x, lane & 3) >> 32;
      if (p_in_range(pv)) {
        J = u32 < inclusion_threshold(pv) ? 1 : 0;
      } else if (r == 0) {
        raise_status(d_status, PAIR_ST_P_RANGE);
      }
      if (mask != nullptr) mask[r * nv + o0 + lane] = (uint8_t)J;
    }
    const uint64_t bits = __ballot(J != 0);
    if (lane == 0) {
      const int32_t k = (int32_t)__popcll(bits);
      if (completed != nullptr) completed[r * B + b] = k;
      if (edge_count != nullptr) edge_count[r * B + b] = k * (k - 1) / 2;
    }
  }
}

int launch_design(int64_t B, int64_t nv, int32_t gmax, const int64_t* offsets, const float* p,
                  uint64_t seed, int64_t rep0, int64_t R, uint8_t* mask, float* pi,
                  int32_t* edge_count, int32_t* completed, int32_t* d_status, hipStream_t stream) {
  const bool draws = mask != nullptr || edge_count != nullptr || completed != nullptr;
  if (!draws && pi == nullptr) return PAIR_OK;
  const int64_t units = draws ? B * R : B;   // the rho block needs replicate 0 only
  const int64_t blocks_needed = (units + 3) / 4;
  const int64_t cap = (int64_t)device_cu_count() * 32;
  const unsigned grid = (unsigned)(blocks_needed < cap ? blocks_needed : cap);
  hipLaunchKernelGGL(design_draw_kernel, dim3(grid), dim3(256), 0, stream, B, nv, gmax, offsets, p,
                     seed, rep0, draws ? R : 1, mask, pi, edge_count, completed, d_status);
  return hipGetLastError() == hipSuccess ? PAIR_OK : PAIR_EHIP;
}

}  // namespace pair
