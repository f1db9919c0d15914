// Device helpers shared by the libpair kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/pair.h"

namespace pair {

constexpr int kWave = 64;

// ---------------------------------------------------------------------------
// Philox4x64-10 counter-based generator (Salmon, Moraes, Dror, Shaw, SC'11).
// Ten rounds; each round forms the full 128-bit products of counter words 0
// and 2 with the two round multipliers, then the new state is
//   (hi(m1*x2) ^ x1 ^ k0, lo(m1*x2), hi(m0*x0) ^ x3 ^ k1, lo(m0*x0)),
// and the key advances by the two Weyl increments between rounds.
// ---------------------------------------------------------------------------
struct Philox4x64 {
  uint64_t w[4];
};

// Full 128-bit product m * c from four 32 x 32 -> 64-bit partial products,
// the high and low halves sharing them: p01 and p10 carry the middle column,
// and no sum can overflow 64 bits (each is at most (2^32 - 1)^2 plus two
// 32-bit values).  Exact; four multiply-adds against about six for a
// separate high product and low product.
__device__ __forceinline__ void mulhilo64(uint64_t m, uint64_t c, uint64_t* hi, uint64_t* lo) {
  const uint32_t c0 = (uint32_t)c, c1 = (uint32_t)(c >> 32);
  const uint32_t m0 = (uint32_t)m, m1 = (uint32_t)(m >> 32);
  const uint64_t p00 = (uint64_t)c0 * m0;
  const uint64_t p01 = (uint64_t)c0 * m1 + (p00 >> 32);
  const uint64_t p10 = (uint64_t)c1 * m0 + (uint32_t)p01;
  *hi = (uint64_t)c1 * m1 + (p01 >> 32) + (p10 >> 32);
  *lo = (p10 << 32) | (uint32_t)p00;
}

__device__ __forceinline__ Philox4x64 philox4x64_10(uint64_t c0, uint64_t c1, uint64_t c2,
                                                    uint64_t c3, uint64_t k0, uint64_t k1) {
  const uint64_t m0 = 0xD2E7470EE14C6C93ull, m1 = 0xCA5A826395121157ull;
  const uint64_t w0 = 0x9E3779B97F4A7C15ull, w1 = 0xBB67AE8584CAA73Bull;
#pragma unroll
  for (int round = 0; round < 10; ++round) {
    if (round > 0) {
      k0 += w0;
      k1 += w1;
    }
    uint64_t hi0, lo0, hi1, lo1;
    mulhilo64(m0, c0, &hi0, &lo0);
    mulhilo64(m1, c2, &hi1, &lo1);
    const uint64_t n0 = hi1 ^ c1 ^ k0;
    const uint64_t n2 = hi0 ^ c3 ^ k1;
    c0 = n0;
    c1 = lo1;
    c2 = n2;
    c3 = lo0;
  }
  Philox4x64 o;
  o.w[0] = c0;
  o.w[1] = c1;
  o.w[2] = c2;
  o.w[3] = c3;
  return o;
}

// Output word q of a block, selected without a dynamic index: indexing the
// array with a lane-dependent q puts the block in memory (a store and a
// reload per lane).  In the one-wave-per-prompt draw and fold of 128 prompts
// that took the launch from 6.1 us with the selects to 14.0 us.
__device__ __forceinline__ uint64_t philox_word(const Philox4x64& x, int q) {
  return q == 0 ? x.w[0] : (q == 1 ? x.w[1] : (q == 2 ? x.w[2] : x.w[3]));
}

// Inclusion threshold floor(p * 2^32) as a 33-bit integer; p >= 1 includes always.
__device__ __forceinline__ uint64_t inclusion_threshold(float p) {
  if (p >= 1.0f) return 0x100000000ull;
  return (uint64_t)(p * 4294967296.0f);  // exact scaling by 2^32, truncation = floor
}

__device__ __forceinline__ bool p_in_range(float p) { return p > 0.0f && p <= 1.0f; }

// Non-temporal 16-byte global accesses for data streamed exactly once.
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2_t __attribute__((ext_vector_type(2)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint4 load_nt16(const void* src) {
  const u32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(src));
  return make_uint4(v.x, v.y, v.z, v.w);
}

__device__ __forceinline__ void store_nt16(void* dst, float a, float b, float c, float d) {
  f32x4_t v = {a, b, c, d};
  __builtin_nontemporal_store(v, reinterpret_cast<f32x4_t*>(dst));
}

// bf16 <-> fp32 bit conversions.
__device__ __forceinline__ float bf16lo_to_f32(uint32_t pair) { return __uint_as_float(pair << 16); }
__device__ __forceinline__ float bf16hi_to_f32(uint32_t pair) {
  return __uint_as_float(pair & 0xffff0000u);
}
// Value of `v` in lane `j` for a wave-uniform j (a scalar read of one lane,
// no LDS round trip).
__device__ __forceinline__ float lane_value(float v, int j) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), j));
}

// DPP move of a float within each row of 16 lanes.
template <int kCtrl>
__device__ __forceinline__ float dpp_f(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), kCtrl, 0xf, 0xf, false));
}

// Sum across the 64 lanes, the same bits in every lane: four DPP steps
// (quad_perm [1,0,3,2], quad_perm [2,3,0,1], row_half_mirror, row_mirror)
// leave each row's total in all its lanes (partner lanes add the same two
// values, and IEEE addition is commutative), then the four row totals are
// added in row order.  Every lane of the wave must be active.
__device__ __forceinline__ float wave_sum(float v) {
  v += dpp_f<0xB1>(v);
  v += dpp_f<0x4E>(v);
  v += dpp_f<0x141>(v);
  v += dpp_f<0x140>(v);
  return ((lane_value(v, 0) + lane_value(v, 16)) + lane_value(v, 32)) + lane_value(v, 48);
}

__device__ __forceinline__ void raise_status(int32_t* d_status, int32_t bits) {
  if (d_status != nullptr) atomicOr(d_status, bits);
}

// Edge weight on vertex i's half of observed edge (i, j) under `rule`
// (PAIR_RULE_*), applied to dr = r_i - r_j; also the edge's own weight (for ESS and the maximum) and
// its share 1/rho of the self-normalised denominator.  Returns false when the
// rule needs rho (or the marginals) and they are outside (0, 1].
__device__ __forceinline__ bool rule_term(int rule, float wmax, float dr, float rho, float pii,
                                          float pij, float* term, float* w_edge, float* inv_rho) {
  *inv_rho = 0.0f;
  switch (rule) {
    case PAIR_RULE_UNWEIGHTED:
    case PAIR_RULE_RATIO_KE:
      *term = dr;
      *w_edge = 1.0f;
      return true;
    case PAIR_RULE_MARGINAL:
      if (!(p_in_range(pii) && p_in_range(pij))) return false;
      *term = dr / pii;
      *w_edge = 0.5f * (1.0f / pii + 1.0f / pij);
      return true;
    default: {  // HT, CLIPPED, SELFNORM
      if (!(rho > 0.0f && rho <= 1.0f)) return false;
      const float w = 1.0f / rho;
      *inv_rho = w;
      if (rule == PAIR_RULE_CLIPPED && w > wmax) {
        *term = dr * wmax;
        *w_edge = wmax;
      } else {
        *term = dr / rho;
        *w_edge = w;
      }
      return true;
    }
  }
}

// 64-bit DPP move of a double (two 32-bit halves), all rows and banks on.
template <int kCtrl>
__device__ __forceinline__ double dpp_d(double v) {
  const uint64_t u = __builtin_bit_cast(uint64_t, v);
  const int lo = __builtin_amdgcn_update_dpp(0, (int)(uint32_t)u, kCtrl, 0xf, 0xf, false);
  const int hi = __builtin_amdgcn_update_dpp(0, (int)(uint32_t)(u >> 32), kCtrl, 0xf, 0xf, false);
  return __builtin_bit_cast(double, ((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo);
}

__device__ __forceinline__ double readlane_d(double v, int lane) {
  const uint64_t u = __builtin_bit_cast(uint64_t, v);
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)u, lane);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(u >> 32), lane);
  return __builtin_bit_cast(double, ((uint64_t)hi << 32) | lo);
}

// Wave sum in a fixed order, the same value in every lane: within each row of
// 16 lanes, pairwise exchanges (quad_perm [1,0,3,2], quad_perm [2,3,0,1],
// row_half_mirror, row_mirror) leave the row total in every lane of the row;
// the four row totals are then added in row order.
__device__ __forceinline__ double wave_sum_d(double v) {
  v += dpp_d<0xB1>(v);     // quad_perm [1,0,3,2]
  v += dpp_d<0x4E>(v);     // quad_perm [2,3,0,1]
  v += dpp_d<0x141>(v);    // row_half_mirror
  v += dpp_d<0x140>(v);    // row_mirror
  return ((readlane_d(v, 0) + readlane_d(v, 16)) + readlane_d(v, 32)) + readlane_d(v, 48);
}

__device__ __forceinline__ double wave_max_d(double v) {
#pragma unroll
  for (int m = 1; m < kWave; m <<= 1) v = fmax(v, __shfl_xor(v, m, kWave));
  return v;
}

// Validated bounds of prompt b: returns false (and sets the status bit) when
// the offsets are not monotone, leave [0, nv], or G_b is outside [gmin, gmax].
__device__ __forceinline__ bool prompt_bounds(const int64_t* offsets, int64_t b, int64_t nv,
                                              int64_t gmin, int64_t gmax, int64_t* o0,
                                              int64_t* g, int32_t* d_status, bool report) {
  const int64_t a = offsets[b], e = offsets[b + 1];
  const bool ok = a >= 0 && e >= a && e <= nv && (e - a) >= gmin && (e - a) <= gmax;
  if (!ok) {
    if (report) raise_status(d_status, PAIR_ST_BAD_GROUP);
    *o0 = 0;
    *g = 0;
    return false;
  }
  *o0 = a;
  *g = e - a;
  return true;
}

}  // namespace pair
