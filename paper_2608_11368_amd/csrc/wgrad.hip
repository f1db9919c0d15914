// Weighted-gradient stream: the induced-edge HT gradient of paper Eq.
// (pair-ht) in its sequence-advantage form (Sec. 3.5),
//     out[b][:] = sum_i A~_{b,i} s_{b,i,:},
// batched over prompts, fp32 accumulation over fp32 or bf16 score rows.
//
// HBM-bound.  A workgroup owns a run of column tiles of one prompt; every
// lane streams one 16-byte chunk per row per tile with non-temporal loads.
// The prompt's nonzero coefficients are found with a ballot (zero rows are
// never read: an uncompleted rollout has no score), the row indices and
// coefficients become wave-uniform scalars, and up to 16 rows are loaded
// back-to-back before any FMA so each lane keeps up to 256 bytes in flight.
// Rows are summed in ascending order, so results are deterministic.
#include "common.hpp"
#include "launch.hpp"

namespace pair {

namespace {

constexpr int kThreads = 256;
constexpr int kBatch = 16;

template <bool BF16>
struct ChunkTraits;
template <>
struct ChunkTraits<true> {
  static constexpr int kElems = 8;  // bf16 per 16-byte chunk
  static constexpr int kBytes = 2;
};
template <>
struct ChunkTraits<false> {
  static constexpr int kElems = 4;  // fp32 per 16-byte chunk
  static constexpr int kBytes = 4;
};

template <bool BF16>
__device__ __forceinline__ void fma_chunk(float (&acc)[ChunkTraits<BF16>::kElems], float c,
                                          const uint4& v) {
  if constexpr (BF16) {
    acc[0] = __builtin_fmaf(c, bf16lo_to_f32(v.x), acc[0]);
    acc[1] = __builtin_fmaf(c, bf16hi_to_f32(v.x), acc[1]);
    acc[2] = __builtin_fmaf(c, bf16lo_to_f32(v.y), acc[2]);
    acc[3] = __builtin_fmaf(c, bf16hi_to_f32(v.y), acc[3]);
    acc[4] = __builtin_fmaf(c, bf16lo_to_f32(v.z), acc[4]);
    acc[5] = __builtin_fmaf(c, bf16hi_to_f32(v.z), acc[5]);
    acc[6] = __builtin_fmaf(c, bf16lo_to_f32(v.w), acc[6]);
    acc[7] = __builtin_fmaf(c, bf16hi_to_f32(v.w), acc[7]);
  } else {
    acc[0] = __builtin_fmaf(c, __uint_as_float(v.x), acc[0]);
    acc[1] = __builtin_fmaf(c, __uint_as_float(v.y), acc[1]);
    acc[2] = __builtin_fmaf(c, __uint_as_float(v.z), acc[2]);
    acc[3] = __builtin_fmaf(c, __uint_as_float(v.w), acc[3]);
  }
}

template <bool BF16>
__device__ __forceinline__ float load_elem(const unsigned char* row, int64_t col) {
  if constexpr (BF16) {
    const uint16_t h = reinterpret_cast<const uint16_t*>(row)[col];
    return __uint_as_float(((uint32_t)h) << 16);
  } else {
    return reinterpret_cast<const float*>(row)[col];
  }
}

template <bool BF16>
__global__ __launch_bounds__(kThreads) void wgrad_kernel(
    int64_t B, int64_t nv, const int64_t* __restrict__ offsets,
    const unsigned char* __restrict__ scores, int64_t row_bytes, const float* __restrict__ coeff,
    float* __restrict__ out, int64_t D, int64_t tiles_per_prompt, int64_t groups_per_prompt,
    int tiles_per_group, int vec_out, int32_t* d_status) {
  using T = ChunkTraits<BF16>;
  constexpr int E = T::kElems;
  constexpr int64_t kTile = (int64_t)kThreads * E;

  const int64_t b = blockIdx.x / groups_per_prompt;
  const int64_t grp = blockIdx.x - b * groups_per_prompt;
  if (b >= B) return;
  const int lane = threadIdx.x & (kWave - 1);
  int64_t o0, g;
  if (!prompt_bounds(offsets, b, nv, 0, nv, &o0, &g, d_status,
                     grp == 0 && threadIdx.x == 0))
    return;

  const unsigned char* base = scores + o0 * row_bytes;
  float* orow = out + b * D;

  for (int t = 0; t < tiles_per_group; ++t) {
    const int64_t tile = grp * tiles_per_group + t;
    if (tile >= tiles_per_prompt) break;
    const int64_t c0 = tile * kTile + (int64_t)threadIdx.x * E;
    const bool full = c0 + E <= D;
    const bool part = !full && c0 < D;

    float acc[E];
#pragma unroll
    for (int e = 0; e < E; ++e) acc[e] = 0.0f;

    for (int64_t w0 = 0; w0 < g; w0 += kWave) {
      const float cv = (w0 + lane < g) ? coeff[o0 + w0 + lane] : 0.0f;
      uint64_t nz = __ballot(cv != 0.0f);
      while (nz != 0ull) {
        int64_t roff[kBatch];
        float cs[kBatch];
        int n = 0;
#pragma unroll
        for (int s = 0; s < kBatch; ++s) {
          roff[s] = 0;
          cs[s] = 0.0f;
          if (nz != 0ull) {
            const int j = __ffsll((unsigned long long)nz) - 1;
            nz &= nz - 1ull;
            roff[s] = (w0 + j) * row_bytes;
            cs[s] = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(cv), j));
            n = s + 1;
          }
        }
        if (full) {
          uint4 v[kBatch];
#pragma unroll
          for (int s = 0; s < kBatch; ++s) {
            if (s < n) {
              v[s] = load_nt16(base + roff[s] + c0 * T::kBytes);
            }
          }
#pragma unroll
          for (int s = 0; s < kBatch; ++s) {
            if (s < n) fma_chunk<BF16>(acc, cs[s], v[s]);
          }
        } else if (part) {
          for (int s = 0; s < n; ++s) {
            const unsigned char* row = base + roff[s];
            for (int e = 0; e < E; ++e)
              if (c0 + e < D) acc[e] = __builtin_fmaf(cs[s], load_elem<BF16>(row, c0 + e), acc[e]);
          }
        }
      }
    }

    if (full && vec_out) {
#pragma unroll
      for (int q = 0; q < E / 4; ++q)
        store_nt16(orow + c0 + 4 * q, acc[4 * q + 0], acc[4 * q + 1], acc[4 * q + 2],
                   acc[4 * q + 3]);
    } else if (full || part) {
      for (int e = 0; e < E; ++e)
        if (c0 + e < D) orow[c0 + e] = acc[e];
    }
  }
}

}  // namespace

int launch_wgrad(int64_t B, int64_t nv, const int64_t* offsets, int64_t D, const void* scores,
                 int32_t dtype, int64_t ld, const float* coeff, float* out, int32_t* d_status,
                 hipStream_t stream) {
  const bool bf16 = dtype == PAIR_BF16;
  const int E = bf16 ? 8 : 4;
  const int64_t tile = (int64_t)kThreads * E;
  const int64_t tiles = (D + tile - 1) / tile;
  int64_t tpg = tiles / 64;
  tpg = tpg < 1 ? 1 : (tpg > 8 ? 8 : tpg);
  const int64_t groups = (tiles + tpg - 1) / tpg;
  const int64_t grid = B * groups;
  if (grid > 0x7fffffffLL) return PAIR_ERANGE;
  const int64_t row_bytes = ld * (bf16 ? 2 : 4);
  const int vec_out = (D % 4 == 0 && (reinterpret_cast<uintptr_t>(out) & 15u) == 0) ? 1 : 0;
  const unsigned char* s = static_cast<const unsigned char*>(scores);
  if (bf16) {
    hipLaunchKernelGGL(wgrad_kernel<true>, dim3((unsigned)grid), dim3(kThreads), 0, stream, B, nv,
                       offsets, s, row_bytes, coeff, out, D, tiles, groups, (int)tpg, vec_out,
                       d_status);
  } else {
    hipLaunchKernelGGL(wgrad_kernel<false>, dim3((unsigned)grid), dim3(kThreads), 0, stream, B,
                       nv, offsets, s, row_bytes, coeff, out, D, tiles, groups, (int)tpg, vec_out,
                       d_status);
  }
  return hipGetLastError() == hipSuccess ? PAIR_OK : PAIR_EHIP;
}

}  // namespace pair
