// Weighted-gradient stream: the induced-edge HT gradient of paper Eq.
// (pair-ht) in its sequence-advantage form (Sec. 4.5),
//     out[b][:] = sum_i A~_{b,i} s_{b,i,:},
// batched over prompts, fp32 accumulation over fp32 or bf16 score rows.
//
// HBM-bound.  A workgroup owns one column tile of one prompt; every
// lane streams 32 bytes per row per tile with non-temporal loads, laid out so
// that each load and store instruction of the workgroup covers one
// contiguous run (full cache lines for the fp32 output).
// The prompt's nonzero coefficients are found with a
// ballot (zero rows are never read: an uncompleted rollout has no score), the
// row indices and coefficients become wave-uniform scalars, and up to 12 rows
// are loaded back-to-back before any FMA so each lane keeps up to 384 bytes
// in flight.  Rows are summed in ascending order, so results are
// deterministic.  Tiles that lie wholly inside the row are one launch of a
// kernel with no tail handling (fewer live registers, three waves per SIMD);
// when D is not a multiple of the tile, the last tile of every prompt is a
// second launch of the variant that guards each column.
#include "common.hpp"
#include "launch.hpp"

namespace pair {

namespace {

constexpr int kThreads = 256;
constexpr int kBatch = 12;   // rows loaded back to back per batch
constexpr int kPieceCols = 4;  // columns per piece: one 16-byte fp32 output store

// A lane owns kPieces pieces of 4 columns per tile; piece p of lane t covers
// columns tile * (kPieces * 1024) + p * 1024 + 4 t .. + 3, so every load and
// store instruction of a workgroup touches one contiguous 4 KB (fp32) or
// 2 KB (bf16 input) run.  Per lane and row: 32 bytes of bf16 or fp32 input.
template <bool BF16>
struct PieceTraits;
template <>
struct PieceTraits<true> {
  static constexpr int kPieces = 4;   // 4 x 8-byte bf16 loads
  static constexpr int kBytes = 2;
  typedef uint2 Vec;
  __device__ static Vec load(const unsigned char* p) {
    const u32x2_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x2_t*>(p));
    return make_uint2(v.x, v.y);
  }
  __device__ static void fma(float (&acc)[kPieceCols], float c, const Vec& v) {
    acc[0] = __builtin_fmaf(c, bf16lo_to_f32(v.x), acc[0]);
    acc[1] = __builtin_fmaf(c, bf16hi_to_f32(v.x), acc[1]);
    acc[2] = __builtin_fmaf(c, bf16lo_to_f32(v.y), acc[2]);
    acc[3] = __builtin_fmaf(c, bf16hi_to_f32(v.y), acc[3]);
  }
  __device__ static float elem(const unsigned char* row, int64_t col) {
    return __uint_as_float(((uint32_t) reinterpret_cast<const uint16_t*>(row)[col]) << 16);
  }
};
template <>
struct PieceTraits<false> {
  static constexpr int kPieces = 2;   // 2 x 16-byte fp32 loads
  static constexpr int kBytes = 4;
  typedef uint4 Vec;
  __device__ static Vec load(const unsigned char* p) { return load_nt16(p); }
  __device__ static void fma(float (&acc)[kPieceCols], float c, const Vec& v) {
    acc[0] = __builtin_fmaf(c, __uint_as_float(v.x), acc[0]);
    acc[1] = __builtin_fmaf(c, __uint_as_float(v.y), acc[1]);
    acc[2] = __builtin_fmaf(c, __uint_as_float(v.z), acc[2]);
    acc[3] = __builtin_fmaf(c, __uint_as_float(v.w), acc[3]);
  }
  __device__ static float elem(const unsigned char* row, int64_t col) {
    return reinterpret_cast<const float*>(row)[col];
  }
};

// TAIL = false: every tile of the launch lies wholly inside [0, D).
// TAIL = true: the launch holds the last tile of each prompt, which may end
// inside a piece; columns past D are neither read nor written.
// Workgroup order of the full-tile launch: groups of `ilv` consecutive
// prompts (fewer in the last group), and within a group consecutive
// workgroups take the group's prompts in turn at the same tile, so that ilv
// prompts' rows stream at once (hardware deals consecutive workgroups to the
// 8 XCDs in turn; 1, 2 or 4 keeps a prompt on a fixed set of XCDs).  The tail
// launch covers prompt x with workgroup x.
template <bool BF16, bool TAIL>
__global__ __launch_bounds__(kThreads) void wgrad_kernel(
    int64_t B, int64_t nv, const int64_t* __restrict__ offsets,
    const unsigned char* __restrict__ scores, int64_t row_bytes, const float* __restrict__ coeff,
    float* __restrict__ out, int64_t D, int64_t tiles_per_prompt, int64_t tile0, int64_t ilv,
    int vec_out, int32_t* d_status) {
  using T = PieceTraits<BF16>;
  constexpr int NP = T::kPieces;
  constexpr int64_t kSpan = (int64_t)kThreads * kPieceCols;   // columns per piece index
  constexpr int64_t kTileCols = kSpan * NP;

  int64_t b, tile;
  if (TAIL) {
    b = blockIdx.x / tiles_per_prompt;
    tile = tile0 + (blockIdx.x - b * tiles_per_prompt);
  } else {
    const int64_t grp = blockIdx.x / (ilv * tiles_per_prompt);
    const int64_t r = blockIdx.x - grp * ilv * tiles_per_prompt;
    const int64_t k = B - ilv * grp < ilv ? B - ilv * grp : ilv;   // prompts in this group
    b = ilv * grp + r % k;
    tile = tile0 + r / k;
  }
  if (b >= B) return;
  const int lane = threadIdx.x & (kWave - 1);
  int64_t o0, g;
  if (!prompt_bounds(offsets, b, nv, 0, nv, &o0, &g, d_status,
                     tile == 0 && threadIdx.x == 0))
    return;

  const unsigned char* base = scores + o0 * row_bytes;
  float* orow = out + b * D;
  int64_t c0[NP];
  bool full[NP], part[NP];
#pragma unroll
  for (int q = 0; q < NP; ++q) {
    c0[q] = tile * kTileCols + q * kSpan + (int64_t)threadIdx.x * kPieceCols;
    full[q] = !TAIL || c0[q] + kPieceCols <= D;
    part[q] = TAIL && !full[q] && c0[q] < D;
  }

  float acc[NP][kPieceCols];
#pragma unroll
  for (int q = 0; q < NP; ++q)
#pragma unroll
    for (int e = 0; e < kPieceCols; ++e) acc[q][e] = 0.0f;

  // Windows of 64 rows: the nonzero coefficients of a window are found with
  // one ballot, then consumed in batches of up to kBatch rows.
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
      typename T::Vec v[kBatch][NP];
#pragma unroll
      for (int s = 0; s < kBatch; ++s)
#pragma unroll
        for (int q = 0; q < NP; ++q)
          if (s < n && full[q]) v[s][q] = T::load(base + roff[s] + c0[q] * T::kBytes);
#pragma unroll
      for (int s = 0; s < kBatch; ++s)
#pragma unroll
        for (int q = 0; q < NP; ++q)
          if (s < n && full[q]) T::fma(acc[q], cs[s], v[s][q]);
#pragma unroll
      for (int q = 0; q < NP; ++q) {
        if (TAIL && part[q]) {   // the ragged tail of the last tile
          for (int s = 0; s < n; ++s) {
            const unsigned char* row = base + roff[s];
            for (int e = 0; e < kPieceCols; ++e)
              if (c0[q] + e < D)
                acc[q][e] = __builtin_fmaf(cs[s], T::elem(row, c0[q] + e), acc[q][e]);
          }
        }
      }
    }
  }

#pragma unroll
  for (int q = 0; q < NP; ++q) {
    if (full[q] && vec_out) {
      store_nt16(orow + c0[q], acc[q][0], acc[q][1], acc[q][2], acc[q][3]);
    } else if (full[q] || (TAIL && part[q])) {
      for (int e = 0; e < kPieceCols; ++e)
        if (c0[q] + e < D) orow[c0[q] + e] = acc[q][e];
    }
  }
}

// Batch mean over prompts, out[d] = (1/B) sum_b g_b[d]: the prompts
// partition the packed rows offsets[0] .. offsets[B]-1, so the mean is one
// flat sum over those rows.  A workgroup owns 1024 output columns (4 per
// thread of a 256-thread row group) and RG row groups.  The rows are taken in
// chunks of kMeanChunk: the chunk's nonzero coefficients are listed in LDS
// in ascending row order (a ballot prefix count per wave, the waves in
// order), the list is split into RG contiguous parts, and row group q sums
// part q with kMeanBatch rows in flight per lane and the next batch's loads
// issued before the current batch's FMAs.  The groups' partial sums are added
// in LDS in group order at the end, so the result is deterministic for a
// given D and score type (RG depends only on them).  Workgroup 0 also checks that the offsets
// are monotone.
constexpr int kMeanBatch = 8;
constexpr int kMeanChunk = 2048;

template <bool BF16, int RG>
__global__ __launch_bounds__(kThreads * RG) void wgrad_mean_kernel(
    int64_t B, int64_t nv, const int64_t* __restrict__ offsets,
    const unsigned char* __restrict__ scores, int64_t row_bytes, const float* __restrict__ coeff,
    float* __restrict__ out, int64_t D, int vec_out, int32_t* d_status) {
  using T = PieceTraits<BF16>;
  constexpr int kN = kThreads * RG;
  constexpr int kWaves = kN / kWave;
  __shared__ int32_t list_row[kMeanChunk];     // row index relative to the chunk start
  __shared__ float list_c[kMeanChunk];
  __shared__ int32_t wcount[kWaves];
  __shared__ float part[RG > 1 ? RG - 1 : 1][kThreads][kPieceCols];
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = tid / kWave;
  const int grp = tid / kThreads;
  const int t = tid - grp * kThreads;
  const int64_t lo = offsets[0], hi = offsets[B];
  if (blockIdx.x == 0) {
    bool bad = false;
    for (int64_t b = tid; b < B; b += kN) {
      const int64_t x = offsets[b], y = offsets[b + 1];
      bad |= x < 0 || y < x || y > nv;
    }
    if (bad) raise_status(d_status, PAIR_ST_BAD_GROUP);
  }
  if (lo < 0 || hi < lo || hi > nv) {
    if (blockIdx.x == 0 && tid == 0) raise_status(d_status, PAIR_ST_BAD_GROUP);
    return;
  }

  const int64_t c0 = (int64_t)blockIdx.x * (kThreads * kPieceCols) + t * kPieceCols;
  const bool full = c0 + kPieceCols <= D;
  const bool part_cols = !full && c0 < D;
  float acc[kPieceCols] = {0.0f, 0.0f, 0.0f, 0.0f};
  const unsigned char* col = scores + c0 * T::kBytes;

  for (int64_t r0 = lo; r0 < hi; r0 += kMeanChunk) {
    const int64_t nrows = hi - r0 < kMeanChunk ? hi - r0 : kMeanChunk;
    // List the chunk's nonzero coefficients in ascending row order.
    int32_t base = 0;
    for (int k0 = 0; k0 < nrows; k0 += kN) {
      const int k = k0 + tid;
      const float cv = k < nrows ? coeff[r0 + k] : 0.0f;
      const uint64_t m = __ballot(cv != 0.0f);
      if (lane == 0) wcount[wave] = __popcll(m);
      __syncthreads();
      int32_t off = base, tot = 0;
      for (int w = 0; w < kWaves; ++w) {
        off += w < wave ? wcount[w] : 0;
        tot += wcount[w];
      }
      if (cv != 0.0f) {
        const int at = off + __popcll(m & ((1ull << lane) - 1ull));
        list_row[at] = k;
        list_c[at] = cv;
      }
      base += tot;
      __syncthreads();
    }
    // Row group grp sums list entries [e0, e1).
    const int n = base;
    const int e0 = (int)((int64_t)n * grp / RG), e1 = (int)((int64_t)n * (grp + 1) / RG);
    const unsigned char* cbase = col + r0 * row_bytes;
    if (full) {
      typename T::Vec va[kMeanBatch], vb[kMeanBatch];
      float ca[kMeanBatch], cb[kMeanBatch];
      auto issue = [&](int e, typename T::Vec (&v)[kMeanBatch], float (&c)[kMeanBatch]) {
#pragma unroll
        for (int s = 0; s < kMeanBatch; ++s) {
          c[s] = 0.0f;
          if (e + s < e1) {
            c[s] = list_c[e + s];
            v[s] = T::load(cbase + (int64_t)list_row[e + s] * row_bytes);
          }
        }
      };
      auto consume = [&](int e, const typename T::Vec (&v)[kMeanBatch], const float (&c)[kMeanBatch]) {
#pragma unroll
        for (int s = 0; s < kMeanBatch; ++s)
          if (e + s < e1) T::fma(acc, c[s], v[s]);
      };
      int e = e0;
      if (e < e1) issue(e, va, ca);
      while (e < e1) {
        const int en = e + kMeanBatch;
        if (en < e1) issue(en, vb, cb);
        consume(e, va, ca);
        if (en >= e1) break;
        const int em = en + kMeanBatch;
        if (em < e1) issue(em, va, ca);
        consume(en, vb, cb);
        e = em;
      }
    } else if (part_cols) {
      for (int e = e0; e < e1; ++e) {
        const float cs = list_c[e];
        const unsigned char* row = scores + (r0 + list_row[e]) * row_bytes;
        for (int q = 0; q < kPieceCols; ++q)
          if (c0 + q < D) acc[q] = __builtin_fmaf(cs, T::elem(row, c0 + q), acc[q]);
      }
    }
    __syncthreads();   // the list is rebuilt for the next chunk
  }

  if (RG > 1) {
    if (grp > 0) {
#pragma unroll
      for (int q = 0; q < kPieceCols; ++q) part[grp - 1][t][q] = acc[q];
    }
    __syncthreads();
    if (grp > 0) return;
#pragma unroll
    for (int g2 = 1; g2 < RG; ++g2)
#pragma unroll
      for (int q = 0; q < kPieceCols; ++q) acc[q] += part[g2 - 1][t][q];
  }
  const float fb = (float)B;
  if (full && vec_out) {
    store_nt16(out + c0, acc[0] / fb, acc[1] / fb, acc[2] / fb, acc[3] / fb);
  } else if (full || part_cols) {
    for (int q = 0; q < kPieceCols; ++q)
      if (c0 + q < D) out[c0 + q] = acc[q] / fb;
  }
}

}  // namespace

int launch_wgrad(int64_t B, int64_t nv, const int64_t* offsets, int64_t D, const void* scores,
                 int32_t dtype, int64_t ld, const float* coeff, float* out, int32_t reduce,
                 int32_t* d_status, hipStream_t stream) {
  const bool bf16 = dtype == PAIR_BF16;
  const int64_t row_bytes = ld * (bf16 ? 2 : 4);
  const int vec_out = (D % 4 == 0 && (reinterpret_cast<uintptr_t>(out) & 15u) == 0) ? 1 : 0;
  const unsigned char* s = static_cast<const unsigned char*>(scores);
  if (reduce) {
    const int64_t grid = (D + kThreads * kPieceCols - 1) / (kThreads * kPieceCols);
    if (grid > 0x7fffffffLL) return PAIR_ERANGE;
    // Row groups per workgroup: enough that the grid holds about 8 waves per
    // SIMD of the chip (4 row groups at most, one 1024-thread workgroup).
    const int64_t simds = 4 * (int64_t)device_cu_count();
    int rg = grid * 4 >= 8 * simds ? 1 : (grid * 8 >= 8 * simds ? 2 : 4);
    // fp32 rows take twice the registers per batch: at four row groups (1024
    // threads, 128 VGPRs a lane) the fp32 kernel would spill, so it stops at two.
    if (!bf16 && rg > 2) rg = 2;
#define PAIR_MEAN(BF, RG_)                                                                       \
  hipLaunchKernelGGL((wgrad_mean_kernel<BF, RG_>), dim3((unsigned)grid), dim3(kThreads * RG_), 0, \
                     stream, B, nv, offsets, s, row_bytes, coeff, out, D, vec_out, d_status)
    if (bf16) {
      if (rg == 1) PAIR_MEAN(true, 1); else if (rg == 2) PAIR_MEAN(true, 2); else PAIR_MEAN(true, 4);
    } else {
      if (rg == 1) PAIR_MEAN(false, 1); else PAIR_MEAN(false, 2);
    }
#undef PAIR_MEAN
    return hipGetLastError() == hipSuccess ? PAIR_OK : PAIR_EHIP;
  }
  const int64_t tile = (int64_t)kThreads * kPieceCols * (bf16 ? 4 : 2);
  const int64_t full_tiles = D / tile;                 // tiles wholly inside [0, D)
  const bool tail = full_tiles * tile < D;
  if (B * full_tiles > 0x7fffffffLL) return PAIR_ERANGE;
  // Prompts streamed at once (see wgrad_kernel): 4 for groups of at most 8
  // rollouts on average, else 2.  Measured on b128 (G = 16), the Qwen3-shaped
  // slice (G = 8) and ragged (mean G 33), against one prompt at a time: +1.5,
  // +2.4 and +0.7 points of HBM peak; 3, 6, 8 and 16 were slower.
  const int64_t ilv = nv <= 8 * B ? 4 : 2;
#define PAIR_WGRAD(BF, TL, GRID, TPP, T0)                                                         \
  hipLaunchKernelGGL((wgrad_kernel<BF, TL>), dim3((unsigned)(GRID)), dim3(kThreads), 0, stream, B, \
                     nv, offsets, s, row_bytes, coeff, out, D, TPP, T0, ilv, vec_out, d_status)
  if (full_tiles > 0) {
    if (bf16) {
      PAIR_WGRAD(true, false, B * full_tiles, full_tiles, 0);
    } else {
      PAIR_WGRAD(false, false, B * full_tiles, full_tiles, 0);
    }
    if (hipGetLastError() != hipSuccess) return PAIR_EHIP;
  }
  if (tail) {
    if (bf16) {
      PAIR_WGRAD(true, true, B, 1, full_tiles);
    } else {
      PAIR_WGRAD(false, true, B, 1, full_tiles);
    }
  }
#undef PAIR_WGRAD
  return hipGetLastError() == hipSuccess ? PAIR_OK : PAIR_EHIP;
}

}  // namespace pair
