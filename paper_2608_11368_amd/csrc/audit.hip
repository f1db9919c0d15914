// Frozen-population estimator audit (paper Sec. 5.2, Table 2; App. D
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
//  1. audit_coeffs  one wave per (prompt, 64 replicates), one lane per
//                   replicate: Philox draw of J^(r) (same counter reading as
//                   the design draw), the coefficient fold over a per-prompt
//                   table W_ij = (r_i - r_j)/rho_ij in LDS, centring over the
//                   completed vertices, delta_r split into two bf16 terms
//                   (hi = RNE(delta), lo = RNE(delta - hi)) so the matrix-core
//                   operand carries ~16 significant bits, and a fixed-order
//                   fp32 partial sum of delta over the 64 lanes.
//  2. audit_mean    delta_bar appended as replicate row R, padding rows zeroed.
//  3. audit_mfma    [rows x 16k] delta (hi and lo terms) times [16k x D] bf16
//                   S_b on v_mfma_f32_32x32x16_bf16, S_b staged through LDS in a
//                   transposed layout (one 128-bit LDS read per operand), the
//                   squared norm of every 32x32 output tile accumulated in the
//                   epilogue, so the rows x D product is never written.
//                   Workgroups of one prompt are placed on one XCD so S_b is
//                   fetched into that XCD's L2 once and reused.
//  4. audit_finalize fp64 fixed-order MSE, bias = sqrt(e[R]), optional copies.
#include "common.hpp"
#include "launch.hpp"

namespace pair {

namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int kCoefThreads = 64;     // replicates per audit_coeffs workgroup
constexpr int kMfmaThreads = 256;    // 4 waves
constexpr int kTilesPerWave = 2;     // 32-row MFMA tiles per wave
constexpr int kRowsPerWave = 32 * kTilesPerWave;
constexpr int kRowsPerGroup = kRowsPerWave * (kMfmaThreads / kWave);  // 256
constexpr int kChunk = 256;          // score columns staged per LDS buffer

inline int64_t round_up(int64_t x, int64_t m) { return (x + m - 1) / m * m; }

struct AuditLayout {
  int ks;            // 16-wide K steps (ceil(gmax / 16))
  int64_t rrows;     // replicate rows per prompt incl. the delta_bar row and padding
  int64_t groups;    // MFMA workgroups per prompt
  int64_t nchunk;    // audit_coeffs workgroups per prompt
  size_t delta_off, e_off, dsum_off, total;
};

AuditLayout audit_layout(int64_t B, int32_t gmax, int64_t R) {
  AuditLayout L;
  L.ks = (gmax + 15) / 16;
  L.groups = (R + 1 + kRowsPerGroup - 1) / kRowsPerGroup;
  L.rrows = L.groups * kRowsPerGroup;
  L.nchunk = (R + kCoefThreads - 1) / kCoefThreads;
  size_t off = 0;
  L.delta_off = off;
  off += (size_t)round_up((int64_t)B * L.rrows * 2 * 16 * L.ks * 2, 256);  // hi + lo bf16
  L.e_off = off;
  off += (size_t)round_up((int64_t)B * L.rrows * 4, 256);
  L.dsum_off = off;
  off += (size_t)round_up((int64_t)B * L.nchunk * gmax * 4, 256);
  L.total = off;
  return L;
}

// ---------------------------------------------------------------------------
// 1. Replicate coefficients.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kCoefThreads) void audit_coeffs_kernel(
    int64_t B, int64_t nv, int32_t gmax, int ks, const int64_t* __restrict__ offsets,
    const float* __restrict__ rewards, const float* __restrict__ p,
    const float* __restrict__ pi_w, uint64_t seed, int64_t rep0, int64_t R, int64_t nchunk,
    int64_t rrows, uint16_t* __restrict__ delta, float* __restrict__ dsum,
    int32_t* __restrict__ edge_count, int32_t* d_status) {
  extern __shared__ float lds[];
  const int64_t b = blockIdx.x / nchunk;
  const int64_t chunk = blockIdx.x - b * nchunk;
  const int lane = threadIdx.x;
  int64_t o0, g;
  if (!prompt_bounds(offsets, b, nv, 2, gmax, &o0, &g, d_status, chunk == 0 && lane == 0)) return;

  const int stride = gmax + 1;
  float* W = lds;                         // [gmax][gmax + 1]  (r_i - r_j) / rho_ij
  float* A = W + gmax * stride;           // [64][gmax + 1]    per-replicate values
  float* pl = A + kCoefThreads * stride;  // [gmax]            continuation probabilities
  float* af = pl + gmax;                  // [gmax]            complete-pair coefficients
  float* rl = af + gmax;                  // [gmax]            rewards

  const bool vert = lane < g;
  const float r_i = vert ? rewards[o0 + lane] : 0.0f;
  const float p_i = vert ? p[o0 + lane] : 1.0f;
  if (vert) {
    pl[lane] = p_i;
    rl[lane] = r_i;
    if (!p_in_range(p_i) && chunk == 0) raise_status(d_status, PAIR_ST_P_RANGE);
  }

  // Complete-pair coefficients: the same fold with every vertex completed
  // and rho = 1, centred over all G vertices.
  float cf = 0.0f;
  for (int j = 0; j < g; ++j) {
    const float r_j = __shfl(r_i, j, kWave);
    if (vert && j != lane) cf += r_i - r_j;
  }
  float a_full = vert ? cf / (float)(g * (g - 1)) : 0.0f;
  const float tot = wave_sum(a_full);
  a_full = vert ? a_full - tot / (float)g : 0.0f;
  if (vert) af[lane] = a_full;
  __syncthreads();

  // Per-prompt edge table.
  bool bad_rho = false;
  for (int64_t idx = lane; idx < g * g; idx += kWave) {
    const int i = (int)(idx / g), j = (int)(idx - (int64_t)i * g);
    float w = 0.0f;
    if (i != j) {
      float rho;
      if (pi_w != nullptr) {
        const int lo = i < j ? i : j, hi = i < j ? j : i;
        rho = pi_w[b * (int64_t)gmax * gmax + lo * gmax + hi];
      } else {
        rho = pl[i] * pl[j];
      }
      if (rho > 0.0f && rho <= 1.0f) {
        w = (rl[i] - rl[j]) / rho;
      } else {
        bad_rho = true;
      }
    }
    W[i * stride + j] = w;
  }
  if (bad_rho && chunk == 0) raise_status(d_status, PAIR_ST_RHO_RANGE);
  __syncthreads();

  // One replicate per lane.
  const int64_t rloc = chunk * kCoefThreads + lane;
  const bool valid = rloc < R;
  uint64_t bits = 0;
  if (valid) {
    const uint64_t rg = (uint64_t)(rep0 + rloc);
    for (int blk = 0; blk * 4 < g; ++blk) {
      const Philox4x64 x = philox4x64_10(rg, (uint64_t)b, (uint64_t)blk, 0ull, seed, 0ull);
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

  // Fold: A~_i = (1/(G(G-1))) sum_{j observed, j != i} W_ij, then centre.
  const float den = (float)(g * (g - 1));
  float sum_obs = 0.0f;
  for (int i = 0; i < g; ++i) {
    float ai = 0.0f;
    if (k >= 2 && ((bits >> i) & 1ull)) {
      float c = 0.0f;
      for (int j = 0; j < g; ++j)
        if (j != i && ((bits >> j) & 1ull)) c += W[i * stride + j];
      ai = c / den;
      sum_obs += ai;
    }
    A[lane * stride + i] = ai;
  }
  const float mean = k >= 2 ? sum_obs / (float)k : 0.0f;

  // delta = A~ - a as two bf16 terms [hi x kp | lo x kp]; the fp32 value is
  // kept for the column sums.
  const int kp = 16 * ks;
  uint16_t* drow = delta + ((b * rrows + rloc) * 2 * kp);
  for (int i0 = 0; i0 < kp; i0 += 8) {
    uint32_t hi_p[4], lo_p[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      uint16_t h[2], l[2];
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        const int i = i0 + 2 * q + hh;
        float dv = 0.0f;
        if (i < g) {
          const float ai = (k >= 2 && ((bits >> i) & 1ull)) ? A[lane * stride + i] - mean : 0.0f;
          dv = valid ? ai - af[i] : 0.0f;
          A[lane * stride + i] = dv;
        }
        h[hh] = f32_to_bf16_rne(dv);
        l[hh] = f32_to_bf16_rne(dv - __uint_as_float((uint32_t)h[hh] << 16));
      }
      hi_p[q] = (uint32_t)h[0] | ((uint32_t)h[1] << 16);
      lo_p[q] = (uint32_t)l[0] | ((uint32_t)l[1] << 16);
    }
    if (valid) {
      *reinterpret_cast<uint4*>(drow + i0) = make_uint4(hi_p[0], hi_p[1], hi_p[2], hi_p[3]);
      *reinterpret_cast<uint4*>(drow + kp + i0) = make_uint4(lo_p[0], lo_p[1], lo_p[2], lo_p[3]);
    }
  }
  __syncthreads();

  // Fixed-order column sums over this workgroup's replicates.
  if (vert) {
    float s = 0.0f;
    for (int t = 0; t < kCoefThreads; ++t) s += A[t * stride + lane];
    dsum[(b * nchunk + chunk) * gmax + lane] = s;
  }
}

// ---------------------------------------------------------------------------
// 2. delta_bar row and zero padding.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void audit_mean_kernel(int64_t B, int64_t nv, int32_t gmax,
                                                         int ks, const int64_t* __restrict__ offsets,
                                                         int64_t R, int64_t nchunk, int64_t rrows,
                                                         const float* __restrict__ dsum,
                                                         uint16_t* __restrict__ delta) {
  const int64_t b = blockIdx.x;
  int64_t o0, g;
  if (!prompt_bounds(offsets, b, nv, 2, gmax, &o0, &g, nullptr, false)) return;
  const int kp = 16 * ks;
  const int tid = threadIdx.x;
  if (tid < kp) {
    float v = 0.0f;
    if (tid < g) {
      float s = 0.0f;
      for (int64_t c = 0; c < nchunk; ++c) s += dsum[(b * nchunk + c) * gmax + tid];
      v = s / (float)R;
    }
    const uint16_t hi = f32_to_bf16_rne(v);
    uint16_t* row = delta + (b * rrows + R) * 2 * kp;
    row[tid] = hi;
    row[kp + tid] = f32_to_bf16_rne(v - __uint_as_float((uint32_t)hi << 16));
  }
  const int64_t pad_elems = (rrows - R - 1) * 2 * kp;
  uint16_t* pad = delta + (b * rrows + R + 1) * 2 * kp;
  for (int64_t idx = tid; idx < pad_elems; idx += blockDim.x) pad[idx] = 0;
}

// ---------------------------------------------------------------------------
// 3. Matrix-core contraction with the squared-norm epilogue.
//
// v_mfma_f32_32x32x16_bf16 operand layout (wave64): lane l holds row l % 32
// of A and column l % 32 of B, with K elements 8*(l/32) .. 8*(l/32)+7.  The
// 16 accumulator registers of lane l hold column l % 32 and rows
// 8*(v/4) + 4*(l/32) + (v%4), v = 0..15.  Here A = delta rows (replicates,
// hi then lo term into the same accumulator), B = S_b^T chunk (columns d), so
// each accumulator register is one (r, d) entry of delta S_b and its square is
// added to a per-register running sum.
// ---------------------------------------------------------------------------
template <int KS>
__global__ __launch_bounds__(kMfmaThreads) void audit_mfma_kernel(
    int64_t B, int64_t nv, int32_t gmax, const int64_t* __restrict__ offsets, int64_t D,
    const uint16_t* __restrict__ scores, int64_t ld, int64_t rrows, int64_t groups,
    int64_t rows_live, const uint16_t* __restrict__ delta, float* __restrict__ e_out) {
  constexpr int KP = 16 * KS;                           // padded K
  constexpr int kPieces = KP * (kChunk / 8);            // 16-byte pieces per chunk
  constexpr int kPiecesPerThread = kPieces / kMfmaThreads;
  __shared__ __align__(16) uint16_t S_lds[2][kChunk * KP];  // [d][i] transposed

  // XCD-aware placement: hardware round-robins workgroup ids over 8 XCDs;
  // give each XCD a contiguous range of logical (prompt, row-group) ids.
  const int64_t per_xcd = gridDim.x / 8;
  const int64_t L = (int64_t)(blockIdx.x % 8) * per_xcd + blockIdx.x / 8;
  if (L >= B * groups) return;
  const int64_t b = L / groups;
  const int64_t grp = L - b * groups;
  int64_t o0, g;
  if (!prompt_bounds(offsets, b, nv, 2, gmax, &o0, &g, nullptr, false)) return;

  const int tid = threadIdx.x;
  const int wave = tid / kWave;
  const int lane = tid & (kWave - 1);
  const int64_t row0 = grp * kRowsPerGroup + wave * kRowsPerWave;

  // A operands: this wave's replicate rows, resident for the whole D loop.
  // A wave whose rows all lie past the live rows (padding of the last row
  // group) still stages score chunks for its workgroup but skips the math.
  const bool wave_live = row0 < rows_live;
  bf16x8_t Ahi[kTilesPerWave][KS], Alo[kTilesPerWave][KS];
#pragma unroll
  for (int t = 0; t < kTilesPerWave; ++t) {
    const uint16_t* src =
        delta + (b * rrows + row0 + t * 32 + (lane & 31)) * 2 * KP + 8 * (lane >> 5);
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      Ahi[t][s] = __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const uint4*>(src + 16 * s));
      Alo[t][s] = __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const uint4*>(src + KP + 16 * s));
    }
  }

  // Staging map: piece p -> (row i = p % KP, 8-column group p / KP); lanes
  // with consecutive i write consecutive LDS halfwords.
  const uint16_t* sb = scores + o0 * ld;
  uint4 stage[kPiecesPerThread];
  auto load_chunk = [&](int64_t c0) {
#pragma unroll
    for (int q = 0; q < kPiecesPerThread; ++q) {
      const int pidx = tid + q * kMfmaThreads;
      const int i = pidx % KP;
      const int64_t col = c0 + 8 * (pidx / KP);
      uint4 v = make_uint4(0u, 0u, 0u, 0u);
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
      stage[q] = v;
    }
  };
  auto store_chunk = [&](int buf) {
#pragma unroll
    for (int q = 0; q < kPiecesPerThread; ++q) {
      const int pidx = tid + q * kMfmaThreads;
      const int i = pidx % KP;
      const int d0 = 8 * (pidx / KP);
      uint16_t* dst = &S_lds[buf][d0 * KP + i];
      const uint4 v = stage[q];
      dst[0 * KP] = (uint16_t)v.x;
      dst[1 * KP] = (uint16_t)(v.x >> 16);
      dst[2 * KP] = (uint16_t)v.y;
      dst[3 * KP] = (uint16_t)(v.y >> 16);
      dst[4 * KP] = (uint16_t)v.z;
      dst[5 * KP] = (uint16_t)(v.z >> 16);
      dst[6 * KP] = (uint16_t)v.w;
      dst[7 * KP] = (uint16_t)(v.w >> 16);
    }
  };
  auto read_b = [&](int buf, int step, bf16x8_t (&Bf)[KS]) {
    const uint16_t* src = &S_lds[buf][(step * 32 + (lane & 31)) * KP + 8 * (lane >> 5)];
#pragma unroll
    for (int s = 0; s < KS; ++s)
      Bf[s] = __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const uint4*>(src + 16 * s));
  };
  auto contract = [&](const bf16x8_t (&Bf)[KS], f32x16_t (&acc)[kTilesPerWave]) {
#pragma unroll
    for (int t = 0; t < kTilesPerWave; ++t) {
      acc[t] = f32x16_t{};
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        acc[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(Ahi[t][s], Bf[s], acc[t], 0, 0, 0);
        acc[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(Alo[t][s], Bf[s], acc[t], 0, 0, 0);
      }
    }
  };

  f32x16_t sq[kTilesPerWave];
#pragma unroll
  for (int t = 0; t < kTilesPerWave; ++t)
#pragma unroll
    for (int v = 0; v < 16; ++v) sq[t][v] = 0.0f;
  auto square_add = [&](const f32x16_t (&acc)[kTilesPerWave]) {
#pragma unroll
    for (int t = 0; t < kTilesPerWave; ++t)
#pragma unroll
      for (int v = 0; v < 16; ++v) sq[t][v] = __builtin_fmaf(acc[t][v], acc[t][v], sq[t][v]);
  };

  const int64_t nchunks = (D + kChunk - 1) / kChunk;
  load_chunk(0);
  store_chunk(0);
  __syncthreads();
  for (int64_t ch = 0; ch < nchunks; ++ch) {
    const int buf = (int)(ch & 1);
    const bool more = ch + 1 < nchunks;
    if (more) load_chunk((ch + 1) * kChunk);
    if (wave_live) {
      // Software pipeline: the matrix core works on step s while the vector
      // ALU squares the outputs of step s - 1.
      bf16x8_t Bf[KS];
      f32x16_t accA[kTilesPerWave], accB[kTilesPerWave];
      read_b(buf, 0, Bf);
      contract(Bf, accA);
#pragma unroll
      for (int step = 1; step < kChunk / 32; step += 2) {
        read_b(buf, step, Bf);
        contract(Bf, accB);
        square_add(accA);
        if (step + 1 < kChunk / 32) {
          read_b(buf, step + 1, Bf);
          contract(Bf, accA);
        }
        square_add(accB);
      }
    }
    if (more) store_chunk(buf ^ 1);
    __syncthreads();
  }

  // Sum each register over the 32 lanes that share its rows (xor over lane
  // bits 0..4), then lane l (l % 32 < 16) writes register v = l % 32.
#pragma unroll
  for (int t = 0; t < kTilesPerWave; ++t) {
    float mine = 0.0f;
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      float x = sq[t][v];
#pragma unroll
      for (int m = 1; m < 32; m <<= 1) x += __shfl_xor(x, m, kWave);
      if ((lane & 31) == v) mine = x;
    }
    const int v = lane & 31;
    if (v < 16) {
      const int64_t row = row0 + t * 32 + 8 * (v / 4) + 4 * (lane >> 5) + (v % 4);
      e_out[b * rrows + row] = mine;
    }
  }
}

// ---------------------------------------------------------------------------
// 4. Fixed-order fp64 reductions.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void audit_finalize_kernel(
    int64_t B, int64_t nv, int32_t gmax, const int64_t* __restrict__ offsets, int64_t R,
    int64_t rrows, const float* __restrict__ e, double* __restrict__ mse,
    double* __restrict__ bias_norm, float* __restrict__ rep_sqerr) {
  __shared__ double part[256];
  const int64_t b = blockIdx.x;
  int64_t o0, g;
  if (!prompt_bounds(offsets, b, nv, 2, gmax, &o0, &g, nullptr, false)) return;
  const float* eb = e + b * rrows;
  double s = 0.0;
  for (int64_t r = threadIdx.x; r < R; r += blockDim.x) {
    s += (double)eb[r];
    if (rep_sqerr != nullptr) rep_sqerr[b * R + r] = eb[r];
  }
  part[threadIdx.x] = s;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) part[threadIdx.x] += part[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    mse[b] = part[0] / (double)R;
    bias_norm[b] = sqrt((double)eb[R]);
  }
}

}  // namespace

size_t audit_workspace_bytes(int64_t B, int32_t gmax, int64_t D, int64_t R) {
  (void)D;
  return audit_layout(B, gmax, R).total;
}

int launch_audit(int64_t B, int64_t nv, int32_t gmax, const int64_t* offsets, int64_t D,
                 const void* scores, int64_t ld, const float* rewards, const float* p,
                 const float* pi_w, uint64_t seed, int64_t rep0, int64_t R, double* mse,
                 double* bias_norm, float* rep_sqerr, int32_t* edge_count, void* workspace,
                 int32_t* d_status, hipStream_t stream) {
  const AuditLayout L = audit_layout(B, gmax, R);
  unsigned char* ws = static_cast<unsigned char*>(workspace);
  uint16_t* delta = reinterpret_cast<uint16_t*>(ws + L.delta_off);
  float* e = reinterpret_cast<float*>(ws + L.e_off);
  float* dsum = reinterpret_cast<float*>(ws + L.dsum_off);

  const int64_t coef_grid = B * L.nchunk;
  if (coef_grid > 0x7fffffffLL) return PAIR_ERANGE;
  const size_t coef_lds =
      ((size_t)gmax * (gmax + 1) + (size_t)kCoefThreads * (gmax + 1) + 3 * (size_t)gmax) *
      sizeof(float);
  hipLaunchKernelGGL(audit_coeffs_kernel, dim3((unsigned)coef_grid), dim3(kCoefThreads), coef_lds,
                     stream, B, nv, gmax, L.ks, offsets, rewards, p, pi_w, seed, rep0, R,
                     L.nchunk, L.rrows, delta, dsum, edge_count, d_status);
  if (hipGetLastError() != hipSuccess) return PAIR_EHIP;

  hipLaunchKernelGGL(audit_mean_kernel, dim3((unsigned)B), dim3(256), 0, stream, B, nv, gmax,
                     L.ks, offsets, R, L.nchunk, L.rrows, dsum, delta);
  if (hipGetLastError() != hipSuccess) return PAIR_EHIP;

  const int64_t logical = B * L.groups;
  const int64_t grid = round_up(logical, 8);
  if (grid > 0x7fffffffLL) return PAIR_ERANGE;
  const uint16_t* s = static_cast<const uint16_t*>(scores);
  const int64_t rows_live = R + 1;
  switch (L.ks) {
    case 1:
      hipLaunchKernelGGL(audit_mfma_kernel<1>, dim3((unsigned)grid), dim3(kMfmaThreads), 0, stream,
                         B, nv, gmax, offsets, D, s, ld, L.rrows, L.groups, rows_live, delta, e);
      break;
    case 2:
      hipLaunchKernelGGL(audit_mfma_kernel<2>, dim3((unsigned)grid), dim3(kMfmaThreads), 0, stream,
                         B, nv, gmax, offsets, D, s, ld, L.rrows, L.groups, rows_live, delta, e);
      break;
    case 3:
      hipLaunchKernelGGL(audit_mfma_kernel<3>, dim3((unsigned)grid), dim3(kMfmaThreads), 0, stream,
                         B, nv, gmax, offsets, D, s, ld, L.rrows, L.groups, rows_live, delta, e);
      break;
    default:
      hipLaunchKernelGGL(audit_mfma_kernel<4>, dim3((unsigned)grid), dim3(kMfmaThreads), 0, stream,
                         B, nv, gmax, offsets, D, s, ld, L.rrows, L.groups, rows_live, delta, e);
      break;
  }
  if (hipGetLastError() != hipSuccess) return PAIR_EHIP;

  hipLaunchKernelGGL(audit_finalize_kernel, dim3((unsigned)B), dim3(256), 0, stream, B, nv, gmax,
                     offsets, R, L.rrows, e, mse, bias_norm, rep_sqerr);
  return hipGetLastError() == hipSuccess ? PAIR_OK : PAIR_EHIP;
}

}  // namespace pair
