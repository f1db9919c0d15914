// The audit for callers that cannot allocate device memory: its workspace is
// a file-scope device array of the library, one per GPU, instead of a
// caller-provided buffer.  The prompts are audited in consecutive chunks
// whose workspace fits the array, each chunk with the kernels pair_audit
// runs and its own prompt-index base for the design draw, so every output is
// bitwise that of pair_audit.
#include <hip/hip_runtime.h>

#include <mutex>

#include "../../include/pair.h"
#include "launch.hpp"

namespace pair {

namespace {

// Nothing on the host may use this name as an address: its device address is
// taken with hipGetSymbolAddress once per device (scratch_address) and only
// that pointer is passed to kernels.
static __device__ __align__(256) unsigned char scratch[PAIR_AUDIT_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];

// Device address of the current device's copy of `scratch`, looked up on the
// first call on that device and kept for the life of the process.
int scratch_address(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return PAIR_EHIP;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || ptr == nullptr)
      return PAIR_EHIP;
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return PAIR_OK;
}

}  // namespace

// Largest number of consecutive prompts whose audit workspace fits the
// scratch array (0 if not even one prompt does).  The workspace grows with
// the prompt count, so a bisection finds it.
int64_t audit_noalloc_chunk(int64_t B, int32_t gmax, int64_t D, int64_t R) {
  if (audit_workspace_bytes(1, gmax, D, R) > PAIR_AUDIT_SCRATCH_BYTES) return 0;
  int64_t lo = 1, hi = B;
  while (lo < hi) {
    const int64_t mid = lo + (hi - lo + 1) / 2;
    if (audit_workspace_bytes(mid, gmax, D, R) <= PAIR_AUDIT_SCRATCH_BYTES)
      lo = mid;
    else
      hi = mid - 1;
  }
  return lo;
}

int launch_audit_noalloc(int64_t B, int64_t nv, int32_t gmax, const int64_t* offsets, int64_t D,
                         const void* scores, int64_t ld, const float* rewards, const float* p,
                         const float* pi_w, uint64_t seed, int64_t rep0, int64_t R, double* mse,
                         double* bias_norm, float* rep_sqerr, int32_t* edge_count,
                         int32_t* d_status, hipStream_t stream) {
  const int64_t chunk = audit_noalloc_chunk(B, gmax, D, R);
  if (chunk < 1) return PAIR_ESCRATCH;
  void* ws = nullptr;
  const int st = scratch_address(&ws);
  if (st != PAIR_OK) return st;
  const int64_t blk = (int64_t)gmax * gmax;
  for (int64_t b0 = 0; b0 < B; b0 += chunk) {
    const int64_t n = B - b0 < chunk ? B - b0 : chunk;
    const int rc = launch_audit(n, nv, gmax, offsets + b0, D, scores, ld, rewards, p,
                                pi_w != nullptr ? pi_w + b0 * blk : nullptr, PAIR_RULE_HT, 0.0f,
                                seed, rep0, b0, R, mse + b0, bias_norm + b0,
                                rep_sqerr != nullptr ? rep_sqerr + b0 * R : nullptr,
                                edge_count != nullptr ? edge_count + b0 * R : nullptr, ws,
                                d_status, stream);
    if (rc != PAIR_OK) return rc;
  }
  return PAIR_OK;
}

}  // namespace pair
