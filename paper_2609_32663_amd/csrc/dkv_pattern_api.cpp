// C-ABI entry points of the exact-budget pattern export (see include/dkv.h).
// Arguments are checked on the host before anything is enqueued.

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <cstring>

#include "dkv_launch.hpp"

extern "C" {

int64_t dkv_budget_entries(double rho, int32_t num_layers, int32_t num_q_heads, int32_t num_bins) {
  if (!std::isfinite(rho) || rho < 0.0 || rho > 1.0 || num_layers < 0 || num_q_heads < 0 || num_bins < 0)
    return -1;
  const double total = (double)num_layers * (double)num_q_heads * (double)num_bins;
  return (int64_t)std::floor(rho * total + 0.5);
}

size_t dkv_topk_workspace_bytes(int32_t num_layers, int32_t num_q_heads, int32_t num_bins) {
  if (num_layers < 0 || num_q_heads < 0 || num_bins < 0) return 0;
  const int64_t n = (int64_t)num_layers * num_q_heads * num_bins;
  if (n == 0 || n > INT32_MAX) return 0;
  return dkv::topk_workspace_bytes(n);
}

dkv_status dkv_topk_pattern(int32_t num_layers, int32_t num_q_heads, int32_t num_bins, const float* probs,
                            int64_t k, uint8_t* pattern, void* workspace, size_t workspace_bytes, void* stream) {
  if (num_layers < 0 || num_q_heads < 0 || num_bins < 0) return DKV_ERR_INVALID_ARG;
  const int64_t n = (int64_t)num_layers * num_q_heads * num_bins;
  if (n > INT32_MAX) return DKV_ERR_UNSUPPORTED;
  if (k < 0 || k > n) return DKV_ERR_INVALID_ARG;
  if (n == 0) return DKV_OK;
  if (probs == nullptr || pattern == nullptr) return DKV_ERR_INVALID_ARG;
  if ((reinterpret_cast<uintptr_t>(probs) & 15u) != 0 || (reinterpret_cast<uintptr_t>(pattern) & 3u) != 0)
    return DKV_ERR_MISALIGNED;
  if (workspace == nullptr || (reinterpret_cast<uintptr_t>(workspace) & 3u) != 0 ||
      workspace_bytes < dkv::topk_workspace_bytes(n))
    return DKV_ERR_WORKSPACE;
  dkv::TopkParams p;
  std::memset(&p, 0, sizeof(p));
  p.probs = probs;
  p.pattern = pattern;
  p.state = static_cast<uint32_t*>(workspace);
  p.n = n;
  p.k = k;
  return dkv::launch_topk_pattern(p, (hipStream_t)stream) == hipSuccess ? DKV_OK : DKV_ERR_HIP;
}

}  // extern "C"
