// Achievable-bandwidth probe: a plain streaming read with the decode
// kernel's load instruction and cache policy (16-byte non-temporal buffer
// loads), used to measure what one launch of a given size reaches on this GPU.

#include <hip/hip_runtime.h>

#include <cstdint>

#include "dkv_probe.h"

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kProbeThreads = 256;
constexpr int kProbeUnroll = 8;                                   // loads in flight per thread
constexpr uint32_t kProbeStride = kProbeThreads * 16;             // bytes per load round of a workgroup
constexpr uint32_t kProbeImpossible = 0x9E3779B9u;

__global__ __launch_bounds__(kProbeThreads) void stream_read_kernel(const char* src, int64_t bytes,
                                                                   u32x4* sink) {
  const int64_t granules = bytes / 16;
  const int64_t per = (granules + gridDim.x - 1) / gridDim.x * 16;  // slice bytes
  const int64_t lo = per * blockIdx.x;
  const int64_t len = lo < bytes ? (bytes - lo < per ? bytes - lo : per) : 0;
  // descriptor over the slice; loads past its end return zeros
  const uint64_t a = reinterpret_cast<uint64_t>(src + lo);
  const uint32_t a_lo = __builtin_amdgcn_readfirstlane((uint32_t)a);
  const uint32_t a_hi = __builtin_amdgcn_readfirstlane((uint32_t)(a >> 32));
  const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(
      reinterpret_cast<void*>(((uint64_t)a_hi << 32) | a_lo), (short)0,
      (int)__builtin_amdgcn_readfirstlane((uint32_t)len), 0x00020000);
  u32x4 acc = {0u, 0u, 0u, 0u};
  for (uint32_t off = threadIdx.x * 16u; off < (uint32_t)len; off += kProbeStride * kProbeUnroll) {
    u32x4 x[kProbeUnroll];
#pragma unroll
    for (int u = 0; u < kProbeUnroll; ++u)
      x[u] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, off + u * kProbeStride, 0, 2));
#pragma unroll
    for (int u = 0; u < kProbeUnroll; ++u) acc ^= x[u];
  }
  if ((acc.x ^ acc.y ^ acc.z ^ acc.w) == kProbeImpossible) *sink = acc;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

}  // namespace

extern "C" dkv_status dkv_probe_stream_read(const void* src, int64_t bytes, void* sink, int32_t workgroups,
                                            void* stream) {
  if (bytes < 0 || bytes % 16 != 0 || workgroups < 1 || workgroups > 65535) return DKV_ERR_INVALID_ARG;
  if (bytes == 0) return DKV_OK;
  if (src == nullptr || sink == nullptr) return DKV_ERR_INVALID_ARG;
  if (!aligned16(src) || !aligned16(sink)) return DKV_ERR_MISALIGNED;
  const int64_t per = (bytes / 16 + workgroups - 1) / workgroups * 16;
  if (per > (int64_t(1) << 31)) return DKV_ERR_UNSUPPORTED;
  hipLaunchKernelGGL(stream_read_kernel, dim3(workgroups), dim3(kProbeThreads), 0, (hipStream_t)stream,
                     static_cast<const char*>(src), bytes, static_cast<u32x4*>(sink));
  return hipGetLastError() == hipSuccess ? DKV_OK : DKV_ERR_HIP;
}
