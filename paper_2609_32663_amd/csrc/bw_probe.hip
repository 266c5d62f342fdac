// Achievable-bandwidth probes: a plain streaming read with the decode
// kernel's load instruction and cache policy (16-byte non-temporal buffer
// loads), and a plain copy (16-byte non-temporal loads and stores), used to
// measure what one launch of a given size reaches on this GPU.

#include <hip/hip_runtime.h>

#include <cstdint>

#include "dkv_probe.h"

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kProbeThreads = 256;
constexpr uint32_t kProbeStride = kProbeThreads * 16;  // bytes per load round of a workgroup
constexpr uint32_t kProbeImpossible = 0x9E3779B9u;

// Read of `bytes` bytes in blocks of 256 x G 16-byte granules, one block per
// workgroup: every thread issues its G loads (the decode kernel's K/V load:
// 16-byte non-temporal buffer loads through a descriptor over the block, so
// loads past the end return zeros) and the workgroup retires.  Over one
// layer-sized launch (185.8 MB) such blocks of 4-32 KiB read 6.59-6.68 TB/s,
// where one contiguous slice per workgroup (256-2048 workgroups, 8 loads in
// flight per thread) read 6.03-6.34.
template <int G>
__global__ __launch_bounds__(kProbeThreads) void stream_read_kernel(const char* src, int64_t bytes,
                                                                   u32x4* sink) {
  constexpr int64_t kBlock = (int64_t)kProbeThreads * G * 16;
  const int64_t lo = (int64_t)blockIdx.x * kBlock;
  const int64_t len = bytes - lo < kBlock ? bytes - lo : kBlock;
  const uint64_t a = reinterpret_cast<uint64_t>(src + lo);
  const uint32_t a_lo = __builtin_amdgcn_readfirstlane((uint32_t)a);
  const uint32_t a_hi = __builtin_amdgcn_readfirstlane((uint32_t)(a >> 32));
  const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(
      reinterpret_cast<void*>(((uint64_t)a_hi << 32) | a_lo), (short)0,
      (int)__builtin_amdgcn_readfirstlane((uint32_t)len), 0x00020000);
  u32x4 x[G];
#pragma unroll
  for (int u = 0; u < G; ++u)
    x[u] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, threadIdx.x * 16u + u * kProbeStride,
                                                                           0, 2));
  u32x4 acc = x[0];
#pragma unroll
  for (int u = 1; u < G; ++u) acc ^= x[u];
  if ((acc.x ^ acc.y ^ acc.z ^ acc.w) == kProbeImpossible) *sink = acc;
}

// Copy of `bytes` bytes in blocks of 256 x G 16-byte granules, one block per
// workgroup (no grid-stride loop): every thread issues its G non-temporal
// loads, then its G stores, and the workgroup retires.  Short workgroups are
// what copies fastest here: with 4-16 KiB per workgroup a copy measured
// 6.0-6.5 TB/s of reads plus writes, with 32 KiB 4.1-4.3 TB/s, and a
// grid-stride sweep with 8 granules per thread per round 5.25-5.36 TB/s.
template <int G>
__global__ __launch_bounds__(kProbeThreads) void copy_kernel(const u32x4* __restrict__ src, u32x4* __restrict__ dst,
                                                             int64_t granules) {
  const int64_t base = (int64_t)blockIdx.x * kProbeThreads * G + threadIdx.x;
  u32x4 x[G];
#pragma unroll
  for (int u = 0; u < G; ++u) {
    const int64_t i = base + (int64_t)u * kProbeThreads;
    if (i < granules) x[u] = __builtin_nontemporal_load(src + i);
  }
#pragma unroll
  for (int u = 0; u < G; ++u) {
    const int64_t i = base + (int64_t)u * kProbeThreads;
    if (i < granules) __builtin_nontemporal_store(x[u], dst + i);
  }
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

}  // namespace

extern "C" dkv_status dkv_probe_stream_read(const void* src, int64_t bytes, void* sink,
                                            int32_t granules_per_thread, void* stream) {
  const int g = granules_per_thread;
  if (bytes < 0 || bytes % 16 != 0 || (g != 1 && g != 2 && g != 4 && g != 8)) return DKV_ERR_INVALID_ARG;
  if (bytes == 0) return DKV_OK;
  if (src == nullptr || sink == nullptr) return DKV_ERR_INVALID_ARG;
  if (!aligned16(src) || !aligned16(sink)) return DKV_ERR_MISALIGNED;
  const int64_t block = (int64_t)kProbeThreads * g * 16;
  const int64_t blocks = (bytes + block - 1) / block;
  if (blocks > 2147483647LL) return DKV_ERR_UNSUPPORTED;
  const dim3 grid((unsigned)blocks);
  const char* s8 = static_cast<const char*>(src);
  u32x4* sk = static_cast<u32x4*>(sink);
  hipStream_t st = (hipStream_t)stream;
  switch (g) {
    case 1: hipLaunchKernelGGL(stream_read_kernel<1>, grid, dim3(kProbeThreads), 0, st, s8, bytes, sk); break;
    case 2: hipLaunchKernelGGL(stream_read_kernel<2>, grid, dim3(kProbeThreads), 0, st, s8, bytes, sk); break;
    case 4: hipLaunchKernelGGL(stream_read_kernel<4>, grid, dim3(kProbeThreads), 0, st, s8, bytes, sk); break;
    default: hipLaunchKernelGGL(stream_read_kernel<8>, grid, dim3(kProbeThreads), 0, st, s8, bytes, sk); break;
  }
  return hipGetLastError() == hipSuccess ? DKV_OK : DKV_ERR_HIP;
}

extern "C" dkv_status dkv_probe_copy(const void* src, void* dst, int64_t bytes, int32_t granules_per_thread,
                                     void* stream) {
  const int g = granules_per_thread;
  if (bytes < 0 || bytes % 16 != 0 || (g != 1 && g != 2 && g != 4 && g != 8)) return DKV_ERR_INVALID_ARG;
  if (bytes == 0) return DKV_OK;
  if (src == nullptr || dst == nullptr) return DKV_ERR_INVALID_ARG;
  if (!aligned16(src) || !aligned16(dst)) return DKV_ERR_MISALIGNED;
  const char* s = static_cast<const char*>(src);
  char* d = static_cast<char*>(dst);
  if (s < d + bytes && d < s + bytes) return DKV_ERR_INVALID_ARG;  // overlapping buffers
  const int64_t granules = bytes / 16;
  const int64_t per = (int64_t)kProbeThreads * g;
  const int64_t blocks = (granules + per - 1) / per;
  if (blocks > 2147483647LL) return DKV_ERR_UNSUPPORTED;
  const dim3 grid((unsigned)blocks);
  const u32x4* s16 = static_cast<const u32x4*>(src);
  u32x4* d16 = static_cast<u32x4*>(dst);
  hipStream_t st = (hipStream_t)stream;
  switch (g) {
    case 1: hipLaunchKernelGGL(copy_kernel<1>, grid, dim3(kProbeThreads), 0, st, s16, d16, granules); break;
    case 2: hipLaunchKernelGGL(copy_kernel<2>, grid, dim3(kProbeThreads), 0, st, s16, d16, granules); break;
    case 4: hipLaunchKernelGGL(copy_kernel<4>, grid, dim3(kProbeThreads), 0, st, s16, d16, granules); break;
    default: hipLaunchKernelGGL(copy_kernel<8>, grid, dim3(kProbeThreads), 0, st, s16, d16, granules); break;
  }
  return hipGetLastError() == hipSuccess ? DKV_OK : DKV_ERR_HIP;
}
