// Exact-budget pattern export (Sec. 3.3, Eq. (topk-pattern); Appendix A,
// exact-budget refinement): the K largest of the L x H x D retention
// probabilities become the pattern's ones, all other entries zeros.
//
// A radix select over the whole grid.  Every entry gets a 32-bit key that
// orders like its value (NaN lowest, -0 equal to +0).  Four rounds of 8-bit
// digits, most significant first, each a histogram kernel (every workgroup
// counts the keys of its contiguous chunk that match the prefix found so far
// in LDS and adds its 256 counts to a global histogram) and a one-workgroup
// select kernel (the digit whose bucket holds the K-th largest key; the
// prefix grows by it), find the K-th largest key v and how many entries equal
// to v must be kept.  Ties go to the lowest flat indices: a count kernel
// gives every chunk its number of entries equal to v, and the write kernel
// ranks its ties after those of the earlier chunks, in index order.
// State lives in a caller-provided workspace; no launch depends on the host.

#include "dkv_device.hpp"
#include "dkv_launch.hpp"

namespace dkv {

namespace {

constexpr int kTkThreads = 256;
constexpr int kTkWaves = kTkThreads / kWave;
constexpr int kTkStep = kTkThreads * 4;     // entries per workgroup iteration (one quadruple per thread)
constexpr int kTkMinChunk = 4 * kTkStep;    // entries per workgroup at least
constexpr int kTkMaxBlocks = 1024;
// workspace (uint32): prefix, entries still to take within it, histogram, per-chunk tie counts
constexpr int kTkPrefix = 0, kTkNeed = 1, kTkHist = 2, kTkTies = kTkHist + 256;

__device__ __forceinline__ uint32_t order_key(float x) {
  if (x != x) return 0u;  // NaN below every number
  uint32_t u = __float_as_uint(x);
  if (u == 0x80000000u) u = 0u;  // -0 ties with +0
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Keys of entries [i, i + 4) below `end`; the rest get valid = 0.  probs is
// 16-byte aligned and i a multiple of 4, so a whole quadruple is one load.
__device__ __forceinline__ uint32_t load_keys(const float* probs, int64_t i, int64_t end, uint32_t (&key)[4]) {
  if (i + 3 < end) {
    const float4 x = *reinterpret_cast<const float4*>(probs + i);
    key[0] = order_key(x.x);
    key[1] = order_key(x.y);
    key[2] = order_key(x.z);
    key[3] = order_key(x.w);
    return 0xFu;
  }
  uint32_t valid = 0u;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    key[e] = i + e < end ? order_key(probs[i + e]) : 0u;
    valid |= (i + e < end ? 1u : 0u) << e;
  }
  return valid;
}

__device__ __forceinline__ void chunk_of(const TopkParams& p, int b, int64_t& c0, int64_t& c1) {
  c0 = (int64_t)b * p.chunk;
  c1 = c0 + p.chunk < p.n ? c0 + p.chunk : p.n;
}

__global__ __launch_bounds__(kTkThreads) void topk_init_kernel(TopkParams p) {
  for (int i = threadIdx.x; i < 256; i += kTkThreads) p.state[kTkHist + i] = 0u;
  if (threadIdx.x == 0) {
    p.state[kTkPrefix] = 0u;
    p.state[kTkNeed] = (uint32_t)p.k;
  }
}

__global__ __launch_bounds__(kTkThreads) void topk_hist_kernel(TopkParams p, int shift) {
  __shared__ uint32_t hist[kTkWaves][256];
  const int tid = threadIdx.x;
  const int wave = tid / kWave;
  for (int i = tid; i < kTkWaves * 256; i += kTkThreads) (&hist[0][0])[i] = 0u;
  __syncthreads();
  const uint32_t prefix = p.state[kTkPrefix];
  const uint32_t mask = shift == 24 ? 0u : 0xFFFFFFFFu << (shift + 8);
  int64_t c0, c1;
  chunk_of(p, blockIdx.x, c0, c1);
  for (int64_t i = c0 + tid * 4; i < c1; i += kTkStep) {
    uint32_t key[4];
    const uint32_t valid = load_keys(p.probs, i, c1, key);
#pragma unroll
    for (int e = 0; e < 4; ++e)
      if (((valid >> e) & 1u) && (key[e] & mask) == prefix) atomicAdd(&hist[wave][(key[e] >> shift) & 255u], 1u);
  }
  __syncthreads();
  if (tid < 256) {
    uint32_t c = 0;
#pragma unroll
    for (int w = 0; w < kTkWaves; ++w) c += hist[w][tid];
    if (c) atomicAdd(&p.state[kTkHist + tid], c);
  }
}

__global__ __launch_bounds__(kTkThreads) void topk_select_kernel(TopkParams p, int shift) {
  __shared__ uint32_t h[256];
  const int tid = threadIdx.x;
  h[tid] = p.state[kTkHist + tid];
  p.state[kTkHist + tid] = 0u;  // ready for the next round
  __syncthreads();
  if (tid == 0) {
    // largest digit first: the bucket that holds the remaining K-th key
    const uint32_t need = p.state[kTkNeed];
    uint32_t above = 0;
    int dgt = 255;
    for (; dgt > 0; --dgt) {
      if (above + h[dgt] >= need) break;
      above += h[dgt];
    }
    p.state[kTkPrefix] |= (uint32_t)dgt << shift;
    p.state[kTkNeed] = need - above;
  }
}

__global__ __launch_bounds__(kTkThreads) void topk_ties_kernel(TopkParams p) {
  __shared__ int64_t red[kTkWaves + 1];
  const uint32_t thr = p.state[kTkPrefix];
  int64_t c0, c1;
  chunk_of(p, blockIdx.x, c0, c1);
  uint32_t ties = 0;
  for (int64_t i = c0 + threadIdx.x * 4; i < c1; i += kTkStep) {
    uint32_t key[4];
    const uint32_t valid = load_keys(p.probs, i, c1, key);
#pragma unroll
    for (int e = 0; e < 4; ++e) ties += ((valid >> e) & 1u) && key[e] == thr ? 1u : 0u;
  }
  int64_t total;
  block_exclusive_scan<kTkThreads>(ties, red, &total);
  if (threadIdx.x == 0) p.state[kTkTies + blockIdx.x] = (uint32_t)total;
}

__global__ __launch_bounds__(kTkThreads) void topk_write_kernel(TopkParams p) {
  __shared__ int64_t red[kTkWaves + 1];
  const int tid = threadIdx.x;
  const uint32_t thr = p.state[kTkPrefix];
  const uint32_t take = p.k > 0 ? p.state[kTkNeed] : 0u;  // entries equal to thr that are kept
  // ties in the chunks before this one
  uint32_t before = 0;
  for (int j = tid; j < (int)blockIdx.x; j += kTkThreads) before += p.state[kTkTies + j];
  int64_t rank;  // the block's total
  block_exclusive_scan<kTkThreads>(before, red, &rank);
  int64_t c0, c1;
  chunk_of(p, blockIdx.x, c0, c1);
  for (int64_t i0 = c0; i0 < c1; i0 += kTkStep) {
    const int64_t i = i0 + tid * 4;
    uint32_t key[4];
    const uint32_t valid = i < c1 ? load_keys(p.probs, i, c1, key) : 0u;
    uint32_t eq = 0u;
#pragma unroll
    for (int e = 0; e < 4; ++e) eq |= (((valid >> e) & 1u) && p.k > 0 && key[e] == thr ? 1u : 0u) << e;
    int64_t step_total;
    int64_t r = rank + block_exclusive_scan<kTkThreads>(__popc(eq), red, &step_total);
    uchar4 out;
    uint8_t* ob = reinterpret_cast<uint8_t*>(&out);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const bool t = (eq >> e) & 1u;
      ob[e] = (p.k > 0 && ((valid >> e) & 1u) && (key[e] > thr || (t && r < (int64_t)take))) ? 1 : 0;
      r += t ? 1 : 0;
    }
    if (valid == 0xFu) {
      *reinterpret_cast<uchar4*>(p.pattern + i) = out;
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if ((valid >> e) & 1u) p.pattern[i + e] = ob[e];
    }
    rank += step_total;
  }
}

}  // namespace

int topk_blocks(int64_t n) {
  const int64_t b = (n + kTkMinChunk - 1) / kTkMinChunk;
  return (int)(b < 1 ? 1 : (b > kTkMaxBlocks ? kTkMaxBlocks : b));
}

size_t topk_workspace_bytes(int64_t n) { return (size_t)(kTkTies + topk_blocks(n)) * sizeof(uint32_t); }

hipError_t launch_topk_pattern(TopkParams p, hipStream_t stream) {
  if (p.n == 0) return hipSuccess;
  const int blocks = topk_blocks(p.n);
  // chunks are whole iterations of the workgroup's quadruples
  p.chunk = ((p.n + blocks - 1) / blocks + kTkStep - 1) / kTkStep * kTkStep;
  hipLaunchKernelGGL(topk_init_kernel, dim3(1), dim3(kTkThreads), 0, stream, p);
  if (p.k > 0) {
    for (int shift = 24; shift >= 0; shift -= 8) {
      hipLaunchKernelGGL(topk_hist_kernel, dim3(blocks), dim3(kTkThreads), 0, stream, p, shift);
      hipLaunchKernelGGL(topk_select_kernel, dim3(1), dim3(kTkThreads), 0, stream, p, shift);
    }
    hipLaunchKernelGGL(topk_ties_kernel, dim3(blocks), dim3(kTkThreads), 0, stream, p);
  }
  hipLaunchKernelGGL(topk_write_kernel, dim3(blocks), dim3(kTkThreads), 0, stream, p);
  return hipGetLastError();
}

}  // namespace dkv
