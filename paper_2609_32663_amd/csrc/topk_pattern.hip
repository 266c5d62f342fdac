// Exact-budget pattern export (Sec. 3.3, Eq. (topk-pattern); Appendix A,
// exact-budget refinement): the K largest of the L x H x D retention
// probabilities become the pattern's ones, all other entries zeros.
//
// A radix select over the whole grid.  Every entry gets a 32-bit key that
// orders like its value (NaN lowest, -0 equal to +0).  Three rounds of
// digits (11, 11 and 10 bits, most significant first) find the K-th largest
// key v and how many entries equal to v must be kept.  In a round every
// workgroup counts the keys of its contiguous chunk that match the prefix
// found so far (one LDS histogram per wave) and adds its counts to the
// round's global histogram.  The digit of a round -- the one whose bucket
// holds the K-th largest key -- is picked at the start of the next launch by
// every workgroup from that histogram (the kernel boundary publishes it; no
// device-scope fence, which costs an L2 write-back per workgroup, and no
// counters); workgroup 0 also stores the grown prefix for the launch after.
// Ties go to the lowest flat indices: in the last round every workgroup also
// stores its own histogram, so the write pass ranks its chunk's ties after
// the earlier chunks' (their count of the final digit), in index order.
// Five launches (clear, three rounds, write); no launch depends on the host.
// State lives in a caller-provided workspace.

#include "dkv_device.hpp"
#include "dkv_launch.hpp"

namespace dkv {

namespace {

constexpr int kTkThreads = 256;
constexpr int kTkWaves = kTkThreads / kWave;
constexpr int kTkStep = kTkThreads * 4;     // entries per workgroup iteration (one quadruple per thread)
constexpr int kTkMinChunk = 4 * kTkStep;    // entries per workgroup at least
constexpr int kTkMaxBlocks = 1024;
constexpr int kTkRounds = 3;
constexpr int kTkShift[kTkRounds] = {21, 10, 0};
constexpr int kTkBits[kTkRounds] = {11, 11, 10};
constexpr int kTkMaxBins = 2048;
constexpr int kTkLastBins = 1 << 10;
// workspace (uint32): the prefix and the entries still to take within it
// after the digits of rounds 0 and 1 (two slots: a launch reads one and
// stores the next), one histogram per round, then the last round's histogram
// of every workgroup
constexpr int kTkSel = 0;  // round r's result: kTkSel + 2r (prefix), + 1 (need)
constexpr int kTkHist = 4;
constexpr int kTkWgHist = kTkHist + kTkRounds * kTkMaxBins;

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
  for (int i = threadIdx.x; i < kTkWgHist; i += kTkThreads) p.state[i] = 0u;
}

// The digit of round R: with the keys of round R's global histogram that
// match `prefix` counted per digit, the largest digit whose bucket holds the
// need-th largest of them.  Thread t takes the bins NB - 1 - per t down to
// NB - per (t + 1); its exclusive scan is the count above its first bin and
// the one thread whose bins cross `need` finds the digit.  Every thread gets
// the grown prefix and what is still to take within it.
template <int R>
__device__ __forceinline__ void select_digit(const TopkParams& p, uint32_t& prefix, uint32_t& need, int64_t* red,
                                             uint32_t* out) {
  constexpr int NB = 1 << kTkBits[R];
  constexpr int per = NB / kTkThreads;
  static_assert(NB % kTkThreads == 0, "bins spread evenly over the threads");
  const uint32_t* g = p.state + kTkHist + R * kTkMaxBins;
  uint32_t h[per];
  int64_t mine = 0;
#pragma unroll
  for (int j = 0; j < per; ++j) {
    h[j] = g[NB - 1 - (per * threadIdx.x + j)];
    mine += h[j];
  }
  int64_t all;
  int64_t above = block_exclusive_scan<kTkThreads>(mine, red, &all);
#pragma unroll
  for (int j = 0; j < per; ++j) {
    if (above < (int64_t)need && above + h[j] >= (int64_t)need) {
      out[0] = prefix | ((uint32_t)(NB - 1 - (per * threadIdx.x + j)) << kTkShift[R]);
      out[1] = need - (uint32_t)above;
    }
    above += h[j];
  }
  __syncthreads();
  prefix = out[0];
  need = out[1];
}

// Round R: the previous round's digit (R > 0), then this round's counts.
template <int R>
__global__ __launch_bounds__(kTkThreads) void topk_round_kernel(TopkParams p) {
  constexpr int shift = kTkShift[R];
  constexpr int NB = 1 << kTkBits[R];
  __shared__ uint32_t hist[kTkWaves][NB];
  __shared__ int64_t red[kTkWaves + 1];
  __shared__ uint32_t sel[2];
  const int tid = threadIdx.x;
  const int wave = tid / kWave;
  for (int i = tid; i < kTkWaves * NB; i += kTkThreads) (&hist[0][0])[i] = 0u;
  uint32_t prefix = 0u, need = (uint32_t)p.k;
  if constexpr (R > 0) {
    if constexpr (R > 1) {
      prefix = p.state[kTkSel + 2 * (R - 2)];
      need = p.state[kTkSel + 2 * (R - 2) + 1];
    }
    select_digit<R - 1>(p, prefix, need, red, sel);
    if (blockIdx.x == 0 && tid == 0) {
      p.state[kTkSel + 2 * (R - 1)] = prefix;
      p.state[kTkSel + 2 * (R - 1) + 1] = need;
    }
  }
  __syncthreads();
  const uint32_t mask = R == 0 ? 0u : 0xFFFFFFFFu << ((shift + kTkBits[R]) & 31);
  int64_t c0, c1;
  chunk_of(p, blockIdx.x, c0, c1);
  for (int64_t i = c0 + tid * 4; i < c1; i += kTkStep) {
    uint32_t key[4];
    const uint32_t valid = load_keys(p.probs, i, c1, key);
#pragma unroll
    for (int e = 0; e < 4; ++e)
      if (((valid >> e) & 1u) && (key[e] & mask) == prefix) atomicAdd(&hist[wave][(key[e] >> shift) & (NB - 1)], 1u);
  }
  __syncthreads();
  uint32_t* g = p.state + kTkHist + R * kTkMaxBins;
  for (int i = tid; i < NB; i += kTkThreads) {
    uint32_t c = 0;
#pragma unroll
    for (int w = 0; w < kTkWaves; ++w) c += hist[w][i];
    if (R == kTkRounds - 1) p.state[kTkWgHist + (int64_t)blockIdx.x * kTkLastBins + i] = c;
    if (c) atomicAdd(&g[i], c);
  }
}

__global__ __launch_bounds__(kTkThreads) void topk_write_kernel(TopkParams p) {
  __shared__ int64_t red[kTkWaves + 1];
  __shared__ uint32_t sel[2];
  const int tid = threadIdx.x;
  // the last digit: thr is the K-th largest key, take the entries equal to
  // it that are kept
  uint32_t thr = 0u, take = 0u;
  if (p.k > 0) {
    thr = p.state[kTkSel + 2 * (kTkRounds - 2)];
    take = p.state[kTkSel + 2 * (kTkRounds - 2) + 1];
    select_digit<kTkRounds - 1>(p, thr, take, red, sel);
  }
  // entries equal to thr in the chunks before this one
  uint32_t before = 0;
  if (p.k > 0)
    for (int j = tid; j < (int)blockIdx.x; j += kTkThreads)
      before += p.state[kTkWgHist + (int64_t)j * kTkLastBins + (thr & (kTkLastBins - 1))];
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

size_t topk_workspace_bytes(int64_t n) {
  return ((size_t)kTkWgHist + (size_t)topk_blocks(n) * kTkLastBins) * sizeof(uint32_t);
}

hipError_t launch_topk_pattern(TopkParams p, hipStream_t stream) {
  if (p.n == 0) return hipSuccess;
  const int blocks = topk_blocks(p.n);
  // chunks are whole iterations of the workgroup's quadruples
  p.chunk = ((p.n + blocks - 1) / blocks + kTkStep - 1) / kTkStep * kTkStep;
  if (p.k > 0) {
    hipLaunchKernelGGL(topk_init_kernel, dim3(1), dim3(kTkThreads), 0, stream, p);
    hipLaunchKernelGGL(topk_round_kernel<0>, dim3(blocks), dim3(kTkThreads), 0, stream, p);
    hipLaunchKernelGGL(topk_round_kernel<1>, dim3(blocks), dim3(kTkThreads), 0, stream, p);
    hipLaunchKernelGGL(topk_round_kernel<2>, dim3(blocks), dim3(kTkThreads), 0, stream, p);
  }
  hipLaunchKernelGGL(topk_write_kernel, dim3(blocks), dim3(kTkThreads), 0, stream, p);
  return hipGetLastError();
}

}  // namespace dkv
