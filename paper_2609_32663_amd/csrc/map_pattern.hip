// Pattern -> per-KV-head keep mask (Distance-KV, Sec. 3.4, Eq. (4)-(5) and the
// GQA union).
//
// One workgroup per (unit, KV head) segment and chunk of kMapChunk positions
// (a 128K context is 8 chunks, so the grid fills the chip).  The group's G
// pattern rows are folded into one G-bit word per bin in LDS (bit h = query
// head g*G+h keeps the bin), so the union over the group is "word != 0" and
// the per-head decision is one bit.  Each thread then owns 16 consecutive
// positions per sweep: it classifies each as sink / recent / binned /
// uncovered, looks the bin up (a division for uniform edges, a binary search
// over the edges in LDS otherwise), and writes 16 mask bytes with one 16-byte
// store when the row is 16-byte aligned.  A run inside one region, or with one
// bin edge inside it (its first b positions in one bin, the rest in the next),
// is settled from its two ends; only runs that cross more (a region boundary,
// or bins narrower than a run) go position by position, and then so does their
// whole wave.  The retained length is not counted
// from the mask: the first chunk of each segment writes it from the closed
// form of Eq. (4)-(5), |sink U recent| plus the width (clipped to the
// compressible span) of every bin some head of the group keeps, with one
// plain store, so the call is one kernel with no atomics or clearing pass.
// In a ragged batch a unit's context is the first unit_len[n] positions of
// its row: distances count from its end and the rest of the row is not
// retained.

#include "dkv_device.hpp"
#include "dkv_launch.hpp"

namespace dkv {

namespace {

constexpr int kMapThreads = 256;
constexpr int kMapPerThread = 16;
constexpr int kMapChunk = 4 * kMapThreads * kMapPerThread;  // positions per workgroup

// Chunks per segment; at least one, whose workgroup writes the length.
__host__ __device__ inline int64_t map_chunks(int32_t T) {
  const int64_t c = ((int64_t)T + kMapChunk - 1) / kMapChunk;
  return c > 0 ? c : 1;
}

__device__ __forceinline__ int find_bin(int32_t u, const int32_t* edges, int D, int uniform_w) {
  if (uniform_w > 0) {
    const int32_t k = u / uniform_w;
    return k < D ? k : -1;
  }
  if (u >= edges[D]) return -1;
  int lo = 0, hi = D;  // edges[lo] <= u < edges[hi]
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (edges[mid] <= u) lo = mid; else hi = mid;
  }
  return lo;
}

__global__ __launch_bounds__(kMapThreads) void map_pattern_kernel(MapParams p) {
  extern __shared__ __align__(16) uint8_t smem[];
  __shared__ int64_t red[kMapThreads / kWave + 1];

  const int chunks = (int)map_chunks(p.T);
  const int seg = (int)(blockIdx.x / chunks);
  const int64_t chunk0 = (int64_t)(blockIdx.x - (int64_t)seg * chunks) * kMapChunk;
  const int64_t chunk1 = chunk0 + kMapChunk < p.T ? chunk0 + kMapChunk : p.T;
  const int unit = seg / p.Hkv;
  const int g = seg - unit * p.Hkv;
  const int tid = threadIdx.x;
  const int D = p.D, T = p.T, G = p.G;

  uint16_t* qbits = reinterpret_cast<uint16_t*>(smem);
  int32_t* edges = reinterpret_cast<int32_t*>(smem + ((D * 2 + 15) & ~15));

  const uint8_t* prow = p.pattern + ((int64_t)unit * p.Hq + (int64_t)g * G) * D;
  for (int k = tid; k < D; k += kMapThreads) {
    uint32_t bits = 0;
    for (int h = 0; h < G; ++h) bits |= (prow[(int64_t)h * D + k] != 0 ? 1u : 0u) << h;
    qbits[k] = (uint16_t)bits;
  }
  if (p.uniform_width == 0)
    for (int k = tid; k <= D; k += kMapThreads) edges[k] = p.edges[k];
  __syncthreads();

  const uint32_t all_heads = (1u << G) - 1u;
  const bool aligned_rows = (T & 15) == 0;
  // this unit's context length (clamped into the row)
  int32_t Tn = T;
  if (p.unit_len != nullptr) {
    Tn = p.unit_len[unit];
    Tn = Tn < 0 ? 0 : (Tn > T ? T : Tn);
  }
  uint8_t* kv_row = p.kv_mask + (int64_t)seg * T;

  if (chunk0 == 0) {
    // retained length, closed form: min(Tn, S + R) always-kept positions,
    // then every kept bin's offsets [E[k], E[k+1]) within the compressible
    // span [0, Tn - S - R)
    const int64_t span = (int64_t)Tn - p.S - p.R;
    int64_t part = 0;
    for (int k = tid; k < D && span > 0; k += kMapThreads) {
      if (qbits[k] == 0) continue;
      const int64_t lo = p.uniform_width > 0 ? (int64_t)p.uniform_width * k : edges[k];
      const int64_t hi_e = p.uniform_width > 0 ? (int64_t)p.uniform_width * (k + 1) : edges[k + 1];
      const int64_t hi = hi_e < span ? hi_e : span;
      if (hi > lo) part += hi - lo;
    }
    int64_t binned;
    block_exclusive_scan<kMapThreads>(part, red, &binned);
    const int64_t always = (int64_t)p.S + p.R < Tn ? (int64_t)p.S + p.R : Tn;
    if (tid == 0) p.kv_len[seg] = (int32_t)(always + binned);
  }

  const int32_t e_end = p.uniform_width > 0 ? 0 : edges[D];  // general edges: the covered span
  // positions fit 31 bits (T is an int32): the sweep runs in 32-bit arithmetic
  const int32_t c0 = (int32_t)chunk0, c1 = (int32_t)chunk1;
  for (int32_t j0 = c0 + tid * kMapPerThread; j0 < c1; j0 += kMapThreads * kMapPerThread) {
    uint32_t hb[kMapPerThread];
    // Most runs lie in one region (sink, recent window, one bin, uncovered, or
    // past the context): classify the run once and give every position the
    // same bits.  Runs across a boundary take the per-position path below.
    const int32_t jl = j0 + kMapPerThread - 1;
    bool one = false;   // every position of the run has the bits rb
    bool two = false;   // one bin edge inside: the first b positions rb, the rest rl
    uint32_t rb = 0, rl = 0;
    int32_t b = kMapPerThread;
    if (j0 >= Tn) {
      one = true;  // past this unit's context: nothing retained
    } else if (jl < Tn) {
      const int32_t d0 = Tn - 1 - j0, dl = Tn - 1 - jl;  // d0 > dl
      if (jl < p.S || d0 < p.R) {
        one = true;
        rb = all_heads;
      } else if (j0 >= p.S && dl >= p.R) {
        const int32_t u0 = d0 - p.R, ul = dl - p.R;  // u0 > ul >= 0
        if (p.uniform_width > 0) {
          const int32_t k0 = u0 / p.uniform_width, kl = ul / p.uniform_width;
          rb = k0 < D ? qbits[k0] : 0u;
          if (k0 == kl) {
            one = true;
          } else if (k0 == kl + 1) {
            two = true;
            rl = kl < D ? qbits[kl] : 0u;
            b = u0 - k0 * p.uniform_width + 1;
          }
        } else if (ul >= e_end) {
          one = true;  // past the last edge: uncovered
        } else if (u0 < e_end) {
          const int k0 = find_bin(u0, edges, D, 0);
          const int32_t e0 = edges[k0];
          rb = qbits[k0];
          if (ul >= e0) {
            one = true;
          } else if (ul >= edges[k0 - 1]) {  // k0 >= 1 here: edges[0] = 0 <= ul
            two = true;
            rl = qbits[k0 - 1];
            b = u0 - e0 + 1;
          }
        }
      }
    }
    if (__builtin_amdgcn_ballot_w64(!one) == 0) {
      // the wave's runs are all uniform
      const uint32_t wb = rb != 0u ? 0x01010101u : 0u;
      const u32x4 w = {wb, wb, wb, wb};
      if (aligned_rows) {
        *reinterpret_cast<u32x4*>(kv_row + j0) = w;
      } else {
#pragma unroll
        for (int e = 0; e < kMapPerThread; ++e)
          if (j0 + e < T) kv_row[j0 + e] = rb != 0u ? 1 : 0;
      }
      if (p.q_mask != nullptr) {
        for (int h = 0; h < G; ++h) {
          uint8_t* q_row = p.q_mask + ((int64_t)unit * p.Hq + (int64_t)g * G + h) * T;
          const uint8_t qb = (uint8_t)((rb >> h) & 1u);
          if (aligned_rows) {
            const uint32_t x = qb ? 0x01010101u : 0u;
            *reinterpret_cast<u32x4*>(q_row + j0) = u32x4{x, x, x, x};
          } else {
#pragma unroll
            for (int e = 0; e < kMapPerThread; ++e)
              if (j0 + e < T) q_row[j0 + e] = qb;
          }
        }
      }
      continue;
    }
    if (__builtin_amdgcn_ballot_w64(!(one || two)) == 0) {
      // every run of the wave has at most one bin edge inside it: the first b
      // positions take rb, the others rl
      if (one) {
        rl = rb;
        b = kMapPerThread;
      }
      u32x4 w;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        uint32_t x = 0;
#pragma unroll
        for (int e4 = 0; e4 < 4; ++e4) x |= ((4 * q + e4 < b ? rb : rl) != 0u ? 1u : 0u) << (8 * e4);
        w[q] = x;
      }
      if (aligned_rows) {
        *reinterpret_cast<u32x4*>(kv_row + j0) = w;
      } else {
#pragma unroll
        for (int e = 0; e < kMapPerThread; ++e)
          if (j0 + e < T) kv_row[j0 + e] = (e < b ? rb : rl) != 0u ? 1 : 0;
      }
      if (p.q_mask != nullptr) {
        for (int h = 0; h < G; ++h) {
          uint8_t* q_row = p.q_mask + ((int64_t)unit * p.Hq + (int64_t)g * G + h) * T;
          if (aligned_rows) {
            u32x4 wq;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              uint32_t x = 0;
#pragma unroll
              for (int e4 = 0; e4 < 4; ++e4) x |= (((4 * q + e4 < b ? rb : rl) >> h) & 1u) << (8 * e4);
              wq[q] = x;
            }
            *reinterpret_cast<u32x4*>(q_row + j0) = wq;
          } else {
#pragma unroll
            for (int e = 0; e < kMapPerThread; ++e)
              if (j0 + e < T) q_row[j0 + e] = (uint8_t)(((e < b ? rb : rl) >> h) & 1u);
          }
        }
      }
      continue;
    }
    // General edges: along the run u = delta - R falls by one per position,
    // so the bin only moves down.  One binary search for the first covered
    // position, then a walk down the edges (usually no step: bins are wider
    // than the run) keeps LDS traffic to about one load per run.
    int kb = -1;       // bin of the previous covered position of the run
    int32_t eb = 0;    // its lower edge
#pragma unroll
    for (int e = 0; e < kMapPerThread; ++e) {
      const int32_t j = j0 + e;
      uint32_t bits = 0;
      if (j < Tn) {
        const int32_t delta = Tn - 1 - j;
        if (j < p.S || delta < p.R) {
          bits = all_heads;
        } else if (p.uniform_width > 0) {
          const int k = find_bin(delta - p.R, edges, D, p.uniform_width);
          if (k >= 0) bits = qbits[k];
        } else {
          const int32_t u = delta - p.R;
          if (u < e_end) {
            if (kb < 0) {
              kb = find_bin(u, edges, D, 0);
              eb = edges[kb];
            }
            while (u < eb) eb = edges[--kb];
            bits = qbits[kb];
          }
        }
      }
      hb[e] = bits;
    }
    u32x4 w;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      w[q] = (hb[4 * q] != 0u ? 1u : 0u) | (hb[4 * q + 1] != 0u ? 1u : 0u) << 8 |
             (hb[4 * q + 2] != 0u ? 1u : 0u) << 16 | (hb[4 * q + 3] != 0u ? 1u : 0u) << 24;
    }
    if (aligned_rows) {
      *reinterpret_cast<u32x4*>(kv_row + j0) = w;
    } else {
#pragma unroll
      for (int e = 0; e < kMapPerThread; ++e)
        if (j0 + e < T) kv_row[j0 + e] = hb[e] != 0u ? 1 : 0;
    }
    if (p.q_mask != nullptr) {
      for (int h = 0; h < G; ++h) {
        uint8_t* q_row = p.q_mask + ((int64_t)unit * p.Hq + (int64_t)g * G + h) * T;
        if (aligned_rows) {
          u32x4 w;
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            uint32_t x = 0;
#pragma unroll
            for (int b = 0; b < 4; ++b) x |= ((hb[4 * q + b] >> h) & 1u) << (8 * b);
            w[q] = x;
          }
          *reinterpret_cast<u32x4*>(q_row + j0) = w;
        } else {
#pragma unroll
          for (int e = 0; e < kMapPerThread; ++e)
            if (j0 + e < T) q_row[j0 + e] = (uint8_t)((hb[e] >> h) & 1u);
        }
      }
    }
  }
}

}  // namespace

int64_t map_blocks(int32_t T, int64_t num_segments) { return map_chunks(T) * num_segments; }

hipError_t launch_map_pattern(const MapParams& p, int num_segments, hipStream_t stream) {
  size_t lds = ((size_t)p.D * 2 + 15) & ~(size_t)15;
  if (p.uniform_width == 0) lds += (size_t)(p.D + 1) * 4;
  const int64_t blocks = map_blocks(p.T, num_segments);
  if (blocks > 0) hipLaunchKernelGGL(map_pattern_kernel, dim3((uint32_t)blocks), dim3(kMapThreads), lds, stream, p);
  return hipGetLastError();
}

}  // namespace dkv
