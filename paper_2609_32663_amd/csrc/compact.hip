// One-time prune and pack of the KV cache (Distance-KV, Sec. 3.4 / Fig. 2(b)),
// and the append of new tokens.
//
// The pack is an order-preserving stream compaction in three passes:
//   count   each (segment, 4096-position tile) counts its retained positions
//           (16 mask bytes per lane, nonzero-byte popcount, block scan) and
//           records where each of its kCompactSub-position sub-tiles starts
//           in the tile's rank order;
//   scan    one workgroup turns tile counts into each tile's first rank within
//           its segment, the segment lengths, and the segment offsets
//           (running sum of length + append capacity, unit-major);
//   gather  two workgroups of 256 lanes per sub-tile, one for K and one for
//           V, each rank the sub-tile's positions with a block scan, list the
//           retained ones in LDS, and copy the rows: LPR lanes move one row
//           with 16-byte non-temporal loads and stores (LPR = row bytes / 16),
//           so a wave moves 64/LPR whole rows per instruction and a lane
//           group moves at most kCompactSub * LPR / 256 rows.
// Short workgroups copy fastest.  On the Llama-3.1-8B-shaped 128K stack (35%
// kept) whole 4096-position tiles per gather workgroup took 2.50-2.55 ms
// whatever the rows in flight per lane group (1 to 8); sub-tiles of 256, 128,
// 64 and 32 positions took 2.18, 2.09-2.10, 2.06-2.07 and 2.48-2.50 ms, and
// on the Qwen-shaped stack 2.78-2.80, 2.65-2.68, 2.81 and 3.72 ms (with 32
// the launch holds two to four million workgroups).  (One workgroup copying both K
// and V ran 6% slower: four interleaved streams per workgroup instead of two.)
// All row arithmetic is 64-bit: a whole-stack cache has more than 2^31 elements.

#include "dkv_device.hpp"
#include "dkv_launch.hpp"

namespace dkv {

namespace {

constexpr int kThreads = 256;
constexpr int kPerThread = 16;
static_assert(kThreads * kPerThread == kCompactTile, "tile = threads x 16 positions");

__global__ __launch_bounds__(kThreads) void compact_count_kernel(CompactParams p) {
  __shared__ int64_t red[kThreads / kWave + 1];
  const int tile = blockIdx.x;
  const int seg = blockIdx.y;
  const uint8_t* row = p.mask + (int64_t)seg * p.T;
  const int64_t j0 = (int64_t)tile * kCompactTile + threadIdx.x * kPerThread;
  const u32x4 w = load_mask16(row, j0, p.T);
  const int64_t c = nonzero_bytes(w[0]) + nonzero_bytes(w[1]) + nonzero_bytes(w[2]) + nonzero_bytes(w[3]);
  int64_t total;
  const int64_t before = block_exclusive_scan<kThreads>(c, red, &total);
  const int64_t ti = (int64_t)seg * p.ntiles + tile;
  if (threadIdx.x == 0) p.tile_cnt[ti] = (int32_t)total;
  constexpr int kLanesPerSub = kCompactSub / kPerThread;
  if (threadIdx.x % kLanesPerSub == 0)  // rank of the sub-tile's first position: < 4096
    p.sub_base[ti * kCompactSubPerTile + threadIdx.x / kLanesPerSub] = (uint16_t)before;
}

constexpr int kScanThreads = 1024;

__global__ __launch_bounds__(kScanThreads) void compact_scan_kernel(CompactParams p) {
  __shared__ int64_t red[kScanThreads / kWave + 1];
  __shared__ int64_t carry;
  if (threadIdx.x == 0) carry = 0;
  __syncthreads();
  for (int64_t s0 = 0; s0 < p.nseg; s0 += kScanThreads) {
    const int64_t s = s0 + threadIdx.x;
    int64_t len = 0;
    if (s < p.nseg) {
      int32_t run = 0;
      const int64_t base = s * p.ntiles;
      for (int t = 0; t < p.ntiles; ++t) {
        const int32_t c = p.tile_cnt[base + t];
        p.tile_base[base + t] = run;
        run += c;
      }
      len = run;
    }
    const int64_t need = s < p.nseg ? len + p.cap : 0;
    int64_t chunk_total;
    const int64_t excl = block_exclusive_scan<kScanThreads>(need, red, &chunk_total);
    if (s < p.nseg) {
      // A segment whose rows and append room do not fit below out_rows is
      // not packed: its length becomes the marker -1 (every call that reads
      // lengths treats it as a segment with no rows and no room) and its
      // offset is clamped to out_rows, so no offset handed out points past
      // the buffer.
      const int64_t off = carry + excl;
      const bool fits = off + need <= p.out_rows;
      p.seg_off[s] = fits ? off : (off < p.out_rows ? off : p.out_rows);
      p.seg_len[s] = fits ? (int32_t)len : -1;
    }
    __syncthreads();
    if (threadIdx.x == 0) carry += chunk_total;
    __syncthreads();
  }
  if (threadIdx.x == 0 && p.rows_needed != nullptr) *p.rows_needed = carry;
}

constexpr int kGatherThreads = 256;  // lanes < kCompactSub each rank one position
static_assert(kCompactSub <= kGatherThreads && kCompactSub % 16 == 0, "sub-tile fits the workgroup");

template <int LPR>
__global__ __launch_bounds__(kGatherThreads) void compact_gather_kernel(CompactParams p) {
  constexpr int kRowsPerPass = kGatherThreads / LPR;
  constexpr int kPasses = (kCompactSub + kRowsPerPass - 1) / kRowsPerPass;
  constexpr int kUnroll = kPasses < 8 ? kPasses : 8;  // rows per lane group in flight
  __shared__ uint16_t list[kCompactSub];
  __shared__ int64_t red[kGatherThreads / kWave + 1];

  const int sub = blockIdx.x >> 1;
  const int which = blockIdx.x & 1;  // 0: K rows (and source positions), 1: V rows
  const int seg = blockIdx.y;
  const int tid = threadIdx.x;
  if (p.seg_len[seg] < 0) return;  // not packed: it does not fit below out_rows
  const int64_t js = (int64_t)sub * kCompactSub;
  const bool keep = tid < kCompactSub && js + tid < p.T && p.mask[(int64_t)seg * p.T + js + tid] != 0;
  int64_t kept;
  const int rank = (int)block_exclusive_scan<kGatherThreads>(keep ? 1 : 0, red, &kept);
  if (keep) list[rank] = (uint16_t)tid;
  __syncthreads();
  if (kept == 0) return;  // (the same for every lane)

  const int tile = sub / kCompactSubPerTile;
  const int64_t ti = (int64_t)seg * p.ntiles + tile;
  const int64_t dst0 = p.seg_off[seg] + p.tile_base[ti] + p.sub_base[ti * kCompactSubPerTile + (sub - tile * kCompactSubPerTile)];
  const int64_t src0 = (int64_t)seg * p.T + js;
  const int lane = tid % LPR;
  const u32x4* src = reinterpret_cast<const u32x4*>(which ? p.v : p.k);
  u32x4* dst = reinterpret_cast<u32x4*>(which ? p.v_out : p.k_out);

  for (int r0 = tid / LPR; r0 < kept; r0 += kRowsPerPass * kUnroll) {
    u32x4 rb[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int r = r0 + u * kRowsPerPass;
      if (r < kept) rb[u] = __builtin_nontemporal_load(&src[(src0 + list[r]) * LPR + lane]);
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int r = r0 + u * kRowsPerPass;
      if (r < kept) {
        __builtin_nontemporal_store(rb[u], &dst[(dst0 + r) * LPR + lane]);
        if (which == 0 && lane == 0 && p.src_pos != nullptr) p.src_pos[dst0 + r] = (int32_t)(js + list[r]);
      }
    }
  }
}

__global__ __launch_bounds__(kThreads) void append_kernel(AppendParams p) {
  const int lpr = p.row_bytes / 16;
  const int64_t gid = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  const int64_t row_id = gid / lpr;
  const int lane = (int)(gid - row_id * lpr);
  if (row_id >= (int64_t)p.nseg * p.n_new) return;
  const int64_t s = row_id / p.n_new;
  const int64_t t = row_id - s * p.n_new;
  if (p.seg_len[s] < 0) return;  // a segment dkv_compact could not pack has no room
  const int64_t drow = p.seg_off[s] + p.seg_len[s] + p.n_tail + t;
  const u32x4* ks = reinterpret_cast<const u32x4*>(p.k_new);
  const u32x4* vs = reinterpret_cast<const u32x4*>(p.v_new);
  reinterpret_cast<u32x4*>(p.k_c)[drow * lpr + lane] = ks[row_id * lpr + lane];
  reinterpret_cast<u32x4*>(p.v_c)[drow * lpr + lane] = vs[row_id * lpr + lane];
}

}  // namespace

size_t compact_workspace_bytes(int64_t nseg, int64_t T) {
  const int64_t ntiles = (T + kCompactTile - 1) / kCompactTile;
  const int64_t n = nseg * (ntiles > 0 ? ntiles : 1);
  return (size_t)(2 * n * 4 + n * kCompactSubPerTile * 2 + 256);  // tile counts, tile bases, sub-tile bases
}

hipError_t launch_compact(const CompactParams& p, hipStream_t stream) {
  const dim3 grid(p.ntiles > 0 ? p.ntiles : 1, p.nseg);
  if (p.ntiles > 0) {
    hipLaunchKernelGGL(compact_count_kernel, grid, dim3(kThreads), 0, stream, p);
  }
  hipLaunchKernelGGL(compact_scan_kernel, dim3(1), dim3(kScanThreads), 0, stream, p);
  if (p.ntiles > 0) {
    const int64_t nsub = ((int64_t)p.T + kCompactSub - 1) / kCompactSub;
    const dim3 ggrid((uint32_t)(2 * nsub), p.nseg);  // a K and a V workgroup per sub-tile
    switch (p.row_bytes) {
      case 128: hipLaunchKernelGGL(compact_gather_kernel<8>, ggrid, dim3(kGatherThreads), 0, stream, p); break;
      case 256: hipLaunchKernelGGL(compact_gather_kernel<16>, ggrid, dim3(kGatherThreads), 0, stream, p); break;
      case 512: hipLaunchKernelGGL(compact_gather_kernel<32>, ggrid, dim3(kGatherThreads), 0, stream, p); break;
      default: return hipErrorInvalidValue;
    }
  }
  return hipGetLastError();
}

hipError_t launch_append(const AppendParams& p, hipStream_t stream) {
  const int64_t threads = (int64_t)p.nseg * p.n_new * (p.row_bytes / 16);
  const int64_t blocks = (threads + kThreads - 1) / kThreads;
  if (blocks > 0) hipLaunchKernelGGL(append_kernel, dim3((uint32_t)blocks), dim3(kThreads), 0, stream, p);
  return hipGetLastError();
}

}  // namespace dkv
