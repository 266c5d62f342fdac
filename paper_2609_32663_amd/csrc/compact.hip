// One-time prune and pack of the KV cache (Distance-KV, Sec. 3.4 / Fig. 2(b)),
// and the append of new tokens.
//
// The pack is an order-preserving stream compaction in three passes over the
// (segment, 4096-position tile) grid:
//   count   each tile counts its retained positions (16 mask bytes per lane,
//           nonzero-byte popcount, block reduction);
//   scan    one workgroup turns tile counts into each tile's first rank within
//           its segment, the segment lengths, and the segment offsets
//           (running sum of length + append capacity, unit-major);
//   gather  two workgroups per tile, one for K and one for V, each rebuild
//           the tile's ranks with a block scan, list its retained positions
//           in rank order in LDS, and copy the rows: LPR lanes move one row
//           with 16-byte loads and stores (LPR = row bytes / 16), so a wave
//           moves 64/LPR whole rows per instruction, 8 rows per lane group in
//           flight.  (One workgroup copying both K and V ran 6% slower: four
//           interleaved streams per workgroup instead of two.)
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
  block_exclusive_scan<kThreads>(c, red, &total);
  if (threadIdx.x == 0) p.tile_cnt[(int64_t)seg * p.ntiles + tile] = (int32_t)total;
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

template <int LPR>
__global__ __launch_bounds__(kThreads) void compact_gather_kernel(CompactParams p) {
  constexpr int kRowsPerPass = kThreads / LPR;
  constexpr int kUnroll = 8;
  __shared__ uint16_t list[kCompactTile];
  __shared__ int64_t red[kThreads / kWave + 1];

  const int tile = blockIdx.x >> 1;
  const int which = blockIdx.x & 1;  // 0: K rows (and source positions), 1: V rows
  const int seg = blockIdx.y;
  const int tid = threadIdx.x;
  if (p.seg_len[seg] < 0) return;  // not packed: it does not fit below out_rows
  const uint8_t* mrow = p.mask + (int64_t)seg * p.T;
  const int64_t jt = (int64_t)tile * kCompactTile;
  const u32x4 w = load_mask16(mrow, jt + tid * kPerThread, p.T);
  const uint32_t bits = nonzero_byte_bits(w);
  int64_t kept;
  int rank = (int)block_exclusive_scan<kThreads>(__popc(bits), red, &kept);
#pragma unroll
  for (int e = 0; e < kPerThread; ++e)
    if ((bits >> e) & 1u) list[rank++] = (uint16_t)(tid * kPerThread + e);
  __syncthreads();

  const int64_t dst0 = p.seg_off[seg] + p.tile_base[(int64_t)seg * p.ntiles + tile];
  const int64_t src0 = (int64_t)seg * p.T + jt;
  const int lane = tid % LPR;
  const int64_t stride16 = p.row_bytes / 16;  // == LPR
  const u32x4* src = reinterpret_cast<const u32x4*>(which ? p.v : p.k);
  u32x4* dst = reinterpret_cast<u32x4*>(which ? p.v_out : p.k_out);

  for (int r0 = tid / LPR; r0 < kept; r0 += kRowsPerPass * kUnroll) {
    u32x4 rb[kUnroll];
    int64_t drow[kUnroll];
    bool ok[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int r = r0 + u * kRowsPerPass;
      drow[u] = dst0 + r;
      ok[u] = r < kept;
      if (ok[u]) rb[u] = src[(src0 + list[r]) * stride16 + lane];
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      if (ok[u]) {
        dst[drow[u] * stride16 + lane] = rb[u];
        if (which == 0 && lane == 0 && p.src_pos != nullptr)
          p.src_pos[drow[u]] = (int32_t)(jt + list[r0 + u * kRowsPerPass]);
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
  return (size_t)(2 * n * 4 + 256);
}

hipError_t launch_compact(const CompactParams& p, hipStream_t stream) {
  const dim3 grid(p.ntiles > 0 ? p.ntiles : 1, p.nseg);
  if (p.ntiles > 0) {
    hipLaunchKernelGGL(compact_count_kernel, grid, dim3(kThreads), 0, stream, p);
  }
  hipLaunchKernelGGL(compact_scan_kernel, dim3(1), dim3(kScanThreads), 0, stream, p);
  if (p.ntiles > 0) {
    const dim3 ggrid(2 * p.ntiles, p.nseg);  // a K and a V workgroup per tile
    switch (p.row_bytes) {
      case 128: hipLaunchKernelGGL(compact_gather_kernel<8>, ggrid, dim3(kThreads), 0, stream, p); break;
      case 256: hipLaunchKernelGGL(compact_gather_kernel<16>, ggrid, dim3(kThreads), 0, stream, p); break;
      case 512: hipLaunchKernelGGL(compact_gather_kernel<32>, ggrid, dim3(kThreads), 0, stream, p); break;
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
