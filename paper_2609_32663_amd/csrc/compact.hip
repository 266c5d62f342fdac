// One-time prune and pack of the KV cache (Distance-KV, Sec. 3.4 / Fig. 2(b)),
// and the append of new tokens.
//
// The pack is an order-preserving stream compaction in four passes:
//   count   each (segment, 4096-position tile) counts its retained positions
//           (16 mask bytes per lane, nonzero-byte popcount, block scan);
//   scan    one workgroup turns tile counts into each tile's first rank within
//           its segment, the segment lengths, and the segment offsets
//           (running sum of length + append capacity, unit-major);
//   list    each tile with retained positions ranks them again (block scan),
//           orders them in LDS and writes them, coalesced, to a per-segment
//           list at their rank: list[s][r] is the position of packed row r;
//   copy    a K and a V workgroup per (segment, chunk of kCopyRows packed
//           rows): LPR lanes move one row with 16-byte non-temporal loads and
//           stores (LPR = row bytes / 16), the source row being the list's
//           entry.
// The copy works on the output side because short workgroups copy fastest on
// this part and every copy workgroup then has whole rows to move: on the
// Llama-3.1-8B-shaped 128K stack (35% kept) the pack takes 1.91-1.97 ms this
// way, against 2.09-2.15 ms for a gather per 128-position input sub-tile (most
// of them empty, the others up to 32 KiB) and 2.50-2.55 ms for one per
// 4096-position tile.  (One workgroup copying both K and
// V ran 6% slower in the block gather: four interleaved streams per
// workgroup instead of two.)
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
      // the segment's tile counts eight at a time, all eight loads in flight
      int32_t run = 0;
      const int64_t base = s * p.ntiles;
      for (int t0 = 0; t0 < p.ntiles; t0 += 8) {
        int32_t c[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) c[e] = p.tile_cnt[base + (t0 + e < p.ntiles ? t0 + e : p.ntiles - 1)];
#pragma unroll
        for (int e = 0; e < 8; ++e)
          if (t0 + e < p.ntiles) {
            p.tile_base[base + t0 + e] = run;
            run += c[e];
          }
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

__global__ __launch_bounds__(kThreads) void compact_list_kernel(CompactParams p) {
  __shared__ int64_t red[kThreads / kWave + 1];
  __shared__ int32_t pos[kCompactTile];
  const int tile = blockIdx.x;
  const int seg = blockIdx.y;
  const int64_t ti = (int64_t)seg * p.ntiles + tile;
  // not packed (it does not fit below out_rows), or nothing kept in this tile
  if (p.seg_len[seg] < 0 || p.tile_cnt[ti] == 0) return;
  const int64_t j0 = (int64_t)tile * kCompactTile + threadIdx.x * kPerThread;
  const u32x4 w = load_mask16(p.mask + (int64_t)seg * p.T, j0, p.T);
  const int64_t c = nonzero_bytes(w[0]) + nonzero_bytes(w[1]) + nonzero_bytes(w[2]) + nonzero_bytes(w[3]);
  int64_t total;
  int r = (int)block_exclusive_scan<kThreads>(c, red, &total);
  const uint32_t bits = nonzero_byte_bits(w);
#pragma unroll
  for (int e = 0; e < kPerThread; ++e)
    if (bits & (1u << e)) pos[r++] = (int32_t)(j0 + e);
  __syncthreads();
  int32_t* dst = p.list + (int64_t)seg * p.T + p.tile_base[ti];
  for (int i = threadIdx.x; i < total; i += kThreads) dst[i] = pos[i];
}

template <int LPR>
__global__ __launch_bounds__(kThreads) void compact_copy_kernel(CompactParams p) {
  constexpr int kRowsPerPass = kThreads / LPR;
  constexpr int kPasses = (kCopyRows + kRowsPerPass - 1) / kRowsPerPass;  // rows per lane group
  static_assert(kPasses <= 8, "rows in flight per lane group");
  const int chunk = blockIdx.x >> 1;
  const int which = blockIdx.x & 1;  // 0: K rows (and source positions), 1: V rows
  const int seg = blockIdx.y;
  const int tid = threadIdx.x;
  const int lane = tid % LPR;
  const int64_t r_lo = (int64_t)chunk * kCopyRows;
  // Most workgroups of the grid lie past their segment's rows: they leave
  // after one scalar load.
  const int32_t len = p.seg_len[seg];
  if (len <= 0 || r_lo >= len) return;  // past the segment's rows, or not packed
  const int64_t r_hi = r_lo + kCopyRows < len ? r_lo + kCopyRows : len;
  const int32_t* list = p.list + (int64_t)seg * p.T;
  int32_t pos[kPasses];
#pragma unroll
  for (int u = 0; u < kPasses; ++u) {
    const int64_t r = r_lo + tid / LPR + (int64_t)u * kRowsPerPass;
    pos[u] = list[r < r_hi ? r : r_lo];
  }
  // Every list entry is waited for at once, then every row load is issued
  // before any is waited for (rows past the chunk's end load its first
  // row): waiting per row would also wait for the row loads before it.
#pragma unroll
  for (int u = 0; u < kPasses; ++u) asm volatile("" ::"v"(pos[u]));
  const int64_t dst0 = p.seg_off[seg];
  const int64_t src0 = (int64_t)seg * p.T;
  const u32x4* src = reinterpret_cast<const u32x4*>(which ? p.v : p.k);
  u32x4* dst = reinterpret_cast<u32x4*>(which ? p.v_out : p.k_out);
  u32x4 rb[kPasses];
#pragma unroll
  for (int u = 0; u < kPasses; ++u) rb[u] = __builtin_nontemporal_load(&src[(src0 + pos[u]) * LPR + lane]);
#pragma unroll
  for (int u = 0; u < kPasses; ++u) {
    const int64_t r = r_lo + tid / LPR + (int64_t)u * kRowsPerPass;
    if (r < r_hi) {
      __builtin_nontemporal_store(rb[u], &dst[(dst0 + r) * LPR + lane]);
      if (which == 0 && lane == 0 && p.src_pos != nullptr) p.src_pos[dst0 + r] = pos[u];
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
  return (size_t)(2 * n * 4 + nseg * T * 4 + 256);  // tile counts, tile bases, position lists
}

hipError_t launch_compact(const CompactParams& p, hipStream_t stream) {
  const dim3 grid(p.ntiles > 0 ? p.ntiles : 1, p.nseg);
  if (p.ntiles > 0) {
    hipLaunchKernelGGL(compact_count_kernel, grid, dim3(kThreads), 0, stream, p);
  }
  hipLaunchKernelGGL(compact_scan_kernel, dim3(1), dim3(kScanThreads), 0, stream, p);
  if (p.ntiles > 0) {
    hipLaunchKernelGGL(compact_list_kernel, grid, dim3(kThreads), 0, stream, p);
    const dim3 cgrid((uint32_t)(2 * compact_chunks(p.T)), p.nseg);  // a K and a V workgroup per chunk
    switch (p.row_bytes) {
      case 128: hipLaunchKernelGGL(compact_copy_kernel<8>, cgrid, dim3(kThreads), 0, stream, p); break;
      case 256: hipLaunchKernelGGL(compact_copy_kernel<16>, cgrid, dim3(kThreads), 0, stream, p); break;
      case 512: hipLaunchKernelGGL(compact_copy_kernel<32>, cgrid, dim3(kThreads), 0, stream, p); break;
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
