// Zero-copy alternative to the pack: list each segment's retained rows where
// they already are, in a cache kept in pages of page_rows consecutive
// positions.
//
// The retained set of a segment is the sink, the recent window and a union of
// whole distance bins (Eq. (4), Eq. (5), union of Sec. 3.4), so its positions
// form a few long runs.  Each run is cut at page boundaries and listed as an
// entry (physical page, logical page, lo, hi) naming slots [lo, hi) of one
// page; decode reads those slots in place.  With the paper's 128-token bins
// and 128-row pages every context entry is a whole page.
//
// Two passes over the (segment, 4096-position tile) grid:
//   count  each thread turns 16 mask bytes into a 16-bit keep mask; a run
//          starts at a kept position whose predecessor is not kept or that
//          opens a page; the tile sums its starts and kept positions;
//   emit   each workgroup adds up the run counts of its segment's earlier
//          tiles (its first entry), and each thread writes the entries whose
//          runs start in its 16 positions (page, logical page, lo) and the
//          end slot of the runs that end there; a run's entry index is its
//          start's rank.  The segment's last tile also writes the retained
//          length, the append region's entries (appended tokens are always
//          kept) and the entry count.
// (A separate scan pass, one thread per segment walking its tiles, took
// ~20 us of dependent loads; the prefix inside emit is one round trip.)
// Contexts of more than kSumTiles tiles (4M positions) keep that scan pass:
// there every emit workgroup summing all earlier tiles would cost work
// quadratic in the context length.
// A context of length 0 has no tile: one small kernel writes those segments.
// Page sizes are multiples of 16 that divide the tile, so a page boundary is
// always the boundary of a thread's 16 positions, and every wave's first
// lane starts a page: neighbouring bits come from the adjacent lane.

#include "dkv_device.hpp"
#include "dkv_launch.hpp"

namespace dkv {

namespace {

constexpr int kThreads = 256;
constexpr int kPerThread = 16;
constexpr int kSumTiles = 1024;  // longest context (in tiles) whose emit pass sums tile counts itself
static_assert(kThreads * kPerThread == kCompactTile, "tile = threads x 16 positions");

// Keep mask of this thread's 16 positions, and the run starts and ends among
// them.  A run starts where the previous position is not kept or a page
// begins, and ends where the next position is not kept or a page ends.
struct RunBits {
  uint32_t keep, starts, ends;
};

__device__ __forceinline__ RunBits run_bits(const PageSelectParams& p, int seg, int tile) {
  const int tid = threadIdx.x;
  const int64_t j0 = (int64_t)tile * kCompactTile + tid * kPerThread;
  const uint32_t keep = nonzero_byte_bits(load_mask16(p.mask + (int64_t)seg * p.T, j0, p.T));
  const uint32_t left = __shfl_up(keep, 1, kWave);
  const uint32_t right = __shfl_down(keep, 1, kWave);
  const bool page_first = (j0 % p.page_rows) == 0;
  const bool page_last = ((j0 + kPerThread) % p.page_rows) == 0;
  const uint32_t prev = page_first ? 0u : (left >> 15) & 1u;
  const uint32_t next = page_last ? 0u : right & 1u;
  RunBits r;
  r.keep = keep;
  r.starts = keep & ~((keep << 1) | prev);
  r.ends = keep & ~((keep >> 1) | (next << 15));
  return r;
}

__global__ __launch_bounds__(kThreads) void page_count_kernel(PageSelectParams p) {
  __shared__ int64_t red[kThreads / kWave + 1];
  const int tile = blockIdx.x;
  const int seg = blockIdx.y;
  const RunBits r = run_bits(p, seg, tile);
  int64_t starts, kept;
  block_exclusive_scan<kThreads>(__popc(r.starts), red, &starts);
  block_exclusive_scan<kThreads>(__popc(r.keep), red, &kept);
  if (threadIdx.x == 0) {
    p.tile_cnt[(int64_t)seg * p.ntiles + tile] = (int32_t)starts;
    p.tile_kept[(int64_t)seg * p.ntiles + tile] = (int32_t)kept;
  }
  // clear the usage flags of this tile's pages; the emit pass sets the used ones
  if (p.page_used != nullptr) {
    const int per_tile = kCompactTile / p.page_rows;
    const int64_t pg0 = (int64_t)tile * per_tile;
    for (int i = threadIdx.x; i < per_tile; i += kThreads)
      if (pg0 + i < p.pages_per_seg) p.page_used[(int64_t)seg * p.pages_per_seg + pg0 + i] = 0;
  }
}

// The append region [T, T + cap) of segment s: one entry per page it touches,
// after the segment's n context entries; returns the segment's entry count.
// Also marks those pages used and clears the flags of pages past the context
// tiles that the region does not use.  One thread.
__device__ int32_t finish_segment(const PageSelectParams& p, int s, int32_t n) {
  const int pr = p.page_rows;
  if (p.cap > 0) {
    const int64_t first = (int64_t)p.T / pr, last = ((int64_t)p.T + p.cap - 1) / pr;
    for (int64_t lp = first; lp <= last; ++lp, ++n) {
      const int32_t page = p.table[(int64_t)s * p.pages_per_seg + lp];
      if (n < p.max_entries) {
        int32_t* e = p.entries + ((int64_t)s * p.max_entries + n) * 4;
        const int64_t lo = (p.T > lp * pr ? p.T : lp * pr) - lp * pr;
        const int64_t end = (int64_t)p.T + p.cap < (lp + 1) * pr ? (int64_t)p.T + p.cap : (lp + 1) * pr;
        e[0] = page;
        e[1] = (int32_t)lp;
        e[2] = (int32_t)lo;
        e[3] = (int32_t)(end - lp * pr);
      }
      if (p.page_used != nullptr) p.page_used[(int64_t)s * p.pages_per_seg + lp] = 1;
    }
  }
  if (p.page_used != nullptr) {
    const int64_t covered = (int64_t)p.ntiles * (kCompactTile / pr);
    const int64_t tail0 = p.cap > 0 ? (int64_t)p.T / pr : p.pages_per_seg;
    const int64_t tail1 = p.cap > 0 ? ((int64_t)p.T + p.cap - 1) / pr : -1;
    for (int64_t lp = covered; lp < p.pages_per_seg; ++lp)
      if (lp < tail0 || lp > tail1) p.page_used[(int64_t)s * p.pages_per_seg + lp] = 0;
  }
  return n;
}

// Long contexts: one thread per segment turns tile counts into each tile's
// first entry, then finishes the segment.
__global__ __launch_bounds__(kThreads) void page_scan_kernel(PageSelectParams p) {
  const int s = blockIdx.x * kThreads + threadIdx.x;
  if (s >= p.nseg) return;
  const int64_t base = (int64_t)s * p.ntiles;
  int32_t run = 0, kept = 0;
  for (int t = 0; t < p.ntiles; ++t) {
    p.tile_base[base + t] = run;
    run += p.tile_cnt[base + t];
    kept += p.tile_kept[base + t];
  }
  p.seg_len[s] = kept;
  p.n_entries[s] = finish_segment(p, s, run);
}

__global__ __launch_bounds__(kThreads) void page_emit_kernel(PageSelectParams p) {
  __shared__ int64_t red[kThreads / kWave + 1];
  const int tile = blockIdx.x;
  const int seg = blockIdx.y;
  // With tile_base (long contexts) the scan pass gave this tile its first
  // entry and finished the segment; otherwise the workgroup adds up the runs
  // that start in the segment's earlier tiles (high 32 bits; low 32 bits:
  // all its tiles' runs, which the last tile needs) and the last tile sums
  // the retained positions.
  const bool summed = p.tile_base == nullptr;
  const bool last_tile = summed && tile == p.ntiles - 1;
  int64_t before = 0, runs = 0, kept_part = 0;
  if (summed) {
    int64_t packed = 0;
    for (int t = threadIdx.x; t < p.ntiles; t += kThreads) {
      const int64_t c = p.tile_cnt[(int64_t)seg * p.ntiles + t];
      packed += (t < tile ? (c << 32) : 0) + c;
      if (last_tile) kept_part += p.tile_kept[(int64_t)seg * p.ntiles + t];
    }
    int64_t sums;
    block_exclusive_scan<kThreads>(packed, red, &sums);
    before = sums >> 32;
    runs = sums & 0xFFFFFFFFLL;
  } else {
    before = p.tile_base[(int64_t)seg * p.ntiles + tile];
  }
  const RunBits r = run_bits(p, seg, tile);
  int64_t total;
  const int64_t rank = block_exclusive_scan<kThreads>(__popc(r.starts), red, &total);
  const int64_t e0 = before + rank;  // entry of this thread's first start
  const int64_t j0 = (int64_t)tile * kCompactTile + threadIdx.x * kPerThread;
  const int pr = p.page_rows;
  int32_t* ent = p.entries + (int64_t)seg * p.max_entries * 4;
  uint32_t st = r.starts, en = r.ends;
  int64_t e = e0;
  while (st != 0u) {
    const int b = __builtin_ctz(st);
    st &= st - 1u;
    const int64_t j = j0 + b;
    const int64_t lp = j / pr;
    if (e < p.max_entries) {
      ent[e * 4 + 0] = p.table[(int64_t)seg * p.pages_per_seg + lp];
      ent[e * 4 + 1] = (int32_t)lp;
      ent[e * 4 + 2] = (int32_t)(j - lp * pr);
    }
    if (p.page_used != nullptr) p.page_used[(int64_t)seg * p.pages_per_seg + lp] = 1;
    ++e;
  }
  // the run ending at bit b is the last one started at or before b
  while (en != 0u) {
    const int b = __builtin_ctz(en);
    en &= en - 1u;
    const int64_t idx = e0 + __popc(r.starts & ((2u << b) - 1u)) - 1;
    const int64_t j = j0 + b;
    if (idx < p.max_entries) ent[idx * 4 + 3] = (int32_t)(j - (j / pr) * pr + 1);
  }
  if (last_tile) {
    int64_t kept;
    block_exclusive_scan<kThreads>(kept_part, red, &kept);
    if (threadIdx.x == 0) {
      p.seg_len[seg] = (int32_t)kept;
      p.n_entries[seg] = finish_segment(p, seg, (int32_t)runs);
    }
  }
}

// Segments of a context of length 0: no retained position, only the append
// region.
__global__ __launch_bounds__(kThreads) void page_empty_kernel(PageSelectParams p) {
  const int s = blockIdx.x * kThreads + threadIdx.x;
  if (s >= p.nseg) return;
  p.seg_len[s] = 0;
  p.n_entries[s] = finish_segment(p, s, 0);
}

}  // namespace

size_t page_select_workspace_bytes(int64_t nseg, int64_t T) {
  const int64_t ntiles = (T + kCompactTile - 1) / kCompactTile;
  return (size_t)((ntiles > kSumTiles ? 3 : 2) * nseg * ntiles) * sizeof(int32_t);
}

hipError_t launch_page_select(PageSelectParams p, hipStream_t stream) {
  if (p.nseg == 0) return hipSuccess;
  if (p.ntiles > 0) {
    // workspace: tile counts, kept positions, and for long contexts each tile's first entry
    p.tile_base = p.ntiles > kSumTiles ? p.tile_kept + (int64_t)p.nseg * p.ntiles : nullptr;
    hipLaunchKernelGGL(page_count_kernel, dim3(p.ntiles, p.nseg), dim3(kThreads), 0, stream, p);
    if (p.tile_base != nullptr)
      hipLaunchKernelGGL(page_scan_kernel, dim3((p.nseg + kThreads - 1) / kThreads), dim3(kThreads), 0, stream, p);
    hipLaunchKernelGGL(page_emit_kernel, dim3(p.ntiles, p.nseg), dim3(kThreads), 0, stream, p);
  } else {
    hipLaunchKernelGGL(page_empty_kernel, dim3((p.nseg + kThreads - 1) / kThreads), dim3(kThreads), 0, stream, p);
  }
  return hipGetLastError();
}

}  // namespace dkv
