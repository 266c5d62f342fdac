// The one-time pack as a block gather, straight from the pattern (Sec. 3.4,
// Fig. 2(b); the union of Sec. 3.4).
//
// A KV head keeps its sink, its recent window and every bin that some query
// head of its group keeps (Eq. (4)-(5)), and bin k is one contiguous range of
// positions: u in [E[k], E[k+1]) with u = T - 1 - j - recent is j in
// [T - recent - E[k+1], T - recent - E[k]), clipped to the compressible span
// u < T - sink - recent.  In token order a segment is the sink, the bins from
// the farthest (k = D - 1) to the nearest (k = 0), and the recent window, so
// its packed rows are the kept ones of these ranges, each a block of
// consecutive rows in the dense cache and in the pack alike.  Three passes:
//   plan  one workgroup per segment: the kept ranges, their first packed row
//         (block scans over the D + 2 ranges), the segment's length, and for
//         every chunk of kBinsChunkRows packed rows the range holding its
//         first row (a binary search per chunk over the ranges' first rows,
//         staged in LDS);
//   scan  one workgroup: offsets from the lengths plus the append room,
//         with dkv_compact's rule for segments that do not fit below
//         out_rows (length -1, offset clamped);
//   copy  a K and a V workgroup per (segment, chunk of packed rows): the
//         chunk's ranges go to LDS, and LPR = row_bytes / 16 lanes move one
//         row with 16-byte non-temporal loads and stores (every byte is read
//         once and written once), walking the ranges in order (the source row
//         of packed row r of range i is its first position plus r minus its
//         first packed row).  Chunks are short, so each workgroup issues its
//         loads once and retires.
// No keep mask is read or written; the outputs are dkv_compact's for
// dkv_map_pattern's mask.  In a ragged batch T is each unit's own context
// length (unit_len), as for dkv_map_pattern_ragged; the dense rows keep the
// layout's context length as their stride.

#include "dkv_bins.hpp"
#include "dkv_device.hpp"

namespace dkv {

namespace {

constexpr int kThreads = 256;
constexpr int kScanThreads = 1024;
constexpr int kMaxUnroll = 8;  // rows per lane group in flight, at most

// Range i of a segment whose unit's context is the first T positions of its
// row, in token order: 0 = sink, 1 .. D = bin D - i, D + 1 = recent window;
// [lo, lo + len) of the dense row (len 0: empty).
__device__ __forceinline__ void range_of(const BinsParams& p, int64_t T, int i, int32_t& lo, int32_t& len) {
  const int64_t S = p.S, R = p.R;
  const int64_t U = T - S - R;  // compressible span
  if (U <= 0) {                 // every position is sink or recent
    const int64_t s_end = S < T ? S : T;
    lo = (i == p.D + 1) ? (int32_t)s_end : 0;
    len = (int32_t)(i == 0 ? s_end : (i == p.D + 1 ? T - s_end : 0));
    return;
  }
  if (i == 0) {
    lo = 0;
    len = (int32_t)S;
    return;
  }
  if (i == p.D + 1) {
    lo = (int32_t)(T - R);
    len = (int32_t)R;
    return;
  }
  const int k = p.D - i;
  const int64_t e0 = p.uniform_width > 0 ? (int64_t)p.uniform_width * k : p.edges[k];
  const int64_t e1r = p.uniform_width > 0 ? (int64_t)p.uniform_width * (k + 1) : p.edges[k + 1];
  const int64_t e1 = e1r < U ? e1r : U;
  lo = e0 < e1 ? (int32_t)(T - R - e1) : 0;
  len = e0 < e1 ? (int32_t)(e1 - e0) : 0;
}

// Whether range i is kept: sink and recent always, a bin when some query
// head of the group keeps it (the union).
__device__ __forceinline__ bool range_kept(const BinsParams& p, const uint8_t* prow, int i) {
  if (i == 0 || i == p.D + 1) return true;
  const int k = p.D - i;
  bool kept = false;
  for (int h = 0; h < p.G; ++h) kept |= prow[(int64_t)h * p.D + k] != 0;
  return kept;
}

// Kept ranges whose first packed rows the plan stages in LDS to fill the chunk
// heads cooperatively (16 KiB); segments with more fall back to the serial fill.
constexpr int kPlanTable = 4096;

__global__ __launch_bounds__(kThreads) void bins_plan_kernel(BinsParams p) {
  __shared__ int64_t red[kThreads / kWave + 1];
  __shared__ int32_t tbl[kPlanTable];
  const int s = blockIdx.x;
  const int n = s / p.Hkv, g = s - n * p.Hkv;
  const int items = p.D + 2;
  const int per = (items + kThreads - 1) / kThreads;
  const int i0 = threadIdx.x * per;
  const int i1 = i0 + per < items ? i0 + per : items;
  const uint8_t* prow = p.pattern + ((int64_t)n * p.Hq + (int64_t)g * p.G) * p.D;
  // this unit's context (a ragged batch: the first unit_len[n] positions)
  int64_t Tn = p.T;
  if (p.unit_len != nullptr) {
    const int32_t u = p.unit_len[n];
    Tn = u < 0 ? 0 : (u > p.T ? p.T : u);
  }
  // this thread's ranges (consecutive, so the scans keep token order)
  int64_t cnt = 0, rows = 0;
  for (int i = i0; i < i1; ++i) {
    int32_t lo, len;
    range_of(p, Tn, i, lo, len);
    if (len > 0 && range_kept(p, prow, i)) {
      ++cnt;
      rows += len;
    }
  }
  int64_t cnt_all, rows_all;
  int64_t c = block_exclusive_scan<kThreads>(cnt, red, &cnt_all);
  int64_t r = block_exclusive_scan<kThreads>(rows, red, &rows_all);
  int32_t* ipos = p.item_pos + (int64_t)s * (p.D + 2);
  int32_t* idst = p.item_dst + (int64_t)s * (p.D + 3);
  int32_t* cf = p.chunk_first + (int64_t)s * p.nchunks;
  const bool staged = cnt_all <= kPlanTable;  // (the same for every lane)
  for (int i = i0; i < i1; ++i) {
    int32_t lo, len;
    range_of(p, Tn, i, lo, len);
    if (len > 0 && range_kept(p, prow, i)) {
      ipos[c] = lo;
      idst[c] = (int32_t)r;
      if (staged) {
        tbl[c] = (int32_t)r;
      } else {
        // chunks whose first packed row lies in this range, by the range's owner
        for (int64_t ch = (r + kBinsChunkRows - 1) / kBinsChunkRows; ch * kBinsChunkRows < r + len; ++ch)
          cf[ch] = (int32_t)c;
      }
      ++c;
      r += len;
    }
  }
  if (threadIdx.x == 0) {
    p.item_cnt[s] = (int32_t)cnt_all;
    p.lens[s] = (int32_t)rows_all;
    idst[cnt_all] = (int32_t)rows_all;  // sentinel: the end of the last range
  }
  if (staged) {
    // every chunk's head: the last kept range whose first packed row is at or
    // before the chunk's first row (a binary search over the ranges' starts)
    __syncthreads();
    const int n = (int)cnt_all;
    const int64_t nch = (rows_all + kBinsChunkRows - 1) / kBinsChunkRows;
    for (int64_t ch = threadIdx.x; ch < nch; ch += kThreads) {
      const int64_t row = ch * kBinsChunkRows;
      int lo_i = 0, hi_i = n - 1;  // tbl[0] = 0 <= row, so the answer exists
      while (lo_i < hi_i) {
        const int mid = (lo_i + hi_i + 1) >> 1;
        if (tbl[mid] <= row) lo_i = mid;
        else hi_i = mid - 1;
      }
      cf[ch] = lo_i;
    }
  }
}

__global__ __launch_bounds__(kScanThreads) void bins_scan_kernel(BinsParams p) {
  __shared__ int64_t red[kScanThreads / kWave + 1];
  __shared__ int64_t carry;
  if (threadIdx.x == 0) carry = 0;
  __syncthreads();
  for (int64_t s0 = 0; s0 < p.nseg; s0 += kScanThreads) {
    const int64_t s = s0 + threadIdx.x;
    const int64_t len = s < p.nseg ? p.lens[s] : 0;
    const int64_t need = s < p.nseg ? len + p.cap : 0;
    int64_t chunk_total;
    const int64_t excl = block_exclusive_scan<kScanThreads>(need, red, &chunk_total);
    if (s < p.nseg) {
      // dkv_compact's rule: a segment whose rows and append room do not lie
      // wholly below out_rows is not packed (length -1, offset clamped)
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
__global__ __launch_bounds__(kThreads) void bins_copy_kernel(BinsParams p) {
  constexpr int kRowsPerPass = kThreads / LPR;
  constexpr int kPasses = (kBinsChunkRows + kRowsPerPass - 1) / kRowsPerPass;
  constexpr int kUnroll = kPasses < kMaxUnroll ? kPasses : kMaxUnroll;
  // the chunk's ranges: at most one per packed row, plus the one after
  __shared__ int32_t tdst[kBinsChunkRows + 2];
  __shared__ int32_t tpos[kBinsChunkRows + 1];
  const int chunk = blockIdx.x >> 1;
  const int which = blockIdx.x & 1;  // 0: K rows (and source positions), 1: V rows
  const int s = blockIdx.y;
  const int tid = threadIdx.x;
  const int32_t len = p.seg_len[s];
  if (len <= 0) return;  // empty, or not packed (does not fit below out_rows)
  const int64_t r_lo = (int64_t)chunk * kBinsChunkRows;
  if (r_lo >= len) return;
  const int64_t r_hi = r_lo + kBinsChunkRows < len ? r_lo + kBinsChunkRows : len;
  const int32_t* cf = p.chunk_first + (int64_t)s * p.nchunks;
  const int32_t* ipos = p.item_pos + (int64_t)s * (p.D + 2);
  const int32_t* idst = p.item_dst + (int64_t)s * (p.D + 3);
  const int f = cf[chunk];
  const int l = r_hi == len ? p.item_cnt[s] - 1 : cf[chunk + 1];  // the range holding the last row (or the next)
  const int nloc = l - f + 1;
  for (int i = tid; i <= nloc; i += kThreads) tdst[i] = idst[f + i];
  for (int i = tid; i < nloc; i += kThreads) tpos[i] = ipos[f + i];
  __syncthreads();

  const int lane = tid % LPR;
  const int64_t dst0 = p.seg_off[s];
  const int64_t src_seg = (int64_t)s * p.T;
  const u32x4* src = reinterpret_cast<const u32x4*>(which ? p.v : p.k);
  u32x4* dst = reinterpret_cast<u32x4*>(which ? p.v_out : p.k_out);
  int it = 0;  // rows only grow along a lane group's sweep: walk the ranges forward
  for (int64_t r0 = r_lo + tid / LPR; r0 < r_hi; r0 += kRowsPerPass * kUnroll) {
    u32x4 rb[kUnroll];
    int32_t pos[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int64_t r = r0 + (int64_t)u * kRowsPerPass;
      pos[u] = -1;
      if (r < r_hi) {
        while (tdst[it + 1] <= r) ++it;
        pos[u] = tpos[it] + (int32_t)(r - tdst[it]);
        rb[u] = __builtin_nontemporal_load(&src[(src_seg + pos[u]) * LPR + lane]);
      }
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int64_t r = r0 + (int64_t)u * kRowsPerPass;
      if (r < r_hi) {
        __builtin_nontemporal_store(rb[u], &dst[(dst0 + r) * LPR + lane]);
        if (which == 0 && lane == 0 && p.src_pos != nullptr) p.src_pos[dst0 + r] = pos[u];
      }
    }
  }
}

}  // namespace

size_t bins_workspace_bytes(int64_t nseg, int32_t D, int32_t T) {
  const int64_t nchunks = ((int64_t)T + kBinsChunkRows - 1) / kBinsChunkRows;
  const int64_t words = nseg * ((int64_t)D + 2 + D + 3 + 2 + (nchunks > 0 ? nchunks : 1));
  return (size_t)(words * 4 + 256);
}

hipError_t launch_compact_bins(const BinsParams& p, hipStream_t stream) {
  hipLaunchKernelGGL(bins_plan_kernel, dim3(p.nseg), dim3(kThreads), 0, stream, p);
  hipLaunchKernelGGL(bins_scan_kernel, dim3(1), dim3(kScanThreads), 0, stream, p);
  if (p.nchunks > 0) {
    const dim3 grid(2 * p.nchunks, p.nseg);  // a K and a V workgroup per chunk
    switch (p.row_bytes) {
      case 128: hipLaunchKernelGGL(bins_copy_kernel<8>, grid, dim3(kThreads), 0, stream, p); break;
      case 256: hipLaunchKernelGGL(bins_copy_kernel<16>, grid, dim3(kThreads), 0, stream, p); break;
      case 512: hipLaunchKernelGGL(bins_copy_kernel<32>, grid, dim3(kThreads), 0, stream, p); break;
      default: return hipErrorInvalidValue;
    }
  }
  return hipGetLastError();
}

}  // namespace dkv
