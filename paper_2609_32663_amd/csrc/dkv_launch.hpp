// Launch interface between the C-ABI layer (argument checks) and the kernels.
// Every launcher assumes its arguments were validated by the caller.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <cmath>

#include "../../include/dkv.h"

namespace dkv {

// The attention kernels take the softmax scale as sm_scale * log2(e) in
// fp32; a scale is accepted when it and that product are finite.
inline bool scale_in_range(float sm_scale) {
  return std::isfinite(sm_scale) && std::isfinite(sm_scale * 1.4426950408889634f);
}

// --------------------------------------------------------------- map pattern
struct MapParams {
  const uint8_t* pattern;  // [N][Hq][D]
  uint8_t* kv_mask;        // [N][Hkv][T]
  int32_t* kv_len;         // [N*Hkv]
  uint8_t* q_mask;         // [N][Hq][T] or null
  const int32_t* unit_len; // [N] context length of each unit, or null (all T)
  int32_t T, S, R, D, Hq, Hkv, G;
  int32_t uniform_width;   // > 0: edges are E[k] = uniform_width * k
  int32_t edges[DKV_MAX_GENERAL_BINS + 1];
};
int64_t map_blocks(int32_t T, int64_t num_segments);  // workgroups of one launch
hipError_t launch_map_pattern(const MapParams& p, int num_segments, hipStream_t stream);

// ---------------------------------------------------------------- compaction
constexpr int kCompactTile = 4096;  // positions per compaction tile (count, scan and list)
// Packed rows one copy workgroup moves (8 KiB of K or V at d = 128, bf16):
// short workgroups copy fastest on this part (the block gather's chunk size).
constexpr int kCopyRows = 32;
// Copy chunks per segment: the most rows a segment can keep is T.
inline int64_t compact_chunks(int64_t T) { return (T + kCopyRows - 1) / kCopyRows; }

struct CompactParams {
  const uint8_t* mask;     // [nseg][T]
  const void* k;           // [nseg][T][d]
  const void* v;
  void* k_out;             // [out_rows][d]
  void* v_out;
  int32_t* tile_cnt;       // [nseg][ntiles] (workspace)
  int32_t* tile_base;      // [nseg][ntiles] (workspace)
  int32_t* list;           // [nseg][T] position of each segment's packed row r, r < its length (workspace)
  int64_t* seg_off;        // [nseg]
  int32_t* seg_len;        // [nseg]
  int32_t* src_pos;        // [out_rows] or null
  int64_t* rows_needed;    // [1] or null
  int64_t out_rows;
  int32_t T, nseg, ntiles, cap, row_bytes;
};
size_t compact_workspace_bytes(int64_t nseg, int64_t T);
hipError_t launch_compact(const CompactParams& p, hipStream_t stream);

struct AppendParams {
  const void* k_new;  // [nseg][n_new][d]
  const void* v_new;
  void* k_c;
  void* v_c;
  const int64_t* seg_off;
  const int32_t* seg_len;
  int32_t nseg, n_new, n_tail, row_bytes;
};
hipError_t launch_append(const AppendParams& p, hipStream_t stream);

// ------------------------------------------------------ zero-copy page select
struct PageSelectParams {
  const uint8_t* mask;     // [nseg][T]
  const int32_t* table;    // [nseg][pages_per_seg]
  int32_t* entries;        // [nseg][max_entries][4]: page, logical page, lo, hi
  int32_t* n_entries;      // [nseg]
  int32_t* seg_len;        // [nseg]
  uint8_t* page_used;      // [nseg][pages_per_seg] or null
  int32_t* tile_cnt;       // [nseg][ntiles] runs starting in each tile (workspace)
  int32_t* tile_kept;      // [nseg][ntiles] retained positions per tile (workspace)
  int32_t* tile_base;      // [nseg][ntiles] first entry of each tile (workspace; set by the launcher)
  int32_t T, nseg, ntiles, page_rows, pages_per_seg, max_entries, cap;
};
size_t page_select_workspace_bytes(int64_t nseg, int64_t T);
hipError_t launch_page_select(PageSelectParams p, hipStream_t stream);

// -------------------------------------------------------- exact-budget export
struct TopkParams {
  const float* probs;  // [n] retention probabilities
  uint8_t* pattern;    // [n] out
  uint32_t* state;     // workspace: selected prefixes, per-round histograms, per-chunk last-round counts
  int64_t n;           // entries, < 2^31
  int64_t k;           // 0 <= k <= n
  int64_t chunk;       // entries per workgroup (set by the launcher)
};
size_t topk_workspace_bytes(int64_t n);
hipError_t launch_topk_pattern(TopkParams p, hipStream_t stream);

// ------------------------------------------------------------ decode attention
constexpr int kDecodeMaxWG = 1024;  // upper bound on the split count

struct DecodeParams {
  const void* q;           // [B][Hq][d]
  const void* k;           // packed (or dense) K rows
  const void* v;
  const int64_t* seg_off;  // null: dense addressing
  const int32_t* seg_len;  // null: dense addressing
  int64_t dense_stride;    // rows between dense segments (t_cap)
  int32_t dense_len;       // rows attended per dense segment (n_valid)
  int32_t n_tail;
  const void* k_new;       // [nseg][n_new][d] tokens appended by this call (or null)
  const void* v_new;
  int32_t n_new;           // 0: attend only
  int32_t nseg, Hkv, Hq, G;
  float scale_log2;        // sm_scale * log2(e)
  float* out;              // [B][Hq][d] fp32
  float* partials;         // [(P + nseg)][GP][d + 2]
  int32_t* seg_meta;       // [nseg][2]: first record slot, piece count
  int32_t P;               // workgroups launched (set by launch_decode)
  // Paged addressing (entries != null): k and v are page pools
  // [num_pages][page_rows][d]; the rows of segment s are the page_rows slots
  // of each of its entries, in entry order, and a slot is attended when it
  // lies in the entry's [lo, hi) and its position (logical page * page_rows
  // + slot) is below ctx_len + n_tail + n_new.
  const int32_t* entries;    // [nseg][max_entries][4]: page, logical page, lo, hi
  const int32_t* n_entries;  // [nseg]
  int64_t num_pages;
  int32_t max_entries, page_rows, page_shift, ctx_len;  // page_rows = 1 << page_shift
  int32_t tail_entries;      // entries of the append region (the last ones of a segment)
#if DKV_PHASE_STAMPS
  int32_t stamp_slot;        // phase-stamp build only: the call's stamp slot
#endif
};
int decode_group_pad(int G);
size_t decode_partials_bytes(int nseg, int G, int head_dim);   // partial records
size_t decode_workspace_bytes(int nseg, int G, int head_dim);  // records + segment metadata
// rows_hint: expected total rows of the call (0 = unknown); sizes the split.
hipError_t launch_decode(const DecodeParams& p, dkv_dtype dtype, int head_dim, int64_t rows_hint,
                         hipStream_t stream);
// Device address of the allocation-free entry point's scratch array
// (DKV_NOALLOC_SCRATCH_BYTES) on the current device, looked up once per device.
hipError_t decode_static_scratch(void** ptr);

}  // namespace dkv
