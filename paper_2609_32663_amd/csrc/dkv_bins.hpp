// Launch interface of the block-gather pack (argument checks live in the
// C-ABI layer; the launcher assumes validated arguments).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/dkv.h"

namespace dkv {

// Packed rows one copy workgroup moves (8 KiB of K or V at d = 128, bf16).
// Short workgroups copy fastest: on the Llama-3.1-8B-shaped 128K stack the
// pack took 1.93-1.97 ms with 32 rows, 2.01 with 64, 2.13-2.15 with 128 and
// 2.50-2.52 with 4,096; with 16 the per-workgroup set-up dominates (2.67).
constexpr int kBinsChunkRows = 32;

struct BinsParams {
  const uint8_t* pattern;  // [N][Hq][D]
  const int32_t* unit_len; // [N] each unit's context length (clamped to [0, T]), or null: every unit T
  const void* k;           // [nseg][T][d]
  const void* v;
  void* k_out;             // [out_rows][d]
  void* v_out;
  // workspace: per segment the kept ranges in token order
  int32_t* item_pos;       // [nseg][D + 2] first position of each kept range
  int32_t* item_dst;       // [nseg][D + 3] its first packed row; entry [count] = the segment's length
  int32_t* item_cnt;       // [nseg] kept ranges
  int32_t* lens;           // [nseg] retained rows
  int32_t* chunk_first;    // [nseg][nchunks] the kept range holding packed row c * kBinsChunkRows
  int64_t* seg_off;        // [nseg]
  int32_t* seg_len;        // [nseg]
  int32_t* src_pos;        // [out_rows] or null
  int64_t* rows_needed;    // [1] or null
  int64_t out_rows;
  int32_t T, S, R, D, Hq, Hkv, G, nseg, cap, row_bytes, nchunks;
  int32_t uniform_width;   // W when E[k] = W k, else 0 (edges below)
  int32_t edges[DKV_MAX_GENERAL_BINS + 1];
};

size_t bins_workspace_bytes(int64_t nseg, int32_t D, int32_t T);
hipError_t launch_compact_bins(const BinsParams& p, hipStream_t stream);

}  // namespace dkv
