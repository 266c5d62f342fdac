// Launch interface of query-block attention (argument checks live in the
// C-ABI layer; the launcher assumes validated arguments).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace dkv {

constexpr int kQueryRowsPerWG = 256;     // query rows (tokens x heads of a group) per workgroup
constexpr int kQueryTargetItems = 512;   // workgroups a split call aims at: two per compute unit
constexpr int kQueryMinTiles = 8;        // 64-key tiles per key range at least
constexpr int kQueryUnknownTiles = 512;  // key tiles per segment assumed when the caller gives no hint
constexpr int kQueryPlanHead = 4;        // plan words before the first-item table

struct QueryParams {
  const void* q;           // [B][n_q][Hq][d] bf16
  const void* k;           // packed K rows (bf16)
  const void* v;
  const int64_t* seg_off;  // [B*Hkv]
  const int32_t* seg_len;  // [B*Hkv]
  int32_t n_tail;          // tokens appended before the block
  int32_t n_q;             // tokens in the block (already appended after them)
  int32_t nseg, Hkv, Hq, G;
  int32_t rows;            // query rows per segment: n_q * G
  int32_t qtiles;          // ceil(rows / kQueryRowsPerWG)
  int32_t tiles_per_range; // C before the plan kernel's check against max_items
  int32_t max_items;       // items the records hold
  float scale_log2;        // sm_scale * log2(e)
  float* out;              // [B][n_q][Hq][d] fp32
  // Split calls only (nullptr otherwise): plan words [0] items, [1] tiles per
  // range, then [kQueryPlanHead + s] first item of segment s (s <= nseg); and
  // the records [max_items][kQueryRowsPerWG][d + 2] (max, sum, output).
  int32_t* plan;
  float* rec;
};

// How a call is split, from the shapes and the caller's hint of the total
// rows (0 = unknown) only, so the workspace size is known before the call.
struct QueryPlanShape {
  int32_t qtiles;
  int64_t tiles_per_range;
  int64_t max_items;   // attention workgroups launched
  size_t plan_bytes;   // 0: no split, one workgroup per (segment, query tile)
  size_t rec_bytes;
};

QueryPlanShape query_plan_shape(int32_t nseg, int32_t rows, int32_t head_dim, int64_t rows_hint);
hipError_t launch_query_attn(const QueryParams& p, int head_dim, int64_t grid, hipStream_t stream);

}  // namespace dkv
