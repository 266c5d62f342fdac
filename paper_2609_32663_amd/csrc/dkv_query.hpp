// Launch interface of query-block attention (argument checks live in the
// C-ABI layer; the launcher assumes validated arguments).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace dkv {

constexpr int kQueryRowsPerWG = 128;  // query rows (tokens x heads of a group) per workgroup
constexpr int kQueryMaxSplit = 16;    // upper bound on key ranges per query tile

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
  int32_t nsplit;          // key ranges per query tile
  float scale_log2;        // sm_scale * log2(e)
  float* out;              // [B][n_q][Hq][d] fp32
  float* rec;              // nsplit > 1: [nseg * qtiles * nsplit][64][d + 2] partial records
};

// Key ranges per query tile for a call: enough workgroups to fill the GPU,
// each range at least a few key tiles long.  A function of the shapes only,
// so the workspace size is known before the call.
int32_t query_split_count(int32_t nseg, int32_t rows, int64_t rows_hint);
size_t query_workspace_bytes(int32_t nseg, int32_t rows, int32_t head_dim, int64_t rows_hint);
hipError_t launch_query_attn(const QueryParams& p, int head_dim, hipStream_t stream);

}  // namespace dkv
