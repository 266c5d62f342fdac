// C-ABI entry points of query-block attention (see include/dkv.h).  Every
// argument is checked on the host before anything is enqueued.

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <cstring>

#include "../../include/dkv.h"
#include "dkv_launch.hpp"
#include "dkv_query.hpp"

namespace {

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Shape checks shared by the call and its workspace query.
dkv_status check_query_shape(int32_t batch, int32_t hq, int32_t hkv, int32_t d, int32_t n_q) {
  if (batch < 0 || hq <= 0 || hkv <= 0 || hq % hkv != 0 || n_q < 0) return DKV_ERR_INVALID_ARG;
  if (hq / hkv > DKV_MAX_GROUP || (d != 64 && d != 128)) return DKV_ERR_UNSUPPORTED;
  if ((int64_t)batch * hkv > DKV_MAX_SEGMENTS) return DKV_ERR_UNSUPPORTED;
  // query rows per segment must fit 31 bits
  if ((int64_t)n_q * (hq / hkv) > INT32_MAX) return DKV_ERR_UNSUPPORTED;
  return DKV_OK;
}

// The split of a call; DKV_ERR_UNSUPPORTED when its dispatches would not fit
// 32-bit work-item counts (workgroups x 512 threads) or the items 31 bits.
dkv_status query_plan(int32_t batch, int32_t hq, int32_t hkv, int32_t d, int32_t n_q, int64_t rows_hint,
                      dkv::QueryPlanShape* sh) {
  *sh = dkv::query_plan_shape(batch * hkv, n_q * (hq / hkv), d, rows_hint);
  if (sh->max_items > 0xFFFFFFFFLL / 512 || sh->max_items > INT32_MAX / 2) return DKV_ERR_UNSUPPORTED;
  // the combine kernel: one work-item per (segment, query row, 4 columns)
  if (sh->plan_bytes > 0 &&
      (int64_t)batch * hkv * sh->qtiles * dkv::kQueryRowsPerWG * (d / 4) > 0xFFFFFFFFLL)
    return DKV_ERR_UNSUPPORTED;
  return DKV_OK;
}

}  // namespace

extern "C" {

size_t dkv_query_workspace_bytes(int32_t batch, int32_t num_q_heads, int32_t num_kv_heads,
                                 int32_t head_dim, int32_t n_q, int64_t rows_hint) {
  if (check_query_shape(batch, num_q_heads, num_kv_heads, head_dim, n_q) != DKV_OK) return 0;
  if (batch == 0 || n_q == 0) return 0;
  dkv::QueryPlanShape sh;
  if (query_plan(batch, num_q_heads, num_kv_heads, head_dim, n_q, rows_hint, &sh) != DKV_OK) return 0;
  return sh.plan_bytes + sh.rec_bytes;
}

dkv_status dkv_query_attn(dkv_dtype dtype, int32_t batch, int32_t num_q_heads, int32_t num_kv_heads,
                          int32_t head_dim, int32_t n_q, const void* q, int32_t n_tail, int32_t append_cap,
                          const void* k_c, const void* v_c, const int64_t* seg_off, const int32_t* seg_len,
                          float sm_scale, int64_t rows_hint, float* out, void* workspace, size_t workspace_bytes,
                          void* stream) {
  if (dtype != DKV_BF16 && dtype != DKV_F32) return DKV_ERR_INVALID_ARG;
  dkv_status st = check_query_shape(batch, num_q_heads, num_kv_heads, head_dim, n_q);
  if (st != DKV_OK) return st;
  if (dtype != DKV_BF16) return DKV_ERR_UNSUPPORTED;
  if (!dkv::scale_in_range(sm_scale) || n_tail < 0 || append_cap < 0) return DKV_ERR_INVALID_ARG;
  if ((int64_t)n_tail + n_q > append_cap) return DKV_ERR_CAPACITY;
  if (batch == 0 || n_q == 0) return DKV_OK;
  if (q == nullptr || k_c == nullptr || v_c == nullptr || out == nullptr || seg_off == nullptr ||
      seg_len == nullptr)
    return DKV_ERR_INVALID_ARG;
  if (!aligned16(q) || !aligned16(k_c) || !aligned16(v_c) || !aligned16(out)) return DKV_ERR_MISALIGNED;
  dkv::QueryPlanShape sh;
  st = query_plan(batch, num_q_heads, num_kv_heads, head_dim, n_q, rows_hint, &sh);
  if (st != DKV_OK) return st;
  const size_t need = sh.plan_bytes + sh.rec_bytes;
  if (need > 0 && (workspace == nullptr || !aligned16(workspace) || workspace_bytes < need))
    return DKV_ERR_WORKSPACE;
  dkv::QueryParams p;
  std::memset(&p, 0, sizeof(p));
  p.q = q;
  p.k = k_c;
  p.v = v_c;
  p.seg_off = seg_off;
  p.seg_len = seg_len;
  p.n_tail = n_tail;
  p.n_q = n_q;
  p.nseg = batch * num_kv_heads;
  p.Hkv = num_kv_heads;
  p.Hq = num_q_heads;
  p.G = num_q_heads / num_kv_heads;
  p.rows = n_q * p.G;
  p.qtiles = sh.qtiles;
  p.tiles_per_range = (int32_t)sh.tiles_per_range;
  p.max_items = (int32_t)sh.max_items;
  p.scale_log2 = sm_scale * 1.4426950408889634f;
  p.out = out;
  if (sh.plan_bytes > 0) {
    p.plan = static_cast<int32_t*>(workspace);
    p.rec = reinterpret_cast<float*>(static_cast<char*>(workspace) + sh.plan_bytes);
  }
  return dkv::launch_query_attn(p, head_dim, sh.max_items, (hipStream_t)stream) == hipSuccess ? DKV_OK
                                                                                               : DKV_ERR_HIP;
}

}  // extern "C"
