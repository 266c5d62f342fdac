// C-ABI entry points of the Distance-KV hot path (see include/dkv.h).
//
// Every argument is checked here, on the host, before any HIP call; a failed
// check returns its status with nothing enqueued.  The launchers in the .hip
// files assume checked arguments.

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <cstring>

#include "dkv_bins.hpp"
#include "dkv_launch.hpp"

namespace {

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

bool head_dim_ok(int32_t d) { return d == 64 || d == 128; }

int elem_bytes(dkv_dtype t) { return t == DKV_BF16 ? 2 : 4; }

bool dtype_ok(int t) { return t == DKV_BF16 || t == DKV_F32; }

dkv_status hip_status(hipError_t e) { return e == hipSuccess ? DKV_OK : DKV_ERR_HIP; }

// Shape checks shared by map and compact.
dkv_status check_shape(const dkv_layout* L) {
  if (L == nullptr) return DKV_ERR_INVALID_ARG;
  if (L->num_units < 0 || L->num_q_heads <= 0 || L->num_kv_heads <= 0 || L->context_len < 0 ||
      L->sink < 0 || L->recent < 0)
    return DKV_ERR_INVALID_ARG;
  if (L->num_q_heads % L->num_kv_heads != 0) return DKV_ERR_INVALID_ARG;
  if (L->num_q_heads / L->num_kv_heads > DKV_MAX_GROUP) return DKV_ERR_UNSUPPORTED;
  return DKV_OK;
}

// Returns the uniform width W when edges are W*k, 0 otherwise.
int32_t uniform_width(const int32_t* e, int32_t D) {
  const int32_t W = e[1] - e[0];
  for (int32_t k = 0; k <= D; ++k)
    if ((int64_t)e[k] != (int64_t)W * k) return 0;
  return W;
}

// Workspace checks are skipped for the allocation-free entry point, whose
// scratch is the library's own (check_ws = false).
dkv_status check_decode_common(int dtype, int32_t batch, int32_t hq, int32_t hkv, int32_t d,
                               const void* q, const void* k, const void* v, const float* out,
                               const void* ws, size_t ws_bytes, float sm_scale, bool check_ws = true) {
  if (!dtype_ok(dtype)) return DKV_ERR_INVALID_ARG;
  if (batch < 0 || hq <= 0 || hkv <= 0 || hq % hkv != 0) return DKV_ERR_INVALID_ARG;
  if (!dkv::scale_in_range(sm_scale)) return DKV_ERR_INVALID_ARG;
  if (hq / hkv > DKV_MAX_GROUP || !head_dim_ok(d)) return DKV_ERR_UNSUPPORTED;
  if ((int64_t)batch * hkv > DKV_MAX_SEGMENTS) return DKV_ERR_UNSUPPORTED;
  if (batch == 0) return DKV_OK;
  if (q == nullptr || k == nullptr || v == nullptr || out == nullptr) return DKV_ERR_INVALID_ARG;
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(out)) return DKV_ERR_MISALIGNED;
  if (!check_ws) return DKV_OK;
  if (ws == nullptr || !aligned16(ws)) return DKV_ERR_WORKSPACE;
  if (ws_bytes < dkv_decode_workspace_bytes(batch, hq, hkv, d)) return DKV_ERR_WORKSPACE;
  return DKV_OK;
}

}  // namespace

extern "C" {

const char* dkv_status_string(dkv_status status) {
  switch (status) {
    case DKV_OK: return "success";
    case DKV_ERR_INVALID_ARG: return "invalid argument";
    case DKV_ERR_UNSUPPORTED: return "unsupported shape";
    case DKV_ERR_MISALIGNED: return "pointer not 16-byte aligned";
    case DKV_ERR_CAPACITY: return "append capacity exceeded";
    case DKV_ERR_WORKSPACE: return "workspace missing or too small";
    case DKV_ERR_HIP: return "HIP launch failed";
  }
  return "unknown status";
}

}  // extern "C"

namespace {

// Bin edges: E[0] = 0 and strictly increasing, within the limits for
// uniform or general edges.  *W is the uniform width (0: general edges).
dkv_status check_edges(const dkv_layout& L, int32_t* W) {
  if (L.num_bins < 1 || L.bin_edges == nullptr) return DKV_ERR_INVALID_ARG;
  const int32_t* e = L.bin_edges;
  if (e[0] != 0) return DKV_ERR_INVALID_ARG;
  for (int32_t k = 0; k < L.num_bins; ++k)
    if (!(e[k + 1] > e[k])) return DKV_ERR_INVALID_ARG;
  *W = uniform_width(e, L.num_bins);
  if (*W > 0 ? L.num_bins > DKV_MAX_UNIFORM_BINS : L.num_bins > DKV_MAX_GENERAL_BINS)
    return DKV_ERR_UNSUPPORTED;
  return DKV_OK;
}

dkv_status map_pattern(const dkv_layout* layout, const int32_t* unit_len, const uint8_t* pattern,
                       uint8_t* kv_mask, int32_t* kv_len, uint8_t* q_mask, void* stream) {
  dkv_status st = check_shape(layout);
  if (st != DKV_OK) return st;
  const dkv_layout& L = *layout;
  int32_t W = 0;
  st = check_edges(L, &W);
  if (st != DKV_OK) return st;
  const int32_t* e = L.bin_edges;
  if (L.num_units == 0) return DKV_OK;
  // With T = 0 there is no mask byte to write, so the mask pointers may be null.
  if (pattern == nullptr || kv_len == nullptr || (kv_mask == nullptr && L.context_len > 0))
    return DKV_ERR_INVALID_ARG;
  if (!aligned16(kv_mask) || (q_mask != nullptr && !aligned16(q_mask))) return DKV_ERR_MISALIGNED;
  const int64_t nseg = (int64_t)L.num_units * L.num_kv_heads;
  // the dispatch's work-item count (workgroups x 256) must fit 32 bits
  if (nseg > 0x7FFFFFFF || dkv::map_blocks(L.context_len, nseg) > 0xFFFFFFFFLL / 256) return DKV_ERR_UNSUPPORTED;
  // the kernel sweeps runs of 16 positions in 32-bit arithmetic
  if (L.context_len > INT32_MAX - 16) return DKV_ERR_UNSUPPORTED;

  dkv::MapParams p;
  std::memset(&p, 0, sizeof(p));
  p.pattern = pattern;
  p.kv_mask = kv_mask;
  p.kv_len = kv_len;
  p.q_mask = q_mask;
  p.T = L.context_len;
  p.S = L.sink;
  p.R = L.recent;
  p.D = L.num_bins;
  p.Hq = L.num_q_heads;
  p.Hkv = L.num_kv_heads;
  p.G = L.num_q_heads / L.num_kv_heads;
  p.uniform_width = W;
  if (W == 0)
    for (int32_t k = 0; k <= L.num_bins; ++k) p.edges[k] = e[k];
  p.unit_len = unit_len;
  return hip_status(dkv::launch_map_pattern(p, (int)nseg, (hipStream_t)stream));
}

}  // namespace

extern "C" {

dkv_status dkv_map_pattern(const dkv_layout* layout, const uint8_t* pattern, uint8_t* kv_mask,
                           int32_t* kv_len, uint8_t* q_mask, void* stream) {
  return map_pattern(layout, nullptr, pattern, kv_mask, kv_len, q_mask, stream);
}

dkv_status dkv_map_pattern_ragged(const dkv_layout* layout, const int32_t* unit_len, const uint8_t* pattern,
                                  uint8_t* kv_mask, int32_t* kv_len, uint8_t* q_mask, void* stream) {
  if (layout != nullptr && layout->num_units > 0 && unit_len == nullptr) return DKV_ERR_INVALID_ARG;
  return map_pattern(layout, unit_len, pattern, kv_mask, kv_len, q_mask, stream);
}

size_t dkv_compact_workspace_bytes(const dkv_layout* layout) {
  if (layout == nullptr || layout->num_units < 0 || layout->num_kv_heads <= 0 || layout->context_len < 0)
    return 0;
  return dkv::compact_workspace_bytes((int64_t)layout->num_units * layout->num_kv_heads,
                                      layout->context_len);
}

dkv_status dkv_compact(const dkv_layout* layout, dkv_dtype dtype, const void* k, const void* v,
                       const uint8_t* kv_mask, int32_t append_cap, void* k_out, void* v_out,
                       int64_t out_rows, int64_t* seg_off, int32_t* seg_len, int32_t* src_pos,
                       int64_t* rows_needed, void* workspace, size_t workspace_bytes, void* stream) {
  dkv_status st = check_shape(layout);
  if (st != DKV_OK) return st;
  const dkv_layout& L = *layout;
  if (!dtype_ok(dtype) || append_cap < 0 || out_rows < 0) return DKV_ERR_INVALID_ARG;
  if (!head_dim_ok(L.head_dim)) return DKV_ERR_UNSUPPORTED;
  const int64_t nseg = (int64_t)L.num_units * L.num_kv_heads;
  if (nseg > 65535) return DKV_ERR_UNSUPPORTED;
  // the copy dispatch (a K and a V workgroup of 256 per 32-row chunk) must
  // hold fewer than 2^32 work-items
  if (2 * dkv::compact_chunks(L.context_len) * 256 > (int64_t)UINT32_MAX) return DKV_ERR_UNSUPPORTED;
  if (nseg == 0) return DKV_OK;
  if (k == nullptr || v == nullptr || kv_mask == nullptr || k_out == nullptr || v_out == nullptr ||
      seg_off == nullptr || seg_len == nullptr)
    return DKV_ERR_INVALID_ARG;
  if (!aligned16(k) || !aligned16(v) || !aligned16(k_out) || !aligned16(v_out) || !aligned16(kv_mask))
    return DKV_ERR_MISALIGNED;
  if (workspace == nullptr || workspace_bytes < dkv_compact_workspace_bytes(layout))
    return DKV_ERR_WORKSPACE;

  dkv::CompactParams p;
  std::memset(&p, 0, sizeof(p));
  const int64_t ntiles = ((int64_t)L.context_len + dkv::kCompactTile - 1) / dkv::kCompactTile;
  p.mask = kv_mask;
  p.k = k;
  p.v = v;
  p.k_out = k_out;
  p.v_out = v_out;
  p.tile_cnt = static_cast<int32_t*>(workspace);
  p.tile_base = p.tile_cnt + nseg * (ntiles > 0 ? ntiles : 1);
  p.list = p.tile_base + nseg * (ntiles > 0 ? ntiles : 1);
  p.seg_off = seg_off;
  p.seg_len = seg_len;
  p.src_pos = src_pos;
  p.rows_needed = rows_needed;
  p.out_rows = out_rows;
  p.T = L.context_len;
  p.nseg = (int32_t)nseg;
  p.ntiles = (int32_t)ntiles;
  p.cap = append_cap;
  p.row_bytes = L.head_dim * elem_bytes(dtype);
  return hip_status(dkv::launch_compact(p, (hipStream_t)stream));
}

size_t dkv_compact_bins_workspace_bytes(const dkv_layout* layout) {
  if (layout == nullptr || layout->num_units < 0 || layout->num_kv_heads <= 0 || layout->context_len < 0 ||
      layout->num_bins < 1)
    return 0;
  const int64_t nseg = (int64_t)layout->num_units * layout->num_kv_heads;
  if (nseg > 65535 || nseg * ((int64_t)layout->num_bins + 3) > (int64_t(1) << 27)) return 0;
  return dkv::bins_workspace_bytes(nseg, layout->num_bins, layout->context_len);
}

namespace {

dkv_status compact_bins(const dkv_layout* layout, const int32_t* unit_len, dkv_dtype dtype, const void* k,
                        const void* v, const uint8_t* pattern, int32_t append_cap, void* k_out, void* v_out,
                        int64_t out_rows, int64_t* seg_off, int32_t* seg_len, int32_t* src_pos,
                        int64_t* rows_needed, void* workspace, size_t workspace_bytes, void* stream) {
  dkv_status st = check_shape(layout);
  if (st != DKV_OK) return st;
  const dkv_layout& L = *layout;
  int32_t W = 0;
  st = check_edges(L, &W);
  if (st != DKV_OK) return st;
  if (!dtype_ok(dtype) || append_cap < 0 || out_rows < 0) return DKV_ERR_INVALID_ARG;
  if (!head_dim_ok(L.head_dim)) return DKV_ERR_UNSUPPORTED;
  const int64_t nseg = (int64_t)L.num_units * L.num_kv_heads;
  if (nseg > 65535 || nseg * ((int64_t)L.num_bins + 3) > (int64_t(1) << 27)) return DKV_ERR_UNSUPPORTED;
  // as for dkv_compact: the copy dispatch must hold fewer than 2^32 work-items
  if (2 * (((int64_t)L.context_len + dkv::kBinsChunkRows - 1) / dkv::kBinsChunkRows) * 256 > (int64_t)UINT32_MAX)
    return DKV_ERR_UNSUPPORTED;
  if (nseg == 0) return DKV_OK;
  if (k == nullptr || v == nullptr || pattern == nullptr || k_out == nullptr || v_out == nullptr ||
      seg_off == nullptr || seg_len == nullptr)
    return DKV_ERR_INVALID_ARG;
  if (!aligned16(k) || !aligned16(v) || !aligned16(k_out) || !aligned16(v_out)) return DKV_ERR_MISALIGNED;
  if (workspace == nullptr || workspace_bytes < dkv_compact_bins_workspace_bytes(layout))
    return DKV_ERR_WORKSPACE;

  dkv::BinsParams p;
  std::memset(&p, 0, sizeof(p));
  const int32_t D = L.num_bins;
  p.pattern = pattern;
  p.unit_len = unit_len;
  p.k = k;
  p.v = v;
  p.k_out = k_out;
  p.v_out = v_out;
  p.item_pos = static_cast<int32_t*>(workspace);
  p.item_dst = p.item_pos + nseg * (D + 2);
  p.item_cnt = p.item_dst + nseg * (D + 3);
  p.lens = p.item_cnt + nseg;
  p.chunk_first = p.lens + nseg;
  p.seg_off = seg_off;
  p.seg_len = seg_len;
  p.src_pos = src_pos;
  p.rows_needed = rows_needed;
  p.out_rows = out_rows;
  p.T = L.context_len;
  p.S = L.sink;
  p.R = L.recent;
  p.D = D;
  p.Hq = L.num_q_heads;
  p.Hkv = L.num_kv_heads;
  p.G = L.num_q_heads / L.num_kv_heads;
  p.nseg = (int32_t)nseg;
  p.cap = append_cap;
  p.row_bytes = L.head_dim * elem_bytes(dtype);
  p.nchunks = (int32_t)(((int64_t)L.context_len + dkv::kBinsChunkRows - 1) / dkv::kBinsChunkRows);
  p.uniform_width = W;
  if (W == 0)
    for (int32_t i = 0; i <= D; ++i) p.edges[i] = L.bin_edges[i];
  return hip_status(dkv::launch_compact_bins(p, (hipStream_t)stream));
}

}  // namespace

dkv_status dkv_compact_bins(const dkv_layout* layout, dkv_dtype dtype, const void* k, const void* v,
                            const uint8_t* pattern, int32_t append_cap, void* k_out, void* v_out,
                            int64_t out_rows, int64_t* seg_off, int32_t* seg_len, int32_t* src_pos,
                            int64_t* rows_needed, void* workspace, size_t workspace_bytes, void* stream) {
  return compact_bins(layout, nullptr, dtype, k, v, pattern, append_cap, k_out, v_out, out_rows, seg_off, seg_len,
                      src_pos, rows_needed, workspace, workspace_bytes, stream);
}

dkv_status dkv_compact_bins_ragged(const dkv_layout* layout, const int32_t* unit_len, dkv_dtype dtype,
                                   const void* k, const void* v, const uint8_t* pattern, int32_t append_cap,
                                   void* k_out, void* v_out, int64_t out_rows, int64_t* seg_off, int32_t* seg_len,
                                   int32_t* src_pos, int64_t* rows_needed, void* workspace,
                                   size_t workspace_bytes, void* stream) {
  if (layout != nullptr && layout->num_units > 0 && unit_len == nullptr) return DKV_ERR_INVALID_ARG;
  return compact_bins(layout, unit_len, dtype, k, v, pattern, append_cap, k_out, v_out, out_rows, seg_off, seg_len,
                      src_pos, rows_needed, workspace, workspace_bytes, stream);
}

dkv_status dkv_append(dkv_dtype dtype, int32_t num_segments, int32_t head_dim, const void* k_new,
                      const void* v_new, int32_t n_new, int32_t n_tail, int32_t append_cap, void* k_c,
                      void* v_c, const int64_t* seg_off, const int32_t* seg_len, void* stream) {
  if (!dtype_ok(dtype) || num_segments < 0 || n_new < 0 || n_tail < 0 || append_cap < 0)
    return DKV_ERR_INVALID_ARG;
  if (!head_dim_ok(head_dim)) return DKV_ERR_UNSUPPORTED;
  if ((int64_t)n_tail + n_new > append_cap) return DKV_ERR_CAPACITY;
  if (num_segments == 0 || n_new == 0) return DKV_OK;
  if (k_new == nullptr || v_new == nullptr || k_c == nullptr || v_c == nullptr || seg_off == nullptr ||
      seg_len == nullptr)
    return DKV_ERR_INVALID_ARG;
  if (!aligned16(k_new) || !aligned16(v_new) || !aligned16(k_c) || !aligned16(v_c))
    return DKV_ERR_MISALIGNED;
  const int row_bytes = head_dim * elem_bytes(dtype);
  if ((int64_t)num_segments * n_new * (row_bytes / 16) > 0x7FFFFFFFLL * 256) return DKV_ERR_UNSUPPORTED;
  dkv::AppendParams p;
  p.k_new = k_new;
  p.v_new = v_new;
  p.k_c = k_c;
  p.v_c = v_c;
  p.seg_off = seg_off;
  p.seg_len = seg_len;
  p.nseg = num_segments;
  p.n_new = n_new;
  p.n_tail = n_tail;
  p.row_bytes = row_bytes;
  return hip_status(dkv::launch_append(p, (hipStream_t)stream));
}

size_t dkv_decode_workspace_bytes(int32_t batch, int32_t num_q_heads, int32_t num_kv_heads,
                                  int32_t head_dim) {
  if (batch < 0 || num_q_heads <= 0 || num_kv_heads <= 0 || num_q_heads % num_kv_heads != 0 ||
      num_q_heads / num_kv_heads > DKV_MAX_GROUP || !head_dim_ok(head_dim) ||
      (int64_t)batch * num_kv_heads > DKV_MAX_SEGMENTS)
    return 0;
  const int nseg = batch * num_kv_heads;
  return dkv::decode_workspace_bytes(nseg, num_q_heads / num_kv_heads, head_dim);
}

}  // extern "C"

namespace {

// Packed-cache attention, optionally appending n_new tokens first.  With
// static_ws the split's scratch is the library's own per-device array (ws
// and ws_bytes are ignored): the allocation-free entry point.
dkv_status decode_packed(dkv_dtype dtype, int32_t batch, int32_t hq, int32_t hkv, int32_t d, const void* q,
                         const void* k_new, const void* v_new, int32_t n_new, int32_t n_tail,
                         int32_t append_cap, const void* k_c, const void* v_c, const int64_t* seg_off,
                         const int32_t* seg_len, float sm_scale, int64_t rows_hint, float* out, void* ws,
                         size_t ws_bytes, void* stream, bool static_ws = false) {
  dkv_status st =
      check_decode_common(dtype, batch, hq, hkv, d, q, k_c, v_c, out, ws, ws_bytes, sm_scale, !static_ws);
  if (st != DKV_OK) return st;
  if (n_tail < 0 || n_new < 0) return DKV_ERR_INVALID_ARG;
  if (n_new > 0 && (int64_t)n_tail + n_new > append_cap) return DKV_ERR_CAPACITY;
  if (batch == 0) return DKV_OK;
  if (seg_off == nullptr || seg_len == nullptr) return DKV_ERR_INVALID_ARG;
  if (n_new > 0 && (k_new == nullptr || v_new == nullptr)) return DKV_ERR_INVALID_ARG;
  if (n_new > 0 && (!aligned16(k_new) || !aligned16(v_new))) return DKV_ERR_MISALIGNED;
  if (static_ws) {
    if (dkv_decode_workspace_bytes(batch, hq, hkv, d) > (size_t)DKV_NOALLOC_SCRATCH_BYTES)
      return DKV_ERR_UNSUPPORTED;
    if (dkv::decode_static_scratch(&ws) != hipSuccess) return DKV_ERR_HIP;
    ws_bytes = DKV_NOALLOC_SCRATCH_BYTES;
  }
  dkv::DecodeParams p;
  std::memset(&p, 0, sizeof(p));
  p.q = q;
  p.k = k_c;
  p.v = v_c;
  p.seg_off = seg_off;
  p.seg_len = seg_len;
  p.n_tail = n_tail;
  p.k_new = k_new;
  p.v_new = v_new;
  p.n_new = n_new;
  p.nseg = batch * hkv;
  p.Hkv = hkv;
  p.Hq = hq;
  p.G = hq / hkv;
  p.scale_log2 = sm_scale * 1.4426950408889634f;
  p.out = out;
  p.partials = static_cast<float*>(ws);
  p.seg_meta = reinterpret_cast<int32_t*>(static_cast<char*>(ws) + dkv::decode_partials_bytes(p.nseg, p.G, d));
  return hip_status(dkv::launch_decode(p, dtype, d, rows_hint, (hipStream_t)stream));
}

// Dense-cache attention over rows [0, n_valid + n_new), optionally writing
// the n_new tokens at rows n_valid.. first.
dkv_status decode_dense(dkv_dtype dtype, int32_t batch, int32_t hq, int32_t hkv, int32_t d, const void* q,
                        const void* k_new, const void* v_new, int32_t n_new, const void* k, const void* v,
                        int64_t t_cap, int32_t n_valid, float sm_scale, float* out, void* ws, size_t ws_bytes,
                        void* stream) {
  dkv_status st = check_decode_common(dtype, batch, hq, hkv, d, q, k, v, out, ws, ws_bytes, sm_scale);
  if (st != DKV_OK) return st;
  if (n_valid < 0 || n_new < 0 || t_cap < 0) return DKV_ERR_INVALID_ARG;
  if ((int64_t)n_valid + n_new > t_cap) return n_new > 0 ? DKV_ERR_CAPACITY : DKV_ERR_INVALID_ARG;
  if (batch == 0) return DKV_OK;
  if (n_new > 0 && (k_new == nullptr || v_new == nullptr)) return DKV_ERR_INVALID_ARG;
  if (n_new > 0 && (!aligned16(k_new) || !aligned16(v_new))) return DKV_ERR_MISALIGNED;
  dkv::DecodeParams p;
  std::memset(&p, 0, sizeof(p));
  p.q = q;
  p.k = k;
  p.v = v;
  p.dense_stride = t_cap;
  p.dense_len = n_valid;
  p.k_new = k_new;
  p.v_new = v_new;
  p.n_new = n_new;
  p.nseg = batch * hkv;
  p.Hkv = hkv;
  p.Hq = hq;
  p.G = hq / hkv;
  p.scale_log2 = sm_scale * 1.4426950408889634f;
  p.out = out;
  p.partials = static_cast<float*>(ws);
  p.seg_meta = reinterpret_cast<int32_t*>(static_cast<char*>(ws) + dkv::decode_partials_bytes(p.nseg, p.G, d));
  return hip_status(dkv::launch_decode(p, dtype, d, (int64_t)p.nseg * ((int64_t)n_valid + n_new),
                                       (hipStream_t)stream));
}

}  // namespace

extern "C" {

dkv_status dkv_decode_attn(dkv_dtype dtype, int32_t batch, int32_t num_q_heads, int32_t num_kv_heads,
                           int32_t head_dim, const void* q, const void* k_c, const void* v_c,
                           const int64_t* seg_off, const int32_t* seg_len, int32_t n_tail, float sm_scale,
                           int64_t rows_hint, float* out, void* workspace, size_t workspace_bytes,
                           void* stream) {
  return decode_packed(dtype, batch, num_q_heads, num_kv_heads, head_dim, q, nullptr, nullptr, 0, n_tail, 0,
                       k_c, v_c, seg_off, seg_len, sm_scale, rows_hint, out, workspace, workspace_bytes, stream);
}

dkv_status dkv_append_decode_attn(dkv_dtype dtype, int32_t batch, int32_t num_q_heads, int32_t num_kv_heads,
                                  int32_t head_dim, const void* q, const void* k_new, const void* v_new,
                                  int32_t n_new, int32_t n_tail, int32_t append_cap, void* k_c, void* v_c,
                                  const int64_t* seg_off, const int32_t* seg_len, float sm_scale,
                                  int64_t rows_hint, float* out, void* workspace, size_t workspace_bytes,
                                  void* stream) {
  return decode_packed(dtype, batch, num_q_heads, num_kv_heads, head_dim, q, k_new, v_new, n_new, n_tail,
                       append_cap, k_c, v_c, seg_off, seg_len, sm_scale, rows_hint, out, workspace,
                       workspace_bytes, stream);
}

dkv_status dkv_append_decode_attn_noalloc(dkv_dtype dtype, int32_t batch, int32_t num_q_heads,
                                          int32_t num_kv_heads, int32_t head_dim, const void* q, const void* k_new,
                                          const void* v_new, int32_t n_new, int32_t n_tail, int32_t append_cap,
                                          void* k_c, void* v_c, const int64_t* seg_off, const int32_t* seg_len,
                                          float sm_scale, int64_t rows_hint, float* out, void* stream) {
  return decode_packed(dtype, batch, num_q_heads, num_kv_heads, head_dim, q, k_new, v_new, n_new, n_tail,
                       append_cap, k_c, v_c, seg_off, seg_len, sm_scale, rows_hint, out, nullptr, 0, stream,
                       /*static_ws=*/true);
}

dkv_status dkv_dense_decode_attn(dkv_dtype dtype, int32_t batch, int32_t num_q_heads, int32_t num_kv_heads,
                                 int32_t head_dim, const void* q, const void* k, const void* v, int64_t t_cap,
                                 int32_t n_valid, float sm_scale, float* out, void* workspace,
                                 size_t workspace_bytes, void* stream) {
  return decode_dense(dtype, batch, num_q_heads, num_kv_heads, head_dim, q, nullptr, nullptr, 0, k, v, t_cap,
                      n_valid, sm_scale, out, workspace, workspace_bytes, stream);
}

dkv_status dkv_dense_append_decode_attn(dkv_dtype dtype, int32_t batch, int32_t num_q_heads,
                                        int32_t num_kv_heads, int32_t head_dim, const void* q,
                                        const void* k_new, const void* v_new, int32_t n_new, void* k, void* v,
                                        int64_t t_cap, int32_t n_valid, float sm_scale, float* out,
                                        void* workspace, size_t workspace_bytes, void* stream) {
  return decode_dense(dtype, batch, num_q_heads, num_kv_heads, head_dim, q, k_new, v_new, n_new, k, v, t_cap,
                      n_valid, sm_scale, out, workspace, workspace_bytes, stream);
}

}  // extern "C"
