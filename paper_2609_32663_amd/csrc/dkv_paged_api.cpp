// C-ABI entry points of the zero-copy paged variant (see include/dkv.h).
// Every argument is checked on the host before anything is enqueued.

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <cstring>

#include "dkv_launch.hpp"

namespace {

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

dkv_status hip_status(hipError_t e) { return e == hipSuccess ? DKV_OK : DKV_ERR_HIP; }

// Page sizes: multiples of the 32-row decode tile that divide the selection's
// 1024-position wave span.
bool page_rows_ok(int32_t pr) {
  return pr == 32 || pr == 64 || pr == 128 || pr == 256 || pr == 512 || pr == 1024;
}

// Entries of the append region [T, T + cap): one per page it touches.
int32_t tail_entry_count(int32_t T, int32_t cap, int32_t pr) {
  if (cap <= 0) return 0;
  return (int32_t)(((int64_t)T + cap - 1) / pr - (int64_t)T / pr + 1);
}

dkv_status paged_decode(dkv_dtype dtype, int32_t batch, int32_t hq, int32_t hkv, int32_t d, const void* q,
                        const void* k_new, const void* v_new, int32_t n_new, int32_t n_tail, int32_t append_cap,
                        const void* k_pages, const void* v_pages, int64_t num_pages, int32_t page_rows,
                        const int32_t* entries, const int32_t* n_entries, int32_t max_entries, int32_t context_len,
                        float sm_scale, int64_t rows_hint, float* out, void* ws, size_t ws_bytes, void* stream) {
  if (dtype != DKV_BF16 && dtype != DKV_F32) return DKV_ERR_INVALID_ARG;
  if (batch < 0 || hq <= 0 || hkv <= 0 || hq % hkv != 0) return DKV_ERR_INVALID_ARG;
  if (!dkv::scale_in_range(sm_scale) || n_tail < 0 || n_new < 0 || context_len < 0 || max_entries < 0 ||
      num_pages < 0)
    return DKV_ERR_INVALID_ARG;
  if (hq / hkv > DKV_MAX_GROUP || (d != 64 && d != 128)) return DKV_ERR_UNSUPPORTED;
  if ((int64_t)batch * hkv > DKV_MAX_SEGMENTS) return DKV_ERR_UNSUPPORTED;
  if (!page_rows_ok(page_rows)) return DKV_ERR_UNSUPPORTED;
  if (n_new > 0 && (append_cap < 0 || (int64_t)n_tail + n_new > append_cap)) return DKV_ERR_CAPACITY;
  if ((int64_t)context_len + n_tail + n_new > INT32_MAX) return DKV_ERR_INVALID_ARG;
  if (batch == 0) return DKV_OK;
  if (q == nullptr || k_pages == nullptr || v_pages == nullptr || out == nullptr || n_entries == nullptr ||
      (max_entries > 0 && entries == nullptr))
    return DKV_ERR_INVALID_ARG;
  if (n_new > 0 && (k_new == nullptr || v_new == nullptr)) return DKV_ERR_INVALID_ARG;
  if (!aligned16(q) || !aligned16(k_pages) || !aligned16(v_pages) || !aligned16(out) || !aligned16(entries))
    return DKV_ERR_MISALIGNED;
  if (n_new > 0 && (!aligned16(k_new) || !aligned16(v_new))) return DKV_ERR_MISALIGNED;
  if (ws == nullptr || !aligned16(ws)) return DKV_ERR_WORKSPACE;
  if (ws_bytes < dkv_decode_workspace_bytes(batch, hq, hkv, d)) return DKV_ERR_WORKSPACE;

  dkv::DecodeParams p;
  std::memset(&p, 0, sizeof(p));
  p.q = q;
  p.k = k_pages;
  p.v = v_pages;
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
  p.entries = entries;
  p.n_entries = n_entries;
  p.num_pages = num_pages;
  p.max_entries = max_entries;
  p.page_rows = page_rows;
  p.page_shift = __builtin_ctz((unsigned)page_rows);
  p.ctx_len = context_len;
  p.tail_entries = n_new > 0 ? tail_entry_count(context_len, append_cap, page_rows) : 0;
  // the kernel tells paged from packed addressing by a non-null entry
  // pointer; with max_entries = 0 no entry is ever read
  if (p.entries == nullptr) p.entries = n_entries;
  return hip_status(dkv::launch_decode(p, dtype, d, rows_hint, (hipStream_t)stream));
}

}  // namespace

extern "C" {

size_t dkv_page_select_workspace_bytes(int32_t num_segments, int32_t context_len) {
  if (num_segments < 0 || context_len < 0) return 0;
  return dkv::page_select_workspace_bytes(num_segments, context_len);
}

int64_t dkv_page_entries_bound(const dkv_layout* layout, int32_t append_cap, int32_t page_rows) {
  if (layout == nullptr || layout->context_len < 0 || layout->num_bins < 0 || append_cap < 0 ||
      !page_rows_ok(page_rows))
    return -1;
  const int64_t T = layout->context_len;
  // runs of a retained set: sink, recent window and one per bin; each is cut
  // at most once per page boundary it crosses
  const int64_t ctx = (T + page_rows - 1) / page_rows + layout->num_bins + 2;
  return ctx + tail_entry_count(layout->context_len, append_cap, page_rows);
}

dkv_status dkv_page_select(int32_t num_segments, int32_t context_len, int32_t append_cap, int32_t page_rows,
                           const uint8_t* kv_mask, const int32_t* page_table, int32_t pages_per_seg,
                           int32_t max_entries, int32_t* entries, int32_t* n_entries, int32_t* seg_len,
                           uint8_t* page_used, void* workspace, size_t workspace_bytes, void* stream) {
  if (num_segments < 0 || context_len < 0 || append_cap < 0 || pages_per_seg < 0 || max_entries < 0)
    return DKV_ERR_INVALID_ARG;
  if (!page_rows_ok(page_rows)) return DKV_ERR_UNSUPPORTED;
  if (num_segments > 65535) return DKV_ERR_UNSUPPORTED;
  if ((int64_t)pages_per_seg * page_rows < (int64_t)context_len + append_cap) return DKV_ERR_INVALID_ARG;
  if (num_segments == 0) return DKV_OK;
  if ((context_len > 0 && kv_mask == nullptr) || page_table == nullptr || n_entries == nullptr ||
      seg_len == nullptr || (max_entries > 0 && entries == nullptr))
    return DKV_ERR_INVALID_ARG;
  if (!aligned16(kv_mask) || !aligned16(entries)) return DKV_ERR_MISALIGNED;
  if (workspace == nullptr || workspace_bytes < dkv_page_select_workspace_bytes(num_segments, context_len))
    return DKV_ERR_WORKSPACE;

  dkv::PageSelectParams p;
  std::memset(&p, 0, sizeof(p));
  const int64_t ntiles = ((int64_t)context_len + dkv::kCompactTile - 1) / dkv::kCompactTile;
  const int64_t n = (int64_t)num_segments * ntiles;
  p.mask = kv_mask;
  p.table = page_table;
  p.entries = entries;
  p.n_entries = n_entries;
  p.seg_len = seg_len;
  p.page_used = page_used;
  p.tile_cnt = static_cast<int32_t*>(workspace);
  p.tile_kept = p.tile_cnt + n;
  p.T = context_len;
  p.nseg = num_segments;
  p.ntiles = (int32_t)ntiles;
  p.page_rows = page_rows;
  p.pages_per_seg = pages_per_seg;
  p.max_entries = max_entries;
  p.cap = append_cap;
  return hip_status(dkv::launch_page_select(p, (hipStream_t)stream));
}

dkv_status dkv_paged_decode_attn(dkv_dtype dtype, int32_t batch, int32_t num_q_heads, int32_t num_kv_heads,
                                 int32_t head_dim, const void* q, const void* k_pages, const void* v_pages,
                                 int64_t num_pages, int32_t page_rows, const int32_t* entries,
                                 const int32_t* n_entries, int32_t max_entries, int32_t context_len,
                                 int32_t n_tail, float sm_scale, int64_t rows_hint, float* out, void* workspace,
                                 size_t workspace_bytes, void* stream) {
  return paged_decode(dtype, batch, num_q_heads, num_kv_heads, head_dim, q, nullptr, nullptr, 0, n_tail, 0,
                      k_pages, v_pages, num_pages, page_rows, entries, n_entries, max_entries, context_len,
                      sm_scale, rows_hint, out, workspace, workspace_bytes, stream);
}

dkv_status dkv_paged_append_decode_attn(dkv_dtype dtype, int32_t batch, int32_t num_q_heads,
                                        int32_t num_kv_heads, int32_t head_dim, const void* q, const void* k_new,
                                        const void* v_new, int32_t n_new, int32_t n_tail, int32_t append_cap,
                                        void* k_pages, void* v_pages, int64_t num_pages, int32_t page_rows,
                                        const int32_t* entries, const int32_t* n_entries, int32_t max_entries,
                                        int32_t context_len, float sm_scale, int64_t rows_hint, float* out,
                                        void* workspace, size_t workspace_bytes, void* stream) {
  return paged_decode(dtype, batch, num_q_heads, num_kv_heads, head_dim, q, k_new, v_new, n_new, n_tail,
                      append_cap, k_pages, v_pages, num_pages, page_rows, entries, n_entries, max_entries,
                      context_len, sm_scale, rows_hint, out, workspace, workspace_bytes, stream);
}

}  // extern "C"
