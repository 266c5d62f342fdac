"""ctypes binding of libdkv.so: argument marshalling only.

Each function has the name and argument order of its C entry point in
include/dkv.h.  Tensors are passed as device pointers (torch is used for
device memory and streams only); every step of the hot path runs in the HIP
kernels of libdkv.so.  There is no fallback: if the library is missing or a
call fails, an exception is raised.
"""

import ctypes
import os

import torch

__all__ = [
    "DKV_OK", "DKV_ERR_INVALID_ARG", "DKV_ERR_UNSUPPORTED", "DKV_ERR_MISALIGNED",
    "DKV_ERR_CAPACITY", "DKV_ERR_WORKSPACE", "DKV_ERR_HIP", "DKV_BF16", "DKV_F32",
    "DkvError", "Layout", "make_layout", "library", "library_at", "library_path", "dtype_code",
    "dkv_map_pattern", "dkv_compact_workspace_bytes", "dkv_compact", "dkv_compact_bins_workspace_bytes",
    "dkv_compact_bins", "dkv_compact_bins_ragged", "dkv_append",
    "dkv_decode_workspace_bytes", "dkv_decode_attn", "dkv_dense_decode_attn",
    "dkv_append_decode_attn", "dkv_append_decode_attn_noalloc", "dkv_dense_append_decode_attn",
    "DKV_NOALLOC_SCRATCH_BYTES",
    "dkv_status_string", "dkv_probe_stream_read", "dkv_probe_copy", "dkv_query_workspace_bytes", "dkv_query_attn",
    "dkv_page_select_workspace_bytes", "dkv_page_entries_bound", "dkv_page_select",
    "dkv_paged_decode_attn", "dkv_paged_append_decode_attn", "dkv_budget_entries",
    "dkv_topk_workspace_bytes", "dkv_topk_pattern", "dkv_map_pattern_ragged",
]

(DKV_OK, DKV_ERR_INVALID_ARG, DKV_ERR_UNSUPPORTED, DKV_ERR_MISALIGNED, DKV_ERR_CAPACITY,
 DKV_ERR_WORKSPACE, DKV_ERR_HIP) = range(7)
DKV_BF16, DKV_F32 = 0, 1
DKV_NOALLOC_SCRATCH_BYTES = 16 << 20  # include/dkv.h: scratch of dkv_append_decode_attn_noalloc

library_path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libdkv.so")


class DkvError(RuntimeError):
    """A libdkv call returned a status other than DKV_OK."""

    def __init__(self, fn, status):
        self.status = status
        super().__init__(f"{fn} failed: {dkv_status_string(status)} (status {status})")


class Layout(ctypes.Structure):
    _fields_ = [
        ("num_units", ctypes.c_int32),
        ("num_q_heads", ctypes.c_int32),
        ("num_kv_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("context_len", ctypes.c_int32),
        ("sink", ctypes.c_int32),
        ("recent", ctypes.c_int32),
        ("num_bins", ctypes.c_int32),
        ("bin_edges", ctypes.POINTER(ctypes.c_int32)),
    ]


def make_layout(num_units, num_q_heads, num_kv_heads, head_dim, context_len, sink, recent,
                bin_edges):
    """A dkv_layout; the host edge array is kept alive on the returned object."""
    edges = (ctypes.c_int32 * len(bin_edges))(*[int(e) for e in bin_edges])
    lay = Layout(int(num_units), int(num_q_heads), int(num_kv_heads), int(head_dim),
                 int(context_len), int(sink), int(recent), len(bin_edges) - 1,
                 ctypes.cast(edges, ctypes.POINTER(ctypes.c_int32)))
    lay._edges = edges
    return lay


_lib = None


def library():
    """The loaded libdkv.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        _lib = library_at(library_path)
    return _lib


def library_at(path):
    """Another build of the same C ABI (e.g. the phase-stamp build), loaded
    with the same signatures; raises if it has not been built."""
    if not os.path.exists(path):
        raise ImportError(
            f"{path} is missing: build it with `python paper_2609_32663_amd/build.py` "
            "(the Distance-KV path has no fallback)")
    lib = ctypes.CDLL(path)
    P, I32, I64, SZ, F32, VP = (ctypes.POINTER(Layout), ctypes.c_int32, ctypes.c_int64,
                                ctypes.c_size_t, ctypes.c_float, ctypes.c_void_p)
    sigs = {
        "dkv_map_pattern": (I32, [P, VP, VP, VP, VP, VP]),
        "dkv_compact_workspace_bytes": (SZ, [P]),
        "dkv_compact": (I32, [P, I32, VP, VP, VP, I32, VP, VP, I64, VP, VP, VP, VP, VP, SZ, VP]),
        "dkv_append": (I32, [I32, I32, I32, VP, VP, I32, I32, I32, VP, VP, VP, VP, VP]),
        "dkv_decode_workspace_bytes": (SZ, [I32, I32, I32, I32]),
        "dkv_decode_attn": (I32, [I32, I32, I32, I32, I32, VP, VP, VP, VP, VP, I32, F32, I64, VP,
                                  VP, SZ, VP]),
        "dkv_dense_decode_attn": (I32, [I32, I32, I32, I32, I32, VP, VP, VP, I64, I32, F32, VP, VP,
                                        SZ, VP]),
        "dkv_append_decode_attn": (I32, [I32, I32, I32, I32, I32, VP, VP, VP, I32, I32, I32, VP, VP,
                                         VP, VP, F32, I64, VP, VP, SZ, VP]),
        "dkv_append_decode_attn_noalloc": (I32, [I32, I32, I32, I32, I32, VP, VP, VP, I32, I32, I32, VP,
                                                 VP, VP, VP, F32, I64, VP, VP]),
        "dkv_dense_append_decode_attn": (I32, [I32, I32, I32, I32, I32, VP, VP, VP, I32, VP, VP, I64,
                                               I32, F32, VP, VP, SZ, VP]),
        "dkv_status_string": (ctypes.c_char_p, [I32]),
        "dkv_probe_stream_read": (I32, [VP, I64, VP, I32, VP]),
        "dkv_probe_copy": (I32, [VP, VP, I64, I32, VP]),
        "dkv_query_workspace_bytes": (SZ, [I32, I32, I32, I32, I32, I64]),
        "dkv_query_attn": (I32, [I32, I32, I32, I32, I32, I32, VP, I32, I32, VP, VP, VP, VP, F32, I64,
                                 VP, VP, SZ, VP]),
        "dkv_page_select_workspace_bytes": (SZ, [I32, I32]),
        "dkv_page_entries_bound": (I64, [P, I32, I32]),
        "dkv_page_select": (I32, [I32, I32, I32, I32, VP, VP, I32, I32, VP, VP, VP, VP, VP, SZ, VP]),
        "dkv_paged_decode_attn": (I32, [I32, I32, I32, I32, I32, VP, VP, VP, I64, I32, VP, VP, I32, I32,
                                        I32, F32, I64, VP, VP, SZ, VP]),
        "dkv_paged_append_decode_attn": (I32, [I32, I32, I32, I32, I32, VP, VP, VP, I32, I32, I32, VP, VP,
                                               I64, I32, VP, VP, I32, I32, F32, I64, VP, VP, SZ, VP]),
        "dkv_budget_entries": (I64, [ctypes.c_double, I32, I32, I32]),
        "dkv_topk_workspace_bytes": (SZ, [I32, I32, I32]),
        "dkv_map_pattern_ragged": (I32, [P, VP, VP, VP, VP, VP, VP]),
        "dkv_topk_pattern": (I32, [I32, I32, I32, VP, I64, VP, VP, SZ, VP]),
        "dkv_compact_bins_workspace_bytes": (SZ, [P]),
        "dkv_compact_bins": (I32, [P, I32, VP, VP, VP, I32, VP, VP, I64, VP, VP, VP, VP, VP, SZ, VP]),
        "dkv_compact_bins_ragged": (I32, [P, VP, I32, VP, VP, VP, I32, VP, VP, I64, VP, VP, VP, VP, VP, SZ, VP]),
    }
    for name, (res, args) in sigs.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    return lib


# ---------------------------------------------------------------------------
# marshalling helpers
# ---------------------------------------------------------------------------

def dtype_code(t):
    if t == torch.bfloat16:
        return DKV_BF16
    if t == torch.float32:
        return DKV_F32
    raise TypeError(f"unsupported element type {t}")


def _dev(t, name, optional=False):
    if t is None:
        if optional:
            return None
        raise ValueError(f"{name} is required")
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t.data_ptr()


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream


def _check(fn, status):
    if status != DKV_OK:
        raise DkvError(fn, status)


# ---------------------------------------------------------------------------
# entry points
# ---------------------------------------------------------------------------

def dkv_status_string(status):
    return library().dkv_status_string(int(status)).decode()


def dkv_map_pattern(layout, pattern, kv_mask, kv_len, q_mask=None, stream=None):
    _check("dkv_map_pattern", library().dkv_map_pattern(
        ctypes.byref(layout), _dev(pattern, "pattern"), _dev(kv_mask, "kv_mask"),
        _dev(kv_len, "kv_len"), _dev(q_mask, "q_mask", True), _stream(stream)))


def dkv_compact_workspace_bytes(layout):
    return int(library().dkv_compact_workspace_bytes(ctypes.byref(layout)))


def dkv_compact(layout, k, v, kv_mask, append_cap, k_out, v_out, seg_off, seg_len, workspace,
                src_pos=None, rows_needed=None, stream=None):
    _check("dkv_compact", library().dkv_compact(
        ctypes.byref(layout), dtype_code(k.dtype), _dev(k, "k"), _dev(v, "v"),
        _dev(kv_mask, "kv_mask"), int(append_cap), _dev(k_out, "k_out"), _dev(v_out, "v_out"),
        k_out.shape[0], _dev(seg_off, "seg_off"), _dev(seg_len, "seg_len"),
        _dev(src_pos, "src_pos", True), _dev(rows_needed, "rows_needed", True),
        _dev(workspace, "workspace"), workspace.numel() * workspace.element_size(),
        _stream(stream)))


def dkv_compact_bins_workspace_bytes(layout):
    return int(library().dkv_compact_bins_workspace_bytes(ctypes.byref(layout)))


def dkv_compact_bins(layout, k, v, pattern, append_cap, k_out, v_out, seg_off, seg_len, workspace,
                     src_pos=None, rows_needed=None, stream=None):
    """Map and pack from the pattern in one call (the block gather); outputs
    as dkv_compact's for dkv_map_pattern's mask."""
    _check("dkv_compact_bins", library().dkv_compact_bins(
        ctypes.byref(layout), dtype_code(k.dtype), _dev(k, "k"), _dev(v, "v"), _dev(pattern, "pattern"),
        int(append_cap), _dev(k_out, "k_out"), _dev(v_out, "v_out"), k_out.shape[0],
        _dev(seg_off, "seg_off"), _dev(seg_len, "seg_len"), _dev(src_pos, "src_pos", True),
        _dev(rows_needed, "rows_needed", True), _dev(workspace, "workspace"),
        workspace.numel() * workspace.element_size(), _stream(stream)))


def dkv_compact_bins_ragged(layout, unit_len, k, v, pattern, append_cap, k_out, v_out, seg_off, seg_len,
                            workspace, src_pos=None, rows_needed=None, stream=None):
    """dkv_compact_bins for contexts of different lengths: unit_len is an
    int32 device tensor [N] (as for dkv_map_pattern_ragged)."""
    _check("dkv_compact_bins_ragged", library().dkv_compact_bins_ragged(
        ctypes.byref(layout), _dev(unit_len, "unit_len"), dtype_code(k.dtype), _dev(k, "k"), _dev(v, "v"),
        _dev(pattern, "pattern"), int(append_cap), _dev(k_out, "k_out"), _dev(v_out, "v_out"), k_out.shape[0],
        _dev(seg_off, "seg_off"), _dev(seg_len, "seg_len"), _dev(src_pos, "src_pos", True),
        _dev(rows_needed, "rows_needed", True), _dev(workspace, "workspace"),
        workspace.numel() * workspace.element_size(), _stream(stream)))


def dkv_append(k_new, v_new, n_tail, append_cap, k_c, v_c, seg_off, seg_len, stream=None):
    """k_new, v_new: [num_segments][n_new][d]."""
    nseg, n_new, d = k_new.shape
    _check("dkv_append", library().dkv_append(
        dtype_code(k_new.dtype), nseg, d, _dev(k_new, "k_new"), _dev(v_new, "v_new"), n_new,
        int(n_tail), int(append_cap), _dev(k_c, "k_c"), _dev(v_c, "v_c"),
        _dev(seg_off, "seg_off"), _dev(seg_len, "seg_len"), _stream(stream)))


def dkv_decode_workspace_bytes(batch, num_q_heads, num_kv_heads, head_dim):
    return int(library().dkv_decode_workspace_bytes(batch, num_q_heads, num_kv_heads, head_dim))


def dkv_decode_attn(q, k_c, v_c, seg_off, seg_len, n_tail, sm_scale, out, workspace,
                    num_kv_heads, rows_hint=0, stream=None):
    """q: [B][Hq][d]; seg_off/seg_len: the B*Hkv segments of this call."""
    B, Hq, d = q.shape
    _check("dkv_decode_attn", library().dkv_decode_attn(
        dtype_code(q.dtype), B, Hq, int(num_kv_heads), d, _dev(q, "q"), _dev(k_c, "k_c"),
        _dev(v_c, "v_c"), _dev(seg_off, "seg_off"), _dev(seg_len, "seg_len"), int(n_tail),
        float(sm_scale), int(rows_hint), _dev(out, "out"), _dev(workspace, "workspace"),
        workspace.numel() * workspace.element_size(), _stream(stream)))


def dkv_append_decode_attn(q, k_new, v_new, n_tail, append_cap, k_c, v_c, seg_off, seg_len,
                           sm_scale, out, workspace, num_kv_heads, rows_hint=0, stream=None):
    """q: [B][Hq][d]; k_new, v_new: [B*Hkv][n_new][d]."""
    B, Hq, d = q.shape
    n_new = k_new.shape[1]
    _check("dkv_append_decode_attn", library().dkv_append_decode_attn(
        dtype_code(q.dtype), B, Hq, int(num_kv_heads), d, _dev(q, "q"), _dev(k_new, "k_new"),
        _dev(v_new, "v_new"), n_new, int(n_tail), int(append_cap), _dev(k_c, "k_c"),
        _dev(v_c, "v_c"), _dev(seg_off, "seg_off"), _dev(seg_len, "seg_len"), float(sm_scale),
        int(rows_hint), _dev(out, "out"), _dev(workspace, "workspace"),
        workspace.numel() * workspace.element_size(), _stream(stream)))


def dkv_append_decode_attn_noalloc(q, k_new, v_new, n_tail, append_cap, k_c, v_c, seg_off, seg_len,
                                   sm_scale, out, num_kv_heads, rows_hint=0, stream=None):
    """dkv_append_decode_attn without a workspace (the library's static scratch)."""
    B, Hq, d = q.shape
    n_new = k_new.shape[1]
    _check("dkv_append_decode_attn_noalloc", library().dkv_append_decode_attn_noalloc(
        dtype_code(q.dtype), B, Hq, int(num_kv_heads), d, _dev(q, "q"), _dev(k_new, "k_new"),
        _dev(v_new, "v_new"), n_new, int(n_tail), int(append_cap), _dev(k_c, "k_c"),
        _dev(v_c, "v_c"), _dev(seg_off, "seg_off"), _dev(seg_len, "seg_len"), float(sm_scale),
        int(rows_hint), _dev(out, "out"), _stream(stream)))


def dkv_dense_append_decode_attn(q, k_new, v_new, k, v, n_valid, sm_scale, out, workspace,
                                 stream=None):
    """q: [B][Hq][d]; k_new, v_new: [B*Hkv][n_new][d]; k, v: [B][Hkv][t_cap][d]."""
    B, Hq, d = q.shape
    _, Hkv, t_cap, _ = k.shape
    _check("dkv_dense_append_decode_attn", library().dkv_dense_append_decode_attn(
        dtype_code(q.dtype), B, Hq, Hkv, d, _dev(q, "q"), _dev(k_new, "k_new"), _dev(v_new, "v_new"),
        k_new.shape[1], _dev(k, "k"), _dev(v, "v"), t_cap, int(n_valid), float(sm_scale),
        _dev(out, "out"), _dev(workspace, "workspace"),
        workspace.numel() * workspace.element_size(), _stream(stream)))


def dkv_dense_decode_attn(q, k, v, n_valid, sm_scale, out, workspace, stream=None):
    """q: [B][Hq][d]; k, v: [B][Hkv][t_cap][d]."""
    B, Hq, d = q.shape
    _, Hkv, t_cap, _ = k.shape
    _check("dkv_dense_decode_attn", library().dkv_dense_decode_attn(
        dtype_code(q.dtype), B, Hq, Hkv, d, _dev(q, "q"), _dev(k, "k"), _dev(v, "v"), t_cap,
        int(n_valid), float(sm_scale), _dev(out, "out"), _dev(workspace, "workspace"),
        workspace.numel() * workspace.element_size(), _stream(stream)))


def dkv_probe_stream_read(src, sink, granules_per_thread, nbytes=None, stream=None):
    """Streaming-read probe (measurement aid): reads `nbytes` (default: all)
    bytes of the device tensor `src`, one block of 256 x granules_per_thread
    16-byte granules per workgroup; `sink` is a device tensor of >= 16 bytes."""
    n = src.numel() * src.element_size() if nbytes is None else int(nbytes)
    _check("dkv_probe_stream_read", library().dkv_probe_stream_read(
        _dev(src, "src"), n, _dev(sink, "sink"), int(granules_per_thread), _stream(stream)))


def dkv_probe_copy(src, dst, granules_per_thread, nbytes=None, stream=None):
    """Copy probe (measurement aid): copies `nbytes` (default: all) bytes of
    the device tensor `src` into the device tensor `dst`, one block of
    256 x granules_per_thread 16-byte granules per workgroup."""
    n = src.numel() * src.element_size() if nbytes is None else int(nbytes)
    _check("dkv_probe_copy", library().dkv_probe_copy(
        _dev(src, "src"), _dev(dst, "dst"), n, int(granules_per_thread), _stream(stream)))


def dkv_query_workspace_bytes(batch, num_q_heads, num_kv_heads, head_dim, n_q, rows_hint=0):
    return library().dkv_query_workspace_bytes(batch, num_q_heads, num_kv_heads, head_dim, n_q,
                                               int(rows_hint))


def dkv_query_attn(q, n_tail, append_cap, k_c, v_c, seg_off, seg_len, sm_scale, out, workspace,
                   num_kv_heads, rows_hint=0, stream=None):
    """q: [B][n_q][Hq][d] bf16 (the block's K/V already appended); out: [B][n_q][Hq][d] fp32;
    workspace: device tensor of dkv_query_workspace_bytes(...) bytes, or None when that is 0."""
    B, n_q, Hq, d = q.shape
    ws_ptr, ws_bytes = (None, 0) if workspace is None else (
        _dev(workspace, "workspace"), workspace.numel() * workspace.element_size())
    _check("dkv_query_attn", library().dkv_query_attn(
        dtype_code(q.dtype), B, Hq, int(num_kv_heads), d, n_q, _dev(q, "q"), int(n_tail),
        int(append_cap), _dev(k_c, "k_c"), _dev(v_c, "v_c"), _dev(seg_off, "seg_off"),
        _dev(seg_len, "seg_len"), float(sm_scale), int(rows_hint), _dev(out, "out"), ws_ptr, ws_bytes,
        _stream(stream)))


def dkv_page_select_workspace_bytes(num_segments, context_len):
    return library().dkv_page_select_workspace_bytes(int(num_segments), int(context_len))


def dkv_page_entries_bound(layout, append_cap, page_rows):
    return library().dkv_page_entries_bound(ctypes.byref(layout), int(append_cap), int(page_rows))


def dkv_page_select(kv_mask, page_table, page_rows, append_cap, entries, n_entries, seg_len, workspace,
                    page_used=None, stream=None):
    """kv_mask: uint8, nseg rows of T positions ([nseg][T] or [N][Hkv][T]);
    page_table: int32 [nseg][pages_per_seg]; entries: int32 [nseg][max_entries][4];
    n_entries, seg_len: int32 [nseg]; page_used: optional uint8 [nseg][pages_per_seg]."""
    nseg, pps = page_table.shape
    T = kv_mask.shape[-1]
    _check("dkv_page_select", library().dkv_page_select(
        nseg, T, int(append_cap), int(page_rows), _dev(kv_mask, "kv_mask"), _dev(page_table, "page_table"),
        pps, entries.shape[1], _dev(entries, "entries"), _dev(n_entries, "n_entries"),
        _dev(seg_len, "seg_len"), _dev(page_used, "page_used", optional=True), _dev(workspace, "workspace"),
        workspace.numel() * workspace.element_size(), _stream(stream)))


def dkv_paged_decode_attn(q, k_pages, v_pages, entries, n_entries, context_len, n_tail, sm_scale, out,
                          workspace, num_kv_heads, rows_hint=0, stream=None):
    """q: [B][Hq][d]; k_pages, v_pages: [num_pages][page_rows][d];
    entries: int32 [B*Hkv][max_entries][4]; n_entries: int32 [B*Hkv]."""
    B, Hq, d = q.shape
    num_pages, page_rows = k_pages.shape[0], k_pages.shape[1]
    _check("dkv_paged_decode_attn", library().dkv_paged_decode_attn(
        dtype_code(q.dtype), B, Hq, int(num_kv_heads), d, _dev(q, "q"), _dev(k_pages, "k_pages"),
        _dev(v_pages, "v_pages"), num_pages, page_rows, _dev(entries, "entries"), _dev(n_entries, "n_entries"),
        entries.shape[1], int(context_len), int(n_tail), float(sm_scale), int(rows_hint), _dev(out, "out"),
        _dev(workspace, "workspace"), workspace.numel() * workspace.element_size(), _stream(stream)))


def dkv_paged_append_decode_attn(q, k_new, v_new, n_tail, append_cap, k_pages, v_pages, entries, n_entries,
                                 context_len, sm_scale, out, workspace, num_kv_heads, rows_hint=0,
                                 stream=None):
    """q: [B][Hq][d]; k_new, v_new: [B*Hkv][n_new][d]; pools and entries as
    dkv_paged_decode_attn."""
    B, Hq, d = q.shape
    num_pages, page_rows = k_pages.shape[0], k_pages.shape[1]
    _check("dkv_paged_append_decode_attn", library().dkv_paged_append_decode_attn(
        dtype_code(q.dtype), B, Hq, int(num_kv_heads), d, _dev(q, "q"), _dev(k_new, "k_new"),
        _dev(v_new, "v_new"), k_new.shape[1], int(n_tail), int(append_cap), _dev(k_pages, "k_pages"),
        _dev(v_pages, "v_pages"), num_pages, page_rows, _dev(entries, "entries"), _dev(n_entries, "n_entries"),
        entries.shape[1], int(context_len), float(sm_scale), int(rows_hint), _dev(out, "out"),
        _dev(workspace, "workspace"), workspace.numel() * workspace.element_size(), _stream(stream)))


def dkv_budget_entries(rho, num_layers, num_q_heads, num_bins):
    return library().dkv_budget_entries(float(rho), int(num_layers), int(num_q_heads), int(num_bins))


def dkv_topk_workspace_bytes(num_layers, num_q_heads, num_bins):
    return library().dkv_topk_workspace_bytes(int(num_layers), int(num_q_heads), int(num_bins))


def dkv_topk_pattern(probs, k, pattern, workspace, stream=None):
    """probs: float32 [L][Hq][D]; pattern: uint8 [L][Hq][D] (out); workspace:
    device tensor of dkv_topk_workspace_bytes(L, Hq, D) bytes."""
    L, H, D = probs.shape
    if probs.dtype != torch.float32 or pattern.dtype != torch.uint8 or tuple(pattern.shape) != (L, H, D):
        raise ValueError("probs must be float32 and pattern uint8 of the same [L][Hq][D] shape")
    _check("dkv_topk_pattern", library().dkv_topk_pattern(
        L, H, D, _dev(probs, "probs"), int(k), _dev(pattern, "pattern"), _dev(workspace, "workspace"),
        workspace.numel() * workspace.element_size(), _stream(stream)))


def dkv_map_pattern_ragged(layout, unit_len, pattern, kv_mask, kv_len, q_mask=None, stream=None):
    """unit_len: int32 [N] device tensor of per-unit context lengths."""
    _check("dkv_map_pattern_ragged", library().dkv_map_pattern_ragged(
        ctypes.byref(layout), _dev(unit_len, "unit_len"), _dev(pattern, "pattern"), _dev(kv_mask, "kv_mask"),
        _dev(kv_len, "kv_len"), _dev(q_mask, "q_mask", optional=True), _stream(stream)))
