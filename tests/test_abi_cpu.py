"""Host-only checks of the C ABI: the library loads, exports every entry point
declared in include/dkv.h, and rejects bad arguments on the host with the
documented status before anything reaches the GPU.

No call here passes validation, so no kernel is launched and no GPU is
needed; fake device addresses are never dereferenced on the host.
"""

import ctypes
import os
import re

import pytest

import paper_2609_32663_amd as d

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADERS = [os.path.join(ROOT, "include", f) for f in sorted(os.listdir(os.path.join(ROOT, "include")))
           if f.endswith(".h")]

A = ctypes.c_void_p(0x10000)      # fake 16-byte-aligned device address
MIS = ctypes.c_void_p(0x10008)    # fake misaligned address
NUL = None


def declared_functions():
    text = "".join(open(h).read() for h in HEADERS)
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(dkv_[a-z_]+)\s*\(", text)))


def test_header_declares_the_hot_path_calls():
    names = declared_functions()
    for n in ("dkv_map_pattern", "dkv_compact", "dkv_append", "dkv_decode_attn",
              "dkv_dense_decode_attn", "dkv_compact_workspace_bytes",
              "dkv_decode_workspace_bytes", "dkv_status_string"):
        assert n in names


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(d.library_path)
    for n in declared_functions():
        assert hasattr(lib, n), n


def test_status_strings():
    for s in range(7):
        assert d.dkv_status_string(s)
    assert d.dkv_status_string(99) == "unknown status"


def _lay(N=1, Hq=8, Hkv=2, dim=128, T=1024, S=4, R=8, edges=(0, 100, 300, 1012)):
    return d.make_layout(N, Hq, Hkv, dim, T, S, R, list(edges))


def _map(lay, pattern=A, kv_mask=A, kv_len=A, q_mask=NUL):
    return d.library().dkv_map_pattern(ctypes.byref(lay) if lay is not None else None,
                                       pattern, kv_mask, kv_len, q_mask, NUL)


def test_map_validation():
    assert _map(None) == d.DKV_ERR_INVALID_ARG
    assert _map(_lay(Hq=6, Hkv=4)) == d.DKV_ERR_INVALID_ARG
    assert _map(_lay(Hq=34, Hkv=2)) == d.DKV_ERR_UNSUPPORTED
    assert _map(_lay(T=-1)) == d.DKV_ERR_INVALID_ARG
    assert _map(_lay(edges=(1, 5, 9))) == d.DKV_ERR_INVALID_ARG
    assert _map(_lay(edges=(0, 5, 5))) == d.DKV_ERR_INVALID_ARG
    assert _map(_lay(edges=(0, 9, 5))) == d.DKV_ERR_INVALID_ARG
    assert _map(_lay(edges=[0] + [k * k + 1 for k in range(1, 514)])) == d.DKV_ERR_UNSUPPORTED
    assert _map(_lay(edges=[3 * k for k in range(16386)])) == d.DKV_ERR_UNSUPPORTED
    assert _map(_lay(), pattern=NUL) == d.DKV_ERR_INVALID_ARG
    assert _map(_lay(), kv_len=NUL) == d.DKV_ERR_INVALID_ARG
    assert _map(_lay(), kv_mask=NUL) == d.DKV_ERR_INVALID_ARG
    assert _map(_lay(), kv_mask=MIS) == d.DKV_ERR_MISALIGNED
    assert _map(_lay(), q_mask=MIS) == d.DKV_ERR_MISALIGNED
    # nothing to do: no launch, success
    assert _map(_lay(N=0), pattern=NUL, kv_mask=NUL, kv_len=NUL) == d.DKV_OK


def _compact(lay, dtype=d.DKV_BF16, k=A, v=A, mask=A, cap=4, k_out=A, v_out=A, out_rows=100,
             seg_off=A, seg_len=A, ws=A, ws_bytes=None):
    if ws_bytes is None:
        ws_bytes = d.dkv_compact_workspace_bytes(lay)
    return d.library().dkv_compact(ctypes.byref(lay), dtype, k, v, mask, cap, k_out, v_out,
                                   out_rows, seg_off, seg_len, NUL, NUL, ws, ws_bytes, NUL)


def test_compact_validation():
    # per segment (2 of them): a count and a base rank per 4096-position tile, and
    # the position list (T entries)
    assert d.dkv_compact_workspace_bytes(_lay()) == 4 * 2 * (1 + 1 + 1024) + 256
    # the copy dispatch (2 workgroups of 256 per 32 rows of T) must stay below 2^32 work-items
    assert _compact(_lay(T=268_435_425, edges=(0, 100, 300, 1012))) == d.DKV_ERR_UNSUPPORTED
    assert _compact(_lay(dim=96)) == d.DKV_ERR_UNSUPPORTED
    assert _compact(_lay(), dtype=7) == d.DKV_ERR_INVALID_ARG
    assert _compact(_lay(), cap=-1) == d.DKV_ERR_INVALID_ARG
    assert _compact(_lay(), out_rows=-1) == d.DKV_ERR_INVALID_ARG
    assert _compact(_lay(), k=NUL) == d.DKV_ERR_INVALID_ARG
    assert _compact(_lay(), seg_off=NUL) == d.DKV_ERR_INVALID_ARG
    assert _compact(_lay(), v=MIS) == d.DKV_ERR_MISALIGNED
    assert _compact(_lay(), k_out=MIS) == d.DKV_ERR_MISALIGNED
    assert _compact(_lay(), mask=MIS) == d.DKV_ERR_MISALIGNED
    assert _compact(_lay(), ws=NUL) == d.DKV_ERR_WORKSPACE
    assert _compact(_lay(), ws_bytes=d.dkv_compact_workspace_bytes(_lay()) - 1) == d.DKV_ERR_WORKSPACE
    assert _compact(_lay(N=40000, Hq=2, Hkv=2)) == d.DKV_ERR_UNSUPPORTED
    assert _compact(_lay(N=0), k=NUL) == d.DKV_OK


def _compact_bins(lay, dtype=d.DKV_BF16, k=A, v=A, pattern=A, cap=4, k_out=A, v_out=A, out_rows=100,
                  seg_off=A, seg_len=A, ws=A, ws_bytes=None):
    if ws_bytes is None:
        ws_bytes = d.dkv_compact_bins_workspace_bytes(lay)
    return d.library().dkv_compact_bins(ctypes.byref(lay), dtype, k, v, pattern, cap, k_out, v_out,
                                        out_rows, seg_off, seg_len, NUL, NUL, ws, ws_bytes, NUL)


def test_compact_bins_validation():
    ws = d.dkv_compact_bins_workspace_bytes(_lay())
    # per segment: kept ranges (D + 2), their packed rows (D + 3), count, length, and the
    # head of every 32-row chunk (T / 32 of them)
    assert ws == 4 * 2 * ((3 + 2) + (3 + 3) + 1 + 1 + 1024 // 32) + 256
    assert d.dkv_compact_bins_workspace_bytes(_lay(N=-1)) == 0
    assert d.dkv_compact_bins_workspace_bytes(_lay(N=40000, Hq=2, Hkv=2)) == 0  # segments
    assert d.dkv_compact_bins_workspace_bytes(_lay(N=30000, Hq=2, Hkv=2, edges=[3 * k for k in range(3001)])) == 0
    assert _compact_bins(_lay(dim=96)) == d.DKV_ERR_UNSUPPORTED
    assert _compact_bins(_lay(), dtype=7) == d.DKV_ERR_INVALID_ARG
    assert _compact_bins(_lay(), cap=-1) == d.DKV_ERR_INVALID_ARG
    assert _compact_bins(_lay(), out_rows=-1) == d.DKV_ERR_INVALID_ARG
    assert _compact_bins(_lay(edges=(0, 9, 5))) == d.DKV_ERR_INVALID_ARG
    assert _compact_bins(_lay(edges=(1, 5, 9))) == d.DKV_ERR_INVALID_ARG
    assert _compact_bins(_lay(edges=[0] + [k * k + 1 for k in range(1, 514)])) == d.DKV_ERR_UNSUPPORTED
    assert _compact_bins(_lay(Hq=6, Hkv=4)) == d.DKV_ERR_INVALID_ARG
    assert _compact_bins(_lay(), k=NUL) == d.DKV_ERR_INVALID_ARG
    assert _compact_bins(_lay(), pattern=NUL) == d.DKV_ERR_INVALID_ARG
    assert _compact_bins(_lay(), seg_len=NUL) == d.DKV_ERR_INVALID_ARG
    assert _compact_bins(_lay(), v=MIS) == d.DKV_ERR_MISALIGNED
    assert _compact_bins(_lay(), v_out=MIS) == d.DKV_ERR_MISALIGNED
    assert _compact_bins(_lay(), ws=NUL) == d.DKV_ERR_WORKSPACE
    assert _compact_bins(_lay(), ws_bytes=ws - 1) == d.DKV_ERR_WORKSPACE
    assert _compact_bins(_lay(N=40000, Hq=2, Hkv=2)) == d.DKV_ERR_UNSUPPORTED
    assert _compact_bins(_lay(N=10000, Hq=2, Hkv=2, edges=list(range(16385)))) == d.DKV_ERR_UNSUPPORTED
    assert _compact_bins(_lay(N=0), k=NUL, pattern=NUL) == d.DKV_OK


def _append(dtype=d.DKV_BF16, nseg=4, dim=128, kn=A, vn=A, n_new=1, n_tail=0, cap=2, kc=A, vc=A,
            so=A, sl=A):
    return d.library().dkv_append(dtype, nseg, dim, kn, vn, n_new, n_tail, cap, kc, vc, so, sl, NUL)


def test_append_validation():
    assert _append(n_tail=2, n_new=1, cap=2) == d.DKV_ERR_CAPACITY
    assert _append(n_tail=-1) == d.DKV_ERR_INVALID_ARG
    assert _append(dim=32) == d.DKV_ERR_UNSUPPORTED
    assert _append(kn=NUL) == d.DKV_ERR_INVALID_ARG
    assert _append(so=NUL) == d.DKV_ERR_INVALID_ARG
    assert _append(vc=MIS) == d.DKV_ERR_MISALIGNED
    assert _append(n_new=0, kn=NUL) == d.DKV_OK


def _decode(dtype=d.DKV_BF16, B=1, Hq=32, Hkv=8, dim=128, q=A, kc=A, vc=A, so=A, sl=A, n_tail=0,
            scale=1.0, out=A, ws=A, ws_bytes=None):
    if ws_bytes is None:
        ws_bytes = d.dkv_decode_workspace_bytes(max(B, 0), Hq, Hkv, dim) if Hq % Hkv == 0 else 0
    return d.library().dkv_decode_attn(dtype, B, Hq, Hkv, dim, q, kc, vc, so, sl, n_tail, scale,
                                       0, out, ws, ws_bytes, NUL)


def test_decode_validation():
    assert d.dkv_decode_workspace_bytes(1, 32, 8, 128) > 0
    assert d.dkv_decode_workspace_bytes(1, 34, 2, 128) == 0
    assert d.dkv_decode_workspace_bytes(1, 32, 8, 80) == 0
    assert _decode(Hq=30, Hkv=8) == d.DKV_ERR_INVALID_ARG
    assert _decode(Hq=34, Hkv=2) == d.DKV_ERR_UNSUPPORTED
    assert _decode(dim=256) == d.DKV_ERR_UNSUPPORTED
    assert _decode(B=300, Hkv=8, Hq=8) == d.DKV_ERR_UNSUPPORTED
    assert _decode(scale=float("nan")) == d.DKV_ERR_INVALID_ARG
    assert _decode(scale=float("inf")) == d.DKV_ERR_INVALID_ARG
    # the kernels take sm_scale * log2(e) in fp32: a finite scale whose product
    # overflows is refused, the largest that does not is accepted (the call then
    # fails later, on the workspace)
    assert _decode(scale=3e38) == d.DKV_ERR_INVALID_ARG
    assert _decode(scale=-3e38) == d.DKV_ERR_INVALID_ARG
    assert _decode(scale=2e38, ws=NUL) == d.DKV_ERR_WORKSPACE
    assert _decode(scale=-2e38, ws=NUL) == d.DKV_ERR_WORKSPACE
    assert _decode(scale=0.0, ws=NUL) == d.DKV_ERR_WORKSPACE
    assert _decode(dtype=5) == d.DKV_ERR_INVALID_ARG
    assert _decode(q=NUL) == d.DKV_ERR_INVALID_ARG
    assert _decode(so=NUL) == d.DKV_ERR_INVALID_ARG
    assert _decode(sl=NUL) == d.DKV_ERR_INVALID_ARG
    assert _decode(n_tail=-1) == d.DKV_ERR_INVALID_ARG
    assert _decode(out=MIS) == d.DKV_ERR_MISALIGNED
    assert _decode(kc=MIS) == d.DKV_ERR_MISALIGNED
    assert _decode(ws=NUL) == d.DKV_ERR_WORKSPACE
    assert _decode(ws=MIS) == d.DKV_ERR_WORKSPACE
    assert _decode(ws_bytes=d.dkv_decode_workspace_bytes(1, 32, 8, 128) - 1) == d.DKV_ERR_WORKSPACE
    assert _decode(B=0, q=NUL, out=NUL) == d.DKV_OK


def test_fused_append_decode_validation():
    lib = d.library()
    ws = d.dkv_decode_workspace_bytes(1, 32, 8, 128)

    def call(n_new=1, n_tail=0, cap=4, kn=A, vn=A):
        return lib.dkv_append_decode_attn(d.DKV_BF16, 1, 32, 8, 128, A, kn, vn, n_new, n_tail, cap, A, A,
                                          A, A, 1.0, 0, A, A, ws, NUL)

    assert call(n_new=2, n_tail=3, cap=4) == d.DKV_ERR_CAPACITY
    assert call(n_new=-1) == d.DKV_ERR_INVALID_ARG
    assert call(kn=NUL) == d.DKV_ERR_INVALID_ARG
    assert call(vn=MIS) == d.DKV_ERR_MISALIGNED
    dws = d.dkv_decode_workspace_bytes(1, 8, 2, 64)
    assert lib.dkv_dense_append_decode_attn(d.DKV_F32, 1, 8, 2, 64, A, A, A, 2, A, A, 100, 99, 1.0, A, A,
                                            dws, NUL) == d.DKV_ERR_CAPACITY
    assert lib.dkv_dense_append_decode_attn(d.DKV_F32, 1, 8, 2, 64, A, NUL, A, 1, A, A, 100, 50, 1.0, A,
                                            A, dws, NUL) == d.DKV_ERR_INVALID_ARG


def test_dense_decode_validation():
    lib = d.library()
    ws = d.dkv_decode_workspace_bytes(1, 8, 2, 64)
    assert lib.dkv_dense_decode_attn(d.DKV_F32, 1, 8, 2, 64, A, A, A, 100, 101, 1.0, A, A, ws,
                                     NUL) == d.DKV_ERR_INVALID_ARG
    assert lib.dkv_dense_decode_attn(d.DKV_F32, 1, 8, 2, 64, A, A, A, 100, -1, 1.0, A, A, ws,
                                     NUL) == d.DKV_ERR_INVALID_ARG
    assert lib.dkv_dense_decode_attn(d.DKV_F32, 1, 8, 2, 64, A, MIS, A, 100, 10, 1.0, A, A, ws,
                                     NUL) == d.DKV_ERR_MISALIGNED
    assert lib.dkv_dense_decode_attn(d.DKV_F32, 1, 8, 2, 64, A, A, A, 100, 10, 1.0, A, A, ws - 4,
                                     NUL) == d.DKV_ERR_WORKSPACE


def test_probe_validation():
    lib = d.library()
    assert lib.dkv_probe_stream_read(A, 0, NUL, 1, NUL) == d.DKV_OK  # nothing to read
    assert lib.dkv_probe_stream_read(A, -16, A, 1, NUL) == d.DKV_ERR_INVALID_ARG
    assert lib.dkv_probe_stream_read(A, 24, A, 1, NUL) == d.DKV_ERR_INVALID_ARG
    for g in (0, 3, 16, -1):
        assert lib.dkv_probe_stream_read(A, 4096, A, g, NUL) == d.DKV_ERR_INVALID_ARG
    assert lib.dkv_probe_stream_read(NUL, 4096, A, 1, NUL) == d.DKV_ERR_INVALID_ARG
    assert lib.dkv_probe_stream_read(A, 4096, NUL, 1, NUL) == d.DKV_ERR_INVALID_ARG
    assert lib.dkv_probe_stream_read(MIS, 4096, A, 1, NUL) == d.DKV_ERR_MISALIGNED
    assert lib.dkv_probe_stream_read(A, 4096, MIS, 1, NUL) == d.DKV_ERR_MISALIGNED
    B = ctypes.c_void_p(A.value + (1 << 20))  # a second, disjoint (never dereferenced) buffer
    assert lib.dkv_probe_copy(A, B, 0, 1, NUL) == d.DKV_OK  # nothing to copy
    assert lib.dkv_probe_copy(A, B, -16, 1, NUL) == d.DKV_ERR_INVALID_ARG
    assert lib.dkv_probe_copy(A, B, 24, 1, NUL) == d.DKV_ERR_INVALID_ARG
    for g in (0, 3, 16, -1):
        assert lib.dkv_probe_copy(A, B, 4096, g, NUL) == d.DKV_ERR_INVALID_ARG
    assert lib.dkv_probe_copy(A, ctypes.c_void_p(A.value + (1 << 44)), (1 << 31) * 4096 + 16, 1,
                              NUL) == d.DKV_ERR_UNSUPPORTED  # 2^31 blocks
    assert lib.dkv_probe_copy(NUL, B, 4096, 1, NUL) == d.DKV_ERR_INVALID_ARG
    assert lib.dkv_probe_copy(A, NUL, 4096, 1, NUL) == d.DKV_ERR_INVALID_ARG
    assert lib.dkv_probe_copy(A, A, 4096, 1, NUL) == d.DKV_ERR_INVALID_ARG  # overlapping
    assert lib.dkv_probe_copy(MIS, B, 4096, 1, NUL) == d.DKV_ERR_MISALIGNED
    assert lib.dkv_probe_copy(A, MIS, 4096, 1, NUL) == d.DKV_ERR_MISALIGNED
    assert lib.dkv_probe_stream_read(A, (1 << 31) * 4096 + 16, A, 1, NUL) == d.DKV_ERR_UNSUPPORTED  # 2^31 blocks


def test_query_validation():
    lib = d.library()
    assert d.dkv_query_workspace_bytes(1, 32, 8, 128, 256, 8 * 50000) > 0
    assert d.dkv_query_workspace_bytes(1, 32, 8, 96, 256, 0) == 0
    assert d.dkv_query_workspace_bytes(1, 32, 8, 128, 256, 8 * 600) == 0  # too few keys to split

    def call(dtype=d.DKV_BF16, B=1, Hq=32, Hkv=8, dim=128, n_q=4, q=A, n_tail=0, cap=8, kc=A, vc=A,
             so=A, sl=A, scale=1.0, hint=0, out=A, ws=A, ws_bytes=1 << 30):
        return lib.dkv_query_attn(dtype, B, Hq, Hkv, dim, n_q, q, n_tail, cap, kc, vc, so, sl, scale, hint,
                                  out, ws, ws_bytes, NUL)

    assert call(dtype=d.DKV_F32) == d.DKV_ERR_UNSUPPORTED
    assert call(dtype=9) == d.DKV_ERR_INVALID_ARG
    assert call(dim=256) == d.DKV_ERR_UNSUPPORTED
    assert call(Hq=30) == d.DKV_ERR_INVALID_ARG
    assert call(Hq=34, Hkv=2) == d.DKV_ERR_UNSUPPORTED
    assert call(n_q=-1) == d.DKV_ERR_INVALID_ARG
    assert call(n_tail=-1) == d.DKV_ERR_INVALID_ARG
    assert call(n_q=5, n_tail=4, cap=8) == d.DKV_ERR_CAPACITY
    assert call(scale=float("nan")) == d.DKV_ERR_INVALID_ARG
    assert call(scale=-3e38) == d.DKV_ERR_INVALID_ARG
    assert call(scale=-2e38, q=NUL) == d.DKV_ERR_INVALID_ARG  # scale accepted, then the null query
    assert call(q=NUL) == d.DKV_ERR_INVALID_ARG
    assert call(sl=NUL) == d.DKV_ERR_INVALID_ARG
    assert call(out=MIS) == d.DKV_ERR_MISALIGNED
    assert call(kc=MIS) == d.DKV_ERR_MISALIGNED
    big = 8 * 50000
    need = d.dkv_query_workspace_bytes(1, 32, 8, 128, 256, big)
    assert call(n_q=256, cap=256, hint=big, ws=NUL) == d.DKV_ERR_WORKSPACE
    assert call(n_q=256, cap=256, hint=big, ws_bytes=need - 1) == d.DKV_ERR_WORKSPACE
    # a split whose combine dispatch would pass 2^32 work-items
    assert call(B=256, Hq=128, Hkv=8, n_q=131072, cap=131072, hint=1 << 36) == d.DKV_ERR_UNSUPPORTED
    assert d.dkv_query_workspace_bytes(256, 128, 8, 128, 131072, 1 << 36) == 0
    assert call(n_q=0, q=NUL, out=NUL) == d.DKV_OK
    assert call(B=0, q=NUL, out=NUL) == d.DKV_OK


def test_page_select_validation():
    lib = d.library()
    assert d.dkv_page_select_workspace_bytes(256, 131072) == 2 * 4 * 256 * 32
    assert d.dkv_page_select_workspace_bytes(-1, 10) == 0
    lay = _lay(T=131072, S=128, R=1024, edges=tuple(128 * k for k in range(1016)))
    # 1024 context pages + 1015 bins + sink + recent, and one page of the append region
    assert d.dkv_page_entries_bound(lay, 64, 128) == 1024 + 1017 + 1
    assert d.dkv_page_entries_bound(lay, 0, 128) == 1024 + 1017
    assert d.dkv_page_entries_bound(lay, 64, 100) == -1

    def call(nseg=4, T=1000, cap=24, pr=128, mask=A, table=A, pps=8, max_e=40, ent=A, ne=A, sl=A,
             used=NUL, ws=A, ws_bytes=1 << 20):
        return lib.dkv_page_select(nseg, T, cap, pr, mask, table, pps, max_e, ent, ne, sl, used, ws, ws_bytes,
                                   NUL)

    assert call(pr=48) == d.DKV_ERR_UNSUPPORTED
    assert call(pr=16) == d.DKV_ERR_UNSUPPORTED
    assert call(nseg=70000) == d.DKV_ERR_UNSUPPORTED
    assert call(pps=7) == d.DKV_ERR_INVALID_ARG        # 7 * 128 < 1000 + 24
    assert call(T=-1) == d.DKV_ERR_INVALID_ARG
    assert call(cap=-1) == d.DKV_ERR_INVALID_ARG
    assert call(max_e=-1) == d.DKV_ERR_INVALID_ARG
    assert call(mask=NUL) == d.DKV_ERR_INVALID_ARG
    assert call(table=NUL) == d.DKV_ERR_INVALID_ARG
    assert call(ent=NUL) == d.DKV_ERR_INVALID_ARG
    assert call(ne=NUL) == d.DKV_ERR_INVALID_ARG
    assert call(sl=NUL) == d.DKV_ERR_INVALID_ARG
    assert call(mask=MIS) == d.DKV_ERR_MISALIGNED
    assert call(ent=MIS) == d.DKV_ERR_MISALIGNED
    assert call(ws=NUL) == d.DKV_ERR_WORKSPACE
    assert call(ws_bytes=2 * 4 * 4 - 1) == d.DKV_ERR_WORKSPACE
    assert call(nseg=0, mask=NUL, table=NUL, ent=NUL, ne=NUL, sl=NUL, ws=NUL) == d.DKV_OK


def test_paged_decode_validation():
    lib = d.library()
    ws = d.dkv_decode_workspace_bytes(1, 32, 8, 128)

    def call(dtype=d.DKV_BF16, B=1, Hq=32, Hkv=8, dim=128, q=A, kn=NUL, vn=NUL, n_new=0, n_tail=0, cap=0,
             kp=A, vp=A, n_pages=100, pr=128, ent=A, ne=A, max_e=10, T=1000, scale=1.0, out=A, w=A,
             w_bytes=ws):
        if n_new == 0 and kn == NUL:
            return lib.dkv_paged_decode_attn(dtype, B, Hq, Hkv, dim, q, kp, vp, n_pages, pr, ent, ne, max_e, T,
                                             n_tail, scale, 0, out, w, w_bytes, NUL)
        return lib.dkv_paged_append_decode_attn(dtype, B, Hq, Hkv, dim, q, kn, vn, n_new, n_tail, cap, kp, vp,
                                                n_pages, pr, ent, ne, max_e, T, scale, 0, out, w, w_bytes, NUL)

    assert call(dtype=9) == d.DKV_ERR_INVALID_ARG
    assert call(dim=96) == d.DKV_ERR_UNSUPPORTED
    assert call(Hq=34, Hkv=2) == d.DKV_ERR_UNSUPPORTED
    assert call(B=300) == d.DKV_ERR_UNSUPPORTED
    assert call(pr=100) == d.DKV_ERR_UNSUPPORTED
    assert call(n_tail=-1) == d.DKV_ERR_INVALID_ARG
    assert call(T=-1) == d.DKV_ERR_INVALID_ARG
    assert call(max_e=-1) == d.DKV_ERR_INVALID_ARG
    assert call(n_pages=-1) == d.DKV_ERR_INVALID_ARG
    assert call(scale=float("inf")) == d.DKV_ERR_INVALID_ARG
    assert call(scale=3e38) == d.DKV_ERR_INVALID_ARG
    assert call(scale=2e38, w=NUL) == d.DKV_ERR_WORKSPACE
    assert call(q=NUL) == d.DKV_ERR_INVALID_ARG
    assert call(kp=NUL) == d.DKV_ERR_INVALID_ARG
    assert call(ne=NUL) == d.DKV_ERR_INVALID_ARG
    assert call(ent=NUL) == d.DKV_ERR_INVALID_ARG
    assert call(out=MIS) == d.DKV_ERR_MISALIGNED
    assert call(vp=MIS) == d.DKV_ERR_MISALIGNED
    assert call(ent=MIS) == d.DKV_ERR_MISALIGNED
    assert call(w=NUL) == d.DKV_ERR_WORKSPACE
    assert call(w_bytes=ws - 1) == d.DKV_ERR_WORKSPACE
    assert call(kn=A, vn=A, n_new=1, n_tail=8, cap=8) == d.DKV_ERR_CAPACITY
    assert call(kn=NUL, vn=A, n_new=1, cap=8) == d.DKV_ERR_INVALID_ARG
    assert call(kn=MIS, vn=A, n_new=1, cap=8) == d.DKV_ERR_MISALIGNED
    assert call(B=0, q=NUL, out=NUL, kp=NUL, vp=NUL) == d.DKV_OK


def test_ragged_map_validation():
    lib = d.library()
    lay = _lay()
    f = lib.dkv_map_pattern_ragged
    assert f(ctypes.byref(lay), NUL, A, A, A, NUL, NUL) == d.DKV_ERR_INVALID_ARG   # unit_len required
    assert f(NUL, A, A, A, A, NUL, NUL) == d.DKV_ERR_INVALID_ARG
    assert f(ctypes.byref(lay), A, A, MIS, A, NUL, NUL) == d.DKV_ERR_MISALIGNED
    assert f(ctypes.byref(_lay(N=0)), NUL, NUL, NUL, NUL, NUL, NUL) == d.DKV_OK


def test_ragged_compact_bins_validation():
    lib = d.library()
    lay = _lay()
    ws = d.dkv_compact_bins_workspace_bytes(lay)

    def f(layout, unit_len, **kw):
        a = dict(dtype=d.DKV_BF16, k=A, v=A, pattern=A, cap=4, k_out=A, v_out=A, out_rows=100, seg_off=A,
                 seg_len=A, ws=A, ws_bytes=ws)
        a.update(kw)
        return lib.dkv_compact_bins_ragged(layout, unit_len, a["dtype"], a["k"], a["v"], a["pattern"], a["cap"],
                                           a["k_out"], a["v_out"], a["out_rows"], a["seg_off"], a["seg_len"],
                                           NUL, NUL, a["ws"], a["ws_bytes"], NUL)
    assert f(ctypes.byref(lay), NUL) == d.DKV_ERR_INVALID_ARG  # unit_len required
    assert f(NUL, A) == d.DKV_ERR_INVALID_ARG
    assert f(ctypes.byref(lay), A, k=MIS) == d.DKV_ERR_MISALIGNED
    assert f(ctypes.byref(lay), A, ws_bytes=ws - 1) == d.DKV_ERR_WORKSPACE
    assert f(ctypes.byref(lay), A, pattern=NUL) == d.DKV_ERR_INVALID_ARG
    assert f(ctypes.byref(_lay(dim=96)), A) == d.DKV_ERR_UNSUPPORTED
    assert f(ctypes.byref(_lay(N=0)), NUL) == d.DKV_OK  # no units: nothing to do


def test_budget_and_topk_validation():
    lib = d.library()
    assert d.dkv_budget_entries(0.2, 32, 32, 1013) == 207462
    assert d.dkv_budget_entries(0.5, 1, 1, 3) == 2
    assert d.dkv_budget_entries(1.0, 2, 3, 4) == 24
    assert d.dkv_budget_entries(-0.1, 1, 1, 1) == -1
    assert d.dkv_budget_entries(1.1, 1, 1, 1) == -1
    assert d.dkv_budget_entries(float("nan"), 1, 1, 1) == -1
    assert d.dkv_budget_entries(0.2, -1, 1, 1) == -1
    ws = d.dkv_topk_workspace_bytes(2, 3, 4)
    assert ws > 0 and d.dkv_topk_workspace_bytes(0, 3, 4) == 0
    assert d.dkv_topk_workspace_bytes(32, 32, 1015) >= d.dkv_topk_workspace_bytes(2, 3, 4)

    def f(L=2, H=3, D=4, probs=A, k=5, pat=A, w=A, w_bytes=ws):
        return lib.dkv_topk_pattern(L, H, D, probs, k, pat, w, w_bytes, NUL)

    assert f(k=-1) == d.DKV_ERR_INVALID_ARG
    assert f(k=25) == d.DKV_ERR_INVALID_ARG
    assert f(probs=NUL) == d.DKV_ERR_INVALID_ARG
    assert f(pat=NUL) == d.DKV_ERR_INVALID_ARG
    assert f(probs=MIS) == d.DKV_ERR_MISALIGNED
    assert f(pat=ctypes.c_void_p(0x10002)) == d.DKV_ERR_MISALIGNED
    assert f(w=NUL) == d.DKV_ERR_WORKSPACE
    assert f(w_bytes=ws - 1) == d.DKV_ERR_WORKSPACE
    assert f(L=-2, k=0) == d.DKV_ERR_INVALID_ARG
    assert f(L=2048, H=2048, D=1024) == d.DKV_ERR_UNSUPPORTED
    assert f(L=0, k=0, probs=NUL, pat=NUL, w=NUL) == d.DKV_OK


def test_build_script_loads_without_the_library():
    """The build runs where no library exists yet: its script must load by
    path without importing the package (which loads the library)."""
    import subprocess
    import sys
    code = ("import importlib.util, sys; "
            f"spec = importlib.util.spec_from_file_location('b', {os.path.join(ROOT, 'paper_2609_32663_amd', 'build.py')!r}); "
            "m = importlib.util.module_from_spec(spec); spec.loader.exec_module(m); "
            "assert callable(m.build); assert 'paper_2609_32663_amd' not in sys.modules")
    subprocess.run([sys.executable, "-c", code], check=True, cwd=ROOT)


def test_binding_rejects_host_tensors():
    import torch
    lay = _lay()
    with pytest.raises(ValueError):
        d.dkv_map_pattern(lay, torch.zeros(1, 8, 3, dtype=torch.uint8),
                          torch.zeros(1, 2, 1024, dtype=torch.uint8),
                          torch.zeros(1, 2, dtype=torch.int32))


def test_noalloc_validation():
    """The allocation-free call checks its arguments like the workspace call,
    and refuses shapes whose workspace exceeds its static scratch, all on the
    host before the scratch is looked up."""
    lib = d.library()

    def call(B=1, Hq=32, Hkv=8, dim=128, q=A, kn=A, vn=A, n_new=1, n_tail=0, cap=4, kc=A, vc=A, so=A, sl=A,
             scale=1.0, out=A):
        return lib.dkv_append_decode_attn_noalloc(d.DKV_BF16, B, Hq, Hkv, dim, q, kn, vn, n_new, n_tail, cap, kc,
                                                  vc, so, sl, scale, 0, out, NUL)

    assert d.dkv_decode_workspace_bytes(128, 128, 8, 128) > d.DKV_NOALLOC_SCRATCH_BYTES
    assert call(B=128, Hq=128, Hkv=8) == d.DKV_ERR_UNSUPPORTED
    assert call(n_new=2, n_tail=3) == d.DKV_ERR_CAPACITY
    assert call(q=NUL) == d.DKV_ERR_INVALID_ARG
    assert call(sl=NUL) == d.DKV_ERR_INVALID_ARG
    assert call(scale=float("inf")) == d.DKV_ERR_INVALID_ARG
    assert call(out=MIS) == d.DKV_ERR_MISALIGNED
    assert call(dim=96) == d.DKV_ERR_UNSUPPORTED
    assert call(B=0, q=NUL, out=NUL) == d.DKV_OK
