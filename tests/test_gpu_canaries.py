"""Guard canaries past (and before) every output buffer of every entry point,
and bitwise reproducibility of the calls the other tests do not repeat.

Each output, in-out cache and workspace is carved out of a larger byte buffer
whose 4 KiB before and after it hold a sentinel; after the call (on small,
ragged shapes: a context of 1,000 positions, rows that are not multiples of
16, odd append capacities) every sentinel byte must be unchanged.  The values
themselves are checked by the parity tests; here only where the kernels write.
"""

import numpy as np
import pytest
import torch

import dkv_inputs as di

pytestmark = pytest.mark.gpu

DEV = "cuda"
GUARD = 4096
SENTINEL = 0xA7


@pytest.fixture(scope="module")
def d():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2609_32663_amd as lib
    return lib


class Guarded:
    """A device tensor with GUARD sentinel bytes on both sides."""

    def __init__(self, shape, dtype, fill=None):
        elem = torch.empty((), dtype=dtype).element_size()
        self.nbytes = int(np.prod(shape)) * elem
        self.base = torch.full((GUARD + self.nbytes + GUARD,), SENTINEL, dtype=torch.uint8, device=DEV)
        self.t = self.base[GUARD:GUARD + self.nbytes].view(dtype).view(shape)
        if fill is not None:
            self.t.fill_(fill)

    def intact(self):
        torch.cuda.synchronize()
        return bool((self.base[:GUARD] == SENTINEL).all()) and bool((self.base[GUARD + self.nbytes:] == SENTINEL).all())


def _ws(nbytes):
    return Guarded((max(int(nbytes), 16),), torch.uint8)


N, HQ, HKV, DIM, T, S, R = 2, 8, 2, 128, 1000, 16, 64
EDGES = [0, 50, 130, 300, 500, 700, 920]
CAP = 37


def _setup(d, seed=5):
    rng = np.random.default_rng(seed)
    lay = d.make_layout(N, HQ, HKV, DIM, T, S, R, EDGES)
    D = len(EDGES) - 1
    pattern = torch.from_numpy(rng.integers(0, 2, size=(N, HQ, D)).astype(np.uint8)).to(DEV)
    g = torch.Generator(device=DEV).manual_seed(seed)
    k = torch.randn((N, HKV, T, DIM), generator=g, device=DEV).to(torch.bfloat16)
    v = torch.randn((N, HKV, T, DIM), generator=g, device=DEV).to(torch.bfloat16)
    return lay, pattern, k, v, g


def _pack(d, lay, pattern, k, v):
    km = Guarded((N, HKV, T), torch.uint8)
    kl = Guarded((N, HKV), torch.int32)
    qm = Guarded((N, HQ, T), torch.uint8)
    d.dkv_map_pattern(lay, pattern, km.t, kl.t, qm.t)
    assert km.intact() and kl.intact() and qm.intact()
    rows = int((kl.t.cpu().to(torch.int64) + CAP).sum())
    pk = {
        "k": Guarded((rows, DIM), torch.bfloat16, 0), "v": Guarded((rows, DIM), torch.bfloat16, 0),
        "off": Guarded((N * HKV,), torch.int64), "len": Guarded((N * HKV,), torch.int32),
        "src": Guarded((rows,), torch.int32), "need": Guarded((1,), torch.int64),
        "ws": _ws(d.dkv_compact_workspace_bytes(lay)),
    }
    d.dkv_compact(lay, k, v, km.t, CAP, pk["k"].t, pk["v"].t, pk["off"].t, pk["len"].t, pk["ws"].t,
                  src_pos=pk["src"].t, rows_needed=pk["need"].t)
    for name, gbuf in pk.items():
        assert gbuf.intact(), f"dkv_compact wrote outside {name}"
    pk["rows"] = rows
    pk["km"] = km
    return pk


def test_map_and_ragged_map_stay_inside(d):
    lay, pattern, k, v, _ = _setup(d)
    _pack(d, lay, pattern, k, v)
    unit_len = torch.tensor([T, 613], dtype=torch.int32, device=DEV)
    km = Guarded((N, HKV, T), torch.uint8)
    kl = Guarded((N, HKV), torch.int32)
    qm = Guarded((N, HQ, T), torch.uint8)
    d.dkv_map_pattern_ragged(lay, unit_len, pattern, km.t, kl.t, qm.t)
    assert km.intact() and kl.intact() and qm.intact()


@pytest.mark.parametrize("short", [False, True])
def test_compact_bins_stays_inside(d, short):
    """The block gather from the pattern, with room for every segment and
    with out_rows one short of it (some segments marked unpacked)."""
    lay, pattern, k, v, _ = _setup(d)
    pk = _pack(d, lay, pattern, k, v)
    _bins_guarded(d, lay, pattern, k, v, pk, short)


def test_compact_bins_ragged_stays_inside(d):
    """The ragged block gather (a full and a short context), exactly fitted."""
    lay, pattern, k, v, _ = _setup(d)
    unit_len = torch.tensor([T, 613], dtype=torch.int32, device=DEV)
    km = torch.empty((N, HKV, T), dtype=torch.uint8, device=DEV)
    kl = torch.empty((N, HKV), dtype=torch.int32, device=DEV)
    d.dkv_map_pattern_ragged(lay, unit_len, pattern, km, kl)
    rows = int((kl.cpu().to(torch.int64) + CAP).sum())
    gb = {
        "k": Guarded((rows, DIM), torch.bfloat16, 0), "v": Guarded((rows, DIM), torch.bfloat16, 0),
        "off": Guarded((N * HKV,), torch.int64), "len": Guarded((N * HKV,), torch.int32),
        "src": Guarded((rows,), torch.int32), "need": Guarded((1,), torch.int64),
        "ws": _ws(d.dkv_compact_bins_workspace_bytes(lay)),
    }
    d.dkv_compact_bins_ragged(lay, unit_len, k, v, pattern, CAP, gb["k"].t, gb["v"].t, gb["off"].t, gb["len"].t,
                              gb["ws"].t, src_pos=gb["src"].t, rows_needed=gb["need"].t)
    for name, gbuf in gb.items():
        assert gbuf.intact(), f"dkv_compact_bins_ragged wrote outside {name}"
    assert int(gb["need"].t.item()) == rows
    assert torch.equal(gb["len"].t.cpu().view(N, HKV), kl.cpu())


def _bins_guarded(d, lay, pattern, k, v, pk, short):
    rows = pk["rows"] - (1 if short else 0)
    gb = {
        "k": Guarded((rows, DIM), torch.bfloat16, 0), "v": Guarded((rows, DIM), torch.bfloat16, 0),
        "off": Guarded((N * HKV,), torch.int64), "len": Guarded((N * HKV,), torch.int32),
        "src": Guarded((rows,), torch.int32), "need": Guarded((1,), torch.int64),
        "ws": _ws(d.dkv_compact_bins_workspace_bytes(lay)),
    }
    d.dkv_compact_bins(lay, k, v, pattern, CAP, gb["k"].t, gb["v"].t, gb["off"].t, gb["len"].t, gb["ws"].t,
                       src_pos=gb["src"].t, rows_needed=gb["need"].t)
    for name, gbuf in gb.items():
        assert gbuf.intact(), f"dkv_compact_bins wrote outside {name}"
    assert int(gb["need"].t.item()) == pk["rows"]
    if not short:
        assert torch.equal(gb["k"].t.view(torch.int16), pk["k"].t.view(torch.int16))
        assert torch.equal(gb["len"].t, pk["len"].t)
    else:
        assert bool((gb["len"].t < 0).any())


def test_append_and_decode_calls_stay_inside(d):
    lay, pattern, k, v, g = _setup(d)
    pk = _pack(d, lay, pattern, k, v)
    nseg = N * HKV
    kn = torch.randn((nseg, 3, DIM), generator=g, device=DEV).to(torch.bfloat16)
    vn = torch.randn((nseg, 3, DIM), generator=g, device=DEV).to(torch.bfloat16)
    d.dkv_append(kn, vn, 0, CAP, pk["k"].t, pk["v"].t, pk["off"].t, pk["len"].t)
    assert pk["k"].intact() and pk["v"].intact()
    rows_u0 = int(pk["len"].t[:HKV].sum()) + HKV * 4
    q = torch.randn((1, HQ, DIM), generator=g, device=DEV).to(torch.bfloat16)
    for rows_hint in (0, rows_u0):
        out = Guarded((1, HQ, DIM), torch.float32)
        ws = _ws(d.dkv_decode_workspace_bytes(1, HQ, HKV, DIM))
        d.dkv_decode_attn(q, pk["k"].t, pk["v"].t, pk["off"].t[:HKV], pk["len"].t[:HKV], 3, 0.1, out.t, ws.t,
                          HKV, rows_hint=rows_hint)
        assert out.intact() and ws.intact()
        out = Guarded((1, HQ, DIM), torch.float32)
        ws = _ws(d.dkv_decode_workspace_bytes(1, HQ, HKV, DIM))
        d.dkv_append_decode_attn(q, kn[:HKV, :1].contiguous(), vn[:HKV, :1].contiguous(), 3, CAP, pk["k"].t,
                                 pk["v"].t, pk["off"].t[:HKV], pk["len"].t[:HKV], 0.1, out.t, ws.t, HKV,
                                 rows_hint=rows_hint)
        assert out.intact() and ws.intact() and pk["k"].intact() and pk["v"].intact()
        out = Guarded((1, HQ, DIM), torch.float32)
        d.dkv_append_decode_attn_noalloc(q, kn[:HKV, :1].contiguous(), vn[:HKV, :1].contiguous(), 4, CAP,
                                         pk["k"].t, pk["v"].t, pk["off"].t[:HKV], pk["len"].t[:HKV], 0.1, out.t,
                                         HKV, rows_hint=rows_hint)
        assert out.intact() and pk["k"].intact() and pk["v"].intact()
    # dense comparator, attend-only and fused
    t_cap = 1003
    kd = Guarded((1, HKV, t_cap, DIM), torch.bfloat16, 0)
    vd = Guarded((1, HKV, t_cap, DIM), torch.bfloat16, 0)
    kd.t[:, :, :T].copy_(k[:1])
    vd.t[:, :, :T].copy_(v[:1])
    out = Guarded((1, HQ, DIM), torch.float32)
    ws = _ws(d.dkv_decode_workspace_bytes(1, HQ, HKV, DIM))
    d.dkv_dense_decode_attn(q, kd.t, vd.t, T, 0.1, out.t, ws.t)
    assert out.intact() and ws.intact()
    first = out.t.clone()
    d.dkv_dense_decode_attn(q, kd.t, vd.t, T, 0.1, out.t, ws.t)
    assert torch.equal(out.t, first)  # fixed merge order
    d.dkv_dense_append_decode_attn(q, kn[:HKV, :3].contiguous(), vn[:HKV, :3].contiguous(), kd.t, vd.t, T, 0.1,
                                   out.t, ws.t)
    assert out.intact() and ws.intact() and kd.intact() and vd.intact()


def test_query_block_stays_inside(d):
    lay, pattern, k, v, g = _setup(d, seed=7)
    pk = _pack(d, lay, pattern, k, v)
    n_q = CAP - 2
    kb = torch.randn((N * HKV, n_q, DIM), generator=g, device=DEV).to(torch.bfloat16)
    vb = torch.randn((N * HKV, n_q, DIM), generator=g, device=DEV).to(torch.bfloat16)
    d.dkv_append(kb, vb, 0, CAP, pk["k"].t, pk["v"].t, pk["off"].t, pk["len"].t)
    qb = torch.randn((N, n_q, HQ, DIM), generator=g, device=DEV).to(torch.bfloat16)
    rows = int(pk["len"].t.sum()) + N * HKV * n_q
    for hint in (0, rows, rows // 20):
        out = Guarded((N, n_q, HQ, DIM), torch.float32)
        nb = d.dkv_query_workspace_bytes(N, HQ, HKV, DIM, n_q, hint)
        ws = _ws(nb) if nb > 0 else None
        d.dkv_query_attn(qb, 0, CAP, pk["k"].t, pk["v"].t, pk["off"].t, pk["len"].t, 0.1, out.t,
                         None if ws is None else ws.t, HKV, rows_hint=hint)
        assert out.intact() and (ws is None or ws.intact())


@pytest.mark.parametrize("page_rows", [32, 128])
def test_page_select_and_paged_decode_stay_inside(d, page_rows):
    lay, pattern, k, v, g = _setup(d, seed=11)
    pk = _pack(d, lay, pattern, k, v)
    nseg = N * HKV
    pps = -(-(T + CAP) // page_rows)
    table, n_pages = di.page_table(nseg, pps, seed=page_rows, spare=3)
    table_d = torch.from_numpy(table).to(DEV)
    max_e = int(d.dkv_page_entries_bound(lay, CAP, page_rows))
    ent = Guarded((nseg, max_e, 4), torch.int32, -5)
    ne = Guarded((nseg,), torch.int32)
    sl = Guarded((nseg,), torch.int32)
    used = Guarded((nseg, pps), torch.uint8)
    ws = _ws(d.dkv_page_select_workspace_bytes(nseg, T))
    d.dkv_page_select(pk["km"].t.view(nseg, T), table_d, page_rows, CAP, ent.t, ne.t, sl.t, ws.t, page_used=used.t)
    assert ent.intact() and ne.intact() and sl.intact() and used.intact() and ws.intact()
    # a list cut short: entries past max_entries are not written
    small = Guarded((nseg, 3, 4), torch.int32, -5)
    d.dkv_page_select(pk["km"].t.view(nseg, T), table_d, page_rows, CAP, small.t, ne.t, sl.t, ws.t)
    assert small.intact()
    kp = Guarded((n_pages, page_rows, DIM), torch.bfloat16, 0)
    vp = Guarded((n_pages, page_rows, DIM), torch.bfloat16, 0)
    di.fill_pages(kp.t, k.reshape(nseg, T, DIM), table, page_rows)
    di.fill_pages(vp.t, v.reshape(nseg, T, DIM), table, page_rows)
    q = torch.randn((1, HQ, DIM), generator=g, device=DEV).to(torch.bfloat16)
    kn = torch.randn((HKV, 2, DIM), generator=g, device=DEV).to(torch.bfloat16)
    vn = torch.randn((HKV, 2, DIM), generator=g, device=DEV).to(torch.bfloat16)
    out = Guarded((1, HQ, DIM), torch.float32)
    dws = _ws(d.dkv_decode_workspace_bytes(1, HQ, HKV, DIM))
    d.dkv_paged_decode_attn(q, kp.t, vp.t, ent.t[:HKV], ne.t[:HKV], T, 0, 0.1, out.t, dws.t, HKV)
    assert out.intact() and dws.intact()
    first = out.t.clone()
    d.dkv_paged_decode_attn(q, kp.t, vp.t, ent.t[:HKV], ne.t[:HKV], T, 0, 0.1, out.t, dws.t, HKV)
    assert torch.equal(out.t, first)  # fixed merge order
    d.dkv_paged_append_decode_attn(q, kn, vn, CAP - 2, CAP, kp.t, vp.t, ent.t[:HKV], ne.t[:HKV], T, 0.1, out.t,
                                   dws.t, HKV)
    assert out.intact() and dws.intact() and kp.intact() and vp.intact()


def test_topk_export_stays_inside(d):
    rng = np.random.default_rng(3)
    L, H, D = 3, 5, 1001  # 15,015 entries: several workgroups and a ragged last chunk
    probs = torch.from_numpy(rng.integers(0, 50, size=(L, H, D)).astype(np.float32) / 50.0).to(DEV)
    for k in (0, 1, 7000, L * H * D):
        pat = Guarded((L, H, D), torch.uint8, 9)
        ws = _ws(d.dkv_topk_workspace_bytes(L, H, D))
        d.dkv_topk_pattern(probs, k, pat.t, ws.t)
        assert pat.intact() and ws.intact()
        assert int(pat.t.to(torch.int64).sum()) == k


def test_query_block_split_stays_inside(d):
    """Segments long enough for the split: the plan and the partial records
    live in the workspace, and the combine writes the output."""
    g = torch.Generator(device=DEV).manual_seed(13)
    n, t = 1, 12000
    lay = d.make_layout(n, HQ, HKV, DIM, t, S, R, [0, 1000, 3000, 6000, t - S - R])
    pattern = torch.ones((n, HQ, 4), dtype=torch.uint8, device=DEV)
    pattern[0, :4, 1] = 0  # one group drops a bin: segments of different lengths
    k = torch.randn((n, HKV, t, DIM), generator=g, device=DEV).to(torch.bfloat16)
    v = torch.randn((n, HKV, t, DIM), generator=g, device=DEV).to(torch.bfloat16)
    km = torch.empty((n, HKV, t), dtype=torch.uint8, device=DEV)
    kl = torch.empty((n, HKV), dtype=torch.int32, device=DEV)
    d.dkv_map_pattern(lay, pattern, km, kl)
    n_q = 61
    rows = int((kl.cpu().to(torch.int64) + n_q).sum())
    kc = Guarded((rows, DIM), torch.bfloat16, 0)
    vc = Guarded((rows, DIM), torch.bfloat16, 0)
    off = torch.empty(n * HKV, dtype=torch.int64, device=DEV)
    ln = torch.empty(n * HKV, dtype=torch.int32, device=DEV)
    cws = torch.empty(d.dkv_compact_workspace_bytes(lay), dtype=torch.uint8, device=DEV)
    d.dkv_compact(lay, k, v, km, n_q, kc.t, vc.t, off, ln, cws)
    kb = torch.randn((n * HKV, n_q, DIM), generator=g, device=DEV).to(torch.bfloat16)
    vb = torch.randn((n * HKV, n_q, DIM), generator=g, device=DEV).to(torch.bfloat16)
    d.dkv_append(kb, vb, 0, n_q, kc.t, vc.t, off, ln)
    assert kc.intact() and vc.intact()
    qb = torch.randn((n, n_q, HQ, DIM), generator=g, device=DEV).to(torch.bfloat16)
    for hint in (0, rows, rows // 3):
        nb = d.dkv_query_workspace_bytes(n, HQ, HKV, DIM, n_q, hint)
        assert nb > 0  # long enough to split
        out = Guarded((n, n_q, HQ, DIM), torch.float32)
        ws = _ws(nb)
        d.dkv_query_attn(qb, 0, n_q, kc.t, vc.t, off, ln, 0.1, out.t, ws.t, HKV, rows_hint=hint)
        assert out.intact() and ws.intact()
        first = out.t.clone()
        d.dkv_query_attn(qb, 0, n_q, kc.t, vc.t, off, ln, 0.1, out.t, ws.t, HKV, rows_hint=hint)
        assert torch.equal(out.t, first)  # ranges combined in a fixed order
