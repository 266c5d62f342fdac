"""GPU parity of the zero-copy paged variant against the CPU oracle.

dkv_page_select must reproduce the oracle's entries, counts, lengths and page
usage bit for bit (from the GPU's own keep masks, which the map tests pin to
the oracle's).  Paged decode must match the oracle's attention over the rows
the oracle's entries name, within ATTN_TOL, and the fused append must place
every token exactly where the oracle does.  Pools are filled from seeded
dense K/V through a shuffled page table, so every read goes through the
indirection.
"""

import numpy as np
import pytest
import torch

import dkv_inputs as di
import oracle as o
from _helpers import ATTN_TOL, bits, odt, row_rel_err

pytestmark = pytest.mark.gpu

DEV = "cuda"


@pytest.fixture(scope="module")
def d():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2609_32663_amd as lib
    return lib


class GpuSelect:
    """dkv_page_select on the GPU, outputs read back."""

    def __init__(self, d, mask, table, page_rows, cap, max_entries):
        nseg, T = mask.shape
        pps = table.shape[1]
        self.mask = mask
        self.table = torch.from_numpy(np.ascontiguousarray(table)).to(DEV)
        self.entries = torch.full((nseg, max(max_entries, 0), 4), -5, dtype=torch.int32, device=DEV)
        self.n_entries = torch.full((nseg,), -5, dtype=torch.int32, device=DEV)
        self.seg_len = torch.full((nseg,), -5, dtype=torch.int32, device=DEV)
        self.page_used = torch.full((nseg, pps), 9, dtype=torch.uint8, device=DEV)
        ws = torch.empty(max(d.dkv_page_select_workspace_bytes(nseg, T), 16), dtype=torch.uint8, device=DEV)
        d.dkv_page_select(mask, self.table, page_rows, cap, self.entries, self.n_entries, self.seg_len, ws,
                          page_used=self.page_used)
        torch.cuda.synchronize()


def _check_select(sel, ref, max_entries):
    ne = sel.n_entries.cpu().numpy()
    np.testing.assert_array_equal(ne, ref["n_entries"])
    np.testing.assert_array_equal(sel.seg_len.cpu().numpy(), ref["seg_len"])
    np.testing.assert_array_equal(sel.page_used.cpu().numpy(), ref["page_used"])
    ent = sel.entries.cpu().numpy()
    for s in range(len(ne)):
        m = min(int(ne[s]), max_entries)
        np.testing.assert_array_equal(ent[s, :m], ref["entries"][s][:m])
        assert (ent[s, m:] == -5).all()  # nothing written past the count or the array


def _mask_tensor(mask_np):
    """Device copy of a [nseg][T] mask with slack, so that T = 0 still has a pointer."""
    nseg, T = mask_np.shape
    flat = torch.zeros(nseg * T + 16, dtype=torch.uint8, device=DEV)
    flat[:nseg * T] = torch.from_numpy(mask_np.reshape(-1))
    return flat[:nseg * T].view(nseg, T)


# ---------------------------------------------------------------------------
# dkv_page_select
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("page_rows", [32, 64, 128, 256, 512, 1024])
@pytest.mark.parametrize("T", [0, 1, 100, 4096, 5000, 9011, 13 * 1024])
def test_page_select_random_masks(d, page_rows, T):
    rng = np.random.default_rng(page_rows * 1000 + T)
    nseg, cap = 5, int(rng.integers(0, 300))
    pps = -(-(T + cap) // page_rows) + 1
    # per segment: empty, full, sparse, dense, and runs of random length
    probs = [0.0, 1.0, 0.2, 0.9]
    m = np.zeros((nseg, T), np.uint8)
    for s in range(4):
        m[s] = (rng.uniform(size=T) < probs[s]) * rng.integers(1, 256, T)
    pos = 0
    while pos < T:
        n = int(rng.integers(1, 700))
        m[4, pos:pos + n] = rng.integers(0, 2)
        pos += n
    table, _ = di.page_table(nseg, pps, seed=T + page_rows, spare=7)
    ref = o.page_select(m, table, page_rows, cap)
    max_e = int(ref["n_entries"].max())
    _check_select(GpuSelect(d, _mask_tensor(m), table, page_rows, cap, max_e), ref, max_e)


@pytest.mark.parametrize("page_rows", [128, 1024])
def test_page_select_long_context(d, page_rows):
    """More than 1,024 tiles of 4,096 positions: the selection takes its
    separate scan pass (each tile's first entry), bit-exact like the short
    contexts that sum tile counts inside the emit pass."""
    rng = np.random.default_rng(page_rows)
    nseg, T, cap = 2, 1025 * 4096 + 777, 40
    m = np.zeros((nseg, T), np.uint8)
    pos = 0
    while pos < T:
        n = int(rng.integers(1, 3000))
        m[:, pos:pos + n] = rng.integers(0, 2, size=(nseg, 1))
        pos += n
    m[1, :T // 3] = 0  # a long empty stretch in one segment
    table, _ = di.page_table(nseg, -(-(T + cap) // page_rows) + 2, seed=page_rows, spare=5)
    ref = o.page_select(m, table, page_rows, cap)
    max_e = int(ref["n_entries"].max())
    _check_select(GpuSelect(d, _mask_tensor(m), table, page_rows, cap, max_e), ref, max_e)


def test_page_select_overflow_reports_true_counts(d):
    """Entries past max_entries are not written; n_entries still says how
    many there are."""
    rng = np.random.default_rng(3)
    nseg, T, pr, cap = 3, 6000, 64, 40
    m = (rng.uniform(size=(nseg, T)) < 0.5).astype(np.uint8)
    table, _ = di.page_table(nseg, -(-(T + cap) // pr), seed=3)
    ref = o.page_select(m, table, pr, cap)
    for max_e in (0, 1, 17, int(ref["n_entries"].min()) - 1):
        _check_select(GpuSelect(d, _mask_tensor(m), table, pr, cap, max_e), ref, max_e)


def test_page_select_from_gpu_map_of_a_workload(d):
    """Keep masks of the Llama-8B-shaped 32K layer from dkv_map_pattern on the
    GPU, 128-row pages: the selection of the real pattern structure."""
    w = di.workload("llama8b_layer_32k")
    pattern, _ = di.make_pattern(w)
    N, Hq, Hkv, T = w.num_units, w.num_q_heads, w.num_kv_heads, w.context_len
    lay = d.make_layout(N, Hq, Hkv, w.head_dim, T, w.sink, w.recent, list(w.bin_edges))
    km = torch.empty((N, Hkv, T), dtype=torch.uint8, device=DEV)
    kl = torch.empty((N, Hkv), dtype=torch.int32, device=DEV)
    d.dkv_map_pattern(lay, torch.from_numpy(pattern).to(DEV), km, kl, None)
    _, okm, okl = o.map_pattern(pattern, T, w.sink, w.recent, w.bin_edges, Hkv)
    np.testing.assert_array_equal(km.cpu().numpy(), okm)
    cap, pr = 16, 128
    nseg = N * Hkv
    table, _ = di.page_table(nseg, -(-(T + cap) // pr), seed=11)
    ref = o.page_select(okm.reshape(nseg, T), table, pr, cap)
    bound = d.dkv_page_entries_bound(lay, cap, pr)
    assert ref["n_entries"].max() <= bound
    sel = GpuSelect(d, km.view(nseg, T), table, pr, cap, bound)
    _check_select(sel, ref, bound)
    np.testing.assert_array_equal(sel.seg_len.cpu().numpy(), okl.reshape(-1))


def test_page_select_paper_layout_whole_pages(d):
    """The paper's layout (128 sink, 1,024 recent, 128-token bins) with
    128-row pages at T = 130,816: every context entry is a whole page."""
    T, S, R, W = 130816, 128, 1024, 128
    D = (T - S - R) // W
    Hq, Hkv = 8, 2
    rng = np.random.default_rng(5)
    pattern = (rng.uniform(size=(1, Hq, D)) < 0.15).astype(np.uint8)
    lay = d.make_layout(1, Hq, Hkv, 128, T, S, R, [W * k for k in range(D + 1)])
    km = torch.empty((1, Hkv, T), dtype=torch.uint8, device=DEV)
    kl = torch.empty((1, Hkv), dtype=torch.int32, device=DEV)
    d.dkv_map_pattern(lay, torch.from_numpy(pattern).to(DEV), km, kl, None)
    cap = 256
    table, _ = di.page_table(Hkv, -(-(T + cap) // W), seed=5)
    _, okm, _ = o.map_pattern(pattern, T, S, R, [W * k for k in range(D + 1)], Hkv)
    ref = o.page_select(okm.reshape(Hkv, T), table, W, cap)
    bound = d.dkv_page_entries_bound(lay, cap, W)
    sel = GpuSelect(d, km.view(Hkv, T), table, W, cap, bound)
    _check_select(sel, ref, bound)
    ent = sel.entries.cpu().numpy()
    ne = sel.n_entries.cpu().numpy()
    for g in range(Hkv):
        e = ent[g, :ne[g]]
        ctx = e[e[:, 1] * W < T]
        assert (ctx[:, 2] == 0).all() and (ctx[:, 3] == W).all()


# ---------------------------------------------------------------------------
# paged decode
# ---------------------------------------------------------------------------

class PagedCase:
    """One layer of a workload in a shuffled page pool, selected on the GPU."""

    def __init__(self, d, w, page_rows, cap, seed, pattern=None, spare=5):
        self.w = w
        B, Hq, Hkv, T, dim = w.batch, w.num_q_heads, w.num_kv_heads, w.context_len, w.head_dim
        nseg = B * Hkv
        self.nseg, self.pr, self.cap = nseg, page_rows, cap
        if pattern is None:
            pattern, _ = di.make_pattern(w)
        pattern = np.ascontiguousarray(pattern[:B])
        lay = d.make_layout(B, Hq, Hkv, dim, T, w.sink, w.recent, list(w.bin_edges))
        self.km = torch.empty((B, Hkv, T), dtype=torch.uint8, device=DEV)
        kl = torch.empty((B, Hkv), dtype=torch.int32, device=DEV)
        d.dkv_map_pattern(lay, torch.from_numpy(pattern).to(DEV), self.km, kl, None)
        _, okm, _ = o.map_pattern(pattern, T, w.sink, w.recent, w.bin_edges, Hkv)
        self.okm = okm.reshape(nseg, T)
        pps = -(-(T + cap) // page_rows)
        self.table, self.num_pages = di.page_table(nseg, pps, seed=seed, spare=spare)
        kv = [di.kv_unit(w, b, device=DEV) for b in range(B)]
        k = torch.stack([a for a, _ in kv]).view(nseg, T, dim)
        v = torch.stack([b for _, b in kv]).view(nseg, T, dim)
        del kv
        # unused slots hold NaN: a masked slot that reached the softmax would show
        nan = float("nan")
        self.kp = torch.full((self.num_pages, page_rows, dim), nan, dtype=k.dtype, device=DEV)
        self.vp = torch.full_like(self.kp, nan)
        # pruned context positions hold NaN too: only retained rows may be read
        km = self.km.view(nseg, T)
        k = torch.where(km.unsqueeze(-1) != 0, k, torch.full_like(k, nan))
        v = torch.where(km.unsqueeze(-1) != 0, v, torch.full_like(v, nan))
        di.fill_pages(self.kp, k, self.table, page_rows)
        di.fill_pages(self.vp, v, self.table, page_rows)
        del k, v
        self.ref = o.page_select(self.okm, self.table, page_rows, cap)
        self.max_e = d.dkv_page_entries_bound(lay, cap, page_rows)
        self.sel = GpuSelect(d, self.km.view(nseg, T), self.table, page_rows, cap, self.max_e)
        _check_select(self.sel, self.ref, self.max_e)
        self.rows = int(self.sel.n_entries.cpu().to(torch.int64).sum()) * page_rows
        self.ws = torch.zeros(d.dkv_decode_workspace_bytes(B, Hq, Hkv, dim), dtype=torch.uint8, device=DEV)

    def pools_np(self):
        return bits(self.kp), bits(self.vp)


def _paged_cases():
    return [
        ("tiny", 32, 16),
        ("tiny", 64, 5),
        ("llama8b_layer_32k", 128, 16),
        ("llama8b_layer_32k", 32, 40),
        ("llama8b_layer_32k", 256, 16),
        ("llama8b_layer_32k", 1024, 16),
        ("llama70b_layer_bs16_32k", 128, 16),
    ]


@pytest.mark.parametrize("name,page_rows,cap", _paged_cases())
def test_paged_decode_matches_oracle(d, name, page_rows, cap):
    w = di.workload(name)
    c = PagedCase(d, w, page_rows, cap, seed=page_rows + cap)
    B, Hq, Hkv, dim, T = w.batch, w.num_q_heads, w.num_kv_heads, w.head_dim, w.context_len
    kp, vp = c.pools_np()
    for n_tail in (0, cap // 2):
        if n_tail:
            # tokens already appended, written by the oracle's rule
            kn, vn = di.kv_new_step(w, 0, 99, n_new=n_tail, device=DEV)
            kn = kn.reshape(c.nseg, n_tail, dim)
            vn = vn.reshape(c.nseg, n_tail, dim)
            kp, vp = o.paged_append(kp, vp, c.table, page_rows, T, bits(kn), bits(vn), 0)
            c.kp.copy_(torch.from_numpy(kp.view(np.int16) if kp.dtype == np.uint16 else kp).view(c.kp.dtype)
                       .to(DEV))
            c.vp.copy_(torch.from_numpy(vp.view(np.int16) if vp.dtype == np.uint16 else vp).view(c.vp.dtype)
                       .to(DEV))
        q = di.q_step(w, 0, n_tail, device=DEV)
        out = torch.full((B, Hq, dim), 7.0, dtype=torch.float32, device=DEV)
        d.dkv_paged_decode_attn(q, c.kp, c.vp, c.sel.entries, c.sel.n_entries, T, n_tail, w.sm_scale, out, c.ws,
                                Hkv, rows_hint=c.rows)
        torch.cuda.synchronize()
        want = o.paged_decode_attn(bits(q), kp, vp, c.ref["entries"], page_rows, T, n_tail, w.sm_scale, Hkv,
                                   odt(q))
        got = out.cpu().numpy()
        assert np.isfinite(got).all()
        err = row_rel_err(got, want)
        assert err <= ATTN_TOL, (name, page_rows, n_tail, err)


@pytest.mark.parametrize("page_rows", [32, 128])
def test_paged_append_decode_steps(d, page_rows):
    """Fused append + decode over several steps, crossing a page boundary of
    the append region: pools bit-exact, outputs within tolerance."""
    w = di.workload("llama8b_layer_32k")
    cap = 48
    c = PagedCase(d, w, page_rows, cap, seed=21)
    B, Hq, Hkv, dim, T = w.batch, w.num_q_heads, w.num_kv_heads, w.head_dim, w.context_len
    kp, vp = c.pools_np()
    out = torch.empty((B, Hq, dim), dtype=torch.float32, device=DEV)
    for step in range(40):
        q = di.q_step(w, 0, step, device=DEV)
        kn, vn = di.kv_new_step(w, 0, step, device=DEV)
        kn = kn.reshape(c.nseg, 1, dim).contiguous()
        vn = vn.reshape(c.nseg, 1, dim).contiguous()
        d.dkv_paged_append_decode_attn(q, kn, vn, step, cap, c.kp, c.vp, c.sel.entries, c.sel.n_entries, T,
                                       w.sm_scale, out, c.ws, Hkv, rows_hint=c.rows)
        kp, vp = o.paged_append(kp, vp, c.table, page_rows, T, bits(kn), bits(vn), step)
        if step % 13 == 0 or step == 39:
            torch.cuda.synchronize()
            want = o.paged_decode_attn(bits(q), kp, vp, c.ref["entries"], page_rows, T, step + 1, w.sm_scale,
                                       Hkv, o.BF16)
            err = row_rel_err(out.cpu().numpy(), want)
            assert err <= ATTN_TOL, (step, err)
    torch.cuda.synchronize()
    gk, gv = c.pools_np()
    # NaN slots compare by bit pattern
    assert np.array_equal(gk, kp) and np.array_equal(gv, vp)


def test_paged_decode_clips_bad_entries_and_truncation(d):
    """An entry naming a page outside the pool, or slots outside a page,
    attends nothing; a segment's entries past max_entries are not read."""
    w = di.workload("llama8b_layer_32k")
    c = PagedCase(d, w, 128, 16, seed=31)
    B, Hq, Hkv, dim, T = w.batch, w.num_q_heads, w.num_kv_heads, w.head_dim, w.context_len
    ent = c.sel.entries.clone()
    ne = c.sel.n_entries.clone()
    ref_ent = [e.copy() for e in c.ref["entries"]]
    # segment 0: a page id past the pool; segment 1: hi beyond the page;
    # segment 2: lo >= hi; segment 3: only the first 5 entries are read
    ent[0, 3, 0] = c.num_pages + 3
    ent[1, 4, 3] = 129
    ent[2, 2, 2] = ent[2, 2, 3]
    for s, i in ((0, 3), (1, 4), (2, 2)):
        ref_ent[s] = np.delete(ref_ent[s], i, axis=0)
    small = torch.full((c.nseg, 5, 4), -5, dtype=torch.int32, device=DEV)
    small.copy_(c.sel.entries[:, :5])
    q = di.q_step(w, 0, 0, device=DEV)
    out = torch.empty((B, Hq, dim), dtype=torch.float32, device=DEV)
    d.dkv_paged_decode_attn(q, c.kp, c.vp, ent, ne, T, 0, w.sm_scale, out, c.ws, Hkv, rows_hint=c.rows)
    torch.cuda.synchronize()
    kp, vp = c.pools_np()
    want = o.paged_decode_attn(bits(q), kp, vp, ref_ent, 128, T, 0, w.sm_scale, Hkv, o.BF16)
    assert row_rel_err(out.cpu().numpy(), want) <= ATTN_TOL
    d.dkv_paged_decode_attn(q, c.kp, c.vp, small, ne, T, 0, w.sm_scale, out, c.ws, Hkv, rows_hint=c.rows)
    torch.cuda.synchronize()
    trunc = [e[:5] for e in c.ref["entries"]]
    want = o.paged_decode_attn(bits(q), kp, vp, trunc, 128, T, 0, w.sm_scale, Hkv, o.BF16)
    assert row_rel_err(out.cpu().numpy(), want) <= ATTN_TOL


def test_paged_decode_empty_segments_are_zero(d):
    """No retained context and no append region: zeros; appended tokens
    only: attention over them."""
    w = di.workload("tiny", context_len=256, sink=0, recent=0)
    pattern = np.zeros((1, w.num_q_heads, w.num_bins), np.uint8)
    for cap in (0, 3):
        c = PagedCase(d, w, 32, cap, seed=41, pattern=pattern)
        assert int(c.sel.seg_len.sum()) == 0
        q = di.q_step(w, 0, 0, device=DEV)
        out = torch.full((1, w.num_q_heads, w.head_dim), 7.0, dtype=torch.float32, device=DEV)
        kp, vp = c.pools_np()
        if cap:
            kn, vn = di.kv_new_step(w, 0, 0, n_new=2, device=DEV)
            kn = kn.reshape(c.nseg, 2, w.head_dim).contiguous()
            vn = vn.reshape(c.nseg, 2, w.head_dim).contiguous()
            d.dkv_paged_append_decode_attn(q, kn, vn, 0, cap, c.kp, c.vp, c.sel.entries, c.sel.n_entries,
                                           w.context_len, w.sm_scale, out, c.ws, w.num_kv_heads, rows_hint=c.rows)
            kp, vp = o.paged_append(kp, vp, c.table, 32, w.context_len, bits(kn), bits(vn), 0)
        else:
            d.dkv_paged_decode_attn(q, c.kp, c.vp, c.sel.entries, c.sel.n_entries, w.context_len, 0,
                                    w.sm_scale, out, c.ws, w.num_kv_heads, rows_hint=c.rows)
        torch.cuda.synchronize()
        want = o.paged_decode_attn(bits(q), kp, vp, c.ref["entries"], 32, w.context_len, 2 if cap else 0,
                                   w.sm_scale, w.num_kv_heads, o.F32)
        got = out.cpu().numpy()
        if cap == 0:
            assert (got == 0).all()
        assert row_rel_err(got, want) <= ATTN_TOL
