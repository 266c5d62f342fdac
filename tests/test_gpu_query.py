"""GPU parity of query-block attention (dkv_query_attn) against the oracle.

Every case runs the GPU path end to end through the C ABI: compaction of a
dense cache under a keep mask, append of the tokens before the block and of
the block itself, then the block's attention.  The oracle packs, appends and
attends on its own from the same inputs.  Output rows ([B][n_q][Hq] rows of
d values) must be within ATTN_TOL (max relative error per row).
"""

import numpy as np
import pytest
import torch

import oracle as o
from _helpers import ATTN_TOL, bits, row_rel_err

pytestmark = pytest.mark.gpu

DEV = "cuda"


@pytest.fixture(scope="module")
def d():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2609_32663_amd as lib
    return lib


def _bf16(rng, shape, scale=1.0):
    return (torch.from_numpy(rng.standard_normal(shape).astype(np.float32)) * scale).to(torch.bfloat16)


def _run(d, rng, B, Hkv, G, T, dim, keep, n_tail, n_q, cap=None, sm_scale=None, hint="exact",
         empty_segments=0, inspect=None):
    """One case; returns (gpu out [B][n_q][Hq][d], oracle out)."""
    Hq = Hkv * G
    cap = n_tail + n_q if cap is None else cap
    sm_scale = 1.0 / np.sqrt(dim) if sm_scale is None else sm_scale
    k = _bf16(rng, (B, Hkv, T, dim))
    v = _bf16(rng, (B, Hkv, T, dim))
    mask = (rng.uniform(size=(B, Hkv, T)) < keep).astype(np.uint8)
    for e in range(empty_segments):
        mask[e % B, (e // B) % Hkv] = 0
    kt = _bf16(rng, (B, Hkv, n_tail, dim))
    vt = _bf16(rng, (B, Hkv, n_tail, dim))
    kb = _bf16(rng, (B, Hkv, n_q, dim))
    vb = _bf16(rng, (B, Hkv, n_q, dim))
    q = _bf16(rng, (B, n_q, Hq, dim))

    # GPU: pack, append the earlier tokens and the block, attend
    lay = d.make_layout(B, Hq, Hkv, dim, T, 0, 0, [0, max(T, 1)])
    rows = int(mask.sum()) + B * Hkv * cap
    k_c = torch.empty((max(rows, 1), dim), dtype=torch.bfloat16, device=DEV)
    v_c = torch.empty_like(k_c)
    seg_off = torch.empty(B * Hkv, dtype=torch.int64, device=DEV)
    seg_len = torch.empty(B * Hkv, dtype=torch.int32, device=DEV)
    cws = torch.empty(d.dkv_compact_workspace_bytes(lay), dtype=torch.uint8, device=DEV)
    d.dkv_compact(lay, k.to(DEV), v.to(DEV), torch.from_numpy(mask).to(DEV), cap, k_c, v_c, seg_off,
                  seg_len, cws)
    if n_tail:
        d.dkv_append(kt.reshape(B * Hkv, n_tail, dim).to(DEV), vt.reshape(B * Hkv, n_tail, dim).to(DEV), 0,
                     cap, k_c, v_c, seg_off, seg_len)
    d.dkv_append(kb.reshape(B * Hkv, n_q, dim).to(DEV), vb.reshape(B * Hkv, n_q, dim).to(DEV), n_tail, cap,
                 k_c, v_c, seg_off, seg_len)
    exact = int(mask.sum()) + B * Hkv * (n_tail + n_q)
    rows_hint = exact if hint == "exact" else (hint(exact) if callable(hint) else hint)
    wsb = d.dkv_query_workspace_bytes(B, Hq, Hkv, dim, n_q, rows_hint)
    ws = torch.empty(wsb, dtype=torch.uint8, device=DEV) if wsb else None
    out = torch.full((B, n_q, Hq, dim), float("nan"), dtype=torch.float32, device=DEV)
    d.dkv_query_attn(q.to(DEV), n_tail, cap, k_c, v_c, seg_off, seg_len, sm_scale, out, ws, Hkv,
                     rows_hint=rows_hint)
    torch.cuda.synchronize()
    if inspect is not None:
        inspect(ws, seg_len.cpu().numpy(), rows_hint, wsb)

    # oracle on its own
    ref = o.compact(bits(k), bits(v), mask, cap)
    new_k = np.concatenate([bits(kt), bits(kb)], axis=2)
    new_v = np.concatenate([bits(vt), bits(vb)], axis=2)
    kc, vc = o.append(ref["k_c"], ref["v_c"], ref["seg_off"], ref["seg_len"], new_k, new_v, 0)
    want = o.query_attn(bits(q), kc, vc, ref["seg_off"], ref["seg_len"], n_tail, sm_scale, Hkv, o.BF16)
    return out.cpu().numpy(), want


@pytest.mark.parametrize("dim", [64, 128])
def test_query_random_shapes(d, dim):
    rng = np.random.default_rng(700 + dim)
    for trial in range(10):
        B = int(rng.integers(1, 3))
        Hkv = int(rng.choice([1, 2, 4]))
        G = int(rng.choice([1, 2, 3, 4, 7, 8]))
        T = int(rng.integers(1, 700))
        n_q = int(rng.choice([1, 2, 5, 16, 17, 33]))
        n_tail = int(rng.integers(0, 3))
        got, want = _run(d, rng, B, Hkv, G, T, dim, float(rng.uniform(0.05, 0.9)), n_tail, n_q,
                         cap=n_tail + n_q + int(rng.integers(0, 3)))
        assert np.isfinite(got).all()
        err = row_rel_err(got.reshape(-1, dim), want.reshape(-1, dim))
        assert err <= ATTN_TOL, (trial, B, Hkv, G, T, n_q, n_tail, err)


@pytest.mark.parametrize("G,n_q,dim", [(1, 64, 128), (4, 64, 128), (4, 100, 128), (7, 40, 128), (8, 128, 128),
                                       (4, 64, 64), (8, 100, 64), (16, 33, 128)])
def test_query_split_key_ranges(d, G, n_q, dim):
    """Long contexts: the keys are split into several ranges and combined."""
    rng = np.random.default_rng(800 + G * 1000 + n_q + dim)
    got, want = _run(d, rng, 1, 2, G, 12000, dim, 0.4, 2, n_q)
    err = row_rel_err(got.reshape(-1, dim), want.reshape(-1, dim))
    assert err <= ATTN_TOL, err


@pytest.mark.parametrize("hint", ["exact", "third", "twentieth", "twenty_times", "none"])
def test_query_unequal_segments_and_wrong_hints(d, hint):
    """Segments from empty to fully kept: the split cuts each into its own
    number of equal ranges.  A hint below the true rows (the plan widens the
    ranges to fit the records), far below it (no split), far above it (fewer,
    longer ranges) or missing changes the split, never the result."""
    rng = np.random.default_rng(905)
    B, Hkv = 2, 4
    keep = rng.permutation(np.array([0.0, 0.001, 0.01, 0.05, 0.2, 0.5, 0.9, 1.0])).reshape(B, Hkv, 1)
    h = {"exact": "exact", "third": lambda x: x // 3, "twentieth": lambda x: x // 20,
         "twenty_times": lambda x: 20 * x, "none": 0}[hint]
    got, want = _run(d, rng, B, Hkv, 4, 20000, 128, keep, 1, 40, hint=h)
    assert np.isfinite(got).all()
    err = row_rel_err(got.reshape(-1, 128), want.reshape(-1, 128))
    assert err <= ATTN_TOL, (hint, err)


# The split's plan, computed independently from its definition: 256-row query
# tiles; C tiles per range from the hint (about 512 items, at least 8 tiles);
# no split when the segments average under 16 tiles; records for
# qtiles * (tiles / C + nseg + 1) items rounded up to 8; C widened on the GPU
# until qtiles * sum_s max(1, round(T_s / C)) fits them.
def _plan_shape(nseg, rows, dim, hint):
    qtiles = -(-rows // 256)
    tiles = (min(hint, 1 << 40) + 63) // 64 + nseg if hint > 0 else nseg * 512
    c = min(max(8, -(-(qtiles * tiles) // 512)), 1 << 30)
    if tiles < nseg * 16:
        return qtiles, c, nseg * qtiles, 0, 0
    max_items = -(-(qtiles * (tiles // c + nseg + 1)) // 8) * 8
    plan_bytes = -(-((4 + nseg + 1) * 4) // 256) * 256
    return qtiles, c, max_items, plan_bytes, max_items * 256 * (dim + 2) * 4


def _plan_expect(seg_tiles, qtiles, c, max_items):
    nseg = len(seg_tiles)
    room = max_items // qtiles - nseg
    c = max(c, -(-int(sum(seg_tiles)) // room))
    ranges = [max(1, (int(t) + c // 2) // c) for t in seg_tiles]
    return c, np.concatenate([[0], np.cumsum(ranges)]).astype(np.int64) * qtiles


@pytest.mark.parametrize("hint", ["exact", "third", "none"])
def test_query_plan_bit_exact(d, hint):
    """The plan kernel's words (items, tiles per range, first item of every
    segment) equal the split computed from its definition, including the
    widening a too-small hint forces, and the workspace size matches."""
    rng = np.random.default_rng(908)
    B, Hkv, G, T, dim, n_tail, n_q = 2, 4, 4, 20000, 128, 1, 300
    keep = rng.permutation(np.array([0.0, 0.01, 0.05, 0.2, 0.4, 0.6, 0.9, 1.0])).reshape(B, Hkv, 1)
    h = {"exact": "exact", "third": lambda x: x // 3, "none": 0}[hint]
    seen = {}

    def inspect(ws, seg_len, rows_hint, wsb):
        qtiles, c, max_items, plan_bytes, rec_bytes = _plan_shape(B * Hkv, n_q * G, dim, rows_hint)
        assert wsb == plan_bytes + rec_bytes
        assert plan_bytes > 0, "the case must split"
        words = ws[:plan_bytes].cpu().view(torch.int32).numpy()
        seg_tiles = (seg_len.astype(np.int64) + n_tail + n_q + 63) // 64
        c_want, first = _plan_expect(seg_tiles, qtiles, c, max_items)
        assert int(words[0]) == int(first[-1]) <= max_items
        assert int(words[1]) == c_want
        np.testing.assert_array_equal(words[4:4 + B * Hkv + 1].astype(np.int64), first)
        seen["c"], seen["c_host"] = c_want, c

    got, want = _run(d, rng, B, Hkv, G, T, dim, keep, n_tail, n_q, hint=h, inspect=inspect)
    assert row_rel_err(got.reshape(-1, dim), want.reshape(-1, dim)) <= ATTN_TOL
    if hint == "third":
        assert seen["c"] > seen["c_host"], "a too-small hint must widen the ranges"


def test_query_more_segments_than_one_plan_pass(d):
    """1,200 segments: the plan scans them in two passes of its workgroup,
    and the items are dealt to the L2 domains in runs."""
    rng = np.random.default_rng(906)
    got, want = _run(d, rng, 300, 4, 1, 1100, 64, 1.0, 0, 2)
    err = row_rel_err(got.reshape(-1, 64), want.reshape(-1, 64))
    assert err <= ATTN_TOL, err


def test_query_unknown_rows_hint_and_empty_context(d):
    """rows_hint 0 (split sized for long segments) with several segments that
    hold no context at all: those rows see only the tokens after it."""
    rng = np.random.default_rng(901)
    got, want = _run(d, rng, 2, 2, 4, 3000, 128, 0.3, 1, 9, hint=0, empty_segments=2)
    err = row_rel_err(got.reshape(-1, 128), want.reshape(-1, 128))
    assert err <= ATTN_TOL, err


def test_query_large_logits(d):
    rng = np.random.default_rng(902)
    got, want = _run(d, rng, 1, 2, 4, 2000, 128, 0.5, 0, 20, sm_scale=3.0)
    assert np.isfinite(got).all()
    assert row_rel_err(got.reshape(-1, 128), want.reshape(-1, 128)) <= ATTN_TOL


@pytest.mark.parametrize("scale", [-0.7, 0.0])
def test_query_negative_and_zero_scale(d, scale):
    """The kernel scores with |scale| and negated queries for a negative
    scale; a zero scale is uniform attention over the visible keys."""
    rng = np.random.default_rng(907)
    got, want = _run(d, rng, 1, 2, 4, 3000, 128, 0.5, 1, 24, sm_scale=scale)
    assert np.isfinite(got).all()
    assert row_rel_err(got.reshape(-1, 128), want.reshape(-1, 128)) <= ATTN_TOL


def test_query_block_of_one_matches_decode_kernel(d):
    """A one-token block is a decode step: both kernels agree with the oracle
    and with each other within the tolerance."""
    rng = np.random.default_rng(903)
    B, Hkv, G, T, dim = 1, 4, 4, 5000, 128
    got, want = _run(d, rng, B, Hkv, G, T, dim, 0.35, 0, 1)
    assert row_rel_err(got.reshape(-1, dim), want.reshape(-1, dim)) <= ATTN_TOL


def test_query_8b_layer_block_of_256(d):
    """An 8B-shaped layer at 32K with a 256-token query block (the paper's
    reserved query/answer length)."""
    import dkv_inputs as di
    w = di.workload("llama8b_layer_32k")
    pattern, _ = di.make_pattern(w)
    _, okm, _ = o.map_pattern(pattern, w.context_len, w.sink, w.recent, w.bin_edges, w.num_kv_heads)
    rng = np.random.default_rng(904)
    n_q = 256
    Hkv, G, dim, T = w.num_kv_heads, w.group, w.head_dim, w.context_len
    k, v = di.kv_unit(w, 0, device=DEV)
    kb = _bf16(rng, (1, Hkv, n_q, dim))
    vb = _bf16(rng, (1, Hkv, n_q, dim))
    q = _bf16(rng, (1, n_q, Hkv * G, dim), 1.0 / np.sqrt(dim))
    lay = d.make_layout(1, Hkv * G, Hkv, dim, T, 0, 0, [0, T])
    rows = int(okm.sum()) + Hkv * n_q
    k_c = torch.empty((rows, dim), dtype=torch.bfloat16, device=DEV)
    v_c = torch.empty_like(k_c)
    seg_off = torch.empty(Hkv, dtype=torch.int64, device=DEV)
    seg_len = torch.empty(Hkv, dtype=torch.int32, device=DEV)
    cws = torch.empty(d.dkv_compact_workspace_bytes(lay), dtype=torch.uint8, device=DEV)
    d.dkv_compact(lay, k[None], v[None], torch.from_numpy(okm).to(DEV), n_q, k_c, v_c, seg_off, seg_len, cws)
    d.dkv_append(kb[0].to(DEV), vb[0].to(DEV), 0, n_q, k_c, v_c, seg_off, seg_len)
    wsb = d.dkv_query_workspace_bytes(1, Hkv * G, Hkv, dim, n_q, rows)
    ws = torch.empty(max(wsb, 16), dtype=torch.uint8, device=DEV)
    out = torch.empty((1, n_q, Hkv * G, dim), dtype=torch.float32, device=DEV)
    d.dkv_query_attn(q.to(DEV), 0, n_q, k_c, v_c, seg_off, seg_len, w.sm_scale, out, ws, Hkv, rows_hint=rows)
    torch.cuda.synchronize()
    ref = o.compact(bits(k[None]), bits(v[None]), okm, n_q)
    kc, vc = o.append(ref["k_c"], ref["v_c"], ref["seg_off"], ref["seg_len"], bits(kb), bits(vb), 0)
    want = o.query_attn(bits(q), kc, vc, ref["seg_off"], ref["seg_len"], 0, w.sm_scale, Hkv, o.BF16)
    assert row_rel_err(out.cpu().numpy().reshape(-1, dim), want.reshape(-1, dim)) <= ATTN_TOL


def test_multi_turn_reuse_of_one_pack(d):
    """Several query rounds over one compacted cache (the shared-context
    multi-turn setting of Sec. 4.2: one fixed pattern and one compression
    serve successive queries).  Each turn appends its query block
    from n_tail = 0, overwriting the previous turn's tokens, attends with the
    block, then decodes a few tokens appended after the block; every call is
    checked against the oracle, which repeats the same bookkeeping."""
    rng = np.random.default_rng(905)
    B, Hkv, G, T, dim = 2, 2, 4, 3000, 128
    Hq = Hkv * G
    turns = [(12, 3), (5, 2), (20, 4)]  # (block tokens, decode steps) per turn
    cap = max(n_q + steps for n_q, steps in turns)
    k = _bf16(rng, (B, Hkv, T, dim))
    v = _bf16(rng, (B, Hkv, T, dim))
    mask = (rng.uniform(size=(B, Hkv, T)) < 0.3).astype(np.uint8)
    lay = d.make_layout(B, Hq, Hkv, dim, T, 0, 0, [0, T])
    rows = int(mask.sum()) + B * Hkv * cap
    k_c = torch.empty((rows, dim), dtype=torch.bfloat16, device=DEV)
    v_c = torch.empty_like(k_c)
    seg_off = torch.empty(B * Hkv, dtype=torch.int64, device=DEV)
    seg_len = torch.empty(B * Hkv, dtype=torch.int32, device=DEV)
    cws = torch.empty(d.dkv_compact_workspace_bytes(lay), dtype=torch.uint8, device=DEV)
    d.dkv_compact(lay, k.to(DEV), v.to(DEV), torch.from_numpy(mask).to(DEV), cap, k_c, v_c, seg_off, seg_len, cws)
    ref = o.compact(bits(k), bits(v), mask, cap)
    dws = torch.zeros(d.dkv_decode_workspace_bytes(B, Hq, Hkv, dim), dtype=torch.uint8, device=DEV)
    for turn, (n_q, steps) in enumerate(turns):
        kb = _bf16(rng, (B, Hkv, n_q, dim))
        vb = _bf16(rng, (B, Hkv, n_q, dim))
        q = _bf16(rng, (B, n_q, Hq, dim), 1.0 / np.sqrt(dim))
        d.dkv_append(kb.reshape(B * Hkv, n_q, dim).to(DEV), vb.reshape(B * Hkv, n_q, dim).to(DEV), 0, cap, k_c,
                     v_c, seg_off, seg_len)
        kc_t, vc_t = o.append(ref["k_c"], ref["v_c"], ref["seg_off"], ref["seg_len"], bits(kb), bits(vb), 0)
        wsb = d.dkv_query_workspace_bytes(B, Hq, Hkv, dim, n_q, 0)
        ws = torch.empty(wsb, dtype=torch.uint8, device=DEV) if wsb else None
        out = torch.empty((B, n_q, Hq, dim), dtype=torch.float32, device=DEV)
        d.dkv_query_attn(q.to(DEV), 0, cap, k_c, v_c, seg_off, seg_len, 1.0, out, ws, Hkv)
        torch.cuda.synchronize()
        want = o.query_attn(bits(q), kc_t, vc_t, ref["seg_off"], ref["seg_len"], 0, 1.0, Hkv, o.BF16)
        assert row_rel_err(out.cpu().numpy().reshape(-1, dim), want.reshape(-1, dim)) <= ATTN_TOL, (turn, "query")
        for step in range(steps):
            kn = _bf16(rng, (B * Hkv, 1, dim))
            vn = _bf16(rng, (B * Hkv, 1, dim))
            qd = _bf16(rng, (B, Hq, dim), 1.0 / np.sqrt(dim))
            od = torch.empty((B, Hq, dim), dtype=torch.float32, device=DEV)
            d.dkv_append_decode_attn(qd.to(DEV), kn.to(DEV), vn.to(DEV), n_q + step, cap, k_c, v_c, seg_off,
                                     seg_len, 1.0, od, dws, Hkv)
            torch.cuda.synchronize()
            kc_t, vc_t = o.append(kc_t, vc_t, ref["seg_off"], ref["seg_len"], bits(kn).reshape(B, Hkv, 1, dim),
                                  bits(vn).reshape(B, Hkv, 1, dim), n_q + step)
            want = o.decode_attn(bits(qd), kc_t, vc_t, ref["seg_off"], ref["seg_len"], n_q + step + 1, 1.0, Hkv,
                                 o.BF16)
            assert row_rel_err(od.cpu().numpy(), want) <= ATTN_TOL, (turn, step)
