"""Pins for the CPU oracle: checks against what the paper and mathematics fix.

Nothing here retypes the oracle's own formulas.  Masks are checked against
the bin counts printed in Appendix A, against the special cases of Sec. 3.2
(all-zero pattern = StreamingLLM's sink + recent, head-level pattern, all-keep)
and against a brute-force construction that paints whole bins instead of
looking up each position.  Packing is checked against a pure-Python loop and
its invariants (order kept, rows bit-identical).  Attention is checked
against torch's scaled_dot_product_attention (a library routine, with and
without a boolean mask, with its own GQA grouping) and against closed forms
(one row, two rows, equal logits).
"""

import json
import os

import numpy as np
import pytest
import torch

import oracle as o
import dkv_inputs as di

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


# ---------------------------------------------------------------------------
# helpers that are independent of the oracle
# ---------------------------------------------------------------------------

def paint_masks(pattern, T, S, R, edges, n_kv):
    """Brute force: paint sink, recent and then whole bins, in pure Python."""
    n_units, n_q, D = pattern.shape
    G = n_q // n_kv
    qm = np.zeros((n_units, n_q, T), dtype=np.uint8)
    for n in range(n_units):
        for h in range(n_q):
            for j in range(min(S, T)):
                qm[n, h, j] = 1
            for j in range(max(0, T - R), T):
                qm[n, h, j] = 1
            for k in range(D):
                for u in range(edges[k], edges[k + 1]):
                    j = T - 1 - R - u          # u counts back from the recent window
                    if S <= j <= T - 1 - R:
                        qm[n, h, j] = pattern[n, h, k]
    km = np.zeros((n_units, n_kv, T), dtype=np.uint8)
    for n in range(n_units):
        for g in range(n_kv):
            for h in range(g * G, g * G + G):
                for j in range(T):
                    if qm[n, h, j]:
                        km[n, g, j] = 1
    return qm, km


def sdpa(q, k, v, scale, mask=None):
    """torch SDPA in float64 on [B][H][1][d] queries with GQA grouping."""
    qt = torch.from_numpy(q)[:, :, None, :]
    kt = torch.from_numpy(k)
    vt = torch.from_numpy(v)
    out = torch.nn.functional.scaled_dot_product_attention(
        qt, kt, vt, attn_mask=mask, scale=scale, enable_gqa=True)
    return out[:, :, 0, :].numpy()


def random_layout(rng):
    T = int(rng.integers(0, 70))
    S = int(rng.integers(0, 5))
    R = int(rng.integers(0, 5))
    D = int(rng.integers(1, 9))
    steps = rng.integers(1, 6, size=D)
    edges = [0] + list(np.cumsum(steps))
    n_kv = int(rng.integers(1, 4))
    G = int(rng.integers(1, 4))
    n_units = int(rng.integers(1, 3))
    pattern = (rng.uniform(size=(n_units, n_kv * G, D)) < rng.uniform()).astype(np.uint8)
    return T, S, R, [int(e) for e in edges], n_kv, pattern


# ---------------------------------------------------------------------------
# bf16 widening
# ---------------------------------------------------------------------------

def test_widen_bf16_known_bits():
    bits = np.array([0x3F80, 0xC000, 0x3F81, 0x0000, 0x8000, 0x7F7F, 0x0001], dtype=np.uint16)
    want = [1.0, -2.0, 1.0 + 2.0 ** -7, 0.0, -0.0, (2 - 2.0 ** -7) * 2.0 ** 127, 2.0 ** -133]
    got = o.widen(bits, o.BF16)
    assert got.dtype == np.float64
    assert list(got) == want


def test_widen_matches_torch_bf16():
    x = torch.randn(1000, generator=torch.Generator().manual_seed(3)).to(torch.bfloat16)
    bits = x.view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(o.widen(bits, o.BF16), x.double().numpy())


# ---------------------------------------------------------------------------
# Eq. (4) / Eq. (5): the paper's printed bin layouts
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("idx", [0, 1])
def test_paper_bin_count(idx):
    g = _golden("paper_layout.json")
    lay = g["layouts"][idx]
    T, S, R, W = lay["context_len"], g["sink"], g["recent"], g["bin_width"]
    D_print = lay["num_bins"]
    D_big = D_print + 40  # more bins than the context can instantiate
    edges = di.uniform_bin_edges(W, D_big)
    # one query head that keeps only the odd bins
    pat = np.zeros((1, 1, D_big), dtype=np.uint8)
    pat[0, 0, 1::2] = 1
    qm = o.q_keep_mask(pat, T, S, R, edges)[0, 0]
    # which bins were instantiated: every bin that covers at least one position
    j = np.arange(S, T - R)
    ks = o.bin_index(T - 1 - j - R, edges)
    assert sorted(set(ks.tolist())) == list(range(D_print))
    # the kept compressible count is 128 per odd instantiated bin
    assert int(qm[S:T - R].sum()) == W * len(range(1, D_print, 2))
    assert int(qm.sum()) == S + R + W * len(range(1, D_print, 2))


@pytest.mark.parametrize("idx", [0, 1])
def test_paper_bin_endpoints(idx):
    g = _golden("paper_layout.json")
    lay = g["layouts"][idx]
    T, S, R, W = lay["context_len"], g["sink"], g["recent"], g["bin_width"]
    D = lay["num_bins"]
    edges = di.uniform_bin_edges(W, D)
    # 1-indexed i = 129 is the first compressible position, in the farthest bin
    j_first = g["first_compressible_position_1idx"] - 1
    j_last = T - g["last_compressible_offset_from_end"] - 1   # i = T_c - 1024
    k_first = o.bin_index(T - 1 - j_first - R, edges)
    k_last = o.bin_index(T - 1 - j_last - R, edges)
    assert int(k_first) == D - 1
    assert int(k_last) == 0
    # their neighbours are sink and recent: kept even by an all-zero pattern
    qm = o.q_keep_mask(np.zeros((1, 1, D), np.uint8), T, S, R, edges)[0, 0]
    assert qm[j_first - 1] == 1 and qm[j_first] == 0
    assert qm[j_last] == 0 and qm[j_last + 1] == 1


def test_streaming_llm_special_case():
    g = _golden("paper_layout.json")
    lay = g["layouts"][0]
    T, S, R, W, D = lay["context_len"], g["sink"], g["recent"], g["bin_width"], lay["num_bins"]
    sl = g["streaming_llm"]
    pat = np.zeros((2, 8, D), dtype=np.uint8)
    _, km, kv_len = o.map_pattern(pat, T, S, R, di.uniform_bin_edges(W, D), 2)
    assert (kv_len == sl["sink"] + sl["recent"]).all()
    assert km[:, :, :sl["sink"]].all() and km[:, :, T - sl["recent"]:].all()
    assert not km[:, :, sl["sink"]:T - sl["recent"]].any()
    cf = o.closed_form_lengths(pat, T, S, R, di.uniform_bin_edges(W, D), 2)
    assert (cf == 1152).all()


def test_all_keep_pattern_keeps_every_position():
    T, S, R = 5000, 128, 1024
    edges = di.log_bin_edges(T - S - R, 12)
    pat = np.ones((1, 4, 12), dtype=np.uint8)
    _, km, kv_len = o.map_pattern(pat, T, S, R, edges, 2)
    assert km.all() and (kv_len == T).all()


def test_head_level_pattern():
    """Sec. 3.2: M[l,h,d] = z_h for all d recovers a head-level policy."""
    T, S, R, W, D = 9000, 128, 1024, 128, (9000 - 1152) // 128 + 1
    rng = np.random.default_rng(0)
    z = (rng.uniform(size=16) < 0.3).astype(np.uint8)
    pat = np.repeat(z[None, :, None], D, axis=2)
    _, _, kv_len = o.map_pattern(pat, T, S, R, di.uniform_bin_edges(W, D), 4)
    for g in range(4):
        want = T if z[4 * g:4 * g + 4].any() else S + R
        assert kv_len[0, g] == want


def test_map_matches_bruteforce_paint():
    rng = np.random.default_rng(1234)
    for _ in range(250):
        T, S, R, edges, n_kv, pat = random_layout(rng)
        qm, km, kv_len = o.map_pattern(pat, T, S, R, edges, n_kv)
        pq, pk = paint_masks(pat, T, S, R, edges, n_kv)
        np.testing.assert_array_equal(qm, pq)
        np.testing.assert_array_equal(km, pk)
        np.testing.assert_array_equal(kv_len, pk.sum(axis=2))
        cf = o.closed_form_lengths(pat, T, S, R, edges, n_kv)
        np.testing.assert_array_equal(cf, kv_len)


def test_sink_recent_overlap_keeps_all():
    for T in range(0, 20):
        pat = np.zeros((1, 2, 3), dtype=np.uint8)
        _, km, kv_len = o.map_pattern(pat, T, 8, 12, [0, 4, 8, 16], 1)
        assert km.all() and kv_len[0, 0] == T


def test_log_bins_with_recent_equal_forced_first_bin():
    """R = 128 with D-1 bins == R = 0 with D bins whose bin 0 is [0,128) kept."""
    T = 3000
    e = di.log_bin_edges(T, 10)                 # E[1] = 128
    rng = np.random.default_rng(5)
    pat = (rng.uniform(size=(1, 6, 10)) < 0.4).astype(np.uint8)
    pat_a = pat.copy()
    pat_a[:, :, 0] = 1
    _, km_a, _ = o.map_pattern(pat_a, T, 0, 0, e, 3)
    e_b = [x - 128 for x in e[1:]]
    _, km_b, _ = o.map_pattern(pat[:, :, 1:], T, 0, 128, e_b, 3)
    np.testing.assert_array_equal(km_a, km_b)


def test_position_beyond_last_bin_is_pruned():
    T, S, R = 400, 4, 8
    edges = [0, 10, 30]                          # covers u < 30 only
    pat = np.ones((1, 1, 2), dtype=np.uint8)
    qm = o.q_keep_mask(pat, T, S, R, edges)[0, 0]
    assert int(qm.sum()) == S + R + 30


# ---------------------------------------------------------------------------
# packing and append
# ---------------------------------------------------------------------------

def _rand_bits(rng, shape):
    return rng.integers(0, 1 << 16, size=shape, dtype=np.uint16)


def test_compact_all_keep_is_dense_bytes():
    rng = np.random.default_rng(2)
    k = _rand_bits(rng, (2, 3, 37, 8))
    v = _rand_bits(rng, (2, 3, 37, 8))
    r = o.compact(k, v, np.ones((2, 3, 37), np.uint8), 0)
    np.testing.assert_array_equal(r["k_c"], k.reshape(-1, 8))
    np.testing.assert_array_equal(r["v_c"], v.reshape(-1, 8))
    assert (r["seg_len"] == 37).all()
    np.testing.assert_array_equal(r["seg_off"], 37 * np.arange(6))


def test_compact_matches_python_loop():
    rng = np.random.default_rng(3)
    for _ in range(40):
        N, H, T, d = rng.integers(1, 3), rng.integers(1, 4), rng.integers(0, 50), 4
        cap = int(rng.integers(0, 4))
        k = rng.standard_normal((N, H, T, d)).astype(np.float32)
        v = rng.standard_normal((N, H, T, d)).astype(np.float32)
        m = (rng.uniform(size=(N, H, T)) < rng.uniform()).astype(np.uint8)
        r = o.compact(k, v, m, cap)
        row = 0
        for n in range(N):
            for g in range(H):
                s = n * H + g
                assert r["seg_off"][s] == row
                cnt = 0
                for j in range(T):
                    if m[n, g, j]:
                        assert (r["k_c"][row + cnt] == k[n, g, j]).all()
                        assert (r["v_c"][row + cnt] == v[n, g, j]).all()
                        assert r["src_pos"][row + cnt] == j
                        cnt += 1
                assert r["seg_len"][s] == cnt
                row += cnt + cap
        assert r["rows"] == row


def test_compact_invariants():
    rng = np.random.default_rng(4)
    k = _rand_bits(rng, (3, 2, 300, 16))
    v = _rand_bits(rng, (3, 2, 300, 16))
    m = (rng.uniform(size=(3, 2, 300)) < 0.3).astype(np.uint8)
    r = o.compact(k, v, m, 5)
    assert int(r["seg_len"].sum()) == int(m.sum())
    for s in range(6):
        n, g = divmod(s, 2)
        lo, ln = int(r["seg_off"][s]), int(r["seg_len"][s])
        sp = r["src_pos"][lo:lo + ln]
        assert (np.diff(sp) > 0).all()
        np.testing.assert_array_equal(r["k_c"][lo:lo + ln], k[n, g, sp])
        assert (r["src_pos"][lo + ln:lo + ln + 5] == -1).all()


def test_append_positions():
    rng = np.random.default_rng(5)
    k = rng.standard_normal((2, 2, 20, 4)).astype(np.float32)
    m = (rng.uniform(size=(2, 2, 20)) < 0.5).astype(np.uint8)
    r = o.compact(k, k, m, 3)
    kn = rng.standard_normal((2, 2, 2, 4)).astype(np.float32)
    kc, _ = o.append(r["k_c"], r["v_c"], r["seg_off"], r["seg_len"], kn, kn, 1)
    want = r["k_c"].copy()
    for s in range(4):
        n, g = divmod(s, 2)
        base = int(r["seg_off"][s]) + int(r["seg_len"][s])
        # slot n_tail = 0 stays free; tokens land in slots 1 and 2
        want[base + 1] = kn[n, g, 0]
        want[base + 2] = kn[n, g, 1]
    np.testing.assert_array_equal(kc, want)


# ---------------------------------------------------------------------------
# attention
# ---------------------------------------------------------------------------

def _attn_case(rng, B=2, n_kv=2, G=3, T=40, d=8):
    q = rng.standard_normal((B, n_kv * G, d)).astype(np.float32)
    k = rng.standard_normal((B, n_kv, T, d)).astype(np.float32)
    v = rng.standard_normal((B, n_kv, T, d)).astype(np.float32)
    return q, k, v


def test_decode_all_keep_matches_sdpa():
    rng = np.random.default_rng(6)
    q, k, v = _attn_case(rng)
    r = o.compact(k, v, np.ones(k.shape[:3], np.uint8), 0)
    out = o.decode_attn(q, r["k_c"], r["v_c"], r["seg_off"], r["seg_len"], 0, 0.37, 2, o.F32)
    ref = sdpa(q.astype(np.float64), k.astype(np.float64), v.astype(np.float64), 0.37)
    np.testing.assert_allclose(out, ref, rtol=1e-12, atol=1e-13)


def test_dense_decode_matches_sdpa():
    rng = np.random.default_rng(7)
    q, k, v = _attn_case(rng, T=50)
    out = o.dense_decode_attn(q, k, v, 31, 0.5, o.F32)
    ref = sdpa(q.astype(np.float64), k[:, :, :31].astype(np.float64),
               v[:, :, :31].astype(np.float64), 0.5)
    np.testing.assert_allclose(out, ref, rtol=1e-12, atol=1e-13)


def test_masked_dense_matches_sdpa_with_bool_mask():
    rng = np.random.default_rng(8)
    B, n_kv, G, T, d = 2, 2, 4, 33, 8
    q, k, v = _attn_case(rng, B, n_kv, G, T, d)
    m = (rng.uniform(size=(B, n_kv, T)) < 0.4).astype(np.uint8)
    m[:, :, 0] = 1
    kt = np.zeros((B, n_kv, 0, d), np.float32)
    out = o.masked_dense_attn(q, k, v, m, kt, kt, 0.3, o.F32)
    mask = torch.from_numpy(np.repeat(m, G, axis=1).astype(bool))[:, :, None, :]
    ref = sdpa(q.astype(np.float64), k.astype(np.float64), v.astype(np.float64), 0.3, mask)
    np.testing.assert_allclose(out, ref, rtol=1e-12, atol=1e-13)


def test_packed_decode_equals_masked_dense_with_tail():
    rng = np.random.default_rng(9)
    for trial in range(10):
        B, n_kv, G, T, d = 2, 3, 2, 64, 16
        q, k, v = _attn_case(rng, B, n_kv, G, T, d)
        m = (rng.uniform(size=(B, n_kv, T)) < 0.35).astype(np.uint8)
        n_tail = int(rng.integers(0, 4))
        kn = rng.standard_normal((B, n_kv, n_tail, d)).astype(np.float32)
        vn = rng.standard_normal((B, n_kv, n_tail, d)).astype(np.float32)
        r = o.compact(k, v, m, 4)
        kc, vc = o.append(r["k_c"], r["v_c"], r["seg_off"], r["seg_len"], kn, vn, 0)
        out = o.decode_attn(q, kc, vc, r["seg_off"], r["seg_len"], n_tail, 0.25, n_kv, o.F32)
        ref = o.masked_dense_attn(q, k, v, m, kn, vn, 0.25, o.F32)
        np.testing.assert_allclose(out, ref, rtol=1e-12, atol=1e-13)


def test_decode_single_row_returns_that_value_row():
    rng = np.random.default_rng(10)
    q, k, v = _attn_case(rng, 1, 1, 2, 10, 8)
    m = np.zeros((1, 1, 10), np.uint8)
    m[0, 0, 6] = 1
    r = o.compact(k, v, m, 0)
    out = o.decode_attn(q, r["k_c"], r["v_c"], r["seg_off"], r["seg_len"], 0, 1.0, 1, o.F32)
    for h in range(2):
        np.testing.assert_array_equal(out[0, h], v[0, 0, 6].astype(np.float64))


def test_decode_zero_query_is_mean_of_retained_values():
    rng = np.random.default_rng(11)
    _, k, v = _attn_case(rng, 1, 2, 2, 30, 8)
    q = np.zeros((1, 4, 8), np.float32)
    m = (rng.uniform(size=(1, 2, 30)) < 0.5).astype(np.uint8)
    r = o.compact(k, v, m, 0)
    out = o.decode_attn(q, r["k_c"], r["v_c"], r["seg_off"], r["seg_len"], 0, 1.0, 2, o.F32)
    for h in range(4):
        g = h // 2
        np.testing.assert_allclose(out[0, h], v[0, g][m[0, g] == 1].astype(np.float64).mean(0),
                                   rtol=1e-13, atol=1e-14)


def test_decode_two_rows_is_logistic_mix():
    q = np.array([[[0.5, -1.0]]], np.float32)
    k = np.array([[[[1.0, 2.0], [3.0, -1.0]]]], np.float32)
    v = np.array([[[[10.0, 0.0], [0.0, 10.0]]]], np.float32)
    r = o.compact(k, v, np.ones((1, 1, 2), np.uint8), 0)
    out = o.decode_attn(q, r["k_c"], r["v_c"], r["seg_off"], r["seg_len"], 0, 0.7, 1, o.F32)
    s1, s2 = 0.7 * (0.5 - 2.0), 0.7 * (1.5 + 1.0)
    w1 = 1.0 / (1.0 + np.exp(s2 - s1))
    np.testing.assert_allclose(out[0, 0], [10 * w1, 10 * (1 - w1)], rtol=1e-14)


def test_decode_empty_segment_is_zero():
    q = np.ones((1, 2, 4), np.float32)
    k = np.ones((1, 1, 5, 4), np.float32)
    r = o.compact(k, k, np.zeros((1, 1, 5), np.uint8), 2)
    out = o.decode_attn(q, r["k_c"], r["v_c"], r["seg_off"], r["seg_len"], 0, 1.0, 1, o.F32)
    assert (out == 0).all()
    out2 = o.masked_dense_attn(q, k, k, np.zeros((1, 1, 5), np.uint8),
                               np.zeros((1, 1, 0, 4), np.float32),
                               np.zeros((1, 1, 0, 4), np.float32), 1.0, o.F32)
    assert (out2 == 0).all()


def test_decode_bf16_matches_sdpa_on_widened_values():
    rng = np.random.default_rng(12)
    x = rng.standard_normal((1, 2, 25, 8)).astype(np.float32)
    kb = di.f32_to_bf16_bits(x)
    vb = di.f32_to_bf16_bits(x[:, :, ::-1])
    qb = di.f32_to_bf16_bits(rng.standard_normal((1, 4, 8)).astype(np.float32))
    r = o.compact(kb, vb, np.ones((1, 2, 25), np.uint8), 0)
    out = o.decode_attn(qb, r["k_c"], r["v_c"], r["seg_off"], r["seg_len"], 0, 0.5, 2, o.BF16)
    ref = sdpa(o.widen(qb, o.BF16), o.widen(kb, o.BF16), o.widen(vb, o.BF16), 0.5)
    np.testing.assert_allclose(out, ref, rtol=1e-12, atol=1e-13)


# ---------------------------------------------------------------------------
# query-block attention
# ---------------------------------------------------------------------------

def _query_case(rng, B, n_kv, G, T, d, n_tail, n_q, keep):
    """Dense context with a keep mask, n_tail appended tokens, then a block of
    n_q query tokens whose K/V are appended after them."""
    k = rng.standard_normal((B, n_kv, T, d)).astype(np.float32)
    v = rng.standard_normal((B, n_kv, T, d)).astype(np.float32)
    m = (rng.uniform(size=(B, n_kv, T)) < keep).astype(np.uint8)
    kt = rng.standard_normal((B, n_kv, n_tail + n_q, d)).astype(np.float32)
    vt = rng.standard_normal((B, n_kv, n_tail + n_q, d)).astype(np.float32)
    q = rng.standard_normal((B, n_q, n_kv * G, d)).astype(np.float32)
    return q, k, v, m, kt, vt


def test_query_attn_matches_sdpa_with_causal_block_mask():
    """Against torch SDPA over the dense cache: pruned context positions
    masked out, earlier appended tokens visible, the block causal."""
    rng = np.random.default_rng(40)
    for trial in range(6):
        B, n_kv, G, T, d = 2, 2, int(rng.integers(1, 4)), 37, 8
        n_tail, n_q = int(rng.integers(0, 3)), int(rng.integers(1, 6))
        q, k, v, m, kt, vt = _query_case(rng, B, n_kv, G, T, d, n_tail, n_q, 0.4)
        r = o.compact(k, v, m, n_tail + n_q)
        kc, vc = o.append(r["k_c"], r["v_c"], r["seg_off"], r["seg_len"], kt, vt, 0)
        out = o.query_attn(q, kc, vc, r["seg_off"], r["seg_len"], n_tail, 0.45, n_kv, o.F32)
        kd = np.concatenate([k, kt], axis=2).astype(np.float64)
        vd = np.concatenate([v, vt], axis=2).astype(np.float64)
        allow = np.zeros((B, n_kv * G, n_q, T + n_tail + n_q), bool)
        for b in range(B):
            for h in range(n_kv * G):
                for i in range(n_q):
                    allow[b, h, i, :T] = m[b, h // G] == 1
                    allow[b, h, i, T:T + n_tail + i + 1] = True
        qt = torch.from_numpy(q.astype(np.float64)).transpose(1, 2)  # [B][Hq][n_q][d]
        ref = torch.nn.functional.scaled_dot_product_attention(
            qt, torch.from_numpy(kd), torch.from_numpy(vd), attn_mask=torch.from_numpy(allow),
            scale=0.45, enable_gqa=True).transpose(1, 2).numpy()
        np.testing.assert_allclose(out, ref, rtol=1e-12, atol=1e-13)


def test_query_attn_zero_query_is_causal_running_mean():
    """q = 0: every visible row has the same weight, so token i's output is
    the mean of the first seg_len + n_tail + i + 1 rows of its segment."""
    rng = np.random.default_rng(41)
    B, n_kv, G, T, d, n_tail, n_q = 1, 2, 2, 20, 4, 2, 4
    _, k, v, m, kt, vt = _query_case(rng, B, n_kv, G, T, d, n_tail, n_q, 0.5)
    q = np.zeros((B, n_q, n_kv * G, d), np.float32)
    r = o.compact(k, v, m, n_tail + n_q)
    kc, vc = o.append(r["k_c"], r["v_c"], r["seg_off"], r["seg_len"], kt, vt, 0)
    out = o.query_attn(q, kc, vc, r["seg_off"], r["seg_len"], n_tail, 1.0, n_kv, o.F32)
    for g in range(n_kv):
        rows = np.concatenate([v[0, g][m[0, g] == 1], vt[0, g]]).astype(np.float64)
        base = int(m[0, g].sum()) + n_tail
        for i in range(n_q):
            for h in range(g * G, g * G + G):
                np.testing.assert_allclose(out[0, i, h], rows[:base + i + 1].mean(0), rtol=1e-13,
                                           atol=1e-14)


def test_query_attn_single_token_is_decode_step():
    """A one-token block is one decode step with the token appended."""
    rng = np.random.default_rng(42)
    B, n_kv, G, T, d, n_tail = 2, 3, 2, 30, 8, 1
    q, k, v, m, kt, vt = _query_case(rng, B, n_kv, G, T, d, n_tail, 1, 0.3)
    r = o.compact(k, v, m, n_tail + 1)
    kc, vc = o.append(r["k_c"], r["v_c"], r["seg_off"], r["seg_len"], kt, vt, 0)
    out = o.query_attn(q, kc, vc, r["seg_off"], r["seg_len"], n_tail, 0.7, n_kv, o.F32)
    dec = o.decode_attn(q[:, 0], kc, vc, r["seg_off"], r["seg_len"], n_tail + 1, 0.7, n_kv, o.F32)
    np.testing.assert_allclose(out[:, 0], dec, rtol=1e-13, atol=1e-14)


# ---------------------------------------------------------------------------
# zero-copy paged variant
# ---------------------------------------------------------------------------

def test_page_select_hand_example():
    g = _golden("page_select_small.json")
    r = o.page_select(np.array([g["kv_mask"]], np.uint8), np.array([g["page_table"]], np.int32),
                      g["page_rows"], g["append_cap"])
    np.testing.assert_array_equal(r["entries"][0], np.array(g["entries"], np.int32))
    assert r["n_entries"][0] == len(g["entries"])
    assert r["seg_len"][0] == g["seg_len"]
    np.testing.assert_array_equal(r["page_used"][0], g["page_used"])


def _walk_positions(mask_row, table_row, pr, T, cap):
    """Brute force, position by position: (page, slot) of every retained
    context position, then of every append position, in position order."""
    out = []
    for pos in range(T + cap):
        if pos >= T or mask_row[pos]:
            out.append((int(table_row[pos // pr]), pos % pr))
    return out


def test_page_select_covers_exactly_the_retained_positions():
    rng = np.random.default_rng(50)
    for trial in range(40):
        nseg = int(rng.integers(1, 4))
        T = int(rng.integers(0, 60))
        pr = int(rng.choice([1, 2, 3, 4, 8]))
        cap = int(rng.integers(0, 10))
        pages = -(-(T + cap) // pr) + int(rng.integers(0, 3))
        m = (rng.uniform(size=(nseg, T)) < rng.uniform()).astype(np.uint8) * rng.integers(1, 255, (nseg, T),
                                                                                              dtype=np.uint8)
        table, _ = di.page_table(nseg, pages, seed=trial, spare=3)
        r = o.page_select(m, table, pr, cap)
        for s in range(nseg):
            e = r["entries"][s]
            want = _walk_positions(m[s], table[s], pr, T, cap)
            got = [(int(p), slot) for p, lp, lo, hi in e for slot in range(lo, hi)]
            assert got == want, (trial, s)
            assert r["seg_len"][s] == int((m[s] != 0).sum())
            assert r["n_entries"][s] == len(e)
            for p, lp, lo, hi in e:
                assert 0 <= lo < hi <= pr and table[s, lp] == p
            # maximal: two entries of one logical page never touch
            for a, b in zip(e[:-1], e[1:]):
                assert a[1] < b[1] or a[3] < b[2] or (a[1] * pr + a[3] == T)
            used = np.zeros(pages, np.uint8)
            for p, slot in want:
                used[list(table[s]).index(p)] = 1
            np.testing.assert_array_equal(r["page_used"][s], used)


def test_page_select_paper_layout_is_whole_pages():
    """The paper's layout (Appendix A: 128 sink, 1,024 recent, 128-token
    bins) at T = 130,816 with 128-row pages: every bin, the sink and the
    recent window are whole pages, so every context entry is a full page and
    the entries hold exactly the retained positions."""
    g = _golden("paper_layout.json")
    T = g["layouts"][0]["context_len"]
    D = g["layouts"][0]["num_bins"]
    S, R, W = g["sink"], g["recent"], g["bin_width"]
    rng = np.random.default_rng(51)
    pattern = (rng.uniform(size=(1, 2, D)) < 0.3).astype(np.uint8)
    _, km = paint_masks(pattern, T, S, R, [W * k for k in range(D + 1)], 1)
    table, _ = di.page_table(1, T // W + 1, seed=1)
    r = o.page_select(km[0], table, W, 64)
    e = r["entries"][0]
    ctx = e[e[:, 1] * W < T]
    assert (ctx[:, 2] == 0).all() and (ctx[:, 3] == W).all()
    assert len(ctx) * W == int(km.sum())


def test_paged_decode_equals_masked_sdpa():
    """Attention through the entries of a shuffled page pool equals torch
    SDPA over the dense cache with pruned positions masked out and the
    appended tokens visible."""
    rng = np.random.default_rng(52)
    for trial in range(8):
        B, n_kv, G, d = 2, 2, int(rng.integers(1, 4)), 8
        T = int(rng.integers(1, 50))
        pr = int(rng.choice([2, 4, 8]))
        cap = int(rng.integers(1, 6))
        n_tail = int(rng.integers(0, cap + 1))
        nseg = B * n_kv
        q = rng.standard_normal((B, n_kv * G, d)).astype(np.float32)
        k = rng.standard_normal((B, n_kv, T + cap, d)).astype(np.float32)
        v = rng.standard_normal((B, n_kv, T + cap, d)).astype(np.float32)
        m = (rng.uniform(size=(B, n_kv, T)) < 0.5).astype(np.uint8)
        table, n_pages = di.page_table(nseg, -(-(T + cap) // pr), seed=100 + trial, spare=2)
        kp = np.zeros((n_pages, pr, d), np.float32)
        vp = np.zeros((n_pages, pr, d), np.float32)
        di.fill_pages(kp, k.reshape(nseg, T + cap, d), table, pr)
        di.fill_pages(vp, v.reshape(nseg, T + cap, d), table, pr)
        sel = o.page_select(m.reshape(nseg, T), table, pr, cap)
        out = o.paged_decode_attn(q, kp, vp, sel["entries"], pr, T, n_tail, 0.6, n_kv, o.F32)
        allow = np.zeros((B, n_kv * G, 1, T + cap), bool)
        for b in range(B):
            for h in range(n_kv * G):
                allow[b, h, 0, :T] = m[b, h // G] == 1
                allow[b, h, 0, T:T + n_tail] = True
        ref = sdpa(q.astype(np.float64), k.astype(np.float64), v.astype(np.float64), 0.6,
                   torch.from_numpy(allow))
        # SDPA yields NaN for a row with nothing visible; the oracle's rule is zeros
        ref = np.nan_to_num(ref, nan=0.0)
        np.testing.assert_allclose(out, ref, rtol=1e-12, atol=1e-13)


def test_paged_append_writes_each_token_at_its_position():
    rng = np.random.default_rng(53)
    nseg, T, pr, cap, d, n_tail, n_new = 3, 13, 4, 7, 2, 2, 3
    table, n_pages = di.page_table(nseg, -(-(T + cap) // pr), seed=7)
    kp = rng.standard_normal((n_pages, pr, d)).astype(np.float32)
    vp = rng.standard_normal((n_pages, pr, d)).astype(np.float32)
    kn = rng.standard_normal((nseg, n_new, d)).astype(np.float32)
    vn = rng.standard_normal((nseg, n_new, d)).astype(np.float32)
    k2, v2 = o.paged_append(kp, vp, table, pr, T, kn, vn, n_tail)
    touched = np.zeros((n_pages, pr), bool)
    for s in range(nseg):
        for t in range(n_new):
            pos = T + n_tail + t          # 15, 16, 17: pages 3 and 4 of the segment
            page, slot = table[s, pos // pr], pos % pr
            assert np.array_equal(k2[page, slot], kn[s, t]) and np.array_equal(v2[page, slot], vn[s, t])
            touched[page, slot] = True
    assert np.array_equal(k2[~touched], kp[~touched]) and np.array_equal(v2[~touched], vp[~touched])


# ---------------------------------------------------------------------------
# exact-budget export and retention report
# ---------------------------------------------------------------------------

def test_budget_of_the_llama31_pattern():
    g = _golden("exact_budget.json")
    # L * H query heads in all; the budget depends only on their product
    assert o.budget_entries(g["rho"], 1, g["query_heads"], g["num_bins"]) == g["k_rho"]
    assert o.budget_entries(g["rho"], 32, 32, g["num_bins"]) == g["k_rho"]


def test_budget_rounds_halves_up_and_hits_the_ends():
    assert o.budget_entries(0.5, 1, 1, 3) == 2      # 1.5
    assert o.budget_entries(0.5, 1, 1, 5) == 3      # 2.5
    assert o.budget_entries(0.25, 1, 2, 5) == 3     # 2.5
    assert o.budget_entries(0.0, 4, 4, 7) == 0
    assert o.budget_entries(1.0, 4, 4, 7) == 112


def _topk_brute(p, k):
    """Sort the flat indices by (NaN last, larger first, lower index first)."""
    flat = [float(x) for x in np.asarray(p, np.float64).reshape(-1)]
    keyed = sorted(range(len(flat)), key=lambda i: (flat[i] != flat[i], -(flat[i] if flat[i] == flat[i] else 0.0), i))
    out = [0] * len(flat)
    for i in keyed[:k]:
        out[i] = 1
    return np.array(out, np.uint8).reshape(np.shape(p))


def test_topk_mask_matches_a_brute_force_sort():
    rng = np.random.default_rng(60)
    for trial in range(60):
        shape = tuple(int(x) for x in rng.integers(1, 6, size=3))
        n = int(np.prod(shape))
        # coarse values give many exact ties; some NaN, some signed zeros
        p = (rng.integers(0, 5, size=shape) / 4.0).astype(np.float32)
        if trial % 3 == 0:
            p[rng.uniform(size=shape) < 0.2] = np.nan
        if trial % 4 == 0:
            p[rng.uniform(size=shape) < 0.3] = -0.0
        k = int(rng.integers(0, n + 1))
        got = o.topk_mask(p, k)
        assert got.dtype == np.uint8 and got.shape == shape
        assert int(got.sum()) == k
        np.testing.assert_array_equal(got, _topk_brute(p, k))


def test_topk_mask_special_cases():
    p = np.full((2, 3, 4), 0.3, np.float32)
    m = o.topk_mask(p, 5)                      # all tied: the first five flat entries
    assert m.reshape(-1).tolist() == [1] * 5 + [0] * 19
    assert o.topk_mask(p, 0).sum() == 0 and o.topk_mask(p, 24).sum() == 24
    q = np.arange(24, dtype=np.float32).reshape(2, 3, 4)
    assert o.topk_mask(q, 3).reshape(-1).tolist() == [0] * 21 + [1] * 3


def test_retention_report_against_painted_masks():
    rng = np.random.default_rng(61)
    for _ in range(30):
        T, S, R, edges, n_kv, pattern = random_layout(rng)
        rep = o.retention_report(pattern, T, S, R, edges, n_kv)
        _, km = paint_masks(pattern, T, S, R, edges, n_kv)
        assert rep["kept_entries"] == int(pattern.sum())
        assert rep["logical"] == pytest.approx(pattern.mean())
        assert rep["retained_positions"] == int(km.sum())
        if T:
            assert rep["physical"] == pytest.approx(km.mean())


def test_ragged_contexts_map_like_separate_contexts():
    """Per-unit context lengths: each unit's mask is the brute-force painting
    of its own context, padded with zeros to the row length."""
    rng = np.random.default_rng(62)
    for _ in range(40):
        T, S, R, edges, n_kv, pattern = random_layout(rng)
        lens = rng.integers(0, T + 1, size=pattern.shape[0])
        qm, km, kl = o.map_pattern(pattern, T, S, R, edges, n_kv, unit_len=lens)
        for n, Tn in enumerate(lens):
            pq, pk = paint_masks(pattern[n:n + 1], int(Tn), S, R, edges, n_kv)
            np.testing.assert_array_equal(qm[n, :, :Tn], pq[0])
            np.testing.assert_array_equal(km[n, :, :Tn], pk[0])
            assert not qm[n, :, Tn:].any() and not km[n, :, Tn:].any()
            np.testing.assert_array_equal(kl[n], pk[0].sum(axis=1))
