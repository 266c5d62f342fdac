"""GPU parity: the HIP path through the C ABI against the CPU oracle.

Masks, lengths, offsets, packed rows and source positions must match
bit-for-bit; attention rows must match within ATTN_TOL (max relative error of
each (batch, head) output row, bf16 in / fp32 accumulate / fp32 out).  Inputs
are seeded; the oracle computes everything it compares from the same inputs
on its own.
"""

import numpy as np
import pytest
import torch

import dkv_inputs as di
import oracle as o
from _helpers import ATTN_TOL, GpuPack, bits, odt, row_rel_err

pytestmark = pytest.mark.gpu

DEV = "cuda"


@pytest.fixture(scope="module")
def d():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2609_32663_amd as lib
    return lib


def _layout(d, N, Hq, Hkv, dim, T, S, R, edges):
    return d.make_layout(N, Hq, Hkv, dim, T, S, R, edges)


def _rand_edges(rng, uniform):
    D = int(rng.integers(1, 40))
    if uniform:
        W = int(rng.integers(1, 200))
        return [W * k for k in range(D + 1)]
    steps = rng.integers(1, 300, size=D)
    return [0] + [int(x) for x in np.cumsum(steps)]


def _check_map(d, N, Hq, Hkv, T, S, R, edges, pattern):
    lay = _layout(d, N, Hq, Hkv, 128, T, S, R, edges)
    pat = torch.from_numpy(pattern).to(DEV)
    # flat buffers with slack so that a zero-length context still has a pointer
    km = torch.full((N * Hkv * T + 16,), 9, dtype=torch.uint8, device=DEV)[:N * Hkv * T].view(N, Hkv, T)
    kl = torch.full((N, Hkv), -1, dtype=torch.int32, device=DEV)
    qm = torch.full((N * Hq * T + 16,), 9, dtype=torch.uint8, device=DEV)[:N * Hq * T].view(N, Hq, T)
    d.dkv_map_pattern(lay, pat, km, kl, qm)
    torch.cuda.synchronize()
    oq, okm, okl = o.map_pattern(pattern, T, S, R, edges, Hkv)
    np.testing.assert_array_equal(km.cpu().numpy(), okm)
    np.testing.assert_array_equal(kl.cpu().numpy(), okl)
    np.testing.assert_array_equal(qm.cpu().numpy(), oq)


# ---------------------------------------------------------------------------
# dkv_map_pattern
# ---------------------------------------------------------------------------

def test_map_random_layouts(d):
    rng = np.random.default_rng(100)
    for trial in range(60):
        N = int(rng.integers(1, 4))
        Hkv = int(rng.integers(1, 4))
        G = int(rng.choice([1, 2, 3, 4, 7, 8, 16]))
        T = int(rng.choice([0, 1, 15, 16, 17, 100, 1000, 4096, 4097, 5000]))
        S = int(rng.integers(0, 300))
        R = int(rng.integers(0, 300))
        edges = _rand_edges(rng, uniform=bool(trial % 2))
        pattern = (rng.uniform(size=(N, Hkv * G, len(edges) - 1)) < rng.uniform()).astype(np.uint8)
        _check_map(d, N, Hkv * G, Hkv, T, S, R, edges, pattern)


def test_map_paper_layout(d):
    """Sink 128, recent 1024, 1013 uniform 128-token bins at T = 130,816."""
    rng = np.random.default_rng(101)
    pattern = (rng.uniform(size=(2, 8, 1013)) < 0.2).astype(np.uint8)
    _check_map(d, 2, 8, 2, 130816, 128, 1024, di.uniform_bin_edges(128, 1013), pattern)


def test_map_nonzero_pattern_values_count_as_keep(d):
    rng = np.random.default_rng(102)
    pattern = rng.integers(0, 4, size=(1, 4, 10)).astype(np.uint8)
    lay = _layout(d, 1, 4, 2, 128, 800, 3, 5, [0, 7, 20, 50, 90, 150, 230, 330, 460, 600, 792])
    km = torch.empty((1, 2, 800), dtype=torch.uint8, device=DEV)
    kl = torch.empty((1, 2), dtype=torch.int32, device=DEV)
    d.dkv_map_pattern(lay, torch.from_numpy(pattern).to(DEV), km, kl, None)
    _, okm, okl = o.map_pattern((pattern != 0).astype(np.uint8), 800, 3, 5, lay._edges[:], 2)
    np.testing.assert_array_equal(km.cpu().numpy(), okm)
    np.testing.assert_array_equal(kl.cpu().numpy(), okl)


@pytest.mark.parametrize("name,units", [
    ("tiny", None), ("llama8b_layer_32k", None), ("llama70b_layer_bs16_32k", None),
    ("llama8b_stack_128k", 4), ("qwen7b_stack_bs4_128k", 8)])
def test_map_workloads(d, name, units):
    w = di.workload(name)
    for b in (w.budgets or (None,)):
        pattern, _ = di.make_pattern(w, budget=b)
        if units is not None:
            pattern = pattern[:units]
        _check_map(d, pattern.shape[0], w.num_q_heads, w.num_kv_heads, w.context_len, w.sink,
                   w.recent, list(w.bin_edges), np.ascontiguousarray(pattern))


# ---------------------------------------------------------------------------
# dkv_compact / dkv_append
# ---------------------------------------------------------------------------

def _rand_kv(rng, shape, dtype):
    x = torch.from_numpy(rng.standard_normal(shape).astype(np.float32))
    return x.to(dtype).to(DEV)


def _check_pack(pack, ref, rows_written=None):
    seg_off = pack.seg_off.cpu().numpy()
    seg_len = pack.seg_len.cpu().numpy()
    np.testing.assert_array_equal(seg_off, ref["seg_off"])
    np.testing.assert_array_equal(seg_len, ref["seg_len"])
    assert int(pack.rows_needed.item()) == ref["rows"]
    kc, vc, sp = bits(pack.k_c), bits(pack.v_c), pack.src_pos.cpu().numpy()
    for s in range(len(seg_off)):
        lo, ln = int(seg_off[s]), int(seg_len[s])
        np.testing.assert_array_equal(kc[lo:lo + ln], ref["k_c"][lo:lo + ln])
        np.testing.assert_array_equal(vc[lo:lo + ln], ref["v_c"][lo:lo + ln])
        np.testing.assert_array_equal(sp[lo:lo + ln], ref["src_pos"][lo:lo + ln])
        assert (sp[lo + ln:lo + ln + pack.cap] == -7).all()  # free rows untouched


def test_compact_random(d):
    rng = np.random.default_rng(200)
    for trial in range(24):
        dtype = torch.bfloat16 if trial % 3 else torch.float32
        dim = 128 if trial % 2 else 64
        N, Hkv, G = int(rng.integers(1, 3)), int(rng.integers(1, 4)), int(rng.choice([1, 2, 4, 8]))
        T = int(rng.choice([1, 33, 1000, 4096, 4100, 9000]))
        S, R = int(rng.integers(0, 64)), int(rng.integers(0, 64))
        edges = _rand_edges(rng, uniform=bool(trial % 2))
        cap = int(rng.integers(0, 5))
        pattern = (rng.uniform(size=(N, Hkv * G, len(edges) - 1)) < rng.uniform()).astype(np.uint8)
        k = _rand_kv(rng, (N, Hkv, T, dim), dtype)
        v = _rand_kv(rng, (N, Hkv, T, dim), dtype)
        lay = _layout(d, N, Hkv * G, Hkv, dim, T, S, R, edges)
        pack = GpuPack(d, lay, pattern, k, v, cap)
        torch.cuda.synchronize()
        _, okm, _ = o.map_pattern(pattern, T, S, R, edges, Hkv)
        ref = o.compact(bits(k), bits(v), okm, cap)
        _check_pack(pack, ref)


def test_compact_zero_and_full_segments(d):
    rng = np.random.default_rng(201)
    N, Hkv, T, dim = 1, 4, 5000, 128
    pattern = np.zeros((N, 4, 5), np.uint8)
    pattern[0, 1] = 1          # head 1 keeps every bin
    pattern[0, 3, 2] = 1
    edges = [0, 100, 700, 1500, 3000, 5000]
    k = _rand_kv(rng, (N, Hkv, T, dim), torch.bfloat16)
    v = _rand_kv(rng, (N, Hkv, T, dim), torch.bfloat16)
    lay = _layout(d, N, 4, Hkv, dim, T, 0, 0, edges)
    pack = GpuPack(d, lay, pattern, k, v, 3)
    torch.cuda.synchronize()
    _, okm, okl = o.map_pattern(pattern, T, 0, 0, edges, Hkv)
    assert okl[0, 0] == 0 and okl[0, 1] == T
    _check_pack(pack, o.compact(bits(k), bits(v), okm, 3))


def test_compact_all_keep_is_dense(d):
    rng = np.random.default_rng(202)
    k = _rand_kv(rng, (2, 2, 3000, 128), torch.bfloat16)
    v = _rand_kv(rng, (2, 2, 3000, 128), torch.bfloat16)
    lay = _layout(d, 2, 4, 2, 128, 3000, 0, 0, [0, 3000])
    pack = GpuPack(d, lay, np.ones((2, 4, 1), np.uint8), k, v, 0)
    torch.cuda.synchronize()
    assert torch.equal(pack.k_c, k.reshape(-1, 128)) and torch.equal(pack.v_c, v.reshape(-1, 128))


@pytest.mark.parametrize("dtype,dim,T", [(torch.bfloat16, 128, 4099), (torch.float32, 128, 4096),
                                         (torch.bfloat16, 64, 8197)])
def test_compact_chunk_boundaries(d, dtype, dim, T):
    """Masks with scattered kept positions and kept counts at the copy's
    32-row chunk edges (0, 1, 31, 32, 33, 63, 64, 65, 4095, T - 33, T - 1, T),
    straight through dkv_compact: rows, offsets, lengths, source positions
    and rows_needed equal the oracle's bit for bit."""
    rng = np.random.default_rng(207)
    counts = [0, 1, 31, 32, 33, 63, 64, 65, 4095, T - 33, T - 1, T]
    N, Hkv, cap = 2, len(counts) // 2, 3
    mask = np.zeros((N, Hkv, T), np.uint8)
    for s, c in enumerate(counts):
        pos = rng.choice(T, size=c, replace=False)
        mask[s // Hkv, s % Hkv, pos] = rng.integers(1, 256, size=c)  # any nonzero byte keeps
    k = _rand_kv(rng, (N, Hkv, T, dim), dtype)
    v = _rand_kv(rng, (N, Hkv, T, dim), dtype)
    ref = o.compact(bits(k), bits(v), mask, cap)
    rows = ref["rows"]
    k_c = torch.zeros((rows, dim), dtype=dtype, device=DEV)
    v_c = torch.zeros_like(k_c)
    seg_off = torch.empty(N * Hkv, dtype=torch.int64, device=DEV)
    seg_len = torch.empty(N * Hkv, dtype=torch.int32, device=DEV)
    src = torch.full((rows,), -7, dtype=torch.int32, device=DEV)
    rn = torch.empty(1, dtype=torch.int64, device=DEV)
    lay = _layout(d, N, Hkv, Hkv, dim, T, 0, 0, [0, T])
    ws = torch.empty(d.dkv_compact_workspace_bytes(lay), dtype=torch.uint8, device=DEV)
    d.dkv_compact(lay, k, v, torch.from_numpy(mask).to(DEV), cap, k_c, v_c, seg_off, seg_len, ws,
                  src_pos=src, rows_needed=rn)
    torch.cuda.synchronize()
    assert int(rn.item()) == rows
    np.testing.assert_array_equal(seg_len.cpu().numpy(), ref["seg_len"])
    np.testing.assert_array_equal(seg_off.cpu().numpy(), ref["seg_off"])
    kc, vc, sp = bits(k_c), bits(v_c), src.cpu().numpy()
    for s in range(N * Hkv):
        lo, ln = int(ref["seg_off"][s]), int(ref["seg_len"][s])
        np.testing.assert_array_equal(kc[lo:lo + ln], ref["k_c"][lo:lo + ln])
        np.testing.assert_array_equal(vc[lo:lo + ln], ref["v_c"][lo:lo + ln])
        np.testing.assert_array_equal(sp[lo:lo + ln], ref["src_pos"][lo:lo + ln])
        assert (sp[lo + ln:lo + ln + cap] == -7).all()  # free rows untouched
        assert not kc[lo + ln:lo + ln + cap].any()


def test_compact_long_context(d):
    """Two segments of a 2^20 + 1-token context (the list and the copy index
    past 2^20 rows of a segment; the copy grid holds 65,538 chunks per
    segment): rows, lengths, offsets and source positions bit-exact."""
    rng = np.random.default_rng(208)
    N, Hkv, T, dim, cap = 1, 2, (1 << 20) + 1, 128, 5
    # runs of kept positions (lengths 1-2,000) with scattered single positions between
    mask = np.zeros((N, Hkv, T), np.uint8)
    for g in range(Hkv):
        j = 0
        while j < T:
            j += int(rng.integers(0, 4000))
            n = int(rng.integers(1, 2000))
            mask[0, g, j:j + n] = 1
            j += n
        mask[0, g, rng.integers(0, T, size=5000)] = 1
    mask[0, 1, T - 1] = 1  # the last position
    gen = torch.Generator(device=DEV).manual_seed(208)
    k = torch.randn((N, Hkv, T, dim), generator=gen, device=DEV).to(torch.bfloat16)
    v = torch.randn((N, Hkv, T, dim), generator=gen, device=DEV).to(torch.bfloat16)
    ref = o.compact(bits(k), bits(v), mask, cap)
    rows = ref["rows"]
    k_c = torch.zeros((rows, dim), dtype=torch.bfloat16, device=DEV)
    v_c = torch.zeros_like(k_c)
    seg_off = torch.empty(N * Hkv, dtype=torch.int64, device=DEV)
    seg_len = torch.empty(N * Hkv, dtype=torch.int32, device=DEV)
    src = torch.full((rows,), -7, dtype=torch.int32, device=DEV)
    rn = torch.empty(1, dtype=torch.int64, device=DEV)
    lay = _layout(d, N, Hkv, Hkv, dim, T, 0, 0, [0, T])
    ws = torch.empty(d.dkv_compact_workspace_bytes(lay), dtype=torch.uint8, device=DEV)
    d.dkv_compact(lay, k, v, torch.from_numpy(mask).to(DEV), cap, k_c, v_c, seg_off, seg_len, ws,
                  src_pos=src, rows_needed=rn)
    torch.cuda.synchronize()
    assert int(rn.item()) == rows
    np.testing.assert_array_equal(seg_len.cpu().numpy(), ref["seg_len"])
    np.testing.assert_array_equal(seg_off.cpu().numpy(), ref["seg_off"])
    assert ref["seg_len"].max() > (1 << 18)
    np.testing.assert_array_equal(bits(k_c), ref["k_c"])
    np.testing.assert_array_equal(bits(v_c), ref["v_c"])
    sp = src.cpu().numpy()
    for s_ in range(N * Hkv):
        lo, ln = int(ref["seg_off"][s_]), int(ref["seg_len"][s_])
        np.testing.assert_array_equal(sp[lo:lo + ln], ref["src_pos"][lo:lo + ln])
        assert (sp[lo + ln:lo + ln + cap] == -7).all()


def test_compact_respects_out_rows(d):
    """Rows at or beyond out_rows are never written; rows_needed reports the need."""
    rng = np.random.default_rng(203)
    N, Hkv, T, dim, cap = 1, 2, 2000, 64, 2
    mask = torch.from_numpy((rng.uniform(size=(N, Hkv, T)) < 0.5).astype(np.uint8)).to(DEV)
    k = _rand_kv(rng, (N, Hkv, T, dim), torch.bfloat16)
    need = int(mask.sum().item()) + Hkv * cap
    out_rows = need - 300
    big_k = torch.full((need + 64, dim), 3.0, dtype=torch.bfloat16, device=DEV)
    big_v = torch.full((need + 64, dim), 3.0, dtype=torch.bfloat16, device=DEV)
    lay = _layout(d, N, 2, Hkv, dim, T, 0, 0, [0, T])
    seg_off = torch.empty(Hkv, dtype=torch.int64, device=DEV)
    seg_len = torch.empty(Hkv, dtype=torch.int32, device=DEV)
    rn = torch.empty(1, dtype=torch.int64, device=DEV)
    ws = torch.empty(d.dkv_compact_workspace_bytes(lay), dtype=torch.uint8, device=DEV)
    d.dkv_compact(lay, k, k, mask, cap, big_k[:out_rows], big_v[:out_rows], seg_off, seg_len, ws,
                  rows_needed=rn)
    torch.cuda.synchronize()
    assert int(rn.item()) == need
    assert (big_k[out_rows:].float() == 3.0).all() and (big_v[out_rows:].float() == 3.0).all()
    ref = o.compact(bits(k), bits(k), mask.cpu().numpy(), cap)
    np.testing.assert_array_equal(bits(big_k[:out_rows])[:ref["seg_len"][0]],
                                  ref["k_c"][:ref["seg_len"][0]])


@pytest.mark.parametrize("short", [0, 1])
def test_compact_out_rows_exact_edge(d, short):
    """out_rows equal to the need packs every segment; one row fewer leaves
    exactly the last segment unpacked (length -1, offset clamped to
    out_rows), and nothing is written at or past out_rows."""
    rng = np.random.default_rng(209)
    N, Hkv, T, dim, cap = 2, 3, 3000, 128, 7
    mask = (rng.uniform(size=(N, Hkv, T)) < 0.4).astype(np.uint8)
    k = _rand_kv(rng, (N, Hkv, T, dim), torch.bfloat16)
    v = _rand_kv(rng, (N, Hkv, T, dim), torch.bfloat16)
    ref = o.compact(bits(k), bits(v), mask, cap)
    need = ref["rows"]
    out_rows = need - short
    big_k = torch.full((need + 64, dim), 3.0, dtype=torch.bfloat16, device=DEV)
    big_v = torch.full((need + 64, dim), 3.0, dtype=torch.bfloat16, device=DEV)
    src = torch.full((need + 64,), -7, dtype=torch.int32, device=DEV)
    seg_off = torch.empty(N * Hkv, dtype=torch.int64, device=DEV)
    seg_len = torch.empty(N * Hkv, dtype=torch.int32, device=DEV)
    rn = torch.empty(1, dtype=torch.int64, device=DEV)
    lay = _layout(d, N, Hkv, Hkv, dim, T, 0, 0, [0, T])
    ws = torch.empty(d.dkv_compact_workspace_bytes(lay), dtype=torch.uint8, device=DEV)
    d.dkv_compact(lay, k, v, torch.from_numpy(mask).to(DEV), cap, big_k[:out_rows], big_v[:out_rows], seg_off,
                  seg_len, ws, src_pos=src[:out_rows], rows_needed=rn)
    torch.cuda.synchronize()
    assert int(rn.item()) == need
    want_len = ref["seg_len"].copy()
    want_off = ref["seg_off"].copy()
    if short:
        want_len[-1] = -1
        want_off[-1] = min(int(want_off[-1]), out_rows)
    np.testing.assert_array_equal(seg_len.cpu().numpy(), want_len)
    np.testing.assert_array_equal(seg_off.cpu().numpy(), want_off)
    kc, vc, sp = bits(big_k), bits(big_v), src.cpu().numpy()
    for s_ in range(N * Hkv):
        if want_len[s_] < 0:
            continue
        lo, ln = int(want_off[s_]), int(want_len[s_])
        np.testing.assert_array_equal(kc[lo:lo + ln], ref["k_c"][lo:lo + ln])
        np.testing.assert_array_equal(vc[lo:lo + ln], ref["v_c"][lo:lo + ln])
        np.testing.assert_array_equal(sp[lo:lo + ln], ref["src_pos"][lo:lo + ln])
    # nothing at or past out_rows, and nothing of the unpacked last segment
    last_lo = int(ref["seg_off"][-1]) if short else out_rows
    assert (big_k[last_lo:].float() == 3.0).all() and (big_v[last_lo:].float() == 3.0).all()
    assert (src[last_lo:] == -7).all()


def test_truncated_compaction_is_safe_downstream(d):
    """A pack that does not fit out_rows: segments that fit are packed whole,
    the others get seg_len -1 and an offset clamped to out_rows; append,
    decode (plain and fused) and query attention then write nothing at or
    past out_rows, skip those segments and give zeros for them."""
    rng = np.random.default_rng(206)
    B, Hkv, G, T, dim, cap, n_q = 1, 3, 2, 2000, 128, 8, 4
    Hq = Hkv * G
    mask = (rng.uniform(size=(B, Hkv, T)) < 0.5).astype(np.uint8)
    lens = mask.reshape(-1, T).sum(-1).astype(np.int64)
    k = _rand_kv(rng, (B, Hkv, T, dim), torch.bfloat16)
    v = _rand_kv(rng, (B, Hkv, T, dim), torch.bfloat16)
    need = int(lens.sum()) + Hkv * cap
    out_rows = int(lens[0]) + cap + int(lens[1]) // 2  # segment 0 fits, 1 and 2 do not
    big_k = torch.full((need + 64, dim), 3.0, dtype=torch.bfloat16, device=DEV)
    big_v = torch.full((need + 64, dim), 3.0, dtype=torch.bfloat16, device=DEV)
    k_c, v_c = big_k[:out_rows], big_v[:out_rows]
    lay = _layout(d, B, Hq, Hkv, dim, T, 0, 0, [0, T])
    seg_off = torch.empty(Hkv, dtype=torch.int64, device=DEV)
    seg_len = torch.empty(Hkv, dtype=torch.int32, device=DEV)
    rn = torch.empty(1, dtype=torch.int64, device=DEV)
    src = torch.full((need + 64,), -7, dtype=torch.int32, device=DEV)
    ws = torch.empty(d.dkv_compact_workspace_bytes(lay), dtype=torch.uint8, device=DEV)
    d.dkv_compact(lay, k, v, torch.from_numpy(mask).to(DEV), cap, k_c, v_c, seg_off, seg_len, ws,
                  src_pos=src[:out_rows], rows_needed=rn)
    torch.cuda.synchronize()
    assert int(rn.item()) == need
    assert seg_len.cpu().tolist() == [int(lens[0]), -1, -1]
    assert seg_off.cpu().tolist() == [0, int(lens[0]) + cap, out_rows]

    def guard_intact():
        torch.cuda.synchronize()
        return bool((big_k[out_rows:].float() == 3.0).all() and (big_v[out_rows:].float() == 3.0).all()
                    and (src[out_rows:] == -7).all()) and bool((src[lens[0]:out_rows] == -7).all())
    assert guard_intact()
    ref = o.compact(bits(k), bits(v), mask, cap)
    n0 = int(lens[0])
    np.testing.assert_array_equal(bits(k_c)[:n0], ref["k_c"][:n0])
    np.testing.assert_array_equal(bits(v_c)[:n0], ref["v_c"][:n0])
    # rows of the unpacked segments below out_rows are not written either
    assert (big_k[n0 + cap:out_rows].float() == 3.0).all()

    # append two tokens, then a fused append + decode of a third
    kn = _rand_kv(rng, (Hkv, 3, dim), torch.bfloat16)
    vn = _rand_kv(rng, (Hkv, 3, dim), torch.bfloat16)
    d.dkv_append(kn[:, :2].contiguous(), vn[:, :2].contiguous(), 0, cap, k_c, v_c, seg_off, seg_len)
    assert guard_intact() and (big_k[n0 + cap:out_rows].float() == 3.0).all()
    q = _rand_kv(rng, (B, Hq, dim), torch.bfloat16)
    out = torch.full((B, Hq, dim), float("nan"), dtype=torch.float32, device=DEV)
    dws = torch.empty(d.dkv_decode_workspace_bytes(B, Hq, Hkv, dim), dtype=torch.uint8, device=DEV)
    d.dkv_append_decode_attn(q, kn[:, 2:].contiguous(), vn[:, 2:].contiguous(), 2, cap, k_c, v_c, seg_off,
                             seg_len, 0.09, out, dws, Hkv, rows_hint=need)
    assert guard_intact() and (big_k[n0 + cap:out_rows].float() == 3.0).all()
    kc_ref, vc_ref = o.append(ref["k_c"], ref["v_c"], ref["seg_off"], ref["seg_len"],
                              bits(kn).reshape(B, Hkv, 3, dim), bits(vn).reshape(B, Hkv, 3, dim), 0)
    want = o.decode_attn(bits(q), kc_ref, vc_ref, ref["seg_off"], ref["seg_len"], 3, 0.09, Hkv, o.BF16)
    got = out.cpu().numpy()
    assert row_rel_err(got[:, :G], want[:, :G]) <= ATTN_TOL
    assert (got[:, G:] == 0).all()
    np.testing.assert_array_equal(bits(k_c)[n0:n0 + 3], bits(kn)[0])

    # query attention of a 4-token block appended after the three tokens
    kb = _rand_kv(rng, (Hkv, n_q, dim), torch.bfloat16)
    vb = _rand_kv(rng, (Hkv, n_q, dim), torch.bfloat16)
    d.dkv_append(kb, vb, 3, cap, k_c, v_c, seg_off, seg_len)
    qb = _rand_kv(rng, (B, n_q, Hq, dim), torch.bfloat16)
    qout = torch.full((B, n_q, Hq, dim), float("nan"), dtype=torch.float32, device=DEV)
    for hint in (0, need):
        wsb = d.dkv_query_workspace_bytes(B, Hq, Hkv, dim, n_q, hint)
        qws = torch.empty(wsb, dtype=torch.uint8, device=DEV) if wsb else None
        d.dkv_query_attn(qb, 3, cap, k_c, v_c, seg_off, seg_len, 0.09, qout, qws, Hkv, rows_hint=hint)
        assert guard_intact()
        kc2, vc2 = o.append(kc_ref, vc_ref, ref["seg_off"], ref["seg_len"], bits(kb).reshape(B, Hkv, n_q, dim),
                            bits(vb).reshape(B, Hkv, n_q, dim), 3)
        qwant = o.query_attn(bits(qb), kc2, vc2, ref["seg_off"], ref["seg_len"], 3, 0.09, Hkv, o.BF16)
        qgot = qout.cpu().numpy()
        assert row_rel_err(qgot[:, :, :G].reshape(-1, dim), qwant[:, :, :G].reshape(-1, dim)) <= ATTN_TOL
        assert (qgot[:, :, G:] == 0).all()


def test_append_matches_oracle(d):
    rng = np.random.default_rng(204)
    for dtype, dim in ((torch.bfloat16, 128), (torch.float32, 64), (torch.bfloat16, 64)):
        N, Hkv, G, T, cap = 2, 3, 2, 700, 6
        edges = [0, 100, 250, 700]
        pattern = (rng.uniform(size=(N, Hkv * G, 3)) < 0.4).astype(np.uint8)
        k = _rand_kv(rng, (N, Hkv, T, dim), dtype)
        v = _rand_kv(rng, (N, Hkv, T, dim), dtype)
        lay = _layout(d, N, Hkv * G, Hkv, dim, T, 4, 8, edges)
        pack = GpuPack(d, lay, pattern, k, v, cap)
        _, okm, _ = o.map_pattern(pattern, T, 4, 8, edges, Hkv)
        ref = o.compact(bits(k), bits(v), okm, cap)
        kc_ref, vc_ref = ref["k_c"], ref["v_c"]
        n_tail = 0
        for n_new in (2, 1, 3):
            kn = _rand_kv(rng, (N * Hkv, n_new, dim), dtype)
            vn = _rand_kv(rng, (N * Hkv, n_new, dim), dtype)
            d.dkv_append(kn, vn, n_tail, cap, pack.k_c, pack.v_c, pack.seg_off, pack.seg_len)
            kc_ref, vc_ref = o.append(kc_ref, vc_ref, ref["seg_off"], ref["seg_len"],
                                      bits(kn).reshape(N, Hkv, n_new, dim),
                                      bits(vn).reshape(N, Hkv, n_new, dim), n_tail)
            n_tail += n_new
        torch.cuda.synchronize()
        kc, vc = bits(pack.k_c), bits(pack.v_c)
        for s in range(N * Hkv):
            lo = int(ref["seg_off"][s])
            hi = lo + int(ref["seg_len"][s]) + n_tail
            np.testing.assert_array_equal(kc[lo:hi], kc_ref[lo:hi])
            np.testing.assert_array_equal(vc[lo:hi], vc_ref[lo:hi])
        with pytest.raises(d.DkvError) as e:
            d.dkv_append(kn, vn, n_tail, cap, pack.k_c, pack.v_c, pack.seg_off, pack.seg_len)
        assert e.value.status == d.DKV_ERR_CAPACITY


# ---------------------------------------------------------------------------
# dkv_decode_attn / dkv_dense_decode_attn
# ---------------------------------------------------------------------------

def _decode_case(d, rng, B, Hkv, G, T, dim, dtype, density, n_tail, cap=8, rows_hint=0,
                 zero_seg=False, sm_scale=None):
    Hq = Hkv * G
    mask = (rng.uniform(size=(B, Hkv, T)) < density).astype(np.uint8)
    if zero_seg:
        mask[0, 0] = 0
    k = _rand_kv(rng, (B, Hkv, T, dim), dtype)
    v = _rand_kv(rng, (B, Hkv, T, dim), dtype)
    q = _rand_kv(rng, (B, Hq, dim), dtype)
    lay = _layout(d, B, Hq, Hkv, dim, T, 0, 0, [0, max(T, 1)])
    mask_d = torch.from_numpy(mask).to(DEV)
    rows = int(mask.sum()) + B * Hkv * cap
    k_c = torch.empty((max(rows, 1), dim), dtype=dtype, device=DEV)
    v_c = torch.empty_like(k_c)
    seg_off = torch.empty(B * Hkv, dtype=torch.int64, device=DEV)
    seg_len = torch.empty(B * Hkv, dtype=torch.int32, device=DEV)
    ws = torch.empty(d.dkv_compact_workspace_bytes(lay), dtype=torch.uint8, device=DEV)
    d.dkv_compact(lay, k, v, mask_d, cap, k_c, v_c, seg_off, seg_len, ws)
    ref = o.compact(bits(k), bits(v), mask, cap)
    kc_ref, vc_ref = ref["k_c"], ref["v_c"]
    if n_tail:
        kn = _rand_kv(rng, (B * Hkv, n_tail, dim), dtype)
        vn = _rand_kv(rng, (B * Hkv, n_tail, dim), dtype)
        d.dkv_append(kn, vn, 0, cap, k_c, v_c, seg_off, seg_len)
        kc_ref, vc_ref = o.append(kc_ref, vc_ref, ref["seg_off"], ref["seg_len"],
                                  bits(kn).reshape(B, Hkv, n_tail, dim),
                                  bits(vn).reshape(B, Hkv, n_tail, dim), 0)
    scale = 1.0 / np.sqrt(dim) if sm_scale is None else sm_scale
    out = torch.full((B, Hq, dim), float("nan"), dtype=torch.float32, device=DEV)
    dws = torch.zeros(d.dkv_decode_workspace_bytes(B, Hq, Hkv, dim), dtype=torch.uint8, device=DEV)
    d.dkv_decode_attn(q, k_c, v_c, seg_off, seg_len, n_tail, scale, out, dws, Hkv, rows_hint=rows_hint)
    torch.cuda.synchronize()
    want = o.decode_attn(bits(q), kc_ref, vc_ref, ref["seg_off"], ref["seg_len"], n_tail, scale,
                         Hkv, odt(q))
    return out.cpu().numpy(), want, (q, k_c, v_c, seg_off, seg_len, out, dws, scale)


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
@pytest.mark.parametrize("dim", [64, 128])
def test_decode_random_shapes(d, dtype, dim):
    rng = np.random.default_rng(300 + dim + (dtype == torch.float32))
    for trial, G in enumerate([1, 2, 3, 4, 5, 7, 8, 16]):
        B, Hkv = int(rng.integers(1, 3)), int(rng.integers(1, 4))
        T = int(rng.choice([5, 31, 33, 200, 1000, 3001]))
        density = float(rng.choice([0.02, 0.3, 0.9]))
        n_tail = int(rng.choice([0, 1, 5]))
        rows_hint = int(rng.choice([0, 1, 10 ** 9]))
        got, want, _ = _decode_case(d, rng, B, Hkv, G, T, dim, dtype, density, n_tail,
                                    rows_hint=rows_hint, zero_seg=trial % 3 == 0)
        assert np.isfinite(got).all()
        err = row_rel_err(got, want)
        assert err <= ATTN_TOL, (G, B, Hkv, T, density, n_tail, rows_hint, err)


def test_decode_empty_segment_gives_zeros(d):
    rng = np.random.default_rng(310)
    got, want, _ = _decode_case(d, rng, 2, 2, 4, 600, 128, torch.bfloat16, 0.4, 0, zero_seg=True)
    assert (got[0, :4] == 0).all() and (want[0, :4] == 0).all()
    assert row_rel_err(got[1], want[1]) <= ATTN_TOL


def test_decode_tail_only_segment(d):
    rng = np.random.default_rng(311)
    got, want, _ = _decode_case(d, rng, 1, 2, 2, 300, 128, torch.bfloat16, 0.5, 3, zero_seg=True)
    assert row_rel_err(got, want) <= ATTN_TOL


@pytest.mark.parametrize("rows_hint", [0, 100, 5000])
def test_decode_many_pieces_and_determinism(d, rows_hint):
    rng = np.random.default_rng(320)
    got, want, args = _decode_case(d, rng, 2, 4, 4, 20000, 128, torch.bfloat16, 0.35, 2,
                                   rows_hint=rows_hint)
    assert row_rel_err(got, want) <= ATTN_TOL
    q, k_c, v_c, seg_off, seg_len, out, dws, scale = args
    for _ in range(3):
        out2 = torch.empty_like(out)
        d.dkv_decode_attn(q, k_c, v_c, seg_off, seg_len, 2, scale, out2, dws, 4, rows_hint=rows_hint)
        torch.cuda.synchronize()
        assert torch.equal(out, out2)  # fixed merge order: bitwise reproducible


def test_decode_workspace_needs_no_clearing(d):
    rng = np.random.default_rng(322)
    got, want, args = _decode_case(d, rng, 2, 4, 4, 6000, 128, torch.bfloat16, 0.35, 1)
    q, k_c, v_c, seg_off, seg_len, out, dws, scale = args
    dws.copy_(torch.from_numpy(rng.integers(0, 256, dws.numel(), dtype=np.uint8)).to(DEV))
    out2 = torch.empty_like(out)
    d.dkv_decode_attn(q, k_c, v_c, seg_off, seg_len, 1, scale, out2, dws, 4)
    torch.cuda.synchronize()
    assert torch.equal(out, out2)
    assert row_rel_err(got, want) <= ATTN_TOL


@pytest.mark.parametrize("dtype,dim,G", [(torch.bfloat16, 128, 4), (torch.float32, 64, 2),
                                         (torch.bfloat16, 128, 8), (torch.bfloat16, 64, 7)])
def test_fused_append_decode_equals_separate_calls(d, dtype, dim, G):
    rng = np.random.default_rng(330 + dim + G)
    B, Hkv, T, cap = 2, 3, 7000, 8
    for rows_hint in (0, 64):
        got, want, args = _decode_case(d, rng, B, Hkv, G, T, dim, dtype, 0.3, 2, cap=cap,
                                       rows_hint=rows_hint)
        q, k_c, v_c, seg_off, seg_len, out, dws, scale = args
        # rows 0..1 of the tail are filled; append 3 more at n_tail = 2 both ways
        kn = _rand_kv(rng, (B * Hkv, 3, dim), dtype)
        vn = _rand_kv(rng, (B * Hkv, 3, dim), dtype)
        k2, v2 = k_c.clone(), v_c.clone()
        sep = torch.empty_like(out)
        d.dkv_append(kn, vn, 2, cap, k_c, v_c, seg_off, seg_len)
        d.dkv_decode_attn(q, k_c, v_c, seg_off, seg_len, 5, scale, sep, dws, Hkv, rows_hint=rows_hint)
        fused = torch.empty_like(out)
        d.dkv_append_decode_attn(q, kn, vn, 2, cap, k2, v2, seg_off, seg_len, scale, fused, dws, Hkv,
                                 rows_hint=rows_hint)
        torch.cuda.synchronize()
        assert torch.equal(sep, fused)
        # the appended rows landed where dkv_append puts them
        for s in range(B * Hkv):
            lo = int(seg_off[s]) + int(seg_len[s])
            assert torch.equal(k2[lo + 2:lo + 5], kn[s]) and torch.equal(v2[lo + 2:lo + 5], vn[s])
        with pytest.raises(d.DkvError) as e:
            d.dkv_append_decode_attn(q, kn, vn, 6, cap, k2, v2, seg_off, seg_len, scale, fused, dws, Hkv)
        assert e.value.status == d.DKV_ERR_CAPACITY


def test_dense_fused_append_decode_matches_oracle(d):
    rng = np.random.default_rng(331)
    B, Hkv, G, t_cap, n_valid, dim = 2, 4, 4, 3000, 2990, 128
    k = _rand_kv(rng, (B, Hkv, t_cap, dim), torch.bfloat16)
    v = _rand_kv(rng, (B, Hkv, t_cap, dim), torch.bfloat16)
    q = _rand_kv(rng, (B, Hkv * G, dim), torch.bfloat16)
    kn = _rand_kv(rng, (B * Hkv, 2, dim), torch.bfloat16)
    vn = _rand_kv(rng, (B * Hkv, 2, dim), torch.bfloat16)
    out = torch.empty((B, Hkv * G, dim), dtype=torch.float32, device=DEV)
    ws = torch.empty(d.dkv_decode_workspace_bytes(B, Hkv * G, Hkv, dim), dtype=torch.uint8, device=DEV)
    d.dkv_dense_append_decode_attn(q, kn, vn, k, v, n_valid, 0.09, out, ws)
    torch.cuda.synchronize()
    kb, vb = bits(k), bits(v)
    kb[:, :, n_valid:n_valid + 2] = bits(kn).reshape(B, Hkv, 2, dim)
    vb[:, :, n_valid:n_valid + 2] = bits(vn).reshape(B, Hkv, 2, dim)
    np.testing.assert_array_equal(bits(k), kb)
    want = o.dense_decode_attn(bits(q), kb, vb, n_valid + 2, 0.09, o.BF16)
    assert row_rel_err(out.cpu().numpy(), want) <= ATTN_TOL
    with pytest.raises(d.DkvError) as e:
        d.dkv_dense_append_decode_attn(q, kn, vn, k, v, t_cap - 1, 0.09, out, ws)
    assert e.value.status == d.DKV_ERR_CAPACITY


def test_append_decode_graph_replays_match_eager(d):
    """append + decode captured in a HIP graph: every replay (with eager work
    and synchronisation in between) equals the eager result bit for bit."""
    rng = np.random.default_rng(323)
    B, Hkv, G, T, dim, cap = 1, 8, 4, 9000, 128, 4
    got, want, args = _decode_case(d, rng, B, Hkv, G, T, dim, torch.bfloat16, 0.35, 0, cap=cap)
    q, k_c, v_c, seg_off, seg_len, out, dws, scale = args
    kn = _rand_kv(rng, (B * Hkv, 1, dim), torch.bfloat16)
    vn = _rand_kv(rng, (B * Hkv, 1, dim), torch.bfloat16)
    d.dkv_append(kn, vn, 0, cap, k_c, v_c, seg_off, seg_len)
    eager = torch.empty_like(out)
    d.dkv_decode_attn(q, k_c, v_c, seg_off, seg_len, 1, scale, eager, dws, Hkv, rows_hint=20000)
    torch.cuda.synchronize()
    s = torch.cuda.Stream()
    g = torch.cuda.CUDAGraph()
    gout = torch.zeros_like(out)
    with torch.cuda.graph(g, stream=s):
        d.dkv_append(kn, vn, 0, cap, k_c, v_c, seg_off, seg_len, stream=s)
        d.dkv_decode_attn(q, k_c, v_c, seg_off, seg_len, 1, scale, gout, dws, Hkv, rows_hint=20000,
                          stream=s)
    for _ in range(3):
        gout.zero_()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(gout, eager)
        scratch = torch.empty_like(out)  # eager work between replays
        d.dkv_decode_attn(q, k_c, v_c, seg_off, seg_len, 0, scale, scratch, dws, Hkv)
        torch.cuda.synchronize()


@pytest.mark.parametrize("scale", [-0.7, 0.0])
@pytest.mark.parametrize("dtype,dim,G", [(torch.bfloat16, 128, 4), (torch.float32, 64, 2),
                                         (torch.bfloat16, 64, 8)])
def test_decode_negative_and_zero_scale(d, scale, dtype, dim, G):
    """A negative scale turns the softmax towards the keys least aligned with
    the query; a zero scale is uniform attention over every attended row.
    Both the attend-only and the fused append + decode call, split over many
    workgroups and in one."""
    rng = np.random.default_rng(350 + dim + G + int(scale == 0.0))
    B, Hkv, T, cap = 2, 3, 4000, 8
    Hq = Hkv * G
    mask = (rng.uniform(size=(B, Hkv, T)) < 0.4).astype(np.uint8)
    k = _rand_kv(rng, (B, Hkv, T, dim), dtype)
    v = _rand_kv(rng, (B, Hkv, T, dim), dtype)
    q = _rand_kv(rng, (B, Hq, dim), dtype)
    kn = _rand_kv(rng, (B * Hkv, 3, dim), dtype)
    vn = _rand_kv(rng, (B * Hkv, 3, dim), dtype)
    lay = _layout(d, B, Hq, Hkv, dim, T, 0, 0, [0, T])
    rows = int(mask.sum()) + B * Hkv * cap
    k_c = torch.empty((rows, dim), dtype=dtype, device=DEV)
    v_c = torch.empty_like(k_c)
    seg_off = torch.empty(B * Hkv, dtype=torch.int64, device=DEV)
    seg_len = torch.empty(B * Hkv, dtype=torch.int32, device=DEV)
    ws = torch.empty(d.dkv_compact_workspace_bytes(lay), dtype=torch.uint8, device=DEV)
    d.dkv_compact(lay, k, v, torch.from_numpy(mask).to(DEV), cap, k_c, v_c, seg_off, seg_len, ws)
    d.dkv_append(kn[:, :2].contiguous(), vn[:, :2].contiguous(), 0, cap, k_c, v_c, seg_off, seg_len)
    dws = torch.empty(d.dkv_decode_workspace_bytes(B, Hq, Hkv, dim), dtype=torch.uint8, device=DEV)
    ref = o.compact(bits(k), bits(v), mask, cap)
    kc_ref, vc_ref = o.append(ref["k_c"], ref["v_c"], ref["seg_off"], ref["seg_len"],
                              bits(kn).reshape(B, Hkv, 3, dim), bits(vn).reshape(B, Hkv, 3, dim), 0)
    want2 = o.decode_attn(bits(q), kc_ref, vc_ref, ref["seg_off"], ref["seg_len"], 2, scale, Hkv, odt(q))
    want3 = o.decode_attn(bits(q), kc_ref, vc_ref, ref["seg_off"], ref["seg_len"], 3, scale, Hkv, odt(q))
    if scale == 0.0:  # uniform weights: the mean of the attended V rows
        vr = o.widen(vc_ref, odt(q))
        for s in range(B * Hkv):
            lo, n = int(ref["seg_off"][s]), int(ref["seg_len"][s]) + 3
            np.testing.assert_allclose(want3[s // Hkv, (s % Hkv) * G:(s % Hkv + 1) * G],
                                       np.broadcast_to(vr[lo:lo + n].mean(0), (G, dim)), rtol=1e-12, atol=1e-12)
    for hint in (0, 1):  # the flat split over every workgroup, and one workgroup
        out = torch.full((B, Hq, dim), float("nan"), dtype=torch.float32, device=DEV)
        d.dkv_decode_attn(q, k_c, v_c, seg_off, seg_len, 2, scale, out, dws, Hkv, rows_hint=hint)
        torch.cuda.synchronize()
        got = out.cpu().numpy()
        assert np.isfinite(got).all()
        assert row_rel_err(got, want2) <= ATTN_TOL, (hint, row_rel_err(got, want2))
        fused = torch.full((B, Hq, dim), float("nan"), dtype=torch.float32, device=DEV)
        d.dkv_append_decode_attn(q, kn[:, 2:].contiguous(), vn[:, 2:].contiguous(), 2, cap, k_c, v_c, seg_off,
                                 seg_len, scale, fused, dws, Hkv, rows_hint=hint)
        torch.cuda.synchronize()
        got = fused.cpu().numpy()
        assert np.isfinite(got).all()
        assert row_rel_err(got, want3) <= ATTN_TOL, (hint, row_rel_err(got, want3))


def test_decode_large_logits_are_stable(d):
    rng = np.random.default_rng(321)
    got, want, _ = _decode_case(d, rng, 1, 2, 4, 5000, 128, torch.bfloat16, 0.5, 1, sm_scale=8.0)
    assert np.isfinite(got).all()
    assert row_rel_err(got, want) <= ATTN_TOL


@pytest.mark.parametrize("dtype,dim", [(torch.bfloat16, 128), (torch.float32, 64),
                                       (torch.bfloat16, 64)])
def test_dense_decode_matches_oracle(d, dtype, dim):
    rng = np.random.default_rng(330)
    for B, Hkv, G, t_cap, n_valid in ((1, 8, 4, 4096, 4000), (3, 2, 8, 900, 900), (2, 1, 7, 50, 17),
                                      (1, 2, 1, 64, 0)):
        k = _rand_kv(rng, (B, Hkv, t_cap, dim), dtype)
        v = _rand_kv(rng, (B, Hkv, t_cap, dim), dtype)
        q = _rand_kv(rng, (B, Hkv * G, dim), dtype)
        out = torch.empty((B, Hkv * G, dim), dtype=torch.float32, device=DEV)
        ws = torch.zeros(d.dkv_decode_workspace_bytes(B, Hkv * G, Hkv, dim), dtype=torch.uint8,
                         device=DEV)
        d.dkv_dense_decode_attn(q, k, v, n_valid, 0.125, out, ws)
        torch.cuda.synchronize()
        want = o.dense_decode_attn(bits(q), bits(k), bits(v), n_valid, 0.125, odt(q))
        assert row_rel_err(out.cpu().numpy(), want) <= ATTN_TOL


def test_all_keep_packed_decode_equals_dense_kernel(d):
    """With every position kept the packed cache is the dense cache, the two
    calls see the same rows and the same split, so they agree bit for bit."""
    rng = np.random.default_rng(340)
    B, Hkv, G, T, dim = 1, 8, 4, 8192, 128
    k = _rand_kv(rng, (B, Hkv, T, dim), torch.bfloat16)
    v = _rand_kv(rng, (B, Hkv, T, dim), torch.bfloat16)
    q = _rand_kv(rng, (B, Hkv * G, dim), torch.bfloat16)
    lay = _layout(d, B, Hkv * G, Hkv, dim, T, 0, 0, [0, T])
    pack = GpuPack(d, lay, np.ones((B, Hkv * G, 1), np.uint8), k, v, 0)
    ws = torch.zeros(d.dkv_decode_workspace_bytes(B, Hkv * G, Hkv, dim), dtype=torch.uint8, device=DEV)
    o1 = torch.empty((B, Hkv * G, dim), dtype=torch.float32, device=DEV)
    o2 = torch.empty_like(o1)
    d.dkv_decode_attn(q, pack.k_c, pack.v_c, pack.seg_off, pack.seg_len, 0, 0.1, o1, ws, Hkv,
                      rows_hint=B * Hkv * T)
    d.dkv_dense_decode_attn(q, k, v, T, 0.1, o2, ws)
    torch.cuda.synchronize()
    assert torch.equal(o1, o2)
    want = o.dense_decode_attn(bits(q), bits(k), bits(v), T, 0.1, o.BF16)
    assert row_rel_err(o1.cpu().numpy(), want) <= ATTN_TOL


# ---------------------------------------------------------------------------
# whole path on the workloads (map -> compact -> append -> decode)
# ---------------------------------------------------------------------------

def _workload_path(d, w, pattern, units, gen_device, steps=1):
    """Run the path for the given unit indices of a workload (one sequence each)."""
    for unit in units:
        k, v = di.kv_unit(w, unit, device=gen_device)
        k, v = k.to(DEV)[None], v.to(DEV)[None]
        pat = np.ascontiguousarray(pattern[unit:unit + 1])
        lay = d.make_layout(1, w.num_q_heads, w.num_kv_heads, w.head_dim, w.context_len, w.sink,
                            w.recent, list(w.bin_edges))
        pack = GpuPack(d, lay, pat, k, v, w.append_cap)
        torch.cuda.synchronize()
        _, okm, _ = o.map_pattern(pat, w.context_len, w.sink, w.recent, w.bin_edges, w.num_kv_heads)
        ref = o.compact(bits(k), bits(v), okm, w.append_cap)
        _check_pack(pack, ref)
        kc_ref, vc_ref = ref["k_c"], ref["v_c"]
        ws = torch.zeros(d.dkv_decode_workspace_bytes(1, w.num_q_heads, w.num_kv_heads, w.head_dim),
                         dtype=torch.uint8, device=DEV)
        for step in range(steps):
            kn, vn = di.kv_new_step(w, unit, step, device=gen_device)
            kn = kn.to(DEV)[0].contiguous()
            vn = vn.to(DEV)[0].contiguous()
            d.dkv_append(kn, vn, step, w.append_cap, pack.k_c, pack.v_c, pack.seg_off, pack.seg_len)
            kc_ref, vc_ref = o.append(kc_ref, vc_ref, ref["seg_off"], ref["seg_len"],
                                      bits(kn)[None], bits(vn)[None], step)
            q = di.q_step(w, unit, step, device=gen_device).to(DEV)[:1].contiguous()
            out = torch.empty((1, w.num_q_heads, w.head_dim), dtype=torch.float32, device=DEV)
            d.dkv_decode_attn(q, pack.k_c, pack.v_c, pack.seg_off, pack.seg_len, step + 1,
                              w.sm_scale, out, ws, w.num_kv_heads, rows_hint=pack.rows)
            torch.cuda.synchronize()
            want = o.decode_attn(bits(q), kc_ref, vc_ref, ref["seg_off"], ref["seg_len"], step + 1,
                                 w.sm_scale, w.num_kv_heads, odt(q))
            err = row_rel_err(out.cpu().numpy(), want)
            assert err <= ATTN_TOL, (w.name, unit, step, err)


def test_path_tiny(d):
    w = di.workload("tiny")
    pattern, _ = di.make_pattern(w)
    _workload_path(d, w, pattern, [0], "cpu", steps=3)


def test_path_llama8b_layer_32k(d):
    w = di.workload("llama8b_layer_32k")
    pattern, _ = di.make_pattern(w)
    _workload_path(d, w, pattern, [0], DEV, steps=2)


@pytest.mark.parametrize("budget", [0.10, 0.20, 0.50])
def test_path_llama70b_batched_budgets(d, budget):
    """Batched 70B-shaped layer: decode all 16 sequences in one call."""
    w = di.workload("llama70b_layer_bs16_32k")
    pattern, _ = di.make_pattern(w, budget=budget)
    B = w.batch
    ks, vs = zip(*(di.kv_unit(w, b, device=DEV) for b in range(B)))
    k, v = torch.stack(ks), torch.stack(vs)
    lay = d.make_layout(B, w.num_q_heads, w.num_kv_heads, w.head_dim, w.context_len, w.sink,
                        w.recent, list(w.bin_edges))
    pack = GpuPack(d, lay, pattern, k, v, w.append_cap)
    torch.cuda.synchronize()
    _, okm, okl = o.map_pattern(pattern, w.context_len, w.sink, w.recent, w.bin_edges, w.num_kv_heads)
    np.testing.assert_array_equal(pack.kv_len.cpu().numpy(), okl)
    ref = o.compact(bits(k), bits(v), okm, w.append_cap)
    _check_pack(pack, ref)
    q = di.q_step(w, 0, 0, device=DEV)
    out = torch.empty((B, w.num_q_heads, w.head_dim), dtype=torch.float32, device=DEV)
    ws = torch.zeros(d.dkv_decode_workspace_bytes(B, w.num_q_heads, w.num_kv_heads, w.head_dim),
                     dtype=torch.uint8, device=DEV)
    d.dkv_decode_attn(q, pack.k_c, pack.v_c, pack.seg_off, pack.seg_len, 0, w.sm_scale, out, ws,
                      w.num_kv_heads, rows_hint=pack.rows)
    torch.cuda.synchronize()
    want = o.decode_attn(bits(q), ref["k_c"], ref["v_c"], ref["seg_off"], ref["seg_len"], 0,
                         w.sm_scale, w.num_kv_heads, o.BF16)
    assert row_rel_err(out.cpu().numpy(), want) <= ATTN_TOL


def test_probe_stream_read_runs(d):
    """The bandwidth probe reads a ragged buffer with every block size, over
    lengths that end inside a block (no result to compare: it only must not
    fail, and the sink keeps its contents since no fold hits the constant)."""
    src = torch.ones((1 << 20) + 48, dtype=torch.uint8, device=DEV)
    sink = torch.zeros(4, dtype=torch.int32, device=DEV)
    for g in (1, 2, 4, 8):
        for n in (16, 4096 * g - 16, (1 << 20) + 48):
            d.dkv_probe_stream_read(src, sink, g, nbytes=n)
    torch.cuda.synchronize()
    assert int(sink.abs().sum()) == 0


def test_probe_copy_copies(d):
    """The copy probe copies every byte, with each block size, over lengths
    that end inside a block, and touches nothing past `nbytes`."""
    g = torch.Generator(device=DEV).manual_seed(5)
    src = torch.randint(0, 256, ((1 << 20) + 4096,), dtype=torch.uint8, device=DEV, generator=g)
    for gpt in (1, 2, 4, 8):
        for n in (16, 4096 * gpt - 16, 4096 * gpt, (1 << 20) + 48):
            dst = torch.full_like(src, 0xA5)
            d.dkv_probe_copy(src, dst, gpt, nbytes=n)
            torch.cuda.synchronize()
            assert torch.equal(dst[:n], src[:n]), (gpt, n)
            assert bool((dst[n:] == 0xA5).all()), (gpt, n)
