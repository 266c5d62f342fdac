"""GPU parity of the block-gather pack (dkv_compact_bins).

Its outputs must equal dkv_map_pattern + dkv_compact's bit for bit for the
same layout and pattern -- packed K and V (free rows untouched alike), offsets,
lengths (with the same -1 marker when out_rows is too small), source positions
and rows_needed -- and, on a case checked independently, the oracle's map and
pack.  Layouts: uniform and irregular edges, contexts shorter than sink +
recent, a farthest bin cut by the compressible span, edges that end before it
(an uncovered gap), G from 1 to 16, d 64 and 128, bf16 and fp32, and the
paper's 1,013-bin layout at 130,816 positions.  The ragged form
(dkv_compact_bins_ragged) must equal dkv_map_pattern_ragged + dkv_compact the
same way.
"""

import numpy as np
import pytest
import torch

import oracle as o
from _helpers import bits

pytestmark = pytest.mark.gpu

DEV = "cuda"


@pytest.fixture(scope="module")
def d():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2609_32663_amd as lib
    return lib


def _both(d, lay, pattern, k, v, cap, out_rows=None):
    """The two routes on the same inputs: (map + compact) and compact_bins."""
    N, Hkv, T = lay.num_units, lay.num_kv_heads, lay.context_len
    nseg = N * Hkv
    dim = k.shape[-1]
    # (with T = 0 no mask byte is read or written; the buffer only has to exist)
    km = torch.empty((N, Hkv, max(T, 1)), dtype=torch.uint8, device=DEV)
    kl = torch.empty((N, Hkv), dtype=torch.int32, device=DEV)
    d.dkv_map_pattern(lay, pattern, km, kl)
    need = int((kl.cpu().to(torch.int64) + cap).sum())
    rows = need if out_rows is None else out_rows
    res = []
    for route in ("mask", "bins"):
        k_out = torch.full((max(rows, 1), dim), 3.0, dtype=k.dtype, device=DEV)[:rows]
        v_out = torch.full((max(rows, 1), dim), -2.0, dtype=k.dtype, device=DEV)[:rows]
        so = torch.full((nseg,), -9, dtype=torch.int64, device=DEV)
        sl = torch.full((nseg,), -9, dtype=torch.int32, device=DEV)
        sp = torch.full((max(rows, 1),), -7, dtype=torch.int32, device=DEV)[:rows]
        rn = torch.full((1,), -9, dtype=torch.int64, device=DEV)
        if route == "mask":
            ws = torch.empty(max(d.dkv_compact_workspace_bytes(lay), 16), dtype=torch.uint8, device=DEV)
            d.dkv_compact(lay, k, v, km, cap, k_out, v_out, so, sl, ws, src_pos=sp, rows_needed=rn)
        else:
            # a workspace full of garbage: nothing may depend on its contents
            ws = torch.full((max(d.dkv_compact_bins_workspace_bytes(lay), 16),), 0x5A, dtype=torch.uint8,
                            device=DEV)
            d.dkv_compact_bins(lay, k, v, pattern, cap, k_out, v_out, so, sl, ws, src_pos=sp, rows_needed=rn)
        torch.cuda.synchronize()
        res.append((k_out, v_out, so, sl, sp, rn))
    return res, km, kl, need


def _assert_same(res):
    (a, b) = res
    for x, y, name in zip(a, b, ("k_out", "v_out", "seg_off", "seg_len", "src_pos", "rows_needed")):
        assert torch.equal(x.view(torch.uint8) if x.dtype == torch.bfloat16 else x,
                           y.view(torch.uint8) if y.dtype == torch.bfloat16 else y), name


def _inputs(rng, N, Hq, Hkv, dim, T, dtype, D, density):
    g = torch.Generator(device=DEV).manual_seed(int(rng.integers(1 << 30)))
    k = torch.randn((N, Hkv, max(T, 1), dim), generator=g, device=DEV).to(dtype)
    v = torch.randn((N, Hkv, max(T, 1), dim), generator=g, device=DEV).to(dtype)
    pattern = torch.from_numpy((rng.uniform(size=(N, Hq, D)) < density).astype(np.uint8)).to(DEV)
    return k, v, pattern


def test_compact_bins_matches_map_and_compact_random(d):
    rng = np.random.default_rng(2024)
    for trial in range(40):
        G = int(rng.choice([1, 2, 3, 4, 7, 8, 16]))
        Hkv = int(rng.integers(1, 4))
        N = int(rng.integers(1, 4))
        dim = int(rng.choice([64, 128]))
        dtype = torch.bfloat16 if trial % 3 else torch.float32
        S, R = int(rng.integers(0, 40)), int(rng.integers(0, 300))
        T = int(rng.choice([0, 1, 15, S + R, S + R + 1, int(rng.integers(2, 9000))]))
        U = max(T - S - R, 1)
        if trial % 2:
            W = int(rng.integers(1, 200))
            D = int(rng.integers(1, 60))
            edges = [W * i for i in range(D + 1)]
        else:
            D = int(rng.integers(1, 40))
            top = int(U * rng.choice([0.5, 1.0, 1.7]))  # edges ending before, at or past the span
            edges = sorted(set([0] + list(rng.integers(1, max(top, 2) + 1, size=D))))
            D = len(edges) - 1
            if D < 1:
                edges, D = [0, 1], 1
        lay = d.make_layout(N, G * Hkv, Hkv, dim, T, S, R, edges)
        k, v, pattern = _inputs(rng, N, G * Hkv, Hkv, dim, T, dtype, D, float(rng.choice([0.0, 0.2, 0.5, 1.0])))
        cap = int(rng.integers(0, 50))
        res, *_ = _both(d, lay, pattern, k, v, cap)
        _assert_same(res)


def test_compact_bins_out_rows_too_small(d):
    rng = np.random.default_rng(7)
    N, Hq, Hkv, dim, T = 2, 8, 2, 128, 3000
    lay = d.make_layout(N, Hq, Hkv, dim, T, 16, 128, [0, 100, 700, 1500, 2856])
    k, v, pattern = _inputs(rng, N, Hq, Hkv, dim, T, torch.bfloat16, 4, 0.5)
    _, _, kl, need = _both(d, lay, pattern, k, v, 11)
    for frac in (0.001, 0.3, 0.75, 0.999):
        res, *_ = _both(d, lay, pattern, k, v, 11, out_rows=max(1, int(need * frac)))
        _assert_same(res)
        assert (res[1][3] < 0).any()


def test_compact_bins_matches_oracle(d):
    """Independent of dkv_compact: the oracle's map and pack of the same inputs."""
    rng = np.random.default_rng(11)
    N, Hq, Hkv, dim, T, S, R = 2, 12, 3, 64, 2500, 32, 256
    edges = [0, 64, 128, 256, 512, 1024, 2048]
    lay = d.make_layout(N, Hq, Hkv, dim, T, S, R, edges)
    k, v, pattern = _inputs(rng, N, Hq, Hkv, dim, T, torch.bfloat16, len(edges) - 1, 0.3)
    cap = 5
    res, km, kl, need = _both(d, lay, pattern, k, v, cap)
    k_out, v_out, so, sl, sp, rn = res[1]
    _, okm, okl = o.map_pattern(pattern.cpu().numpy(), T, S, R, edges, Hkv)
    ref = o.compact(bits(k), bits(v), okm, cap)
    np.testing.assert_array_equal(sl.cpu().numpy(), ref["seg_len"])
    np.testing.assert_array_equal(so.cpu().numpy(), ref["seg_off"])
    assert int(rn.item()) == need
    ko, vo, spo = bits(k_out), bits(v_out), sp.cpu().numpy()
    for s_ in range(N * Hkv):
        o0, n0 = int(ref["seg_off"][s_]), int(ref["seg_len"][s_])
        np.testing.assert_array_equal(ko[o0:o0 + n0], ref["k_c"][o0:o0 + n0])
        np.testing.assert_array_equal(vo[o0:o0 + n0], ref["v_c"][o0:o0 + n0])
        np.testing.assert_array_equal(spo[o0:o0 + n0], ref["src_pos"][o0:o0 + n0])


def test_compact_bins_paper_layout(d):
    """Appendix A's layout: 128 sink, 1,024 recent, 128-token bins, D = 1,013 at
    130,816 positions; one unit of 8 KV heads, every bin a 128-row block."""
    rng = np.random.default_rng(1013)
    T, S, R, W = 130816, 128, 1024, 128
    D = (T - S - R) // W
    assert D == 1013
    N, Hq, Hkv, dim = 1, 32, 8, 128
    lay = d.make_layout(N, Hq, Hkv, dim, T, S, R, [W * i for i in range(D + 1)])
    k, v, pattern = _inputs(rng, N, Hq, Hkv, dim, T, torch.bfloat16, D, 0.1)
    res, *_ = _both(d, lay, pattern, k, v, 64)
    _assert_same(res)


def test_compact_bins_one_row_bins(d):
    """Bins one position wide: every kept bin is a range of one row, so a
    copy chunk spans as many ranges as it has rows (the most its range table
    holds), and chunk boundaries fall between and inside the sink and recent
    ranges; densities from sparse to full, several contexts, up to more kept
    ranges per segment (8,986) than the plan pass stages in LDS (4,096)."""
    rng = np.random.default_rng(1)
    N, Hq, Hkv, dim = 2, 4, 2, 128
    # (the last case keeps more ranges than the plan stages in LDS: the serial fill)
    for T, S, R, density in ((2100, 5, 37, 0.5), (2100, 0, 0, 0.9), (4133, 31, 33, 1.0), (700, 64, 64, 0.05),
                             (9000, 8, 8, 1.0)):
        D = T - S - R
        lay = d.make_layout(N, Hq, Hkv, dim, T, S, R, list(range(D + 1)))
        k, v, pattern = _inputs(rng, N, Hq, Hkv, dim, T, torch.bfloat16, D, density)
        res, *_ = _both(d, lay, pattern, k, v, 3)
        _assert_same(res)


def test_compact_bins_ragged_matches_map_ragged_and_compact(d):
    """dkv_compact_bins_ragged equals dkv_map_pattern_ragged + dkv_compact in
    every output, bit for bit: per-unit lengths below zero, zero, shorter than
    sink + recent, in between, equal to and past the row length (clamped);
    uniform and irregular edges; and once against the oracle's ragged map and
    pack."""
    rng = np.random.default_rng(99)
    for trial in range(20):
        G = int(rng.choice([1, 2, 4, 7, 8]))
        Hkv = int(rng.integers(1, 4))
        N = int(rng.integers(1, 7))
        dim = int(rng.choice([64, 128]))
        S, R = int(rng.integers(0, 40)), int(rng.integers(0, 300))
        T = int(rng.integers(S + R + 2, 6000))
        if trial % 2:
            W = int(rng.integers(1, 150))
            D = int(rng.integers(1, 50))
            edges = [W * i for i in range(D + 1)]
        else:
            D = int(rng.integers(1, 30))
            edges = sorted(set([0] + list(rng.integers(1, T + 1, size=D))))
            D = len(edges) - 1
            if D < 1:
                edges, D = [0, 1], 1
        lay = d.make_layout(N, G * Hkv, Hkv, dim, T, S, R, edges)
        k, v, pattern = _inputs(rng, N, G * Hkv, Hkv, dim, T, torch.bfloat16, D, float(rng.choice([0.1, 0.5, 1.0])))
        cands = [-5, 0, max(S + R - 3, 0), S + R, int(rng.integers(0, T + 1)), T, T + 40]
        ulen = torch.tensor([int(rng.choice(cands)) for _ in range(N)], dtype=torch.int32, device=DEV)
        cap = int(rng.integers(0, 20))
        km = torch.empty((N, Hkv, T), dtype=torch.uint8, device=DEV)
        kl = torch.empty((N, Hkv), dtype=torch.int32, device=DEV)
        d.dkv_map_pattern_ragged(lay, ulen, pattern, km, kl)
        need = int((kl.cpu().to(torch.int64) + cap).sum())
        res = []
        for route in ("mask", "bins"):
            k_out = torch.full((max(need, 1), dim), 3.0, dtype=k.dtype, device=DEV)[:need]
            v_out = torch.full((max(need, 1), dim), -2.0, dtype=k.dtype, device=DEV)[:need]
            so = torch.full((N * Hkv,), -9, dtype=torch.int64, device=DEV)
            sl = torch.full((N * Hkv,), -9, dtype=torch.int32, device=DEV)
            sp = torch.full((max(need, 1),), -7, dtype=torch.int32, device=DEV)[:need]
            rn = torch.full((1,), -9, dtype=torch.int64, device=DEV)
            if route == "mask":
                ws = torch.empty(max(d.dkv_compact_workspace_bytes(lay), 16), dtype=torch.uint8, device=DEV)
                d.dkv_compact(lay, k, v, km, cap, k_out, v_out, so, sl, ws, src_pos=sp, rows_needed=rn)
            else:
                ws = torch.full((max(d.dkv_compact_bins_workspace_bytes(lay), 16),), 0x5A, dtype=torch.uint8,
                                device=DEV)
                d.dkv_compact_bins_ragged(lay, ulen, k, v, pattern, cap, k_out, v_out, so, sl, ws, src_pos=sp,
                                          rows_needed=rn)
            torch.cuda.synchronize()
            res.append((k_out, v_out, so, sl, sp, rn))
        _assert_same(res)
        if trial == 0:
            _, okm, okl = o.map_pattern(pattern.cpu().numpy(), T, S, R, edges, Hkv, unit_len=ulen.cpu().numpy())
            ref = o.compact(bits(k), bits(v), okm, cap)
            np.testing.assert_array_equal(res[1][3].cpu().numpy(), ref["seg_len"])
            np.testing.assert_array_equal(res[1][2].cpu().numpy(), ref["seg_off"])
            ko = bits(res[1][0])
            for s_ in range(N * Hkv):
                o0, n0 = int(ref["seg_off"][s_]), int(ref["seg_len"][s_])
                np.testing.assert_array_equal(ko[o0:o0 + n0], ref["k_c"][o0:o0 + n0])


def test_compact_bins_many_segments(d):
    """65,520 segments (4,095 units x 16 KV heads), near the 65,535 limit of
    the segment grid: the plan and copy grids at their largest, and the offset
    scan over 64 chunks of 1,024 segments; equal to map + compact."""
    rng = np.random.default_rng(65520)
    N, Hq, Hkv, dim, T, S, R = 4095, 32, 16, 64, 100, 4, 8
    lay = d.make_layout(N, Hq, Hkv, dim, T, S, R, [0, 10, 30, 88])
    k, v, pattern = _inputs(rng, N, Hq, Hkv, dim, T, torch.bfloat16, 3, 0.4)
    res, *_ = _both(d, lay, pattern, k, v, 2)
    _assert_same(res)
