"""GPU parity of the exact-budget pattern export, and of the hot path on
exported patterns and their ablation families.

dkv_topk_pattern must equal the oracle's TopKMask bit for bit: exactly k ones,
ties at the k-th value to the lowest flat indices, NaN below every number,
-0 equal to +0.  Patterns exported on the GPU then go through the GPU's map,
pack and decode on the paper's bin layout (128-token bins, 1,015 bins at
131,072 tokens), checked against the oracle's own export, lengths and
attention; so does every ablation family of the exported pattern.
"""

import numpy as np
import pytest
import torch

import dkv_inputs as di
import oracle as o
from _helpers import ATTN_TOL, GpuPack, bits, row_rel_err

pytestmark = pytest.mark.gpu

DEV = "cuda"


@pytest.fixture(scope="module")
def d():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2609_32663_amd as lib
    return lib


def _gpu_topk(d, p, k):
    probs = torch.from_numpy(np.ascontiguousarray(p, dtype=np.float32)).to(DEV)
    out = torch.full(p.shape, 7, dtype=torch.uint8, device=DEV)
    # a workspace full of garbage: nothing may depend on its contents
    ws = torch.full((d.dkv_topk_workspace_bytes(*p.shape),), 0xA5, dtype=torch.uint8, device=DEV)
    d.dkv_topk_pattern(probs, k, out, ws)
    torch.cuda.synchronize()
    return out.cpu().numpy()


def test_topk_random_shapes_ties_and_specials(d):
    rng = np.random.default_rng(70)
    for trial in range(40):
        shape = (int(rng.integers(1, 5)), int(rng.integers(1, 40)), int(rng.integers(1, 300)))
        n = int(np.prod(shape))
        levels = int(rng.choice([2, 5, 64, 100000]))
        p = (rng.integers(0, levels, size=shape) / float(levels)).astype(np.float32)
        if trial % 3 == 0:
            p[rng.uniform(size=shape) < 0.1] = np.nan
        if trial % 4 == 1:
            p[rng.uniform(size=shape) < 0.2] = -0.0
        if trial % 5 == 2:
            p[rng.uniform(size=shape) < 0.05] = -np.inf
            p[rng.uniform(size=shape) < 0.05] = np.inf
            p[rng.uniform(size=shape) < 0.1] *= -1.0
        for k in sorted({0, 1, n // 5, n // 2, max(n - 1, 0), n, int(rng.integers(0, n + 1))}):
            got = _gpu_topk(d, p, k)
            np.testing.assert_array_equal(got, o.topk_mask(p, k), err_msg=f"trial {trial} k {k}")


def test_topk_paper_shape(d):
    """32 layers x 32 query heads x 1,015 bins (the paper's layout at 131,072
    tokens), the exact budget at rho = 0.2 and values around it."""
    w = di.workload("llama8b_stack_128k_paper_bins")
    L, H, D = w.num_layers, w.num_q_heads, w.num_bins
    p = di.retention_probs(L, H, w.num_kv_heads, D, seed=w.cfg_id)
    k = d.dkv_budget_entries(w.rho, L, H, D)
    assert k == o.budget_entries(w.rho, L, H, D)
    for kk in (k - 1, k, k + 1, 0, L * H * D):
        got = _gpu_topk(d, p, kk)
        np.testing.assert_array_equal(got, o.topk_mask(p, kk))
        assert int(got.sum()) == kk


def _layer_slice_case(w, layers):
    """The exported pattern of the paper-bins workload, restricted to a few layers."""
    L, H, D = w.num_layers, w.num_q_heads, w.num_bins
    p = di.retention_probs(L, H, w.num_kv_heads, D, seed=w.cfg_id)
    return p, o.topk_mask(p, o.budget_entries(w.rho, L, H, D))


@pytest.mark.parametrize("kind", ("exported",) + di.PATTERN_FAMILIES)
def test_exported_pattern_families_through_the_path(d, kind):
    """Map, pack and decode two layers of the paper-bins stack with the
    GPU-exported pattern (or one of its ablation families)."""
    w = di.workload("llama8b_stack_128k_paper_bins")
    layers = (3, 17)
    H, Hkv, dim, T, cap = w.num_q_heads, w.num_kv_heads, w.head_dim, w.context_len, 8
    p, want_pat = _layer_slice_case(w, layers)
    got_pat = _gpu_topk(d, p, d.dkv_budget_entries(w.rho, w.num_layers, H, w.num_bins))
    np.testing.assert_array_equal(got_pat, want_pat)
    pat = got_pat if kind == "exported" else di.pattern_family(got_pat, kind, Hkv, seed=5)
    pat = np.ascontiguousarray(pat[list(layers)])
    units = len(layers)
    kv = [di.kv_unit(w, layer, device=DEV) for layer in layers]
    k = torch.stack([a for a, _ in kv])
    v = torch.stack([b for _, b in kv])
    del kv
    lay = d.make_layout(units, H, Hkv, dim, T, w.sink, w.recent, list(w.bin_edges))
    pack = GpuPack(d, lay, pat, k, v, cap)
    olen = o.closed_form_lengths(pat, T, w.sink, w.recent, w.bin_edges, Hkv)
    np.testing.assert_array_equal(pack.kv_len.cpu().numpy(), olen)
    rep = o.retention_report(pat, T, w.sink, w.recent, w.bin_edges, Hkv)
    assert rep["retained_positions"] == int(pack.kv_len.sum())
    _, okm, _ = o.map_pattern(pat, T, w.sink, w.recent, w.bin_edges, Hkv)
    ws = torch.zeros(d.dkv_decode_workspace_bytes(1, H, Hkv, dim), dtype=torch.uint8, device=DEV)
    out = torch.empty((1, H, dim), dtype=torch.float32, device=DEV)
    for u, layer in enumerate(layers):
        segs = slice(u * Hkv, (u + 1) * Hkv)
        q = di.q_step(w, layer, 0, device=DEV)
        d.dkv_decode_attn(q, pack.k_c, pack.v_c, pack.seg_off[segs], pack.seg_len[segs], 0, w.sm_scale, out, ws,
                          Hkv, rows_hint=int(pack.kv_len[u].sum()))
        torch.cuda.synchronize()
        ref = o.compact(bits(k[u:u + 1]), bits(v[u:u + 1]), okm[u:u + 1], 0)
        want = o.decode_attn(bits(q), ref["k_c"], ref["v_c"], ref["seg_off"], ref["seg_len"], 0, w.sm_scale, Hkv,
                             o.BF16)
        assert row_rel_err(out.cpu().numpy(), want) <= ATTN_TOL, (kind, layer)
