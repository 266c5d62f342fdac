"""GPU parity for batches of contexts of different lengths (ragged batches).

dkv_map_pattern_ragged must give the oracle's masks and lengths bit for bit,
with each unit's distances counted from the end of its own context; the
pack, the appends and decode then follow the lengths unchanged, checked
against the oracle on the 70B-shaped batch (16 sequences of 4K-32K tokens).
"""

import numpy as np
import pytest
import torch

import dkv_inputs as di
import oracle as o
from _helpers import ATTN_TOL, bits, row_rel_err

pytestmark = pytest.mark.gpu

DEV = "cuda"


@pytest.fixture(scope="module")
def d():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2609_32663_amd as lib
    return lib


def _edges(rng, uniform):
    D = int(rng.integers(1, 40))
    if uniform:
        W = int(rng.integers(1, 200))
        return [W * k for k in range(D + 1)]
    return [0] + [int(x) for x in np.cumsum(rng.integers(1, 300, size=D))]


@pytest.mark.parametrize("seed", range(30))
def test_ragged_map_matches_oracle(d, seed):
    rng = np.random.default_rng(900 + seed)
    N = int(rng.integers(1, 6))
    Hkv = int(rng.integers(1, 4))
    G = int(rng.choice([1, 2, 4, 8]))
    Hq = Hkv * G
    T = int(rng.choice([0, 1, 15, 16, 17, 200, 1000, 4096, 5003]))
    S, R = int(rng.integers(0, 40)), int(rng.integers(0, 300))
    edges = _edges(rng, seed % 2 == 0)
    pattern = (rng.uniform(size=(N, Hq, len(edges) - 1)) < 0.4).astype(np.uint8)
    lens = rng.integers(0, T + 1, size=N).astype(np.int32)
    if T:
        lens[0] = T
    # out-of-range lengths are clamped into the row
    raw = lens.copy()
    if N > 1:
        raw[-1] = -5 if seed % 3 == 0 else T + 7
        lens[-1] = 0 if seed % 3 == 0 else T
    lay = d.make_layout(N, Hq, Hkv, 128, T, S, R, edges)
    km = torch.full((N * Hkv * T + 16,), 9, dtype=torch.uint8, device=DEV)[:N * Hkv * T].view(N, Hkv, T)
    qm = torch.full((N * Hq * T + 16,), 9, dtype=torch.uint8, device=DEV)[:N * Hq * T].view(N, Hq, T)
    kl = torch.full((N, Hkv), -1, dtype=torch.int32, device=DEV)
    d.dkv_map_pattern_ragged(lay, torch.from_numpy(raw).to(DEV), torch.from_numpy(pattern).to(DEV), km, kl, qm)
    torch.cuda.synchronize()
    oq, okm, okl = o.map_pattern(pattern, T, S, R, edges, Hkv, unit_len=lens)
    np.testing.assert_array_equal(km.cpu().numpy(), okm)
    np.testing.assert_array_equal(qm.cpu().numpy(), oq)
    np.testing.assert_array_equal(kl.cpu().numpy(), okl)


def test_ragged_batch_pack_append_decode(d):
    """The 70B-shaped batch (16 sequences, 64q/8kv, 20% physical budget) with
    per-sequence contexts of 4K-32K tokens: one ragged map and pack, then 16
    fused append + decode steps, against the oracle's map, pack, appends and
    attention at the first and the last step."""
    w = di.workload("llama70b_layer_bs16_32k")
    B, Hq, Hkv, dim, T, cap = w.batch, w.num_q_heads, w.num_kv_heads, w.head_dim, w.context_len, 16
    lens = di.sequence_lengths(w, seed=1)
    pattern, _ = di.make_pattern(w)
    k = torch.empty((B, Hkv, T, dim), dtype=torch.bfloat16, device=DEV)
    v = torch.empty_like(k)
    for b in range(B):
        kb, vb = di.kv_unit(w, b, device=DEV)
        k[b].copy_(kb)
        v[b].copy_(vb)
    lay = d.make_layout(B, Hq, Hkv, dim, T, w.sink, w.recent, list(w.bin_edges))
    km = torch.empty((B, Hkv, T), dtype=torch.uint8, device=DEV)
    kl = torch.empty((B, Hkv), dtype=torch.int32, device=DEV)
    d.dkv_map_pattern_ragged(lay, torch.from_numpy(lens).to(DEV), torch.from_numpy(pattern).to(DEV), km, kl)
    _, okm, okl = o.map_pattern(pattern, T, w.sink, w.recent, w.bin_edges, Hkv, unit_len=lens)
    np.testing.assert_array_equal(kl.cpu().numpy(), okl)
    rows = int((kl.cpu().to(torch.int64) + cap).sum())
    k_c = torch.empty((rows, dim), dtype=torch.bfloat16, device=DEV)
    v_c = torch.empty_like(k_c)
    so = torch.empty(B * Hkv, dtype=torch.int64, device=DEV)
    sl = torch.empty(B * Hkv, dtype=torch.int32, device=DEV)
    cws = torch.empty(d.dkv_compact_workspace_bytes(lay), dtype=torch.uint8, device=DEV)
    d.dkv_compact(lay, k, v, km, cap, k_c, v_c, so, sl, cws)
    ref = o.compact(bits(k), bits(v), okm, cap)
    np.testing.assert_array_equal(so.cpu().numpy(), ref["seg_off"])
    ws = torch.zeros(d.dkv_decode_workspace_bytes(B, Hq, Hkv, dim), dtype=torch.uint8, device=DEV)
    out = torch.empty((B, Hq, dim), dtype=torch.float32, device=DEV)
    steps = w.decode_steps
    outs, news = {}, []
    hint = int(kl.sum())
    for s in range(steps):
        q = di.q_step(w, 0, s, device=DEV)
        kn, vn = di.kv_new_step(w, 0, s, device=DEV)
        news.append((bits(kn), bits(vn)))
        d.dkv_append_decode_attn(q, kn.reshape(B * Hkv, 1, dim).contiguous(), vn.reshape(B * Hkv, 1, dim).contiguous(),
                                 s, cap, k_c, v_c, so, sl, w.sm_scale, out, ws, Hkv, rows_hint=hint + B * Hkv * (s + 1))
        if s in (0, steps - 1):
            outs[s] = out.clone()
    torch.cuda.synchronize()
    kn_all = np.concatenate([a for a, _ in news], axis=2)
    vn_all = np.concatenate([b_ for _, b_ in news], axis=2)
    kc_all, vc_all = o.append(ref["k_c"], ref["v_c"], ref["seg_off"], ref["seg_len"], kn_all, vn_all, 0)
    np.testing.assert_array_equal(bits(k_c), kc_all)
    for s, got in outs.items():
        q = bits(di.q_step(w, 0, s, device=DEV))
        want = o.decode_attn(q, kc_all, vc_all, ref["seg_off"], ref["seg_len"], s + 1, w.sm_scale, Hkv, o.BF16)
        assert row_rel_err(got.cpu().numpy(), want) <= ATTN_TOL, s
