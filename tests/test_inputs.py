"""Checks of the seeded workload generators (host only)."""

import numpy as np
import pytest
import torch

import dkv_inputs as di
import oracle as o


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(20000).astype(np.float32) * 10.0 ** rng.integers(-8, 8, 20000),
                        np.array([1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8, -(1.0 + 2.0 ** -8)], np.float32)])
    x = x.astype(np.float32)
    got = di.f32_to_bf16_bits(x)
    want = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(got, want)


@pytest.mark.parametrize("span,D", [(32768, 24), (129920, 32), (1000, 6)])
def test_log_bin_edges(span, D):
    e = di.log_bin_edges(span, D)
    assert e[0] == 0 and e[1] == 128 and e[-1] == span and len(e) == D + 1
    assert all(b > a for a, b in zip(e, e[1:]))


def test_seeds_are_distinct_and_stable():
    s = {di.seed_of(c, u, st) for c in range(3) for u in range(10) for st in range(6)}
    assert len(s) == 180
    assert di.seed_of(3, 1, 2) == di.seed_of(3, 1, 2)


@pytest.mark.parametrize("name", [n for n, w in di.WORKLOADS.items() if w.family != "topk"])
def test_pattern_budget_and_union_structure(name):
    w = di.WORKLOADS[name]
    for b in (w.budgets or (None,)):
        pat, info = di.make_pattern(w, budget=b)
        assert pat.shape == (w.num_units, w.num_q_heads, w.num_bins)
        assert set(np.unique(pat)) <= {0, 1}
        L = o.closed_form_lengths(pat, w.context_len, w.sink, w.recent, w.bin_edges,
                                  w.num_kv_heads)
        frac = L.sum() / (w.num_units * w.num_kv_heads * w.context_len)
        if info["target"] is not None:
            # the generator's own bookkeeping agrees with the oracle's count
            assert abs(frac - info["achieved"]) < 1e-12
            # and the target is hit within the bin granularity
            assert abs(frac - info["target"]) < 0.01
        for k in w.always_keep_bins:
            assert pat[:, :, k].all()


def test_pattern_is_deterministic():
    w = di.WORKLOADS["llama8b_layer_32k"]
    a, _ = di.make_pattern(w)
    b, _ = di.make_pattern(w)
    np.testing.assert_array_equal(a, b)


def test_recent_only_groups_exist_in_batched_workload():
    w = di.WORKLOADS["llama70b_layer_bs16_32k"]
    pat, _ = di.make_pattern(w, budget=0.2)
    L = o.closed_form_lengths(pat, w.context_len, w.sink, w.recent, w.bin_edges, w.num_kv_heads)
    assert (L == 128).sum() >= 0.1 * L.size


def test_tensor_generators_shapes_and_seeding():
    w = di.workload("tiny")
    k1, v1 = di.kv_unit(w, 0)
    k2, _ = di.kv_unit(w, 0)
    assert k1.shape == (2, 1024, 64) and k1.dtype == torch.float32
    assert torch.equal(k1, k2) and not torch.equal(k1, v1)
    q = di.q_step(w, 0, 0)
    assert q.shape == (1, 4, 64)
    kn, vn = di.kv_new_step(w, 0, 3, n_new=2)
    assert kn.shape == (1, 2, 2, 64)


def test_topk_workload_pattern_is_not_an_input_recipe():
    with pytest.raises(ValueError):
        di.make_pattern(di.workload("llama8b_stack_128k_paper_bins"))


def test_retention_probs_range_ties_and_seeding():
    p = di.retention_probs(4, 8, 2, 50, seed=3)
    assert p.dtype == np.float32 and p.shape == (4, 8, 50)
    assert p.min() >= 0.001 and p.max() <= 0.999
    assert len(np.unique(p)) < p.size // 2          # quantised: many exact ties
    np.testing.assert_array_equal(p, di.retention_probs(4, 8, 2, 50, seed=3))
    assert not np.array_equal(p, di.retention_probs(4, 8, 2, 50, seed=4))


def test_paper_bins_workload_retention():
    """The exact-budget export at rho = 0.2 over the stand-in probabilities
    gives a physical retention near the paper's 34.6% at 128K."""
    w = di.workload("llama8b_stack_128k_paper_bins")
    assert w.num_bins == 1015 and w.bin_edges[1] == 128
    p = di.retention_probs(w.num_layers, w.num_q_heads, w.num_kv_heads, w.num_bins, seed=w.cfg_id)
    m = o.topk_mask(p, o.budget_entries(w.rho, w.num_layers, w.num_q_heads, w.num_bins))
    rep = o.retention_report(m, w.context_len, w.sink, w.recent, w.bin_edges, w.num_kv_heads)
    assert rep["logical"] == pytest.approx(0.2, abs=1e-6)
    assert 0.30 < rep["physical"] < 0.40


def _cells(pat, n_kv):
    N, H, D = pat.shape
    return (pat.reshape(N, n_kv, H // n_kv, D) != 0).any(axis=2)


@pytest.mark.parametrize("kind", di.PATTERN_FAMILIES)
def test_pattern_families_structure_and_cost(kind):
    rng = np.random.default_rng(9)
    N, H, n_kv, D = 3, 8, 2, 40
    base = (rng.uniform(size=(N, H, D)) < 0.25).astype(np.uint8)
    f = di.pattern_family(base, kind, n_kv, seed=1)
    assert f.shape == base.shape and f.dtype == np.uint8 and set(np.unique(f)) <= {0, 1}
    np.testing.assert_array_equal(f, di.pattern_family(base, kind, n_kv, seed=1))
    cb, cf = _cells(base, n_kv), _cells(f, n_kv)
    G = H // n_kv
    if kind == "head_only":
        assert all(f[n, h].all() or not f[n, h].any() for n in range(N) for h in range(H))
        assert abs(int(cf.sum()) - int(cb.sum())) <= D // 2
    elif kind == "distance_only":
        assert all((f[n] == f[n, 0]).all() for n in range(N))
        for n in range(N):
            assert abs(int(cf[n].sum()) - int(cb[n].sum())) <= n_kv // 2 + n_kv
    elif kind == "distance_shuffled":
        np.testing.assert_array_equal(f.sum(axis=2), base.sum(axis=2))        # per-head counts
        np.testing.assert_array_equal(cf.sum(axis=2), cb.sum(axis=2))        # per-group cells
        # the same permutation for every head of a group
        for n in range(N):
            for g in range(n_kv):
                hb = base[n, g * G:(g + 1) * G]
                hf = f[n, g * G:(g + 1) * G]
                assert sorted(map(tuple, hb.T.tolist())) == sorted(map(tuple, hf.T.tolist()))
    else:
        assert int(f.sum()) == int(base.sum()) and int(cf.sum()) == int(cb.sum())
        assert not np.array_equal(f, base)
