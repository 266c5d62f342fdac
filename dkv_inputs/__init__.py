"""Seeded synthetic workloads for the Distance-KV hot path.

This module only makes inputs: bin layouts, binary retention patterns and
K/V/q tensors with the shapes, value distributions and raggedness of the
workloads the method is measured on.  It performs none of the method's own
arithmetic (no position-to-bin mapping, no keep masks, no union over query
heads, no packing, no attention), so it can feed the oracle and the HIP
library alike without coupling them.

Stand-ins: the paper measures on NIAH, LongBench, RULER and SCBench prompts
with trained Llama / Qwen weights.  None of that is used here.  The cost of
the hot path depends only on shapes, retained counts and how ragged the
per-head lengths are, so K, V and q are i.i.d. Gaussian and the retention
patterns are drawn to hit the stated budgets.

Pattern recipe (the same for every workload): each (unit, KV head) group
first gets a physical keep decision per distance bin, chosen by a global
threshold on a per-(unit, group, bin) key so that the token-weighted
fraction of kept positions, sink and recent included, comes as close as the
bin granularity allows to the workload's budget.  Each kept group bin is then
given to a random non-empty subset of the group's query heads, and a dropped
group bin to none of them, so the query-head pattern's GQA union is the
group decision by construction.  Bins a workload always keeps (the most
recent 128-token bin when sink and recent are zero) are kept by every query
head.
"""

from dataclasses import dataclass, field
import math

import numpy as np

__all__ = [
    "Workload",
    "WORKLOADS",
    "workload",
    "seed_of",
    "f32_to_bf16_bits",
    "uniform_bin_edges",
    "log_bin_edges",
    "make_pattern",
    "bin_widths",
    "kv_unit",
    "q_step",
    "kv_new_step",
    "query_block",
    "page_table",
    "fill_pages",
    "retention_probs",
    "PATTERN_FAMILIES",
    "pattern_family",
    "sequence_lengths",
]

# stream ids of the seed derivation
STREAM_PATTERN, STREAM_K, STREAM_V, STREAM_Q, STREAM_NEW_K, STREAM_NEW_V = range(6)
STREAM_BLOCK_Q, STREAM_BLOCK_K, STREAM_BLOCK_V = 6, 7, 8
STREAM_PAGES = 9
STREAM_PROBS, STREAM_FAMILY = 10, 11
STREAM_LENGTHS = 12


def seed_of(*parts):
    """64-bit seed from a tuple of small non-negative integers."""
    ss = np.random.SeedSequence([int(p) for p in parts])
    return int(ss.generate_state(1, dtype=np.uint64)[0] & np.uint64(0x7FFFFFFFFFFFFFFF))


def f32_to_bf16_bits(x):
    """Round float32 values to bf16 (round to nearest, ties to even).

    Returns the uint16 bit patterns.  Inputs are finite.
    """
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    lsb = (b >> np.uint64(16)) & np.uint64(1)
    r = (b + np.uint64(0x7FFF) + lsb) >> np.uint64(16)
    return r.astype(np.uint16)


def uniform_bin_edges(width, num_bins):
    """Edges E[k] = width * k, k = 0..D (the paper's 128-token layout)."""
    return tuple(int(width) * k for k in range(num_bins + 1))


def log_bin_edges(span, num_bins, first=128):
    """Log-spaced edges over a compressible span.

    E[0] = 0, E[1] = first and E[k] = round(first * (span/first)^((k-1)/(D-1)))
    for k = 1..D, so E[D] = span.  Raises if the rounding makes two edges
    equal.
    """
    if num_bins < 2:
        raise ValueError("need at least two bins")
    e = [0]
    ratio = span / first
    for k in range(1, num_bins + 1):
        e.append(int(round(first * ratio ** ((k - 1) / (num_bins - 1)))))
    for a, b in zip(e, e[1:]):
        if not b > a:
            raise ValueError("log-spaced edges are not strictly increasing")
    return tuple(e)


def bin_widths(bin_edges, span):
    """Token width of each bin clipped to a compressible span (input design)."""
    e = list(bin_edges)
    return np.array([max(0, min(e[k + 1], span) - e[k]) for k in range(len(e) - 1)],
                    dtype=np.int64)


@dataclass(frozen=True)
class Workload:
    """Shape, dtype and pattern recipe of one synthetic workload."""

    name: str
    cfg_id: int
    num_layers: int
    batch: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    context_len: int
    sink: int
    recent: int
    bin_edges: tuple
    dtype: str                    # "bf16" or "f32"
    sm_scale: float
    q_std: float
    budget: float = None          # physical retained fraction; None: Bernoulli rate
    keep_prob: float = None       # plain Bernoulli(p) per (q head, bin) when budget is None
    family: str = "bernoulli"     # "bernoulli", "mixture" or "topk" (exact-budget export)
    always_keep_bins: tuple = ()  # bins kept by every query head
    recent_only_frac: float = 0.0  # fraction of groups that keep only always_keep_bins
    decode_steps: int = 1
    append_cap: int = 16
    budgets: tuple = field(default=())  # extra budgets measured on the same shape
    rho: float = None             # logical retention ratio of a "topk" workload

    @property
    def num_units(self):
        return self.num_layers * self.batch

    @property
    def group(self):
        return self.num_q_heads // self.num_kv_heads

    @property
    def num_bins(self):
        return len(self.bin_edges) - 1

    @property
    def elem_bytes(self):
        return 2 if self.dtype == "bf16" else 4

    def unit(self, layer, seq):
        """Units are layer-major: unit = layer * batch + seq."""
        return layer * self.batch + seq


_SPAN_8B = 131072 - 128 - 1024

WORKLOADS = {
    "tiny": Workload(
        name="tiny", cfg_id=1, num_layers=1, batch=1, num_q_heads=4, num_kv_heads=2,
        head_dim=64, context_len=1024, sink=0, recent=0,
        bin_edges=uniform_bin_edges(64, 16), dtype="f32", sm_scale=1.0 / 8.0,
        q_std=1.0, keep_prob=0.35, decode_steps=1, append_cap=16),
    "llama8b_layer_32k": Workload(
        name="llama8b_layer_32k", cfg_id=2, num_layers=1, batch=1, num_q_heads=32,
        num_kv_heads=8, head_dim=128, context_len=32768, sink=0, recent=0,
        bin_edges=log_bin_edges(32768, 24), dtype="bf16", sm_scale=1.0,
        q_std=1.0 / math.sqrt(128), budget=0.35, always_keep_bins=(0,),
        decode_steps=1, append_cap=16),
    "llama8b_stack_128k": Workload(
        name="llama8b_stack_128k", cfg_id=3, num_layers=32, batch=1, num_q_heads=32,
        num_kv_heads=8, head_dim=128, context_len=131072, sink=128, recent=1024,
        bin_edges=log_bin_edges(_SPAN_8B, 32), dtype="bf16", sm_scale=1.0,
        q_std=1.0 / math.sqrt(128), budget=0.346, decode_steps=64, append_cap=64),
    "llama70b_layer_bs16_32k": Workload(
        name="llama70b_layer_bs16_32k", cfg_id=4, num_layers=1, batch=16, num_q_heads=64,
        num_kv_heads=8, head_dim=128, context_len=32768, sink=0, recent=0,
        bin_edges=log_bin_edges(32768, 24), dtype="bf16", sm_scale=1.0,
        q_std=1.0 / math.sqrt(128), budget=0.20, always_keep_bins=(0,),
        recent_only_frac=0.2, decode_steps=16, append_cap=16, budgets=(0.10, 0.20, 0.50)),
    "llama8b_stack_128k_paper_bins": Workload(
        name="llama8b_stack_128k_paper_bins", cfg_id=6, num_layers=32, batch=1, num_q_heads=32,
        num_kv_heads=8, head_dim=128, context_len=131072, sink=128, recent=1024,
        bin_edges=uniform_bin_edges(128, (131072 - 128 - 1024) // 128), dtype="bf16", sm_scale=1.0,
        q_std=1.0 / math.sqrt(128), family="topk", rho=0.2, decode_steps=64, append_cap=64),
    "qwen7b_stack_bs4_128k": Workload(
        name="qwen7b_stack_bs4_128k", cfg_id=5, num_layers=28, batch=4, num_q_heads=28,
        num_kv_heads=4, head_dim=128, context_len=131072, sink=128, recent=1024,
        bin_edges=log_bin_edges(_SPAN_8B, 32), dtype="bf16", sm_scale=1.0,
        q_std=1.0 / math.sqrt(128), budget=0.25, family="mixture",
        decode_steps=256, append_cap=256),
}


def workload(name, **overrides):
    """A named workload, optionally with fields replaced (for scaled-down tests)."""
    import dataclasses
    w = WORKLOADS[name]
    return dataclasses.replace(w, **overrides) if overrides else w


# ---------------------------------------------------------------------------
# retention patterns
# ---------------------------------------------------------------------------

def _group_keys(w, rng_of_unit, rates):
    """Per-(unit, group, bin) threshold keys; smaller keys are kept first."""
    N, Hkv, D = w.num_units, w.num_kv_heads, w.num_bins
    G = w.group
    keys = np.empty((N, Hkv, D), dtype=np.float64)
    for n in range(N):
        rng = rng_of_unit(n)
        if w.family == "mixture":
            fam = rng.integers(0, 3, size=Hkv)
            z = rng.uniform(0.5, 1.5, size=Hkv)
            for g in range(Hkv):
                if fam[g] == 0:        # near-only: nearest bins first
                    order = list(range(D))
                elif fam[g] == 1:      # far-only: farthest bins first
                    order = list(range(D - 1, -1, -1))
                else:                  # bimodal: alternate near and far
                    order = []
                    lo, hi = 0, D - 1
                    while lo <= hi:
                        order.append(lo)
                        if hi != lo:
                            order.append(hi)
                        lo, hi = lo + 1, hi - 1
                for rank, k in enumerate(order):
                    keys[n, g, k] = (rank + 1) / z[g]
        else:
            v = rng.uniform(0.0, 1.0, size=(Hkv, D))
            for g in range(Hkv):
                r = rates[n, g * G:(g + 1) * G]
                group_rate = 1.0 - np.prod(1.0 - r)
                keys[n, g] = v[g] / group_rate
    return keys


def make_pattern(w, budget=None, all_keep=False):
    """Binary pattern uint8 [N][Hq][D] for a workload (see module docstring).

    Returns (pattern, info) where info records the recipe's achieved physical
    fraction as seen by the generator's own accounting.
    """
    N, Hq, Hkv, D = w.num_units, w.num_q_heads, w.num_kv_heads, w.num_bins
    G = w.group
    if all_keep:
        return np.ones((N, Hq, D), dtype=np.uint8), {"target": 1.0}
    if w.family == "topk":
        raise ValueError(f"{w.name}: the pattern is the exact-budget export of retention_probs "
                         "(dkv_topk_pattern, or the oracle's topk_mask), not an input recipe")

    def rng_of_unit(n, sub=0):
        return np.random.default_rng(seed_of(w.cfg_id, n, STREAM_PATTERN, sub))

    if budget is None and w.budget is None:
        # plain Bernoulli(keep_prob) per (query head, bin)
        pat = np.zeros((N, Hq, D), dtype=np.uint8)
        for n in range(N):
            pat[n] = (rng_of_unit(n).uniform(size=(Hq, D)) < w.keep_prob).astype(np.uint8)
        for k in w.always_keep_bins:
            pat[:, :, k] = 1
        return pat, {"target": None, "keep_prob": w.keep_prob}

    target = w.budget if budget is None else budget
    rates = np.stack([rng_of_unit(n, 1).uniform(0.1, 0.7, size=Hq) for n in range(N)])
    keys = _group_keys(w, rng_of_unit, rates)

    T = w.context_len
    span = max(0, T - w.sink - w.recent)
    width = bin_widths(w.bin_edges, span)
    forced = np.zeros((N, Hkv, D), dtype=bool)
    for k in w.always_keep_bins:
        forced[:, :, k] = True
    banned = np.zeros((N, Hkv, D), dtype=bool)
    if w.recent_only_frac > 0:
        for n in range(N):
            sel = rng_of_unit(n, 2).uniform(size=Hkv) < w.recent_only_frac
            banned[n, sel, :] = True
    banned &= ~forced

    total = N * Hkv * T
    base = N * Hkv * min(T, w.sink + w.recent) + int((forced * width).sum())
    want = target * total - base
    free = ~(forced | banned)
    k_flat = keys[free]
    w_flat = np.broadcast_to(width, keys.shape)[free]
    order = np.argsort(k_flat, kind="stable")
    ks = k_flat[order]
    cum = np.concatenate([[0], np.cumsum(w_flat[order])])
    # candidate cut points: only between distinct key values
    cuts = [0] + [i for i in range(1, len(ks) + 1) if i == len(ks) or ks[i] != ks[i - 1]]
    best = min(cuts, key=lambda i: abs(cum[i] - want))
    thresh = ks[best - 1] if best > 0 else -np.inf
    group_keep = forced | (free & (keys <= thresh))

    pat = np.zeros((N, Hq, D), dtype=np.uint8)
    for n in range(N):
        rng = rng_of_unit(n, 3)
        x = rng.uniform(size=(Hq, D))
        for g in range(Hkv):
            hs = slice(g * G, (g + 1) * G)
            r = rates[n, hs]
            for k in range(D):
                if forced[n, g, k]:
                    pat[n, hs, k] = 1
                elif group_keep[n, g, k]:
                    pick = (x[hs, k] < r)
                    if not pick.any():
                        pick[np.argmin(x[hs, k] / r)] = True
                    pat[n, hs, k] = pick.astype(np.uint8)
    achieved = (base + ((group_keep & free) * width).sum()) / total
    return pat, {"target": target, "achieved": float(achieved)}


# ---------------------------------------------------------------------------
# K / V / q tensors (torch generators: fast on the GPU at 16 GiB scale)
# ---------------------------------------------------------------------------

def _torch_dtype(w):
    import torch
    return torch.bfloat16 if w.dtype == "bf16" else torch.float32


def _randn(shape, seed, device, std, dtype):
    import torch
    gen = torch.Generator(device=device)
    gen.manual_seed(seed)
    x = torch.randn(shape, generator=gen, device=device, dtype=torch.float32)
    if std != 1.0:
        x.mul_(std)
    return x.to(dtype)


def kv_unit(w, unit, device="cpu"):
    """Dense K and V of one unit: two tensors [Hkv][T][d], N(0, 1)."""
    shape = (w.num_kv_heads, w.context_len, w.head_dim)
    dt = _torch_dtype(w)
    k = _randn(shape, seed_of(w.cfg_id, unit, STREAM_K), device, 1.0, dt)
    v = _randn(shape, seed_of(w.cfg_id, unit, STREAM_V), device, 1.0, dt)
    return k, v


def q_step(w, layer, step, device="cpu"):
    """Decode queries of one layer at one step: [B][Hq][d], N(0, q_std^2)."""
    shape = (w.batch, w.num_q_heads, w.head_dim)
    return _randn(shape, seed_of(w.cfg_id, layer, STREAM_Q, step), device, w.q_std,
                  _torch_dtype(w))


def kv_new_step(w, layer, step, n_new=1, device="cpu"):
    """K/V of the n_new tokens appended at a step: [B][Hkv][n_new][d]."""
    shape = (w.batch, w.num_kv_heads, n_new, w.head_dim)
    dt = _torch_dtype(w)
    k = _randn(shape, seed_of(w.cfg_id, layer, STREAM_NEW_K, step), device, 1.0, dt)
    v = _randn(shape, seed_of(w.cfg_id, layer, STREAM_NEW_V, step), device, 1.0, dt)
    return k, v


def query_block(w, layer, n_q, device="cpu"):
    """The n_q query tokens after the context (the question), one layer:
    q [B][n_q][Hq][d] ~ N(0, q_std^2), token-major, and the block's own
    K, V [B][Hkv][n_q][d] ~ N(0, 1), which are appended to the cache."""
    dt = _torch_dtype(w)
    q = _randn((w.batch, n_q, w.num_q_heads, w.head_dim), seed_of(w.cfg_id, layer, STREAM_BLOCK_Q, n_q),
               device, w.q_std, dt)
    shape = (w.batch, w.num_kv_heads, n_q, w.head_dim)
    k = _randn(shape, seed_of(w.cfg_id, layer, STREAM_BLOCK_K, n_q), device, 1.0, dt)
    v = _randn(shape, seed_of(w.cfg_id, layer, STREAM_BLOCK_V, n_q), device, 1.0, dt)
    return q, k, v


# ---------------------------------------------------------------------------
# paged caches (the layout a page allocator leaves behind after prefill)
# ---------------------------------------------------------------------------

def page_table(num_segments, pages_per_segment, seed, spare=0):
    """Physical page of every (segment, logical page): the first
    num_segments * pages_per_segment values of a seeded permutation of
    range(num_pages), num_pages = that product + spare, as an allocator that
    hands out pages in no particular order would leave them.
    Returns (int32 [num_segments][pages_per_segment], num_pages)."""
    n = num_segments * pages_per_segment
    num_pages = n + int(spare)
    perm = np.random.default_rng(seed_of(STREAM_PAGES, seed)).permutation(num_pages)[:n]
    return perm.reshape(num_segments, pages_per_segment).astype(np.int32), num_pages


def fill_pages(pool, x, table, page_rows):
    """Store dense per-segment rows in their pages: page table[s][p] of `pool`
    ([num_pages][page_rows][...], numpy or torch) receives rows
    [p * page_rows, (p + 1) * page_rows) of x[s] (x: [n][rows][...], n =
    len(table)); slots past the end of x's rows are left as they are."""
    table = np.asarray(table)
    n, rows = x.shape[0], x.shape[1]
    full = min(rows // page_rows, table.shape[1])
    rest = tuple(x.shape[2:])
    is_torch = not isinstance(pool, np.ndarray)
    if full > 0:
        idx = table[:, :full].reshape(-1)
        src = x[:, :full * page_rows].reshape((n * full, page_rows) + rest)
        if is_torch:
            import torch
            pool[torch.as_tensor(idx, dtype=torch.long, device=pool.device)] = src
        else:
            pool[idx] = src
    r0 = full * page_rows
    if r0 < rows and full < table.shape[1]:
        for s in range(n):
            pool[int(table[s, full]), :rows - r0] = x[s, r0:rows]


# ---------------------------------------------------------------------------
# retention probabilities and the ablation pattern families
# ---------------------------------------------------------------------------

def retention_probs(num_layers, num_q_heads, num_kv_heads, num_bins, seed, group_weight=1.5):
    """Stand-in for learned gate probabilities p[layer][query head][bin] in
    [0.001, 0.999] (the clip range of the paper's gates), float32.

    Each (layer, KV group) draws a distance profile -- near-favouring,
    far-favouring or bimodal, with random strength -- shared by its query
    heads with weight `group_weight`; each query head adds its own noise, so
    heads of a group agree more than independent heads would (the union then
    keeps fewer positions).  Probabilities are quantised to steps of 1/1024,
    so exact ties occur.
    """
    rng = np.random.default_rng(seed_of(STREAM_PROBS, seed))
    L, H, Hkv, D = int(num_layers), int(num_q_heads), int(num_kv_heads), int(num_bins)
    G = H // Hkv
    x = np.arange(D, dtype=np.float64) / max(D - 1, 1)
    prof = np.empty((L, Hkv, D))
    for layer in range(L):
        for g in range(Hkv):
            kind = rng.integers(3)
            a = rng.uniform(2.0, 8.0)
            if kind == 0:
                prof[layer, g] = -a * x
            elif kind == 1:
                prof[layer, g] = -a * (1.0 - x)
            else:
                prof[layer, g] = -a * np.minimum(x, 1.0 - x) * 2.0
            prof[layer, g] += rng.normal(0.0, 0.5, size=D)
    logits = group_weight * np.repeat(prof, G, axis=1) + rng.normal(0.0, 1.0, size=(L, H, D))
    p = 1.0 / (1.0 + np.exp(-logits))
    p = np.clip(np.round(p * 1024.0) / 1024.0, 0.001, 0.999)
    return p.astype(np.float32)


PATTERN_FAMILIES = ("head_only", "distance_only", "distance_shuffled", "fully_shuffled")


def pattern_family(base, kind, num_kv_heads, seed):
    """Structural variants of a pattern [N][Hq][D], built to keep its physical
    cost (the number of (unit, KV group, bin) cells some query head of the
    group keeps) when bins have equal widths -- the controls of the paper's
    ablation (Sec. 4.4; Appendix, task-level ablation):

    head_only          each query head keeps all of its bins or none: the
                       groups with the most kept cells keep every bin, with
                       the heads that kept anything (n_keep = round(cells/D));
    distance_only      one bin set per unit shared by all query heads: the
                       round(cells_n / Hkv) bins the most groups keep (ties to
                       the lower bin);
    distance_shuffled  one random bin permutation per (unit, group), applied
                       to all its heads: per-head counts and the group's cell
                       count are kept, the distances are not;
    fully_shuffled     the (unit, group, bin) cells, each the G-bit vector of
                       the group's heads, are permuted over all units, groups
                       and bins, and each vector's bits among its heads:
                       logical entries and kept cells are kept, nothing else.
    """
    base = np.asarray(base, dtype=np.uint8) != 0
    N, H, D = base.shape
    Hkv = int(num_kv_heads)
    G = H // Hkv
    rng = np.random.default_rng(seed_of(STREAM_FAMILY, PATTERN_FAMILIES.index(kind), seed))
    cells = base.reshape(N, Hkv, G, D)            # [unit][group][head in group][bin]
    kept = cells.any(axis=2)                      # [unit][group][bin]
    out = np.zeros((N, Hkv, G, D), dtype=bool)
    if kind == "head_only":
        n_keep = int(round(kept.sum() / float(D)))
        score = kept.sum(axis=2).reshape(-1)      # cells per (unit, group)
        order = np.lexsort((np.arange(score.size), -score))[:n_keep]
        heads = cells.any(axis=3).reshape(N * Hkv, G)
        flat = out.reshape(N * Hkv, G, D)
        for c in order:
            who = heads[c] if heads[c].any() else np.eye(G, dtype=bool)[0]
            flat[c, who, :] = True
    elif kind == "distance_only":
        for n in range(N):
            c = int(round(kept[n].sum() / float(Hkv)))
            votes = kept[n].sum(axis=0)           # groups keeping each bin
            bins = np.lexsort((np.arange(D), -votes))[:c]
            out[n, :, :, bins] = True
    elif kind == "distance_shuffled":
        for n in range(N):
            for g in range(Hkv):
                out[n, g] = cells[n, g][:, rng.permutation(D)]
    elif kind == "fully_shuffled":
        vec = cells.transpose(0, 1, 3, 2).reshape(-1, G)   # one G-bit vector per cell
        vec = vec[rng.permutation(vec.shape[0])]
        vec = np.array([v[rng.permutation(G)] for v in vec])
        out = vec.reshape(N, Hkv, D, G).transpose(0, 1, 3, 2)
    else:
        raise ValueError(f"unknown pattern family {kind!r}")
    return np.ascontiguousarray(out.reshape(N, H, D)).astype(np.uint8)


def sequence_lengths(w, seed=0, shortest=0.125):
    """Context length of every unit for a ragged batch: sequence b draws T_b
    uniformly from [shortest * T, T] (T = the workload's context length) and
    every layer of that sequence shares it (units are layer-major), int32 [N].
    The longest sequence is always T."""
    rng = np.random.default_rng(seed_of(STREAM_LENGTHS, w.cfg_id, seed))
    T = int(w.context_len)
    per_seq = rng.integers(int(shortest * T), T + 1, size=w.batch)
    per_seq[int(rng.integers(w.batch))] = T
    return np.tile(per_seq, w.num_layers).astype(np.int32)
