"""CPU oracle for the Distance-KV inference hot path.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import, call or
execute this module: it is used by the tests, by the package's smoke check and
by the benchmark's CPU-baseline leg, and by nothing else.  It shares no code
with the HIP library and imports nothing from it.

What it computes (Distance-KV, Sec. 3.4 "Static-Pattern Inference"):

* the distance bin of a context position, Eq. (4), and the per-query-head
  retention decision, Eq. (5): sink and recent positions are always kept, the
  learned pattern decides every other position through its bin;
* the union over the query heads that share one KV head (last paragraph of
  Sec. 3.4), which gives the physical per-KV-head keep mask;
* the one-time prune-and-pack of the KV cache, which keeps retained rows in
  their original token order (Sec. 3.4, Fig. 2(b));
* the append of new tokens, which are always retained (Sec. 3.4);
* attention of the query block (the tokens after the context, Sec. 3.4):
  each query token attends to the packed context, the tokens appended before
  the block, and causally to the block's own tokens, which are appended like
  any new token;
* decode attention over the packed cache.  Attention restricted to a fixed
  retained set is exactly dense attention with every other position masked to
  -inf, so the oracle writes out that plain definition twice, once over the
  packed rows and once over the dense cache with a mask;
* the exact-budget export of a pattern from retention probabilities (Sec. 3.3,
  Eq. (topk-pattern) and Appendix A's exact-budget refinement): K = round(rho L H D)
  entries, the K largest probabilities, kept; and the logical (pattern entries)
  against physical (retained positions after the union) retention report of
  Sec. 3.4 and the experimental setup;
* the zero-copy alternative to the pack: the retained set of a segment is a
  union of contiguous distance bins plus the sink and the recent window
  (Eq. (4), Eq. (5), union of Sec. 3.4), so in a cache kept in fixed pages of
  consecutive positions it can be listed in place as runs within pages, and
  decode can read those rows where they are.  The oracle lists the runs from
  their definition and attends to exactly the rows they name.

Everything is plain NumPy in float64; bf16 inputs are carried as their uint16
bit patterns and widened exactly.  Loops are over segments and heads only, so
the code can be read against the equations line by line; it is slow on
purpose.

Readings of points the paper leaves open (the same list is kept with the
design notes):

* positions are 0-indexed, j = i - 1.  The distance of position j from the
  end of a context of length T is delta = T - 1 - j, the sink is j < S, the
  recent window is delta < R, and the compressible offset is
  u = delta - R.  With S = 128, R = 1024 and 128-token bins, bin(u) =
  floor(u / 128) is Eq. (4) with i = j + 1;
* bins are given by edges E[0] = 0 < E[1] < ... < E[D] in units of u; a
  position whose u is not covered by any bin (u >= E[D]) is pruned;
* if T <= S + R every position is sink or recent and is kept;
* query head h belongs to KV head h // G with G = Hq / Hkv (contiguous GQA
  groups);
* every query head of a group attends to the union of the group's keep masks,
  i.e. to every row of the shared packed segment;
* appended tokens are attended after the packed context rows;
* the softmax scale is an explicit argument;
* an empty segment (no rows at all) produces a zero output.
"""

import math

import numpy as np

__all__ = [
    "BF16",
    "F32",
    "widen",
    "bin_index",
    "q_keep_mask",
    "kv_keep_mask",
    "map_pattern",
    "closed_form_lengths",
    "compact",
    "append",
    "decode_attn",
    "dense_decode_attn",
    "query_attn",
    "masked_dense_attn",
    "budget_entries",
    "topk_mask",
    "retention_report",
    "PAGE_ENTRY_FIELDS",
    "page_select",
    "paged_append",
    "paged_decode_attn",
]

BF16 = "bf16"
F32 = "f32"


def widen(x, dtype):
    """Exact float64 value of a bf16 (uint16 bits) or float32 array."""
    if dtype == BF16:
        x = np.asarray(x, dtype=np.uint16)
        return (x.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)
    if dtype == F32:
        return np.asarray(x, dtype=np.float32).astype(np.float64)
    raise ValueError(f"unknown dtype {dtype!r}")


# ---------------------------------------------------------------------------
# Eq. (4): distance bin of a compressible position
# ---------------------------------------------------------------------------

def bin_index(u, bin_edges):
    """Bin k with E[k] <= u < E[k+1] for every offset u, or -1 if none.

    Eq. (4) of Sec. 3.4 with the bin boundaries made explicit: u is the
    distance past the recent window, and bin k covers the half-open range
    [E[k], E[k+1]).  The paper's layout is E[k] = 128 k.  A library binary
    search stands in for the comparison against every edge.
    """
    e = np.asarray(bin_edges, dtype=np.int64)
    u = np.asarray(u, dtype=np.int64)
    k = np.searchsorted(e, u, side="right") - 1
    covered = (u >= e[0]) & (u < e[-1])
    return np.where(covered, k, -1)


# ---------------------------------------------------------------------------
# Eq. (5): retention decision of each query head at each position
# ---------------------------------------------------------------------------

def q_keep_mask(pattern, context_len, sink, recent, bin_edges, unit_len=None):
    """Logical keep mask m[n, h, j] (uint8), Eq. (5) of Sec. 3.4.

    pattern: uint8 [N][Hq][D], the binary Distance-KV pattern of Sec. 3.2.
    A position is kept if it is a sink position (j < S) or a recent position
    (delta < R); otherwise the pattern entry of its bin decides, and a
    position that no bin covers is dropped.

    unit_len (optional, [N]): a batch of contexts of different lengths.
    Unit n's context is its first unit_len[n] positions of the
    context_len-long rows; distances are measured from the end of that
    context, and the positions after it are not retained.
    """
    pattern = np.asarray(pattern, dtype=np.uint8)
    n_units, n_q, n_bins = pattern.shape
    assert len(bin_edges) == n_bins + 1
    T = int(context_len)
    lens = [T] * n_units if unit_len is None else [int(x) for x in unit_len]
    out = np.zeros((n_units, n_q, T), dtype=np.uint8)
    for n in range(n_units):
        Tn = lens[n]
        assert 0 <= Tn <= T
        j = np.arange(Tn, dtype=np.int64)
        delta = Tn - 1 - j
        always = (j < sink) | (delta < recent)
        u = delta - recent
        k = bin_index(np.maximum(u, 0), bin_edges)
        has_bin = (~always) & (k >= 0)
        for h in range(n_q):
            row = np.zeros(Tn, dtype=np.uint8)
            row[always] = 1
            row[has_bin] = pattern[n, h, k[has_bin]]
            out[n, h, :Tn] = row
    return out


def kv_keep_mask(q_mask, num_kv_heads):
    """Physical keep mask of each KV head: union over its query heads.

    Last paragraph of Sec. 3.4: for GQA a position is retained whenever any
    query head of the group selects it.  Query heads g*G .. g*G+G-1 share KV
    head g.
    """
    q_mask = np.asarray(q_mask, dtype=np.uint8)
    n_units, n_q, T = q_mask.shape
    assert n_q % num_kv_heads == 0
    G = n_q // num_kv_heads
    out = np.zeros((n_units, num_kv_heads, T), dtype=np.uint8)
    for n in range(n_units):
        for g in range(num_kv_heads):
            acc = np.zeros(T, dtype=np.uint8)
            for h in range(g * G, (g + 1) * G):
                acc = acc | q_mask[n, h]
            out[n, g] = acc
    return out


def map_pattern(pattern, context_len, sink, recent, bin_edges, num_kv_heads, unit_len=None):
    """Pattern -> (q_mask, kv_mask, kv_len): Eq. (5) then the GQA union.

    kv_len[n, g] is the number of retained positions of KV head g, the
    physical per-head cache length after pruning.  unit_len: as in
    q_keep_mask.
    """
    qm = q_keep_mask(pattern, context_len, sink, recent, bin_edges, unit_len)
    km = kv_keep_mask(qm, num_kv_heads)
    kv_len = km.sum(axis=2, dtype=np.int64).astype(np.int32)
    return qm, km, kv_len


def closed_form_lengths(pattern, context_len, sink, recent, bin_edges, num_kv_heads):
    """Per-KV-head retained length without building a mask.

    The always-kept part is |sink U recent| = min(T, S + R).  The
    compressible offsets are u in [0, T - S - R); bin k contributes its
    width clipped to that span, w_k = max(0, min(E[k+1], T-S-R) - E[k]),
    once for a KV head if any query head of its group keeps bin k.
    """
    pattern = np.asarray(pattern, dtype=np.uint8)
    n_units, n_q, n_bins = pattern.shape
    G = n_q // num_kv_heads
    T = int(context_len)
    span = max(0, T - sink - recent)
    e = [int(x) for x in bin_edges]
    width = [max(0, min(e[k + 1], span) - e[k]) for k in range(n_bins)]
    out = np.zeros((n_units, num_kv_heads), dtype=np.int64)
    for n in range(n_units):
        for g in range(num_kv_heads):
            total = min(T, sink + recent)
            for k in range(n_bins):
                if any(pattern[n, h, k] for h in range(g * G, (g + 1) * G)):
                    total += width[k]
            out[n, g] = total
    return out


# ---------------------------------------------------------------------------
# One-time prune and pack (Sec. 3.4, Fig. 2(b))
# ---------------------------------------------------------------------------

def compact(k, v, kv_mask, append_cap):
    """Pack the retained rows of every (unit, KV head) segment.

    k, v: [N][Hkv][T][d] arrays (bf16 bits or float32), kv_mask uint8
    [N][Hkv][T].  Segments are laid out unit-major then head; segment
    (n, g) starts at seg_off = sum over earlier segments of (len + cap)
    and holds its retained rows in original token order, followed by `cap`
    free rows for appended tokens.  Rows are copied unchanged, so the
    packed cache is bit-identical to the retained dense rows.

    Returns dict(k_c, v_c [rows][d] with free rows zero, seg_off int64
    [N*Hkv], seg_len int32 [N*Hkv], src_pos int32 [rows] with -1 in free
    rows, rows = total row count).
    """
    k = np.asarray(k)
    v = np.asarray(v)
    kv_mask = np.asarray(kv_mask, dtype=np.uint8)
    n_units, n_kv, T, d = k.shape
    n_seg = n_units * n_kv
    seg_off = np.zeros(n_seg, dtype=np.int64)
    seg_len = np.zeros(n_seg, dtype=np.int32)
    kept = []
    running = 0
    for n in range(n_units):
        for g in range(n_kv):
            s = n * n_kv + g
            pos = np.flatnonzero(kv_mask[n, g])
            kept.append(pos)
            seg_off[s] = running
            seg_len[s] = len(pos)
            running += len(pos) + int(append_cap)
    rows = running
    k_c = np.zeros((rows, d), dtype=k.dtype)
    v_c = np.zeros((rows, d), dtype=v.dtype)
    src_pos = np.full(rows, -1, dtype=np.int32)
    for n in range(n_units):
        for g in range(n_kv):
            s = n * n_kv + g
            pos = kept[s]
            o = int(seg_off[s])
            k_c[o:o + len(pos)] = k[n, g, pos]
            v_c[o:o + len(pos)] = v[n, g, pos]
            src_pos[o:o + len(pos)] = pos
    return dict(k_c=k_c, v_c=v_c, seg_off=seg_off, seg_len=seg_len,
                src_pos=src_pos, rows=rows)


def append(k_c, v_c, seg_off, seg_len, k_new, v_new, n_tail):
    """Write new tokens after the packed rows of every segment (Sec. 3.4).

    Appended tokens are retained in full.  k_new, v_new: [N][Hkv][n_new][d];
    token t of segment s goes to row seg_off[s] + seg_len[s] + n_tail + t.
    Returns updated copies of k_c and v_c.
    """
    k_c = np.array(k_c, copy=True)
    v_c = np.array(v_c, copy=True)
    n_units, n_kv, n_new, d = np.asarray(k_new).shape
    for n in range(n_units):
        for g in range(n_kv):
            s = n * n_kv + g
            base = int(seg_off[s]) + int(seg_len[s]) + int(n_tail)
            for t in range(n_new):
                k_c[base + t] = k_new[n, g, t]
                v_c[base + t] = v_new[n, g, t]
    return k_c, v_c


# ---------------------------------------------------------------------------
# Decode attention
# ---------------------------------------------------------------------------

def _softmax_attend(q_vec, k_rows, v_rows, sm_scale):
    """softmax(sm_scale * K q) V in float64; zeros when there is no row."""
    if k_rows.shape[0] == 0:
        return np.zeros(v_rows.shape[1], dtype=np.float64)
    s = sm_scale * (k_rows @ q_vec)
    s = s - s.max()
    p = np.exp(s)
    return (p @ v_rows) / p.sum()


def decode_attn(q, k_c, v_c, seg_off, seg_len, n_tail, sm_scale, num_kv_heads, dtype):
    """One decode step over the packed cache (Sec. 3.4; union of Sec. 3.4).

    q: [B][Hq][d]; segment s = b * Hkv + g holds rows
    [seg_off[s], seg_off[s] + seg_len[s] + n_tail): the packed context
    rows followed by the appended tokens.  Every query head of group g
    attends to all of them.  Returns float64 [B][Hq][d].
    """
    qf = widen(q, dtype)
    B, Hq, d = qf.shape
    G = Hq // num_kv_heads
    out = np.zeros((B, Hq, d), dtype=np.float64)
    for b in range(B):
        for g in range(num_kv_heads):
            s = b * num_kv_heads + g
            lo = int(seg_off[s])
            hi = lo + int(seg_len[s]) + int(n_tail)
            kr = widen(k_c[lo:hi], dtype)
            vr = widen(v_c[lo:hi], dtype)
            for h in range(g * G, (g + 1) * G):
                out[b, h] = _softmax_attend(qf[b, h], kr, vr, sm_scale)
    return out


def dense_decode_attn(q, k, v, n_valid, sm_scale, dtype):
    """Dense-cache decode (the comparator of Sec. 4.3): rows [0, n_valid).

    k, v: [B][Hkv][T_cap][d].  Returns float64 [B][Hq][d].
    """
    qf = widen(q, dtype)
    B, Hq, d = qf.shape
    n_kv = np.asarray(k).shape[1]
    G = Hq // n_kv
    out = np.zeros((B, Hq, d), dtype=np.float64)
    for b in range(B):
        for g in range(n_kv):
            kr = widen(k[b, g, :n_valid], dtype)
            vr = widen(v[b, g, :n_valid], dtype)
            for h in range(g * G, (g + 1) * G):
                out[b, h] = _softmax_attend(qf[b, h], kr, vr, sm_scale)
    return out


def query_attn(q, k_c, v_c, seg_off, seg_len, n_tail, sm_scale, num_kv_heads, dtype):
    """Attention of a query block over the packed cache (Sec. 3.4).

    After the one-time compaction the query tokens attend to the compressed
    context; their own K/V are appended like every new token and kept.
    q: [B][n_q][Hq][d], token-major; the block's K/V must already sit in the
    segment's rows [seg_len + n_tail, seg_len + n_tail + n_q) (after the
    packed context and the n_tail tokens appended before the block).  Query
    token i attends to rows [seg_off, seg_off + seg_len + n_tail + i + 1): the
    context, the earlier appended tokens, and the block causally up to
    itself.  Every query head of group g attends to segment b * Hkv + g.
    Returns float64 [B][n_q][Hq][d].
    """
    qf = widen(q, dtype)
    B, n_q, Hq, d = qf.shape
    G = Hq // num_kv_heads
    out = np.zeros((B, n_q, Hq, d), dtype=np.float64)
    for b in range(B):
        for g in range(num_kv_heads):
            s = b * num_kv_heads + g
            lo = int(seg_off[s])
            base = int(seg_len[s]) + int(n_tail)
            kr = widen(k_c[lo:lo + base + n_q], dtype)
            vr = widen(v_c[lo:lo + base + n_q], dtype)
            for i in range(n_q):
                for h in range(g * G, (g + 1) * G):
                    out[b, i, h] = _softmax_attend(qf[b, i, h], kr[:base + i + 1], vr[:base + i + 1],
                                                   sm_scale)
    return out


def masked_dense_attn(q, k, v, kv_mask, k_tail, v_tail, sm_scale, dtype):
    """Second, independent decode path: dense attention with pruned -> -inf.

    Scores are taken against every dense position of the KV head; positions
    with kv_mask = 0 get -inf before the softmax.  The appended tokens
    k_tail, v_tail ([B][Hkv][n_tail][d]) are always attended.  Equal to
    `decode_attn` over the packed cache up to float64 rounding.
    """
    qf = widen(q, dtype)
    B, Hq, d = qf.shape
    kf = widen(k, dtype)
    vf = widen(v, dtype)
    ktf = widen(k_tail, dtype)
    vtf = widen(v_tail, dtype)
    n_kv = kf.shape[1]
    G = Hq // n_kv
    out = np.zeros((B, Hq, d), dtype=np.float64)
    for b in range(B):
        for h in range(Hq):
            g = h // G
            s_ctx = sm_scale * (kf[b, g] @ qf[b, h])
            s_ctx = np.where(np.asarray(kv_mask[b, g]) != 0, s_ctx, -np.inf)
            s_tail = sm_scale * (ktf[b, g] @ qf[b, h])
            s = np.concatenate([s_ctx, s_tail])
            vals = np.concatenate([vf[b, g], vtf[b, g]], axis=0)
            if not np.isfinite(s).any():
                continue
            p = np.exp(s - s.max())
            out[b, h] = (p @ vals) / p.sum()
    return out


# ---------------------------------------------------------------------------
# Exact-budget pattern export (Sec. 3.3; Appendix A, exact-budget refinement)
# ---------------------------------------------------------------------------

def budget_entries(rho, num_layers, num_q_heads, num_bins):
    """K_rho = round(rho * L * H * D), the number of active pattern entries at
    logical retention ratio rho.  The paper does not say how halves round;
    they round up here (floor(x + 0.5) of the float64 product)."""
    return int(math.floor(float(rho) * int(num_layers) * int(num_q_heads) * int(num_bins) + 0.5))


def topk_mask(probs, k):
    """TopKMask(P, K): the k largest entries of P set to one, all others zero,
    globally over every (layer, query head, bin) entry.  Ties (equal
    probabilities, +0 and -0 alike) go to the lower flat index in row-major
    (layer, head, bin) order; NaN ranks below every number.  Returns uint8 of
    P's shape."""
    p = np.asarray(probs, dtype=np.float64)
    flat = p.reshape(-1)
    nan = np.isnan(flat)
    value = np.where(nan, 0.0, flat)
    # lexsort orders by the last key first: numbers before NaN, then larger
    # probability first, then lower index
    order = np.lexsort((np.arange(flat.size), -value, nan))
    out = np.zeros(flat.size, dtype=np.uint8)
    out[order[:int(k)]] = 1
    return out.reshape(p.shape)


def retention_report(pattern, context_len, sink, recent, bin_edges, num_kv_heads):
    """Logical against physical retention (Sec. 3.4, last paragraph).

    logical: fraction of pattern entries that are one, ||M||_0 / (N Hq D);
    physical: fraction of cache positions a KV head keeps after the union,
    sink and recent included, sum of retained lengths / (N Hkv T).
    Returns dict(logical, physical, kept_entries, retained_positions).
    """
    pattern = np.asarray(pattern, dtype=np.uint8)
    n_units, n_q, n_bins = pattern.shape
    lengths = closed_form_lengths(pattern, context_len, sink, recent, bin_edges, num_kv_heads)
    kept = int(np.count_nonzero(pattern))
    positions = int(lengths.sum())
    total = n_units * num_kv_heads * int(context_len)
    return dict(logical=kept / float(pattern.size) if pattern.size else 0.0,
                physical=positions / float(total) if total else 0.0,
                kept_entries=kept, retained_positions=positions)


# ---------------------------------------------------------------------------
# Zero-copy paged variant
# ---------------------------------------------------------------------------
#
# A paged cache keeps the rows of segment s in pages of `page_rows`
# consecutive positions: logical page p (positions [p * page_rows,
# (p + 1) * page_rows)) lives in physical page page_table[s][p] of a pool
# [num_pages][page_rows][d].  Nothing about this layout comes from the paper;
# it is the paged-cache idea the paper cites as prior art, used to keep the
# retained rows in place instead of packing them.

PAGE_ENTRY_FIELDS = ("page", "logical_page", "lo", "hi")


def page_select(kv_mask, page_table, page_rows, append_cap):
    """Runs of retained positions of every segment, referenced in place.

    kv_mask uint8 [nseg][T] (nonzero = retained), page_table int32
    [nseg][pages_per_seg].  For each segment, in position order: every
    maximal run of retained context positions that stays within one logical
    page, as the entry (physical page, logical page, lo, hi) covering slots
    [lo, hi) of that page; then the append region [T, T + append_cap), one
    entry per logical page it touches (appended tokens are always retained,
    Sec. 3.4).  A page is used when some entry names it.

    Returns dict(entries = list per segment of int32 [n][4] arrays,
    n_entries int32 [nseg], seg_len int32 [nseg] (retained context
    positions), page_used uint8 [nseg][pages_per_seg]).
    """
    kv_mask = np.asarray(kv_mask)
    table = np.asarray(page_table)
    nseg, T = kv_mask.shape
    pr = int(page_rows)
    n_pages = table.shape[1]
    ctx_pages = -(-T // pr)
    entries = []
    n_entries = np.zeros(nseg, dtype=np.int32)
    seg_len = np.zeros(nseg, dtype=np.int32)
    page_used = np.zeros((nseg, n_pages), dtype=np.uint8)
    for s in range(nseg):
        kept = np.zeros(ctx_pages * pr, dtype=np.int8)
        kept[:T] = kv_mask[s] != 0
        seg_len[s] = int(kept.sum())
        # one row per logical page, a zero on either side: a run can then
        # neither start before a page nor end after it
        framed = np.zeros((ctx_pages, pr + 2), dtype=np.int8)
        framed[:, 1:-1] = kept.reshape(ctx_pages, pr)
        step = np.diff(framed, axis=1)
        starts = np.argwhere(step == 1)   # (logical page, first slot), row-major = position order
        ends = np.argwhere(step == -1)    # (logical page, end slot)
        rows = [(int(table[s, lp]), int(lp), int(lo), int(hi))
                for (lp, lo), (_, hi) in zip(starts, ends)]
        if append_cap > 0:
            for lp in range(T // pr, (T + append_cap - 1) // pr + 1):
                lo = max(T, lp * pr) - lp * pr
                hi = min(T + append_cap, (lp + 1) * pr) - lp * pr
                rows.append((int(table[s, lp]), lp, lo, hi))
        e = np.array(rows, dtype=np.int32).reshape(-1, 4)
        entries.append(e)
        n_entries[s] = len(e)
        page_used[s, e[:, 1]] = 1
    return dict(entries=entries, n_entries=n_entries, seg_len=seg_len, page_used=page_used)


def paged_append(k_pages, v_pages, page_table, page_rows, context_len, k_new, v_new, n_tail):
    """Write new tokens into their pages (Sec. 3.4: appended and retained).

    k_new, v_new [nseg][n_new][d]; token t of segment s is position
    P = context_len + n_tail + t, stored at slot P % page_rows of page
    page_table[s][P // page_rows].  Returns updated copies of the pools.
    """
    k_pages = np.array(k_pages, copy=True)
    v_pages = np.array(v_pages, copy=True)
    nseg, n_new = np.asarray(k_new).shape[:2]
    for s in range(nseg):
        for t in range(n_new):
            pos = int(context_len) + int(n_tail) + t
            page = int(page_table[s][pos // page_rows])
            k_pages[page, pos % page_rows] = k_new[s][t]
            v_pages[page, pos % page_rows] = v_new[s][t]
    return k_pages, v_pages


def paged_decode_attn(q, k_pages, v_pages, entries, page_rows, context_len, n_tail, sm_scale,
                      num_kv_heads, dtype):
    """One decode step over a paged cache, through page_select's entries.

    Segment s = b * Hkv + g attends to every slot [lo, hi) of every entry
    whose position (logical page * page_rows + slot) is below
    context_len + n_tail: the retained context and the tokens appended so
    far.  Every query head of group g attends to all of them (union of
    Sec. 3.4).  Returns float64 [B][Hq][d].
    """
    qf = widen(q, dtype)
    B, Hq, d = qf.shape
    G = Hq // num_kv_heads
    limit = int(context_len) + int(n_tail)
    out = np.zeros((B, Hq, d), dtype=np.float64)
    for b in range(B):
        for g in range(num_kv_heads):
            s = b * num_kv_heads + g
            pages, slots = [], []
            for page, lp, lo, hi in np.asarray(entries[s]).reshape(-1, 4):
                for slot in range(int(lo), int(hi)):
                    if int(lp) * page_rows + slot < limit:
                        pages.append(int(page))
                        slots.append(slot)
            kr = widen(np.asarray(k_pages)[pages, slots].reshape(len(pages), d), dtype)
            vr = widen(np.asarray(v_pages)[pages, slots].reshape(len(pages), d), dtype)
            for h in range(g * G, (g + 1) * G):
                out[b, h] = _softmax_attend(qf[b, h], kr, vr, sm_scale)
    return out
