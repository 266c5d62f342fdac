"""GPU parity at the full sizes of the two stack workloads, in the launch
configuration bench.py times.

The whole stack is mapped and packed by one call each; then every decode step
runs one dkv_append_decode_attn per layer (append the step's token, attend),
with the same rows_hint and workspace as the benchmark.  Checked against the
oracle, layer by layer (dense K/V streamed back one layer at a time):

* packing: lengths, offsets and every packed row bit-exact, and after the
  last step the appended rows too; the block gather (dkv_compact_bins) of
  the same stack equal to map + compact's pack in every output;
* attention: every layer at the first and at the last step, and sampled
  (step, layer) pairs in between: for each intermediate step of the 8B stack
  one layer drawn by a seeded generator, for every 32nd intermediate step of
  the Qwen stack likewise.

The all-keep pattern on one Qwen layer must give the dense kernel's result
bit for bit, and the oracle's within tolerance.
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


def _check_steps(w, steps, every, seed):
    """(step, layer) pairs whose attention output is compared."""
    L = w.num_layers
    checks = {(0, layer) for layer in range(L)} | {(steps - 1, layer) for layer in range(L)}
    rng = np.random.default_rng(seed)
    for s in range(1, steps - 1):
        layer = int(rng.integers(L))
        if s % every == 0:
            checks.add((s, layer))
    return checks


class StackRun:
    """The GPU side of a full-size run: inputs, pack, all decode steps."""

    def __init__(self, d, name, steps, every):
        w = di.workload(name)
        self.w, self.steps = w, steps
        L, B, Hq, Hkv, dim, T = (w.num_layers, w.batch, w.num_q_heads, w.num_kv_heads, w.head_dim,
                                 w.context_len)
        N, cap = w.num_units, w.append_cap
        assert steps <= cap
        self.pattern, _ = di.make_pattern(w)
        self.k = torch.empty((N, Hkv, T, dim), dtype=torch.bfloat16, device=DEV)
        self.v = torch.empty_like(self.k)
        for u in range(N):
            ku, vu = di.kv_unit(w, u, device=DEV)
            self.k[u].copy_(ku)
            self.v[u].copy_(vu)
        lay = d.make_layout(N, Hq, Hkv, dim, T, w.sink, w.recent, list(w.bin_edges))
        self.pack = GpuPack(d, lay, self.pattern, self.k, self.v, cap)
        self.bins_equal = self._bins_pack(d, lay, cap)
        lens = self.pack.kv_len.cpu().to(torch.int64)
        nseg = B * Hkv
        layer_rows = [int(lens[layer * B:(layer + 1) * B].sum()) for layer in range(L)]
        ws = torch.zeros(d.dkv_decode_workspace_bytes(B, Hq, Hkv, dim), dtype=torch.uint8, device=DEV)
        out = torch.empty((B, Hq, dim), dtype=torch.float32, device=DEV)
        self.checks = _check_steps(w, steps, every, seed=w.cfg_id)
        self.outs = {}
        for s in range(steps):
            for layer in range(L):
                q = di.q_step(w, layer, s, device=DEV)
                kn, vn = di.kv_new_step(w, layer, s, device=DEV)
                segs = slice(layer * nseg, (layer + 1) * nseg)
                d.dkv_append_decode_attn(q, kn.reshape(nseg, 1, dim).contiguous(),
                                         vn.reshape(nseg, 1, dim).contiguous(), s, cap, self.pack.k_c,
                                         self.pack.v_c, self.pack.seg_off[segs], self.pack.seg_len[segs],
                                         w.sm_scale, out, ws, Hkv,
                                         rows_hint=layer_rows[layer] + nseg * (s + 1))
                if (s, layer) in self.checks:
                    self.outs[(s, layer)] = out.clone()
        torch.cuda.synchronize()
        self._okm = None

    def _bins_pack(self, d, lay, cap):
        """The same stack packed by the block gather straight from the pattern,
        compared with map + compact's pack (before any append): offsets,
        lengths, rows_needed, every source position and every packed row."""
        pk = self.pack
        kb, vb = torch.empty_like(pk.k_c), torch.empty_like(pk.v_c)
        so, sl = torch.empty_like(pk.seg_off), torch.empty_like(pk.seg_len)
        sp = torch.full_like(pk.src_pos, -7)
        rn = torch.empty_like(pk.rows_needed)
        ws = torch.empty(d.dkv_compact_bins_workspace_bytes(lay), dtype=torch.uint8, device=DEV)
        d.dkv_compact_bins(lay, self.k, self.v, pk.pattern, cap, kb, vb, so, sl, ws, src_pos=sp, rows_needed=rn)
        kept = pk.src_pos >= 0  # the packed rows (free append rows keep -7)
        eq = {"seg_off": torch.equal(so, pk.seg_off), "seg_len": torch.equal(sl, pk.seg_len),
              "rows_needed": torch.equal(rn, pk.rows_needed), "src_pos": torch.equal(sp, pk.src_pos),
              "k": torch.equal(kb[kept].view(torch.int16), pk.k_c[kept].view(torch.int16)),
              "v": torch.equal(vb[kept].view(torch.int16), pk.v_c[kept].view(torch.int16)),
              "packed_rows": int(kept.sum())}
        del kb, vb, ws
        torch.cuda.empty_cache()
        return eq

    def _oracle_map(self):
        """The oracle's masks for the whole stack (computed once), after checking
        the GPU's lengths and whole-stack offsets against them."""
        if self._okm is None:
            w = self.w
            _, okm, okl = o.map_pattern(self.pattern, w.context_len, w.sink, w.recent, w.bin_edges,
                                        w.num_kv_heads)
            # whole-stack offsets: segments unit-major, each len + cap rows
            base = np.concatenate([[0], np.cumsum(okl.reshape(-1).astype(np.int64) + w.append_cap)])
            self.gpu_off = self.pack.seg_off.cpu().numpy()
            self.gpu_len = self.pack.seg_len.cpu().numpy()
            np.testing.assert_array_equal(self.gpu_len, okl.reshape(-1))
            np.testing.assert_array_equal(self.gpu_off, base[:-1])
            self._okm = okm
        return self._okm

    def check_layers(self, layers):
        """Compare the listed layers with the oracle."""
        w, steps = self.w, self.steps
        B, Hkv, cap = w.batch, w.num_kv_heads, w.append_cap
        nseg = B * Hkv
        okm = self._oracle_map()
        gpu_off, gpu_len = self.gpu_off, self.gpu_len
        for layer in layers:
            units = slice(layer * B, (layer + 1) * B)
            segs = slice(layer * nseg, (layer + 1) * nseg)
            ref = o.compact(bits(self.k[units]), bits(self.v[units]), okm[units], cap)
            # all appended tokens of this layer, steps 0 .. steps-1: [B][Hkv][steps][d]
            new = [di.kv_new_step(w, layer, s, device=DEV) for s in range(steps)]
            kn = np.concatenate([bits(a) for a, _ in new], axis=2)
            vn = np.concatenate([bits(b) for _, b in new], axis=2)
            # packed rows and appended rows, bit-exact (one contiguous read-back)
            lo = int(gpu_off[segs][0])
            hi = int(gpu_off[segs][-1]) + int(gpu_len[segs][-1]) + cap
            gk = bits(self.pack.k_c[lo:hi])
            gv = bits(self.pack.v_c[lo:hi])
            kc_all, vc_all = o.append(ref["k_c"], ref["v_c"], ref["seg_off"], ref["seg_len"], kn, vn, 0)
            for i in range(nseg):
                n = int(ref["seg_len"][i]) + steps
                r0, g0 = int(ref["seg_off"][i]), int(gpu_off[segs][i]) - lo
                assert np.array_equal(gk[g0:g0 + n], kc_all[r0:r0 + n]), (w.name, layer, i)
                assert np.array_equal(gv[g0:g0 + n], vc_all[r0:r0 + n]), (w.name, layer, i)
            del gk, gv
            # step s attends the packed rows and tokens 0..s: the first s + 1
            # appended rows, so the fully appended pack serves every step
            for s in sorted(st for st, ly in self.checks if ly == layer):
                q = bits(di.q_step(w, layer, s, device=DEV))
                want = o.decode_attn(q, kc_all, vc_all, ref["seg_off"], ref["seg_len"], s + 1,
                                     w.sm_scale, Hkv, o.BF16)
                err = row_rel_err(self.outs[(s, layer)].cpu().numpy(), want)
                assert err <= ATTN_TOL, (w.name, layer, s, err)


@pytest.fixture(scope="module")
def headline(d):
    w = di.workload("llama8b_stack_128k")
    return StackRun(d, w.name, steps=w.decode_steps, every=1)


@pytest.fixture(scope="module")
def qwen(d):
    w = di.workload("qwen7b_stack_bs4_128k")
    return StackRun(d, w.name, steps=w.decode_steps, every=32)


@pytest.mark.parametrize("chunk", range(4))
def test_headline_stack_full_size(headline, chunk):
    """8B stack at 128K, 32 layers, 64 steps: layers 8*chunk .. 8*chunk+7."""
    headline.check_layers(range(8 * chunk, 8 * chunk + 8))


def test_headline_stack_bins_pack(headline):
    """dkv_compact_bins packs the whole 8B stack exactly as map + compact,
    whose rows the layer tests compare with the oracle."""
    eq = headline.bins_equal
    assert eq["packed_rows"] == int(headline.pack.kv_len.sum())
    assert all(v for key, v in eq.items() if key != "packed_rows"), eq


@pytest.mark.parametrize("chunk", range(7))
def test_qwen_stack_full_size(qwen, chunk):
    """Qwen-7B-shaped stack at 128K, 28 layers x 4 sequences, 256 steps:
    layers 4*chunk .. 4*chunk+3."""
    qwen.check_layers(range(4 * chunk, 4 * chunk + 4))


def test_qwen_stack_bins_pack(qwen):
    """The same for the Qwen-shaped stack (G = 7, four sequences per layer)."""
    eq = qwen.bins_equal
    assert eq["packed_rows"] == int(qwen.pack.kv_len.sum())
    assert all(v for key, v in eq.items() if key != "packed_rows"), eq


def test_qwen_all_keep_layer_equals_dense(d):
    """One Qwen layer (4 sequences) with every position kept: the packed
    decode is the dense kernel's result bit for bit, and the oracle's within
    tolerance."""
    w = di.workload("qwen7b_stack_bs4_128k")
    B, Hq, Hkv, dim, T, cap = w.batch, w.num_q_heads, w.num_kv_heads, w.head_dim, w.context_len, 8
    layer = 11
    pattern, _ = di.make_pattern(w, all_keep=True)
    pattern = np.ascontiguousarray(pattern[layer * B:(layer + 1) * B])
    kv = [di.kv_unit(w, layer * B + b, device=DEV) for b in range(B)]
    k = torch.stack([a for a, _ in kv])
    v = torch.stack([b for _, b in kv])
    del kv
    lay = d.make_layout(B, Hq, Hkv, dim, T, w.sink, w.recent, list(w.bin_edges))
    pack = GpuPack(d, lay, pattern, k, v, cap)
    assert pack.rows == B * Hkv * (T + cap)
    q = di.q_step(w, layer, 0, device=DEV)
    ws = torch.zeros(d.dkv_decode_workspace_bytes(B, Hq, Hkv, dim), dtype=torch.uint8, device=DEV)
    out_p = torch.empty((B, Hq, dim), dtype=torch.float32, device=DEV)
    out_d = torch.empty_like(out_p)
    d.dkv_decode_attn(q, pack.k_c, pack.v_c, pack.seg_off, pack.seg_len, 0, w.sm_scale, out_p, ws,
                      Hkv, rows_hint=B * Hkv * T)
    d.dkv_dense_decode_attn(q, k, v, T, w.sm_scale, out_d, ws)
    torch.cuda.synchronize()
    assert torch.equal(out_p, out_d)
    want = o.dense_decode_attn(bits(q), bits(k), bits(v), T, w.sm_scale, o.BF16)
    assert row_rel_err(out_p.cpu().numpy(), want) <= ATTN_TOL
