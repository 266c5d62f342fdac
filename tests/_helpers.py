"""Shared helpers for the GPU parity tests (host side only)."""

import numpy as np
import torch

import oracle as o

ATTN_TOL = 2e-3  # max relative error of an attention output row (bf16 in, fp32 accumulate)


def bits(t):
    """Host numpy copy of a tensor: uint16 bit patterns for bf16, float32 otherwise."""
    t = t.detach().cpu().contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


def odt(t):
    return o.BF16 if t.dtype == torch.bfloat16 else o.F32


def row_rel_err(got, ref):
    """max over (b, h) of |got - ref|_inf / max(|ref|_inf, 1e-30)."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    num = np.abs(got - ref).max(axis=-1)
    den = np.maximum(np.abs(ref).max(axis=-1), 1e-30)
    return float((num / den).max())


class GpuPack:
    """Map + compact on the GPU through the C ABI, with exact allocation.

    kv_len is read back once (the caller-side sync the one-time compaction
    allows) to size the packed buffers.
    """

    def __init__(self, d, layout, pattern, k, v, cap, with_q_mask=False, stream=None):
        N, Hq, Hkv, T = layout.num_units, layout.num_q_heads, layout.num_kv_heads, layout.context_len
        dev = k.device
        self.pattern = torch.from_numpy(np.ascontiguousarray(pattern)).to(dev)
        self.kv_mask = torch.empty((N, Hkv, T), dtype=torch.uint8, device=dev)
        self.kv_len = torch.empty((N, Hkv), dtype=torch.int32, device=dev)
        self.q_mask = torch.empty((N, Hq, T), dtype=torch.uint8, device=dev) if with_q_mask else None
        d.dkv_map_pattern(layout, self.pattern, self.kv_mask, self.kv_len, self.q_mask, stream=stream)
        self.rows = int((self.kv_len.cpu().to(torch.int64) + cap).sum())
        rows = self.rows
        dim = k.shape[-1]
        self.k_c = torch.empty((max(rows, 1), dim), dtype=k.dtype, device=dev)
        self.v_c = torch.empty((max(rows, 1), dim), dtype=k.dtype, device=dev)
        self.seg_off = torch.empty(N * Hkv, dtype=torch.int64, device=dev)
        self.seg_len = torch.empty(N * Hkv, dtype=torch.int32, device=dev)
        self.src_pos = torch.full((max(rows, 1),), -7, dtype=torch.int32, device=dev)
        self.rows_needed = torch.empty(1, dtype=torch.int64, device=dev)
        ws = torch.empty(d.dkv_compact_workspace_bytes(layout), dtype=torch.uint8, device=dev)
        d.dkv_compact(layout, k, v, self.kv_mask, cap, self.k_c, self.v_c, self.seg_off,
                      self.seg_len, ws, src_pos=self.src_pos, rows_needed=self.rows_needed,
                      stream=stream)
        self.cap = cap
