"""Benchmark: decode attention over the packed Distance-KV cache vs dense decode.

Workload: Llama-3.1-8B-shaped stack at 128K context -- 32 layers x (32 query
heads, 8 KV heads, head_dim 128), batch 1, bf16, sink 128 + recent 1024, 32
log-spaced distance bins, 34.6% of the KV positions retained after the GQA
union (the 65.4% reduction the paper reports at 128K).  Inputs are seeded
synthetic tensors generated on the GPU.

One step is one decode step of the whole stack: for each layer, append the new
token's K/V (dkv_append) and attend over the packed cache (dkv_decode_attn).
The one-time pattern mapping and compaction, and the same step over the dense
cache (dkv_dense_decode_attn), are timed in the same run.  Every number comes
from HIP events on the stream the kernels run on.

    python bench.py [--gpus 1] [--steps K] [--warmup W]

Prints one JSON line.
"""

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "compacted-KV decode attn: HBM GB/s + µs/step vs dense decode, 8B-shape @128K"
WORKLOAD = "llama8b_stack_128k"
PEAK_HBM_GBPS = 8000.0
PMC_FILE = os.path.join(ROOT, "profiles", "decode_attn_llama8b_stack_128k_pmc.json")
KERNEL_SRC = os.path.join(ROOT, "paper_2609_32663_amd", "csrc", "decode_attn.hip")


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true",
                    help="skip the oracle timing (for profiler runs)")
    ap.add_argument("--copy-probe", action="store_true",
                    help="also run a plain 1 GiB device copy (HBM-counter calibration)")
    return ap.parse_args()


def kernel_hash():
    with open(KERNEL_SRC, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py runs on one GPU only: the Distance-KV path here is a single-GPU "
              "build (no collectives); use --gpus 1", file=sys.stderr)
        sys.exit(2)

    import ctypes
    import numpy as np
    import torch

    import dkv_inputs as di
    import paper_2609_32663_amd as d

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream()
    sh = stream.cuda_stream
    lib = d.library()

    w = di.workload(WORKLOAD)
    L, B, Hq, Hkv, dim, T = w.num_layers, w.batch, w.num_q_heads, w.num_kv_heads, w.head_dim, w.context_len
    cap = w.append_cap
    nseg_layer = B * Hkv
    N = w.num_units
    elem = 2

    def ev():
        return torch.cuda.Event(enable_timing=True)

    # ---------------- inputs (untimed) ------------------------------------
    log("generating inputs")
    pattern, pinfo = di.make_pattern(w)
    k = torch.empty((N, Hkv, T, dim), dtype=torch.bfloat16, device=dev)
    v = torch.empty_like(k)
    for u in range(N):
        ku, vu = di.kv_unit(w, u, device=dev)
        k[u].copy_(ku)
        v[u].copy_(vu)
        del ku, vu
    q_layers = [di.q_step(w, layer, 0, device=dev) for layer in range(L)]
    new_kv = [di.kv_new_step(w, layer, 0, device=dev) for layer in range(L)]
    new_kv = [(a[0].contiguous(), b[0].contiguous()) for a, b in new_kv]  # [B*Hkv][1][d] (B = 1)

    # ---------------- one-time map + compaction (timed, reported apart) ----
    lay = d.make_layout(N, Hq, Hkv, dim, T, w.sink, w.recent, list(w.bin_edges))
    pat_d = torch.from_numpy(pattern).to(dev)
    kv_mask = torch.empty((N, Hkv, T), dtype=torch.uint8, device=dev)
    kv_len = torch.empty((N, Hkv), dtype=torch.int32, device=dev)
    e0, e1, e2 = ev(), ev(), ev()
    e0.record(stream)
    d.dkv_map_pattern(lay, pat_d, kv_mask, kv_len)
    e1.record(stream)
    torch.cuda.synchronize()
    map_us = e0.elapsed_time(e1) * 1e3
    lens = kv_len.cpu().to(torch.int64)
    rows = int((lens + cap).sum())
    k_c = torch.empty((rows, dim), dtype=torch.bfloat16, device=dev)
    v_c = torch.empty_like(k_c)
    seg_off = torch.empty(N * Hkv, dtype=torch.int64, device=dev)
    seg_len = torch.empty(N * Hkv, dtype=torch.int32, device=dev)
    cws = torch.empty(d.dkv_compact_workspace_bytes(lay), dtype=torch.uint8, device=dev)
    e1.record(stream)
    d.dkv_compact(lay, k, v, kv_mask, cap, k_c, v_c, seg_off, seg_len, cws)
    e2.record(stream)
    torch.cuda.synchronize()
    compact_us = e1.elapsed_time(e2) * 1e3
    retained = int(lens.sum())
    compact_bytes = 2 * 2 * retained * dim * elem + N * Hkv * T  # K,V read+write + mask
    phys_frac = retained / float(N * Hkv * T)
    log(f"map {map_us:.0f} us, compact {compact_us:.0f} us, retained {phys_frac:.4f}")

    # ---------------- CPU oracle baseline + parity sample (layer 0) --------
    cpu = None
    parity = None
    dws = torch.zeros(d.dkv_decode_workspace_bytes(B, Hq, Hkv, dim), dtype=torch.uint8, device=dev)
    out = torch.empty((B, Hq, dim), dtype=torch.float32, device=dev)
    if not args.no_cpu_baseline:
        import oracle as o
        from threadpoolctl import threadpool_limits
        log("oracle baseline: one decode step over all layers")
        cpu_s, sample_bytes, worst, same_pack = 0.0, 0, 0.0, True
        for layer in range(L):
            units = slice(layer * B, (layer + 1) * B)
            segs = slice(layer * nseg_layer, (layer + 1) * nseg_layer)
            d.dkv_decode_attn(q_layers[layer], k_c, v_c, seg_off[segs], seg_len[segs], 0, w.sm_scale,
                              out, dws, Hkv, rows_hint=int(lens[units].sum()))
            torch.cuda.synchronize()
            got = out.cpu().numpy().astype(np.float64)
            kb = k[units].cpu().view(torch.int16).numpy().view(np.uint16)
            vb = v[units].cpu().view(torch.int16).numpy().view(np.uint16)
            qb = q_layers[layer].cpu().view(torch.int16).numpy().view(np.uint16)
            _, okm, _ = o.map_pattern(pattern[units], T, w.sink, w.recent, w.bin_edges, Hkv)
            ref = o.compact(kb, vb, okm, cap)
            with threadpool_limits(1):
                t0 = time.perf_counter()
                want = o.decode_attn(qb, ref["k_c"], ref["v_c"], ref["seg_off"], ref["seg_len"], 0,
                                     w.sm_scale, Hkv, o.BF16)
                cpu_s += time.perf_counter() - t0
            sample_bytes += int(ref["seg_len"].sum()) * dim * elem * 2 + B * Hq * dim * (elem + 4)
            err = float((np.abs(got - want).max(-1) / np.maximum(np.abs(want).max(-1), 1e-30)).max())
            worst = max(worst, err)
            same_pack &= bool(np.array_equal(seg_len[segs].cpu().numpy(), ref["seg_len"]))
            del kb, vb, ref
        cpu = {"value": round(sample_bytes / cpu_s / 1e9, 4), "unit": "GB/s", "cores": 1,
               "kind": "oracle",
               "sample": f"one full decode step (all {L} layers, n_tail 0) by the fp64 NumPy "
                         f"oracle with 1 BLAS thread: {cpu_s:.2f} s for {sample_bytes / 1e9:.2f} GB "
                         f"of packed K/V"}
        parity = {"layers": L, "max_rel_err": worst, "seg_len_equal": same_pack}
        log(f"oracle {cpu_s:.2f} s, worst parity err {worst:.2e}")

    # ---------------- dense comparator cache [L][B*Hkv][T+cap][d] ----------
    t_cap = T + cap
    kd = torch.zeros((N, Hkv, t_cap, dim), dtype=torch.bfloat16, device=dev)
    vd = torch.zeros_like(kd)
    kd[:, :, :T].copy_(k)
    vd[:, :, :T].copy_(v)
    del k, v  # the dense input is no longer needed once packed
    torch.cuda.empty_cache()
    dseg_off = torch.arange(N * Hkv, dtype=torch.int64, device=dev) * t_cap
    dseg_len = torch.full((N * Hkv,), T, dtype=torch.int32, device=dev)

    # ---------------- pre-marshalled launch arguments ----------------------
    P = ctypes.c_void_p
    ws_bytes = dws.numel()
    layer_rows = [int(lens[layer * B:(layer + 1) * B].sum()) for layer in range(L)]

    def packed_args(layer, n_tail, sh):
        """dkv_append_decode_attn: append this step's token at n_tail, attend."""
        off = layer * nseg_layer
        kn, vn = new_kv[layer]
        return (d.DKV_BF16, B, Hq, Hkv, dim, P(q_layers[layer].data_ptr()), P(kn.data_ptr()),
                P(vn.data_ptr()), 1, n_tail, cap, P(k_c.data_ptr()), P(v_c.data_ptr()),
                P(seg_off.data_ptr() + 8 * off), P(seg_len.data_ptr() + 4 * off), w.sm_scale,
                layer_rows[layer] + nseg_layer * (n_tail + 1), P(out.data_ptr()), P(dws.data_ptr()),
                ws_bytes, P(sh))

    def dense_args(layer, n_valid, sh):
        """dkv_dense_append_decode_attn: write the token at row n_valid, attend."""
        kl = kd[layer * B:(layer + 1) * B]
        vl = vd[layer * B:(layer + 1) * B]
        kn, vn = new_kv[layer]
        return (d.DKV_BF16, B, Hq, Hkv, dim, P(q_layers[layer].data_ptr()), P(kn.data_ptr()),
                P(vn.data_ptr()), 1, P(kl.data_ptr()), P(vl.data_ptr()), t_cap, n_valid, w.sm_scale,
                P(out.data_ptr()), P(dws.data_ptr()), ws_bytes, P(sh))

    def step_args(step, dense, sh):
        """One decode step: per layer, one call that appends the step's token
        and attends over the cache."""
        slot = step % cap
        acts = []
        for layer in range(L):
            if dense:
                acts.append((lib.dkv_dense_append_decode_attn, dense_args(layer, T + slot, sh)))
            else:
                acts.append((lib.dkv_append_decode_attn, packed_args(layer, slot, sh)))
        return acts

    def run(acts):
        for fn, a in acts:
            st = fn(*a)
            if st != 0:
                raise d.DkvError(fn.__name__, st)

    def decode_bytes(step, dense):
        n_tail = step % cap + 1
        rows_step = (N * Hkv * (T + n_tail)) if dense else (retained + N * Hkv * n_tail)
        return rows_step * dim * elem * 2 + L * B * Hq * dim * (elem + 4) + L * nseg_layer * 12

    cap_stream = torch.cuda.Stream()

    def timed(dense, steps, warmup):
        """Step time as HIP-graph replays (one graph per step: each keeps its
        own append slot), plus the same steps launched eagerly."""
        run(step_args(0, dense, sh))  # warm: first launches load code objects
        torch.cuda.synchronize()
        graphs = []
        for s in range(warmup + steps):
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g, stream=cap_stream):
                run(step_args(s, dense, cap_stream.cuda_stream))
            graphs.append(g)
        for s in range(warmup):
            graphs[s].replay()
        torch.cuda.synchronize()
        a, b = ev(), ev()
        a.record(stream)
        for s in range(warmup, warmup + steps):
            graphs[s].replay()
        b.record(stream)
        torch.cuda.synchronize()
        ms = a.elapsed_time(b) / steps
        plans = [step_args(s, dense, sh) for s in range(warmup + steps)]
        for s in range(warmup):
            run(plans[s])
        torch.cuda.synchronize()
        a.record(stream)
        for s in range(warmup, warmup + steps):
            run(plans[s])
        b.record(stream)
        torch.cuda.synchronize()
        eager_ms = a.elapsed_time(b) / steps
        nbytes = sum(decode_bytes(s, dense) for s in range(warmup, warmup + steps)) / steps
        return ms, eager_ms, nbytes

    log("timing packed decode")
    ms, eager_ms, nbytes = timed(False, args.steps, args.warmup)
    log("timing dense decode")
    dms, deager_ms, dbytes = timed(True, args.steps, args.warmup)
    # A step is exactly one attention call per layer on one stream, so the
    # average duration of a call (split + combine kernel, with the gaps
    # between them) is the timed region's event interval over L calls.
    launch_ms = ms / L
    dlaunch_ms = dms / L

    if args.copy_probe:
        src = torch.empty(1 << 29, dtype=torch.int16, device=dev)  # 1 GiB
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()

    per_launch_bytes = nbytes / L
    achieved = per_launch_bytes / (launch_ms * 1e-3) / 1e9
    traffic = None
    if os.path.exists(PMC_FILE):
        with open(PMC_FILE) as f:
            pmc = json.load(f)
        if pmc.get("kernel_sha256_16") == kernel_hash():
            traffic = pmc.get("traffic_bytes_per_launch")

    res = {
        "metric": METRIC,
        "value": round(nbytes / (ms * 1e-3) / 1e9, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "eager_ms_per_step": round(eager_ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": WORKLOAD, "layers": L, "batch": B, "q_heads": Hq, "kv_heads": Hkv,
                   "head_dim": dim, "context_len": T, "sink": w.sink, "recent": w.recent,
                   "bins": w.num_bins, "retained_fraction": round(phys_frac, 4),
                   "step": "per layer: dkv_append_decode_attn (append 1 token, attend); timed as HIP-graph "
                           "replays, one graph per step"},
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBPS,
                     "unit": "GB/s", "frac": round(achieved / PEAK_HBM_GBPS, 4),
                     "traffic": traffic,
                     "kernel": "dkv_append_decode_attn call: decode_kernel<bf16,128,4> + "
                               "decode_merge_kernel",
                     "avg_launch_us": round(launch_ms * 1e3, 2),
                     "bytes_per_launch": int(per_launch_bytes)},
        "cpu_baseline": cpu,
        "us_per_step": round(ms * 1e3, 1),
        "dense": {"ms_per_step": round(dms, 4), "eager_ms_per_step": round(deager_ms, 4),
                  "gb_per_s": round(dbytes / (dms * 1e-3) / 1e9, 2),
                  "avg_launch_us": round(dlaunch_ms * 1e3, 2),
                  "launch_frac_of_peak": round(dbytes / L / (dlaunch_ms * 1e-3) / 1e9 / PEAK_HBM_GBPS, 4)},
        "speedup_vs_dense": round(dms / ms, 3),
        "one_time": {"map_us": round(map_us, 1), "compact_us": round(compact_us, 1),
                     "compact_gb_per_s": round(compact_bytes / (compact_us * 1e-6) / 1e9, 1)},
        "kv_cache_gib": {"dense": round(N * Hkv * T * dim * elem * 2 / 2 ** 30, 3),
                         "packed": round(retained * dim * elem * 2 / 2 ** 30, 3)},
        "parity_layer0": parity,
        "pattern": pinfo,
    }
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
