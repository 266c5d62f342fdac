"""Benchmark: decode attention over the packed Distance-KV cache vs dense decode.

Workload: Llama-3.1-8B-shaped stack at 128K context -- 32 layers x (32 query
heads, 8 KV heads, head_dim 128), batch 1, bf16, sink 128 + recent 1024, 32
log-spaced distance bins, 34.6% of the KV positions retained after the GQA
union (the 65.4% reduction the paper reports at 128K).  Inputs are seeded
synthetic tensors generated on the GPU.

One step is one decode step of the whole stack: for each layer, append the new
token's K/V (dkv_append) and attend over the packed cache (dkv_decode_attn).
The one-time pattern mapping and compaction, and the same step over the dense
cache (dkv_dense_decode_attn), are timed in the same run, and so are the
zero-copy paged variant (the stack in 128-row pages, the retained runs listed
in place by dkv_page_select, one dkv_paged_append_decode_attn per layer) and
the query block after the context.  Every number comes from HIP events on the
stream the kernels run on.

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
PEAK_BF16_TFLOPS = 2500.0  # dense bf16 matrix peak
QUERY_TOKENS = 256
MT_TURNS, MT_STEPS = 4, 16  # multi-turn row: query rounds over one pack, tokens generated per round
PAGE_ROWS = 128  # rows per page of the zero-copy paged variant
SPREAD_REPS = 50  # single-step replays, at least, behind the median / p10 / p90 of a step
PMC_FILE = os.path.join(ROOT, "profiles", "decode_attn_llama8b_stack_128k_pmc.json")
KERNEL_SRCS = [os.path.join(ROOT, "paper_2609_32663_amd", "csrc", f)
               for f in ("decode_attn.hip", "dkv_device.hpp", "dkv_launch.hpp")]
QUERY_SRCS = [os.path.join(ROOT, "paper_2609_32663_amd", "csrc", f)
              for f in ("query_attn.hip", "dkv_device.hpp", "dkv_query.hpp")]
COMPACT_SRCS = [os.path.join(ROOT, "paper_2609_32663_amd", "csrc", f)
                for f in ("compact.hip", "dkv_device.hpp", "dkv_launch.hpp")]
BINS_SRCS = [os.path.join(ROOT, "paper_2609_32663_amd", "csrc", f)
             for f in ("compact_bins.hip", "dkv_device.hpp", "dkv_bins.hpp")]


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true",
                    help="skip the oracle timing (for profiler runs)")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the other configurations' rows (counter runs: rocprofv3 --pmc has crashed on the "
                         "host in that section)")
    ap.add_argument("--no-full-generation", action="store_true",
                    help="skip the full-generation row (counter runs: the profiler process has crashed on the "
                         "host in that section under rocprofv3 --pmc)")
    ap.add_argument("--copy-probe", action="store_true",
                    help="also run a plain 1 GiB device copy (HBM-counter calibration)")
    ap.add_argument("--no-sustain", action="store_true",
                    help="skip the untimed load runs before each timed measurement (for runs under a "
                         "profiler, which serialises every dispatch: the load runs would multiply them)")
    ap.add_argument("--pmc-summary", nargs=3, metavar=("FETCH_CSV", "WRITE_CSV", "BENCH_LOG"),
                    help="summarise two rocprofv3 --pmc runs of this script (FETCH_SIZE, then "
                         "WRITE_SIZE, each with --copy-probe --no-cpu-baseline) and the JSON line one of "
                         "them printed into the traffic file")
    ap.add_argument("--trace-summary", nargs=2, metavar=("TRACE_DIR", "BENCH_LOG"),
                    help="summarise a rocprofv3 --kernel-trace --stats run of this script (csv output "
                         "named run_*) and its JSON line into the kernel-trace profile")
    ap.add_argument("--phase-budget", action="store_true",
                    help="per-phase time budget of the headline call from the phase-stamp build "
                         "(python paper_2609_32663_amd/build.py --phase-stamps first); writes the profile")
    ap.add_argument("--power-sample", action="store_true",
                    help="sample socket power, engine clock and temperature (amd-smi, read only) while the "
                         "query-block kernel and, for comparison, the decode call run continuously on one "
                         "layer of the headline stack; writes the query kernel's power profile")
    ap.add_argument("--query-counters", nargs=2, metavar=("SQ_DIR", "BENCH_LOG"),
                    help="summarise a rocprofv3 run of this script with --kernel-trace and --pmc GRBM_GUI_ACTIVE "
                         "SQ_VALU_MFMA_BUSY_CYCLES SQ_INSTS_VALU_MFMA_MOPS_BF16 SQ_BUSY_CYCLES (csv output named "
                         "run_*) into the query kernel's clock and matrix-unit profile")
    ap.add_argument("--pmc-command", default="",
                    help="command line recorded by --pmc-summary / --trace-summary")
    args = ap.parse_args()
    if args.steps < 1 or args.warmup < 0:
        ap.error("--steps must be at least 1 and --warmup at least 0")
    return args


def host_info():
    """The host the oracle ran on: CPU model, cores this process may use, NumPy's BLAS."""
    model = None
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    blas = None
    try:
        from threadpoolctl import threadpool_info
        blas = [f"{i.get('internal_api')} {i.get('version')} ({i.get('num_threads')} threads)"
                for i in threadpool_info() if i.get("user_api") == "blas"]
    except Exception:
        pass
    return {"cpu_model": model, "cores_available": len(os.sched_getaffinity(0)), "blas": blas}


def kernel_hash(srcs=None):
    """Hash of the decode kernels' sources (the kernel file and the headers it
    includes; or of other sources): stored counter results apply only to the
    code they measured."""
    h = hashlib.sha256()
    for path in (KERNEL_SRCS if srcs is None else srcs):
        with open(path, "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def timed_calls_per_mode(b):
    """Decode calls one timed mode (packed or dense) issues: a warm step, the
    graph replays, the replays of the per-step spread pass (when the line
    reports one) and the eager steps, one call per layer each."""
    spread = b["step_ms_spread"].get("reps", b["steps"]) if b.get("step_ms_spread") else 0
    return b["config"]["layers"] * (1 + 2 * (b["warmup"] + b["steps"]) + spread)


def last_json(path):
    b = None
    for line in open(path):
        if line.startswith("{"):
            b = json.loads(line)
    return b


def is_paged_kernel(name):
    """Whether a decode_kernel instantiation is the paged one (its last
    template argument)."""
    import re
    m = re.search(r"decode_kernel<([^>]*)>", name)
    return bool(m) and m.group(1).replace(" ", "").split(",")[-1] == "true"


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


# Untimed load run before every timed decode, query and probe measurement, so
# that each is taken in the steady state of that same work.  A timed region
# that started right after the one-time section (its multi-GiB buffers freed
# just before) measured the packed step at 1.225-1.238 ms; after an idle
# period or after continuous replays at 1.17-1.19, and a 10 s trace of
# continuous replays holds 1.170-1.178 from its second 20-step window on.
SUSTAIN_S = 1.5
SUSTAIN_ON = True  # cleared by --no-sustain


def sustain(replay, seconds=SUSTAIN_S):
    """Calls `replay` (one untimed unit of GPU work) until `seconds` of wall
    time have passed, synchronising every 16 calls."""
    import time
    import torch
    if not SUSTAIN_ON:
        return
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < seconds:
        for _ in range(16):
            replay()
        torch.cuda.synchronize()


def pmc_per_dispatch(path, counter):
    """{dispatch id: (kernel name, counter value)} from a rocprofv3 counter CSV."""
    import csv
    out = {}
    with open(path) as f:
        for r in csv.DictReader(f):
            if r["Counter_Name"] != counter:
                continue
            i = int(r["Dispatch_Id"])
            name, val = out.get(i, (r["Kernel_Name"], 0.0))
            out[i] = (name, val + float(r["Counter_Value"]))
    return [out[i] for i in sorted(out)]


TRACE_FILE = os.path.join(ROOT, "profiles", "decode_attn_llama8b_stack_128k.txt")
QUERY_TRACE_FILE = os.path.join(ROOT, "profiles", "query_attn_llama8b_stack_128k.txt")
CONFIGS_TRACE_FILE = os.path.join(ROOT, "profiles", "decode_attn_other_configs.txt")
PHASE_FILE = os.path.join(ROOT, "profiles", "decode_phase_budget_llama8b_stack_128k.txt")
PHASE_LIB = os.path.join(ROOT, "paper_2609_32663_amd", "libdkv_phase.so")


def trace_summary(trace_dir, bench_log, command):
    """Per-kernel durations of a kernel-trace run of this script, next to the
    JSON line that run printed.  After the parity calls (one per layer, when
    the oracle baseline runs) the packed calls come first in the trace and
    the dense comparator's calls follow, equally many."""
    import csv
    import statistics as st
    stats = list(csv.DictReader(open(os.path.join(trace_dir, "run_kernel_stats.csv"))))
    rows = sorted(csv.DictReader(open(os.path.join(trace_dir, "run_kernel_trace.csv"))),
                  key=lambda r: int(r["Start_Timestamp"]))
    b = last_json(bench_log)
    pairs, paged = [], []
    for i in range(len(rows) - 1):
        a, m = rows[i], rows[i + 1]
        if "decode_kernel" in a["Kernel_Name"] and "decode_merge_kernel" in m["Kernel_Name"]:
            s0, e0 = int(a["Start_Timestamp"]), int(a["End_Timestamp"])
            s1, e1 = int(m["Start_Timestamp"]), int(m["End_Timestamp"])
            (paged if is_paged_kernel(a["Kernel_Name"]) else pairs).append(
                ((e0 - s0) / 1e3, (e1 - s1) / 1e3, (e1 - s0) / 1e3))
    # with the oracle baseline, one parity call per layer precedes the timing;
    # then the packed and the dense calls, equally many (later sections of
    # the run make other decode calls)
    front = b["config"]["layers"] if b.get("parity_layer0") else 0
    m = timed_calls_per_mode(b)
    packed, dense = pairs[front:front + m], pairs[front + m:front + 2 * m]
    lines = [f"# rocprofv3 kernel trace of bench.py ({WORKLOAD}: 32 layers x 32q/8kv x d128, "
             f"T=131072, {b['config']['retained_fraction'] * 100:.1f}% retained)",
             f"# command: {command}",
             f"# sources measured: decode kernel sha256/16 {kernel_hash()} (decode_attn.hip, dkv_device.hpp, "
             f"dkv_launch.hpp)",
             "# per-kernel statistics (rocprofv3 --stats, dkv kernels only; us):",
             f"{'kernel':58s} {'calls':>6s} {'avg':>9s} {'min':>9s} {'max':>9s}"]
    for r in stats:
        if "dkv" in r["Name"]:
            nm = r["Name"].replace("(anonymous namespace)::", "").replace("dkv::", "")
            lines.append(f"{nm[:58]:58s} {r['Calls']:>6s} {float(r['AverageNs']) / 1e3:9.2f} "
                         f"{float(r['MinNs']) / 1e3:9.2f} {float(r['MaxNs']) / 1e3:9.2f}")
    groups = [("packed", packed), ("dense", dense)] + ([("paged", paged)] if paged else [])
    for name, ps in groups:
        lines.append(f"{name:6s} calls {len(ps):4d}: decode_kernel mean {st.mean(p[0] for p in ps):7.2f}  "
                     f"decode_merge_kernel mean {st.mean(p[1] for p in ps):6.2f}  "
                     f"call (split start to combine end) mean {st.mean(p[2] for p in ps):7.2f} us")
    lines += ["",
              "# JSON line of the same run (timed region = HIP-graph replays; the profiler adds overhead):",
              f"ms_per_step {b['ms_per_step']}  value {b['value']} GB/s  roofline.avg_launch_us "
              f"{b['roofline']['avg_launch_us']}  frac {b['roofline']['frac']}",
              f"dense ms_per_step {b['dense']['ms_per_step']}  speedup_vs_dense {b['speedup_vs_dense']}",
              *([f"paged ms_per_step {b['paged']['ms_per_step']}  avg_launch_us {b['paged']['avg_launch_us']}  "
                 f"select_us {b['paged']['select_us']}"] if b.get("paged") else []),
              f"cpu_baseline {json.dumps(b['cpu_baseline'])}",
              f"parity_layer0 {json.dumps(b['parity_layer0'])}"]
    with open(TRACE_FILE, "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))

    # query-block attention: (plan +) attention kernel (+ combine) per layer call
    qpairs = []
    for i, r in enumerate(rows):
        if "query_attn_kernel" in r["Kernel_Name"]:
            s0, e0 = int(r["Start_Timestamp"]), int(r["End_Timestamp"])
            sp, e1 = s0, e0
            if i > 0 and "query_plan_kernel" in rows[i - 1]["Kernel_Name"]:
                sp = int(rows[i - 1]["Start_Timestamp"])
            if i + 1 < len(rows) and "query_merge_kernel" in rows[i + 1]["Kernel_Name"]:
                e1 = int(rows[i + 1]["End_Timestamp"])
            qpairs.append(((e0 - s0) / 1e3, (e1 - e0) / 1e3, (e1 - sp) / 1e3, (s0 - sp) / 1e3))
    if qpairs and b.get("query_block"):
        qb = b["query_block"]
        ql = [f"# rocprofv3 kernel trace of bench.py, query-block attention ({WORKLOAD}: {qb['n_q']} tokens after "
              f"the context, every layer)",
              f"# command: {command}",
              f"# sources measured: query kernel sha256/16 {kernel_hash(QUERY_SRCS)} (query_attn.hip, "
              f"dkv_device.hpp, dkv_query.hpp)",
              "# per-kernel statistics (rocprofv3 --stats; us):",
              f"{'kernel':58s} {'calls':>6s} {'avg':>9s} {'min':>9s} {'max':>9s}"]
        for r in stats:
            if "query" in r["Name"]:
                nm = r["Name"].replace("(anonymous namespace)::", "").replace("dkv::", "")
                ql.append(f"{nm[:58]:58s} {r['Calls']:>6s} {float(r['AverageNs']) / 1e3:9.2f} "
                          f"{float(r['MinNs']) / 1e3:9.2f} {float(r['MaxNs']) / 1e3:9.2f}")
        ql += [f"calls {len(qpairs)}: plan (start to start) mean {st.mean(x[3] for x in qpairs):6.2f}  "
               f"query_attn_kernel mean {st.mean(x[0] for x in qpairs):8.2f}  "
               f"combine (end to end) mean {st.mean(x[1] for x in qpairs):6.2f}  call mean "
               f"{st.mean(x[2] for x in qpairs):8.2f} us",
               "",
               "# JSON line of the same run (timed region = HIP-graph replays; the profiler adds overhead):",
               f"query_block us_per_layer {qb['us_per_layer']}  roofline {json.dumps(qb['roofline'])}",
               f"cpu_baseline {json.dumps(qb['cpu_baseline'])}",
               f"parity_layer0 {json.dumps(qb['parity_layer0'])}"]
        with open(QUERY_TRACE_FILE, "w") as f:
            f.write("\n".join(ql) + "\n")
        print("\n".join(ql))

    # the other configurations: their decode calls are the run's last
    # non-paged ones, issued in the order the JSON line lists them
    seq = b.get("configs_decode_calls")
    if seq:
        n = sum(c for _, c in seq)
        tail = pairs[len(pairs) - n:]
        cl = ["# rocprofv3 kernel trace of bench.py, the other configurations (decode calls in issue order: "
              "the eager call, warm-up and timed graph replays of each row)",
              f"# command: {command}",
              f"# sources measured: decode kernel sha256/16 {kernel_hash()}",
              f"{'row':34s} {'calls':>6s} {'decode_kernel':>14s} {'merge':>8s} {'call':>9s}  (means, us)"]
        i = 0
        for label, c in seq:
            ps = tail[i:i + c]
            i += c
            cl.append(f"{label:34s} {len(ps):6d} {st.mean(p[0] for p in ps):14.2f} {st.mean(p[1] for p in ps):8.2f} "
                      f"{st.mean(p[2] for p in ps):9.2f}")
        cl += ["", "# JSON rows of the same run (timed region = HIP-graph replays; the profiler adds overhead):"]
        for name, r in b["configs"].items():
            keep = {k: r[k] for k in r if k in ("us_per_step", "gb_per_s", "frac_of_peak", "speedup_vs_dense",
                                                "dense", "parity", "one_time")}
            for k, r2 in r.items():
                if k.startswith("budget_"):
                    keep[k] = {k2: r2[k2] for k2 in ("us_per_step", "gb_per_s", "frac_of_peak", "speedup_vs_dense",
                                                      "parity", "one_time")}
            cl.append(f"{name} {json.dumps(keep)}")
        with open(CONFIGS_TRACE_FILE, "w") as f:
            f.write("\n".join(cl) + "\n")
        print("\n".join(cl))


def pmc_summary(fetch_csv, write_csv, bench_log, command):
    """HBM traffic of one packed attention call from FETCH_SIZE / WRITE_SIZE
    (KiB per dispatch).  Each counter is scaled by what it reads for the
    1 GiB device copy run at the end (which reads and writes exactly 1 GiB),
    and the packed calls are the first non-paged decode/combine dispatch pairs
    of the run (the script times the packed path first; their number follows
    from the steps of the JSON line); the paged calls, told apart by the
    kernel's template flag, are averaged on their own."""
    import statistics
    res = {"kernel_sha256_16": kernel_hash(), "command": command, "unit": "bytes per call"}
    b = last_json(bench_log)
    m = timed_calls_per_mode(b)
    front = b["config"]["layers"] if b.get("parity_layer0") else 0  # parity calls of an oracle run
    per_call, per_paged = {}, {}
    for key, path, counter in (("fetch", fetch_csv, "FETCH_SIZE"), ("write", write_csv, "WRITE_SIZE")):
        rows = pmc_per_dispatch(path, counter)
        copies = [v for n, v in rows if "copy" in n.lower() or "elementwise" in n.lower()]
        calib = (1 << 30) / (copies[-1] * 1024.0)
        pairs = [(is_paged_kernel(rows[i][0]), rows[i][1] + rows[i + 1][1]) for i in range(len(rows) - 1)
                 if "decode_kernel" in rows[i][0] and "decode_merge_kernel" in rows[i + 1][0]]
        calls = [v for pg, v in pairs if not pg]
        packed = calls[front:front + m]
        paged = [v for pg, v in pairs if pg]
        per_call[key] = statistics.mean(packed) * 1024.0 * calib
        res[f"{key}_calibration"] = round(calib, 4)
        res[f"{key}_bytes_per_call"] = int(per_call[key])
        res[f"{key}_calls_counted"] = len(packed)
        if paged:
            per_paged[key] = statistics.mean(paged) * 1024.0 * calib
            res[f"paged_{key}_bytes_per_call"] = int(per_paged[key])
    res["traffic_bytes_per_launch"] = int(per_call["fetch"] + per_call["write"])
    # query-block calls: plan + attention (d 128) + combine dispatches in a row
    res["query_kernel_sha256_16"] = kernel_hash(QUERY_SRCS)
    q_bytes = {}
    for key, path, counter in (("fetch", fetch_csv, "FETCH_SIZE"), ("write", write_csv, "WRITE_SIZE")):
        rows = pmc_per_dispatch(path, counter)
        calib = res[f"{key}_calibration"]
        calls = [rows[i][1] + rows[i + 1][1] + rows[i + 2][1] for i in range(len(rows) - 2)
                 if "query_plan_kernel" in rows[i][0] and "query_attn_kernel<128>" in rows[i + 1][0]
                 and "query_merge_kernel" in rows[i + 2][0]]
        if calls:
            q_bytes[key] = statistics.mean(calls) * 1024.0 * calib
            res[f"query_{key}_bytes_per_call"] = int(q_bytes[key])
            res["query_calls_counted"] = len(calls)
    if len(q_bytes) == 2:
        res["query_traffic_bytes_per_call"] = int(q_bytes["fetch"] + q_bytes["write"])
    if len(per_paged) == 2:
        res["paged_traffic_bytes_per_launch"] = int(per_paged["fetch"] + per_paged["write"])
    # the headline's timed one-time compaction: the second count / scan /
    # list / copy sequence of the run (the first is its warm-up call), against
    # its algorithmic bytes (retained K and V rows read and written, mask read)
    res["compact_kernel_sha256_16"] = kernel_hash(COMPACT_SRCS)
    names = ("compact_count_kernel", "compact_scan_kernel", "compact_list_kernel", "compact_copy_kernel")
    for key, path, counter in (("fetch", fetch_csv, "FETCH_SIZE"), ("write", write_csv, "WRITE_SIZE")):
        rows = pmc_per_dispatch(path, counter)
        calib = res[f"{key}_calibration"]
        packs = [sum(rows[i + j][1] for j in range(4)) for i in range(len(rows) - 3)
                 if all(names[j] in rows[i + j][0] for j in range(4))]
        if len(packs) >= 2:
            res[f"compact_{key}_bytes"] = int(packs[1] * 1024.0 * calib)
    if "compact_fetch_bytes" in res and "compact_write_bytes" in res:
        res["compact_traffic_bytes"] = res["compact_fetch_bytes"] + res["compact_write_bytes"]
        oc = b.get("one_time", {})
        if oc.get("compact_bytes"):
            res["compact_algorithmic_bytes"] = oc["compact_bytes"]
            res["compact_traffic_over_algorithmic"] = round(res["compact_traffic_bytes"] / oc["compact_bytes"], 4)
    # the block gather from the pattern: the second plan / scan / copy triple
    # (the first is its warm-up call), against its algorithmic bytes
    res["compact_bins_kernel_sha256_16"] = kernel_hash(BINS_SRCS)
    for key, path, counter in (("fetch", fetch_csv, "FETCH_SIZE"), ("write", write_csv, "WRITE_SIZE")):
        rows = pmc_per_dispatch(path, counter)
        calib = res[f"{key}_calibration"]
        triples = [rows[i][1] + rows[i + 1][1] + rows[i + 2][1] for i in range(len(rows) - 2)
                   if "bins_plan_kernel" in rows[i][0] and "bins_scan_kernel" in rows[i + 1][0]
                   and "bins_copy_kernel" in rows[i + 2][0]]
        if len(triples) >= 2:
            res[f"compact_bins_{key}_bytes"] = int(triples[1] * 1024.0 * calib)
    if "compact_bins_fetch_bytes" in res and "compact_bins_write_bytes" in res:
        res["compact_bins_traffic_bytes"] = res["compact_bins_fetch_bytes"] + res["compact_bins_write_bytes"]
        oc = b.get("one_time", {})
        if oc.get("compact_bins_bytes"):
            res["compact_bins_algorithmic_bytes"] = oc["compact_bins_bytes"]
            res["compact_bins_traffic_over_algorithmic"] = round(
                res["compact_bins_traffic_bytes"] / oc["compact_bins_bytes"], 4)
    with open(PMC_FILE, "w") as f:
        json.dump(res, f, indent=1)
        f.write("\n")
    print(json.dumps(res))


QUERY_COUNTERS_FILE = os.path.join(ROOT, "profiles", "query_attn_counters_llama8b_stack_128k.txt")
POWER_FILE = os.path.join(ROOT, "profiles", "query_attn_power_llama8b_stack_128k.txt")


def power_sample(seconds=8.0):
    """Socket power, engine clocks and hotspot temperature (`amd-smi metric
    --json`, polled every 0.5 s; read only) while, on layer 0 of the headline
    stack, the query-block call (256 tokens) and then the decode call run
    back to back for `seconds` each, with an idle period first."""
    import ctypes
    import statistics as st
    import subprocess
    import threading
    import time
    import torch

    import dkv_inputs as di
    import paper_2609_32663_amd as d
    dev = torch.device("cuda:0")
    P = ctypes.c_void_p
    w = di.workload(WORKLOAD)
    T, Hq, Hkv, dim = w.context_len, w.num_q_heads, w.num_kv_heads, w.head_dim
    nq = QUERY_TOKENS
    pattern, _ = di.make_pattern(w)
    k, v = di.kv_unit(w, 0, device=dev)
    lay = d.make_layout(1, Hq, Hkv, dim, T, w.sink, w.recent, list(w.bin_edges))
    km = torch.empty((1, Hkv, T), dtype=torch.uint8, device=dev)
    kl = torch.empty((1, Hkv), dtype=torch.int32, device=dev)
    d.dkv_map_pattern(lay, torch.from_numpy(pattern[:1]).to(dev), km, kl)
    lens = kl.cpu().long().reshape(-1)
    rows = int((lens + nq).sum())
    k_q = torch.empty((rows, dim), dtype=torch.bfloat16, device=dev)
    v_q = torch.empty_like(k_q)
    so = torch.empty(Hkv, dtype=torch.int64, device=dev)
    sl = torch.empty(Hkv, dtype=torch.int32, device=dev)
    cws = torch.empty(d.dkv_compact_workspace_bytes(lay), dtype=torch.uint8, device=dev)
    d.dkv_compact(lay, k[None], v[None], km, nq, k_q, v_q, so, sl, cws)
    qb, kb, vb = di.query_block(w, 0, nq, device=dev)
    d.dkv_append(kb.reshape(Hkv, nq, dim).contiguous(), vb.reshape(Hkv, nq, dim).contiguous(), 0, nq, k_q, v_q,
                 so, sl)
    qb = qb.contiguous()
    hint = int(lens.sum()) + Hkv * nq
    ws = torch.empty(d.dkv_query_workspace_bytes(1, Hq, Hkv, dim, nq, hint), dtype=torch.uint8, device=dev)
    out = torch.empty((1, nq, Hq, dim), dtype=torch.float32, device=dev)
    lib = d.library()
    cs = torch.cuda.Stream()
    gq = torch.cuda.CUDAGraph()
    with torch.cuda.graph(gq, stream=cs):
        for _ in range(8):
            st_ = lib.dkv_query_attn(d.DKV_BF16, 1, Hq, Hkv, dim, nq, P(qb.data_ptr()), 0, nq, P(k_q.data_ptr()),
                                     P(v_q.data_ptr()), P(so.data_ptr()), P(sl.data_ptr()), w.sm_scale, hint,
                                     P(out.data_ptr()), P(ws.data_ptr()), ws.numel(), P(cs.cuda_stream))
            if st_ != 0:
                raise d.DkvError("dkv_query_attn", st_)
    q1 = di.q_step(w, 0, 0, device=dev)
    dws = torch.zeros(d.dkv_decode_workspace_bytes(1, Hq, Hkv, dim), dtype=torch.uint8, device=dev)
    o1 = torch.empty((1, Hq, dim), dtype=torch.float32, device=dev)
    gd = torch.cuda.CUDAGraph()
    with torch.cuda.graph(gd, stream=cs):
        for _ in range(64):
            d.dkv_decode_attn(q1, k_q, v_q, so, sl, 0, w.sm_scale, o1, dws, Hkv, rows_hint=int(lens.sum()),
                              stream=cs)
    torch.cuda.synchronize()

    def get(g, path):
        for p_ in path.split("/"):
            g = g.get(p_) if isinstance(g, dict) else None
        return g

    def poll(stop, samples):
        while not stop.is_set():
            r = subprocess.run(["amd-smi", "metric", "--json"], capture_output=True, text=True, timeout=20)
            try:
                g = json.loads(r.stdout)["gpu_data"][0]
                clocks = [get(g, f"clock/gfx_{i}/clk/value") for i in range(8)]
                samples.append((get(g, "power/socket_power/value"),
                                st.mean(c for c in clocks if isinstance(c, (int, float))),
                                get(g, "temperature/hotspot/value")))
            except (ValueError, KeyError, IndexError, TypeError, st.StatisticsError):
                pass
            time.sleep(0.5)

    lines = [f"# socket power and engine clock while one call kind runs continuously ({WORKLOAD}, layer 0: "
             f"{nq} query tokens after the context; decode: the attend-only call over the same packed layer)",
             "# command: python bench.py --power-sample",
             "# source: amd-smi metric --json, polled every 0.5 s (read only); the first second of each run "
             "is left out (the samples while the load ramps up)", ""]
    for tag, g, per in (("idle", None, 0), ("query", gq, 8), ("decode", gd, 64)):
        samples, stop = [], threading.Event()
        th = threading.Thread(target=poll, args=(stop, samples))
        t0 = time.perf_counter()
        th.start()
        n = 0
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        if g is None:
            time.sleep(seconds / 2)
        else:
            a.record()
            while time.perf_counter() - t0 < seconds:
                for _ in range(4):
                    g.replay()
                torch.cuda.synchronize()
                n += 4
            b.record()
            torch.cuda.synchronize()
        stop.set()
        th.join()
        keep = samples[2:] if len(samples) > 4 else samples
        pw = [x[0] for x in keep if isinstance(x[0], (int, float))]
        ck = [x[1] for x in keep]
        hs = [x[2] for x in keep if isinstance(x[2], (int, float))]
        call = f"; {a.elapsed_time(b) * 1e3 / (n * per):.1f} us per call over {n * per} calls" if g is not None else ""
        lines.append(f"{tag:6s}: {len(keep)} samples; socket power median {st.median(pw):.0f} W (min {min(pw):.0f}, "
                     f"max {max(pw):.0f}); engine clock median {st.median(ck):.0f} MHz (min {min(ck):.0f}, max "
                     f"{max(ck):.0f}; the part's maximum is 2,400); hotspot {min(hs)}-{max(hs)} C{call}")
        log(lines[-1])
    with open(POWER_FILE, "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def query_counters(sq_dir, bench_log, command):
    """Clock and matrix-unit use of the query-block attention kernel (d 128)
    from one rocprofv3 run with --pmc GRBM_GUI_ACTIVE SQ_VALU_MFMA_BUSY_CYCLES
    SQ_INSTS_VALU_MFMA_MOPS_BF16 SQ_BUSY_CYCLES and --kernel-trace: per
    dispatch, the GPU's busy cycles (GRBM_GUI_ACTIVE is reported summed over
    the XCDs), the matrix units' busy cycles (summed over the SIMDs) and the
    bf16 matrix operations issued, against the same dispatch's duration."""
    import csv
    import statistics as st
    agent = next(r for r in csv.DictReader(open(os.path.join(sq_dir, "run_agent_info.csv")))
                 if r["Agent_Type"] == "GPU")
    xcc, simds, fmax = int(agent["Num_Xcc"]), int(agent["Simd_Count"]), float(agent["Max_Engine_Clk_Fcompute"])
    per = {}
    for r in csv.DictReader(open(os.path.join(sq_dir, "run_counter_collection.csv"))):
        if "query_attn_kernel<128>" in r["Kernel_Name"]:
            d_ = per.setdefault(int(r["Dispatch_Id"]), {})
            d_[r["Counter_Name"]] = d_.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
    dur = {int(r["Dispatch_Id"]): (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
           for r in csv.DictReader(open(os.path.join(sq_dir, "run_kernel_trace.csv")))
           if "query_attn_kernel<128>" in r["Kernel_Name"]}
    rows = [dict(v, us=dur[i]) for i, v in per.items() if len(v) == 4 and i in dur]
    b = last_json(bench_log)
    qb = b["query_block"]
    alg_flops = qb["tflop_per_step"] * 1e12 / b["config"]["layers"]
    us = st.mean(r["us"] for r in rows)
    cyc = st.mean(r["GRBM_GUI_ACTIVE"] / xcc for r in rows)  # per XCD
    clocks = sorted(r["GRBM_GUI_ACTIVE"] / xcc / r["us"] / 1e3 for r in rows)
    busy = st.mean(r["SQ_VALU_MFMA_BUSY_CYCLES"] / (r["GRBM_GUI_ACTIVE"] / xcc * simds) for r in rows)
    issued = st.mean(r["SQ_INSTS_VALU_MFMA_MOPS_BF16"] * 512 for r in rows)
    clock = st.mean(clocks)
    rate = issued / (us * 1e-6) / 1e12
    lines = ["# query-block attention kernel (query_attn_kernel<128>, llama8b_stack_128k: 256 tokens after the "
             "context, every layer): clock and matrix-unit counters",
             f"# command: {command}",
             f"# sources measured: query kernel sha256/16 {kernel_hash(QUERY_SRCS)}",
             f"# device: {xcc} XCDs, {simds} SIMDs, engine clock up to {fmax:.0f} MHz; dispatches with all four "
             f"counters and a duration: {len(rows)} (counter collection runs the dispatches one at a time)",
             f"duration per dispatch (same run): {us:.2f} us; GRBM_GUI_ACTIVE per XCD {cyc:.0f} cycles",
             f"effective clock (busy cycles / duration): mean {clock:.3f} GHz, min {clocks[0]:.3f}, "
             f"max {clocks[-1]:.3f}",
             f"matrix units busy (SQ_VALU_MFMA_BUSY_CYCLES / (busy cycles x {simds} SIMDs)): {busy:.1%}",
             f"bf16 matrix operations issued (SQ_INSTS_VALU_MFMA_MOPS_BF16 x 512): {issued / 1e9:.1f} GFLOP per "
             f"dispatch; algorithmic {alg_flops / 1e9:.1f} GFLOP per call (ratio {issued / alg_flops:.3f}: the bf16 "
             "remainder products of P, and key slots past a row's causal limit)",
             f"issued rate {rate:.0f} TFLOP/s = {rate / 2500:.1%} of 2.5 PFLOP/s (a {fmax / 1e3:.1f} GHz figure) and "
             f"{rate / (2500 * clock / (fmax / 1e3)):.1%} of the peak at the measured clock; algorithmic "
             f"{alg_flops / (us * 1e-6) / 1e12:.0f} TFLOP/s",
             "",
             f"JSON line of the counter run (dispatches serialised by counter collection): query_block us_per_layer "
             f"{qb['us_per_layer']}"]
    with open(QUERY_COUNTERS_FILE, "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def rel_err(got, want):
    """Max over output rows of |got - want|_inf / max(|want|_inf, 1e-30)."""
    import numpy as np
    got = np.asarray(got, np.float64)
    want = np.asarray(want, np.float64)
    return float((np.abs(got - want).max(-1) / np.maximum(np.abs(want).max(-1), 1e-30)).max())


def bench_configs(ctx):
    """The other configurations of the measurement plan, one row each: the
    8B-shaped layer at 32K, the 70B-shaped batch at each budget and the
    Qwen-shaped stack.  Every row times the packed step and the same build's
    dense decode, the one-time compaction, checks a sample of outputs against
    the oracle and (with the oracle baseline on) times the oracle on the same
    sample.  Caches whose step reads less than 1 GiB are rotated over
    copies, so no timed call finds its bytes in the 256 MB last-level cache
    from the call before.  Returns the rows and the decode calls they issued,
    in order (for the kernel-trace summary)."""
    import ctypes
    import numpy as np
    import torch

    import dkv_inputs as di
    d, lib, dev, stream, args = ctx["d"], ctx["lib"], ctx["dev"], ctx["stream"], ctx["args"]
    o = ctx.get("oracle")
    P = ctypes.c_void_p
    elem = 2
    gstream = torch.cuda.Stream()
    calls = []  # (label, decode calls issued), in issue order

    def ev():
        return torch.cuda.Event(enable_timing=True)

    def check(fn, *a):
        st = fn(*a)
        if st != 0:
            raise d.DkvError(fn.__name__, st)

    def replay_ms(g, reps, warm):
        sustain(g.replay)
        for _ in range(warm):
            g.replay()
        torch.cuda.synchronize()
        a, b = ev(), ev()
        a.record(stream)
        for _ in range(reps):
            g.replay()
        b.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(b) / reps

    def capture(fn):
        fn(stream.cuda_stream)  # eager once: code objects loaded, results defined
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=gstream):
            fn(gstream.cuda_stream)
        return g

    def timed_event(fn, reps=3):
        fn()  # warm
        torch.cuda.synchronize()
        a, b = ev(), ev()
        a.record(stream)
        for _ in range(reps):
            fn()
        b.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(b) * 1e3 / reps

    def pack(w, pattern, k, v, cap, lay):
        N, Hkv, T = w.num_units, w.num_kv_heads, w.context_len
        km = torch.empty((N, Hkv, T), dtype=torch.uint8, device=dev)
        kl = torch.empty((N, Hkv), dtype=torch.int32, device=dev)
        pat = torch.from_numpy(np.ascontiguousarray(pattern)).to(dev)
        map_us = timed_event(lambda: d.dkv_map_pattern(lay, pat, km, kl))
        lens = kl.cpu().to(torch.int64)
        rows = int((lens + cap).sum())
        # zeroed, so the two packs' buffers agree on the free rows neither writes
        k_c = torch.zeros((rows, w.head_dim), dtype=torch.bfloat16, device=dev)
        v_c = torch.zeros_like(k_c)
        so = torch.empty(N * Hkv, dtype=torch.int64, device=dev)
        sl = torch.empty(N * Hkv, dtype=torch.int32, device=dev)
        ws = torch.empty(d.dkv_compact_workspace_bytes(lay), dtype=torch.uint8, device=dev)
        c_us = timed_event(lambda: d.dkv_compact(lay, k, v, km, cap, k_c, v_c, so, sl, ws), reps=2)
        retained = int(lens.sum())
        c_bytes = 2 * 2 * retained * w.head_dim * elem + N * Hkv * T
        # the block gather from the pattern into a second buffer, checked against it
        k_b, v_b = torch.zeros_like(k_c), torch.zeros_like(v_c)
        so_b, sl_b = torch.empty_like(so), torch.empty_like(sl)
        bws = torch.empty(d.dkv_compact_bins_workspace_bytes(lay), dtype=torch.uint8, device=dev)
        b_us = timed_event(lambda: d.dkv_compact_bins(lay, k, v, pat, cap, k_b, v_b, so_b, sl_b, bws), reps=2)
        b_equal = bool(torch.equal(so_b, so) and torch.equal(sl_b, sl)
                       and torch.equal(k_b.view(torch.int16), k_c.view(torch.int16))
                       and torch.equal(v_b.view(torch.int16), v_c.view(torch.int16)))
        del k_b, v_b, bws
        b_bytes = 2 * 2 * retained * w.head_dim * elem
        one_time = {"map_us": round(map_us, 1), "compact_us": round(c_us, 1),
                    "compact_gb_per_s": round(c_bytes / (c_us * 1e-6) / 1e9, 1),
                    "map_write_gb_per_s": round(N * Hkv * T / (map_us * 1e-6) / 1e9, 1),
                    "compact_bins_us": round(b_us, 1),
                    "compact_bins_gb_per_s": round(b_bytes / (b_us * 1e-6) / 1e9, 1),
                    "compact_bins_equal_to_compact": b_equal}
        return dict(km=km, lens=lens, rows=rows, k_c=k_c, v_c=v_c, so=so, sl=sl, retained=retained,
                    one_time=one_time)

    def bits(t):
        return t.cpu().view(torch.int16).numpy().view(np.uint16)

    def copies_for(step_bytes):
        # enough copies that a call's bytes were last read >= 1 GiB earlier
        return max(1, -(-(1 << 30) // max(1, int(step_bytes))))

    rows = {}

    # ---------------- 8B-shaped layer at 32K ------------------------------
    w = di.workload("llama8b_layer_32k")
    B, Hq, Hkv, dim, T, cap = w.batch, w.num_q_heads, w.num_kv_heads, w.head_dim, w.context_len, w.append_cap
    nseg = B * Hkv
    pattern, pinfo = di.make_pattern(w)
    ku, vu = di.kv_unit(w, 0, device=dev)
    k, v = ku[None].contiguous(), vu[None].contiguous()
    del ku, vu
    lay = d.make_layout(1, Hq, Hkv, dim, T, w.sink, w.recent, list(w.bin_edges))
    pk = pack(w, pattern, k, v, cap, lay)
    q = di.q_step(w, 0, 0, device=dev).contiguous()
    kn, vn = (t.reshape(nseg, 1, dim).contiguous() for t in di.kv_new_step(w, 0, 0, device=dev))
    out = torch.empty((B, Hq, dim), dtype=torch.float32, device=dev)
    dws = torch.empty(d.dkv_decode_workspace_bytes(B, Hq, Hkv, dim), dtype=torch.uint8, device=dev)
    p_bytes = (pk["retained"] + nseg) * dim * elem * 2 + B * Hq * dim * (elem + 4) + nseg * 12
    d_bytes = nseg * (T + 1) * dim * elem * 2 + B * Hq * dim * (elem + 4)
    Rp, Rd = copies_for(p_bytes), copies_for(d_bytes)
    kcs = [pk["k_c"]] + [pk["k_c"].clone() for _ in range(Rp - 1)]
    vcs = [pk["v_c"]] + [pk["v_c"].clone() for _ in range(Rp - 1)]
    kds, vds = [], []
    for _ in range(Rd):
        kd_ = torch.zeros((B, Hkv, T + cap, dim), dtype=torch.bfloat16, device=dev)
        vd_ = torch.zeros_like(kd_)
        kd_[:, :, :T].copy_(k)
        vd_[:, :, :T].copy_(v)
        kds.append(kd_)
        vds.append(vd_)
    hint = pk["retained"] + nseg

    def packed_calls(shp):
        for r in range(Rp):
            check(lib.dkv_append_decode_attn, d.DKV_BF16, B, Hq, Hkv, dim, P(q.data_ptr()), P(kn.data_ptr()),
                  P(vn.data_ptr()), 1, 0, cap, P(kcs[r].data_ptr()), P(vcs[r].data_ptr()),
                  P(pk["so"].data_ptr()), P(pk["sl"].data_ptr()), w.sm_scale, hint, P(out.data_ptr()),
                  P(dws.data_ptr()), dws.numel(), P(shp))

    def dense_calls(shp):
        for r in range(Rd):
            check(lib.dkv_dense_append_decode_attn, d.DKV_BF16, B, Hq, Hkv, dim, P(q.data_ptr()),
                  P(kn.data_ptr()), P(vn.data_ptr()), 1, P(kds[r].data_ptr()), P(vds[r].data_ptr()), T + cap, T,
                  w.sm_scale, P(out.data_ptr()), P(dws.data_ptr()), dws.numel(), P(shp))

    g = capture(packed_calls)
    p_us = replay_ms(g, args.steps, args.warmup) * 1e3 / Rp
    calls.append(("llama8b_layer_32k packed", Rp * (1 + args.warmup + args.steps)))
    got = out.cpu().numpy()
    del g
    g = capture(dense_calls)
    dn_us = replay_ms(g, args.steps, args.warmup) * 1e3 / Rd
    calls.append(("llama8b_layer_32k dense", Rd * (1 + args.warmup + args.steps)))
    del g
    row = {"workload": w.name, "step": "one dkv_append_decode_attn (append 1 token, attend); HIP-graph replays "
                                      f"cycling over {Rp} copies of the packed cache ({Rd} of the dense one)",
           "retained_fraction": round(pk["retained"] / float(nseg * T), 4),
           "us_per_step": round(p_us, 2), "gb_per_s": round(p_bytes / (p_us * 1e-6) / 1e9, 1),
           "frac_of_peak": round(p_bytes / (p_us * 1e-6) / 1e9 / ctx["peak_hbm"], 4), "bytes_per_step": int(p_bytes),
           "dense": {"us_per_step": round(dn_us, 2), "gb_per_s": round(d_bytes / (dn_us * 1e-6) / 1e9, 1)},
           "speedup_vs_dense": round(dn_us / p_us, 3), "copies": {"packed": Rp, "dense": Rd},
           "one_time": pk["one_time"], "parity": None, "cpu_baseline": None}
    if o is not None:
        from threadpoolctl import threadpool_limits
        kb, vb = bits(k), bits(v)
        _, okm, _ = o.map_pattern(pattern, T, w.sink, w.recent, w.bin_edges, Hkv)
        with threadpool_limits(1):
            t0 = time.perf_counter()
            ref = o.compact(kb, vb, okm, cap)
            t_pack = time.perf_counter() - t0
            kc1, vc1 = o.append(ref["k_c"], ref["v_c"], ref["seg_off"], ref["seg_len"],
                                bits(kn).reshape(B, Hkv, 1, dim), bits(vn).reshape(B, Hkv, 1, dim), 0)
            t0 = time.perf_counter()
            want = o.decode_attn(bits(q), kc1, vc1, ref["seg_off"], ref["seg_len"], 1, w.sm_scale, Hkv, o.BF16)
            t_dec = time.perf_counter() - t0
        # the retained rows and the appended token of every segment (the rest
        # of the append room is never written)
        live = np.concatenate([np.arange(int(ref["seg_off"][s_]), int(ref["seg_off"][s_] + ref["seg_len"][s_]) + 1)
                               for s_ in range(nseg)])
        row["parity"] = {"max_rel_err": rel_err(got, want),
                         "seg_len_equal": bool(np.array_equal(pk["sl"].cpu().numpy(), ref["seg_len"])),
                         "packed_rows_equal": bool(np.array_equal(bits(pk["k_c"])[live], kc1[live]))}
        row["cpu_baseline"] = {"value": round(p_bytes / t_dec / 1e9, 4), "unit": "GB/s", "cores": 1, "kind": "oracle",
                               "sample": f"the whole step (one decode over the packed layer plus the appended token) "
                                         f"by the fp64 NumPy oracle, 1 BLAS thread: {t_dec:.3f} s",
                               "compaction_s": round(t_pack, 3)}
        del kb, vb, ref, kc1, vc1
    rows[w.name] = row
    del kcs, vcs, kds, vds, k, v, pk
    torch.cuda.empty_cache()

    # ---------------- 70B-shaped batch at each budget ---------------------
    w = di.workload("llama70b_layer_bs16_32k")
    B, Hq, Hkv, dim, T, cap, S = (w.batch, w.num_q_heads, w.num_kv_heads, w.head_dim, w.context_len,
                                  w.append_cap, w.decode_steps)
    nseg = B * Hkv
    k = torch.empty((B, Hkv, T, dim), dtype=torch.bfloat16, device=dev)
    v = torch.empty_like(k)
    for b_ in range(B):
        ku, vu = di.kv_unit(w, b_, device=dev)
        k[b_].copy_(ku)
        v[b_].copy_(vu)
    del ku, vu
    lay = d.make_layout(B, Hq, Hkv, dim, T, w.sink, w.recent, list(w.bin_edges))
    qs = [di.q_step(w, 0, s_, device=dev).contiguous() for s_ in range(S)]
    news = [tuple(t.reshape(nseg, 1, dim).contiguous() for t in di.kv_new_step(w, 0, s_, device=dev))
            for s_ in range(S)]
    k_all = torch.cat([kn_ for kn_, _ in news], dim=1).contiguous()  # [nseg][S][d]
    v_all = torch.cat([vn_ for _, vn_ in news], dim=1).contiguous()
    out = torch.empty((B, Hq, dim), dtype=torch.float32, device=dev)
    dws = torch.empty(d.dkv_decode_workspace_bytes(B, Hq, Hkv, dim), dtype=torch.uint8, device=dev)
    kd = torch.zeros((B, Hkv, T + cap, dim), dtype=torch.bfloat16, device=dev)
    vd = torch.zeros_like(kd)
    kd[:, :, :T].copy_(k)
    vd[:, :, :T].copy_(v)
    d_bytes = sum(nseg * (T + s_ + 1) * dim * elem * 2 for s_ in range(S)) / S + B * Hq * dim * (elem + 4)

    def dense_steps(shp):
        for s_ in range(S):
            kn_, vn_ = news[s_]
            check(lib.dkv_dense_append_decode_attn, d.DKV_BF16, B, Hq, Hkv, dim, P(qs[s_].data_ptr()),
                  P(kn_.data_ptr()), P(vn_.data_ptr()), 1, P(kd.data_ptr()), P(vd.data_ptr()), T + cap, T + s_,
                  w.sm_scale, P(out.data_ptr()), P(dws.data_ptr()), dws.numel(), P(shp))

    g = capture(dense_steps)
    dn_us = replay_ms(g, max(1, args.steps // 4), 1) * 1e3 / S
    calls.append(("llama70b dense", S * (1 + 1 + max(1, args.steps // 4))))
    del g, kd, vd
    torch.cuda.empty_cache()
    brow = {"workload": w.name, "steps": S, "step": "one dkv_append_decode_attn per step (append 1 token, attend "
                                                      "the whole batch); the 16 steps as one HIP graph",
            "dense": {"us_per_step": round(dn_us, 2), "gb_per_s": round(d_bytes / (dn_us * 1e-6) / 1e9, 1),
                      "frac_of_peak": round(d_bytes / (dn_us * 1e-6) / 1e9 / ctx["peak_hbm"], 4)}}
    for budget in w.budgets:
        pattern, pinfo = di.make_pattern(w, budget=budget)
        pk = pack(w, pattern, k, v, cap, lay)
        # every step's token written once up front (untimed), so each copy
        # holds what the sequential steps would have appended before it
        d.dkv_append(k_all, v_all, 0, cap, pk["k_c"], pk["v_c"], pk["so"], pk["sl"])
        p_bytes = (sum((pk["retained"] + nseg * (s_ + 1)) for s_ in range(S)) / S * dim * elem * 2
                   + B * Hq * dim * (elem + 4) + nseg * 12)
        R = copies_for(p_bytes)
        kcs = [pk["k_c"]] + [pk["k_c"].clone() for _ in range(R - 1)]
        vcs = [pk["v_c"]] + [pk["v_c"].clone() for _ in range(R - 1)]

        def packed_steps(shp):
            for s_ in range(S):
                kn_, vn_ = news[s_]
                r = s_ % R
                check(lib.dkv_append_decode_attn, d.DKV_BF16, B, Hq, Hkv, dim, P(qs[s_].data_ptr()),
                      P(kn_.data_ptr()), P(vn_.data_ptr()), 1, s_, cap, P(kcs[r].data_ptr()), P(vcs[r].data_ptr()),
                      P(pk["so"].data_ptr()), P(pk["sl"].data_ptr()), w.sm_scale, pk["retained"] + nseg * (s_ + 1),
                      P(out.data_ptr()), P(dws.data_ptr()), dws.numel(), P(shp))

        g = capture(packed_steps)
        p_us = replay_ms(g, args.steps, args.warmup) * 1e3 / S
        calls.append((f"llama70b packed {budget}", S * (1 + args.warmup + args.steps)))
        got = out.cpu().numpy()  # the last step: every sequence, all 16 tokens appended
        del g
        seg = pk["lens"].view(-1).to(torch.float64)
        r_ = {"retained_fraction": round(pk["retained"] / float(nseg * T), 4),
              "us_per_step": round(p_us, 2), "gb_per_s": round(p_bytes / (p_us * 1e-6) / 1e9, 1),
              "frac_of_peak": round(p_bytes / (p_us * 1e-6) / 1e9 / ctx["peak_hbm"], 4),
              "bytes_per_step": int(p_bytes), "speedup_vs_dense": round(dn_us / p_us, 3), "copies": R,
              "segment_rows": {"min": int(seg.min()), "max": int(seg.max()),
                               "cv": round(float(seg.std() / seg.mean()), 3)},
              "one_time": pk["one_time"], "parity": None, "cpu_baseline": None}
        if o is not None:
            from threadpoolctl import threadpool_limits
            ns = 2  # sample: the first two sequences, at the last step
            _, okm, _ = o.map_pattern(pattern[:ns], T, w.sink, w.recent, w.bin_edges, Hkv)
            with threadpool_limits(1):
                t0 = time.perf_counter()
                ref = o.compact(bits(k[:ns]), bits(v[:ns]), okm, cap)
                t_pack = time.perf_counter() - t0
                kc1, vc1 = o.append(ref["k_c"], ref["v_c"], ref["seg_off"], ref["seg_len"],
                                    bits(k_all[:ns * Hkv]).reshape(ns, Hkv, S, dim),
                                    bits(v_all[:ns * Hkv]).reshape(ns, Hkv, S, dim), 0)
                t0 = time.perf_counter()
                want = o.decode_attn(bits(qs[S - 1][:ns]), kc1, vc1, ref["seg_off"], ref["seg_len"], S, w.sm_scale,
                                     Hkv, o.BF16)
                t_dec = time.perf_counter() - t0
            s_bytes = (int(ref["seg_len"].sum()) + ns * Hkv * S) * dim * elem * 2
            r_["parity"] = {"sequences": ns, "step": S - 1, "max_rel_err": rel_err(got[:ns], want),
                            "seg_len_equal": bool(np.array_equal(pk["sl"].cpu().numpy()[:ns * Hkv], ref["seg_len"]))}
            r_["cpu_baseline"] = {"value": round(s_bytes / t_dec / 1e9, 4), "unit": "GB/s", "cores": 1,
                                  "kind": "oracle",
                                  "sample": f"the last decode step of sequences 0-{ns - 1} by the fp64 NumPy oracle, "
                                            f"1 BLAS thread: {t_dec:.3f} s", "compaction_s_sample": round(t_pack, 3)}
        brow[f"budget_{budget}"] = r_
        del kcs, vcs, pk
        torch.cuda.empty_cache()
    rows[w.name] = brow
    del k, v, k_all, v_all
    torch.cuda.empty_cache()

    # ---------------- Qwen-shaped stack, batch 4, 128K --------------------
    w = di.workload("qwen7b_stack_bs4_128k")
    L, B, Hq, Hkv, dim, T, cap = (w.num_layers, w.batch, w.num_q_heads, w.num_kv_heads, w.head_dim, w.context_len,
                                  w.append_cap)
    N, S, nsl = w.num_units, w.decode_steps, B * Hkv
    k = torch.empty((N, Hkv, T, dim), dtype=torch.bfloat16, device=dev)
    v = torch.empty_like(k)
    for u in range(N):
        ku, vu = di.kv_unit(w, u, device=dev)
        k[u].copy_(ku)
        v[u].copy_(vu)
        del ku, vu
    pattern, pinfo = di.make_pattern(w)
    lay = d.make_layout(N, Hq, Hkv, dim, T, w.sink, w.recent, list(w.bin_edges))
    pk = pack(w, pattern, k, v, cap, lay)
    qs = [di.q_step(w, layer, 0, device=dev).contiguous() for layer in range(L)]
    news = [tuple(t.reshape(nsl, 1, dim).contiguous() for t in di.kv_new_step(w, layer, 0, device=dev))
            for layer in range(L)]
    outs = torch.empty((L, B, Hq, dim), dtype=torch.float32, device=dev)
    dws = torch.empty(d.dkv_decode_workspace_bytes(B, Hq, Hkv, dim), dtype=torch.uint8, device=dev)
    lrows = [int(pk["lens"][layer * B:(layer + 1) * B].sum()) for layer in range(L)]

    def gen_steps(shp):  # all 256 steps of the generation, 28 layers each
        for s_ in range(S):
            for layer in range(L):
                off = layer * nsl
                kn_, vn_ = news[layer]
                check(lib.dkv_append_decode_attn, d.DKV_BF16, B, Hq, Hkv, dim, P(qs[layer].data_ptr()),
                      P(kn_.data_ptr()), P(vn_.data_ptr()), 1, s_, cap, P(pk["k_c"].data_ptr()),
                      P(pk["v_c"].data_ptr()), P(pk["so"].data_ptr() + 8 * off), P(pk["sl"].data_ptr() + 4 * off),
                      w.sm_scale, lrows[layer] + nsl * (s_ + 1), P(outs[layer].data_ptr()), P(dws.data_ptr()),
                      dws.numel(), P(shp))

    g = capture(gen_steps)
    reps = max(1, args.steps // 10)
    p_us = replay_ms(g, reps, 1) * 1e3 / S
    calls.append(("qwen packed", S * L * (1 + 1 + reps)))
    got_last = outs[0].cpu().numpy()  # layer 0 after the last of the 256 steps
    del g
    p_bytes = (sum(pk["retained"] + N * Hkv * (s_ + 1) for s_ in range(S)) / S * dim * elem * 2
               + L * B * Hq * dim * (elem + 4) + N * Hkv * 12)

    def dense_step(shp):  # attend-only over the dense cache (no room to append in it)
        for layer in range(L):
            u = slice(layer * B, (layer + 1) * B)
            check(lib.dkv_dense_decode_attn, d.DKV_BF16, B, Hq, Hkv, dim, P(qs[layer].data_ptr()),
                  P(k[u].data_ptr()), P(v[u].data_ptr()), T, T, w.sm_scale, P(outs[layer].data_ptr()),
                  P(dws.data_ptr()), dws.numel(), P(shp))

    g = capture(dense_step)
    dreps = max(2, args.steps // 4)
    dn_us = replay_ms(g, dreps, 1) * 1e3
    calls.append(("qwen dense", L * (1 + 1 + dreps)))
    del g
    d_bytes = N * Hkv * T * dim * elem * 2 + L * B * Hq * dim * (elem + 4)
    seg = pk["lens"].view(-1).to(torch.float64)
    qrow = {"workload": w.name, "layers": L, "batch": B, "steps": S,
            "step": "per layer one dkv_append_decode_attn (append 1 token per sequence, attend); the 256 steps of "
                    "the generation as one HIP graph",
            "retained_fraction": round(pk["retained"] / float(N * Hkv * T), 4),
            "us_per_step": round(p_us, 1), "us_per_layer": round(p_us / L, 2),
            "gb_per_s": round(p_bytes / (p_us * 1e-6) / 1e9, 1),
            "frac_of_peak": round(p_bytes / (p_us * 1e-6) / 1e9 / ctx["peak_hbm"], 4),
            "bytes_per_step": int(p_bytes),
            "dense": {"us_per_step": round(dn_us, 1), "gb_per_s": round(d_bytes / (dn_us * 1e-6) / 1e9, 1),
                      "frac_of_peak": round(d_bytes / (dn_us * 1e-6) / 1e9 / ctx["peak_hbm"], 4),
                      "step": "per layer one dkv_dense_decode_attn over the 131,072 context rows (attend only)"},
            "speedup_vs_dense": round(dn_us / p_us, 3),
            "segment_rows": {"min": int(seg.min()), "max": int(seg.max()), "cv": round(float(seg.std() / seg.mean()), 3)},
            "one_time": pk["one_time"], "all_keep_equals_dense": None, "parity": None, "cpu_baseline": None}
    # all-keep pattern on layer 0: the packed decode must give the dense kernel's result bit for bit
    lay0 = d.make_layout(B, Hq, Hkv, dim, T, w.sink, w.recent, list(w.bin_edges))
    wk = di.workload(w.name, num_layers=1)
    pk1 = pack(wk, np.ones((B, Hq, w.num_bins), np.uint8), k[:B], v[:B], 0, lay0)
    o_p = torch.empty((B, Hq, dim), dtype=torch.float32, device=dev)
    o_d = torch.empty_like(o_p)
    d.dkv_decode_attn(qs[0], pk1["k_c"], pk1["v_c"], pk1["so"], pk1["sl"], 0, w.sm_scale, o_p, dws, Hkv,
                      rows_hint=pk1["rows"])
    d.dkv_dense_decode_attn(qs[0], k[:B], v[:B], T, w.sm_scale, o_d, dws)
    torch.cuda.synchronize()
    calls.append(("qwen all-keep check", 2))
    qrow["all_keep_equals_dense"] = bool(torch.equal(o_p, o_d))
    del pk1
    if o is not None:
        from threadpoolctl import threadpool_limits
        _, okm, _ = o.map_pattern(pattern[:B], T, w.sink, w.recent, w.bin_edges, Hkv)
        with threadpool_limits(1):
            t0 = time.perf_counter()
            ref = o.compact(bits(k[:B]), bits(v[:B]), okm, cap)
            t_pack = time.perf_counter() - t0
            kn0 = np.repeat(bits(news[0][0]).reshape(B, Hkv, 1, dim), S, axis=2)
            vn0 = np.repeat(bits(news[0][1]).reshape(B, Hkv, 1, dim), S, axis=2)
            kc1, vc1 = o.append(ref["k_c"], ref["v_c"], ref["seg_off"], ref["seg_len"], kn0, vn0, 0)
            t0 = time.perf_counter()
            want = o.decode_attn(bits(qs[0]), kc1, vc1, ref["seg_off"], ref["seg_len"], S, w.sm_scale, Hkv, o.BF16)
            t_dec = time.perf_counter() - t0
        l_bytes = (int(ref["seg_len"].sum()) + nsl * S) * dim * elem * 2
        qrow["parity"] = {"layer": 0, "step": S - 1, "max_rel_err": rel_err(got_last, want),
                          "seg_len_equal": bool(np.array_equal(pk["sl"].cpu().numpy()[:nsl], ref["seg_len"]))}
        qrow["cpu_baseline"] = {"value": round(l_bytes / t_dec / 1e9, 4), "unit": "GB/s", "cores": 1, "kind": "oracle",
                                "sample": f"the last step of layer 0 (4 sequences) by the fp64 NumPy oracle, 1 BLAS "
                                          f"thread: {t_dec:.3f} s; a 28-layer step scales to {t_dec * L:.2f} s",
                                "compaction_s_layer0": round(t_pack, 3)}
    rows[w.name] = qrow
    del k, v, pk
    torch.cuda.empty_cache()
    return rows, calls


def phase_budget(args):
    """Where the time of one decode call goes, for the headline stack, the
    70B-shaped batch (20% budget) and the Qwen-shaped stack: their decode
    steps (fused append + decode calls) captured as graphs through the
    phase-stamp build and replayed; per-workgroup clock stamps (100 MHz, one
    clock for the whole chip) give, per call, the prologue, the stream, the
    tail of the slowest workgroups, the fold, the combine kernel and the gaps
    between kernels.  The product library's graphs of the same steps are
    timed in the same run, and so is the streaming-read probe over the same
    bytes."""
    import ctypes
    import numpy as np
    import torch

    import dkv_inputs as di
    import paper_2609_32663_amd as d
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream()
    lib = d.library()
    plib = d.library_at(PHASE_LIB)
    plib.dkv_phase_stamps.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
    plib.dkv_phase_stamps.restype = ctypes.c_int
    plib.dkv_phase_reset.argtypes = []
    plib.dkv_phase_reset.restype = None
    P = ctypes.c_void_p
    cs = torch.cuda.Stream()

    def ev():
        return torch.cuda.Event(enable_timing=True)

    def case(name, budget=None):
        w = di.workload(name)
        L, B, Hq, Hkv, dim, T, cap, N = (w.num_layers, w.batch, w.num_q_heads, w.num_kv_heads, w.head_dim,
                                         w.context_len, w.append_cap, w.num_units)
        nsl = B * Hkv
        log(f"phase budget: {name}")
        pattern, _ = di.make_pattern(w, budget=budget)
        k = torch.empty((N, Hkv, T, dim), dtype=torch.bfloat16, device=dev)
        v = torch.empty_like(k)
        for u in range(N):
            ku, vu = di.kv_unit(w, u, device=dev)
            k[u].copy_(ku)
            v[u].copy_(vu)
            del ku, vu
        lay = d.make_layout(N, Hq, Hkv, dim, T, w.sink, w.recent, list(w.bin_edges))
        km = torch.empty((N, Hkv, T), dtype=torch.uint8, device=dev)
        kl = torch.empty((N, Hkv), dtype=torch.int32, device=dev)
        d.dkv_map_pattern(lay, torch.from_numpy(pattern).to(dev), km, kl)
        lens = kl.cpu().to(torch.int64)
        rows = int((lens + cap).sum())
        k_c = torch.empty((rows, dim), dtype=torch.bfloat16, device=dev)
        v_c = torch.empty_like(k_c)
        so = torch.empty(N * Hkv, dtype=torch.int64, device=dev)
        sl = torch.empty(N * Hkv, dtype=torch.int32, device=dev)
        cws = torch.empty(d.dkv_compact_workspace_bytes(lay), dtype=torch.uint8, device=dev)
        d.dkv_compact(lay, k, v, km, cap, k_c, v_c, so, sl, cws)
        del k, v, km
        torch.cuda.empty_cache()
        qs = [di.q_step(w, layer, 0, device=dev) for layer in range(L)]
        news = [tuple(t.reshape(nsl, 1, dim).contiguous() for t in di.kv_new_step(w, layer, 0, device=dev))
                for layer in range(L)]
        out = torch.empty((B, Hq, dim), dtype=torch.float32, device=dev)
        dws = torch.zeros(d.dkv_decode_workspace_bytes(B, Hq, Hkv, dim), dtype=torch.uint8, device=dev)
        lrows = [int(lens[layer * B:(layer + 1) * B].sum()) for layer in range(L)]
        # a graph of `per_graph` calls: whole steps of the stack, or (one layer) several steps
        steps_per_graph = max(1, 32 // L)
        per_graph = L * steps_per_graph

        def graph_calls(lb, g_idx, shp):
            for j in range(steps_per_graph):
                s_ = (g_idx * steps_per_graph + j) % cap
                for layer in range(L):
                    kn, vn = news[layer]
                    st_ = lb.dkv_append_decode_attn(d.DKV_BF16, B, Hq, Hkv, dim, P(qs[layer].data_ptr()),
                                                    P(kn.data_ptr()), P(vn.data_ptr()), 1, s_, cap, P(k_c.data_ptr()),
                                                    P(v_c.data_ptr()), P(so.data_ptr() + 8 * layer * nsl),
                                                    P(sl.data_ptr() + 4 * layer * nsl), w.sm_scale,
                                                    lrows[layer] + nsl * (s_ + 1), P(out.data_ptr()),
                                                    P(dws.data_ptr()), dws.numel(), P(shp))
                    if st_ != 0:
                        raise d.DkvError("dkv_append_decode_attn", st_)

        n_graphs, n_warm = 8, 5

        def graphs_of(lb):
            gs = []
            for gi in range(n_graphs):
                g = torch.cuda.CUDAGraph()
                with torch.cuda.graph(g, stream=cs):
                    graph_calls(lb, gi, cs.cuda_stream)
                gs.append(g)
            return gs

        graph_calls(lib, 0, stream.cuda_stream)
        torch.cuda.synchronize()
        prod = graphs_of(lib)
        for g in prod[:n_warm]:
            g.replay()
        torch.cuda.synchronize()
        a, b = ev(), ev()
        a.record(stream)
        for g in prod[n_warm:]:
            g.replay()
        b.record(stream)
        torch.cuda.synchronize()
        prod_us = a.elapsed_time(b) * 1e3 / (n_graphs - n_warm) / per_graph
        del prod

        plib.dkv_phase_reset()  # graph g, call c -> slot (g * per_graph + c) % 64
        stamped = graphs_of(plib)
        for g in stamped[:n_warm]:
            g.replay()
        torch.cuda.synchronize()
        split = np.zeros((64, 1024, 8), dtype=np.uint64)
        merge = np.zeros((64, 4096, 2), dtype=np.uint64)
        calls, stamped_us = [], []
        rel_by_layer = {}  # layer -> per-call arrays of each workgroup's last tile minus the call's median
        for gi in range(n_warm, n_graphs):
            a.record(stream)
            stamped[gi].replay()
            b.record(stream)
            torch.cuda.synchronize()
            stamped_us.append(a.elapsed_time(b) * 1e3 / per_graph)
            st_ = plib.dkv_phase_stamps(P(split.ctypes.data), P(merge.ctypes.data))
            if st_ != 0:
                raise RuntimeError(f"dkv_phase_stamps: {st_}")
            for c in range(min(per_graph, 64) - 1):  # the last call of a graph has no next call in it
                sl_ = (gi * per_graph + c) % 64
                nx = (sl_ + 1) % 64
                t = split[sl_].astype(np.int64)
                used = t[:, 0] > 0
                wg = np.nonzero(used)[0]
                t = t[used]
                m = merge[sl_][:nsl * w.group].astype(np.int64)
                t0 = t[:, 0].min()
                us = lambda x: (x - t0) * 0.01  # 100 MHz
                nt = split[nx].astype(np.int64)
                nt = nt[nt[:, 0] > 0]
                loop_end = us(t[:, 3:7].max(1))
                rel = np.full(split.shape[1], np.nan)
                rel[wg] = loop_end - np.median(loop_end)
                rel_by_layer.setdefault(c % L, []).append(rel)
                calls.append({
                    "workgroups": float(used.sum()),
                    "last_start": float(us(t[:, 0]).max()),
                    "prologue_p50": float(np.median(us(t[:, 1]))),
                    "first_tile_p50": float(np.median(us(t[:, 2]))),
                    "loop_end_p50": float(np.median(loop_end)),
                    "loop_end_max": float(loop_end.max()),
                    "fold_p50": float(np.median(us(t[:, 7]) - loop_end)),
                    "wg_end_p10": float(np.percentile(us(t[:, 7]), 10)),
                    "wg_end_p50": float(np.median(us(t[:, 7]))),
                    "wg_end_max": float(us(t[:, 7]).max()),
                    "combine_start": float(us(m[:, 0]).min()),
                    "combine_end": float(us(m[:, 1]).max()),
                    "next_start": float(us(nt[:, 0]).min()),
                    "xcd": [float(np.median(us(t[wg % 8 == x, 7]))) for x in range(8)],
                })
        c = {k_: float(np.mean([x[k_] for x in calls])) for k_ in calls[0] if k_ != "xcd"}
        # spread of the workgroups' last tiles within a call, and the part of it
        # that stays with a workgroup over calls of the same layer
        within = float(np.mean([np.nanstd(r) for v in rel_by_layer.values() for r in v]))
        persist = float(np.mean([np.nanstd(np.nanmean(np.array(v), 0)) for v in rel_by_layer.values() if len(v) > 1]))
        xcd = np.mean([x["xcd"] for x in calls], axis=0)
        # bytes of a call of the stamped replays
        tails = [(gi * steps_per_graph + j) % cap + 1 for gi in range(n_warm, n_graphs) for j in range(steps_per_graph)]
        nbytes = int(np.mean([(lrows[layer] + nsl * t_) * dim * 2 * 2 + B * Hq * dim * 6 + nsl * 12
                              for layer in range(L) for t_ in tails]))
        del stamped, k_c, v_c
        torch.cuda.empty_cache()

        # the streaming-read probe over the same bytes, one launch per call, graph-replayed
        per = (nbytes + 15) // 16 * 16
        pbuf = torch.ones(32 * per // 2, dtype=torch.int16, device=dev)
        psink = torch.zeros(4, dtype=torch.int32, device=dev)
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=cs):
            for i in range(32):
                lib.dkv_probe_stream_read(P(pbuf.data_ptr() + i * per), per, P(psink.data_ptr()), 2,
                                          P(cs.cuda_stream))
        for _ in range(3):
            g.replay()
        torch.cuda.synchronize()
        a.record(stream)
        for _ in range(5):
            g.replay()
        b.record(stream)
        torch.cuda.synchronize()
        probe_us = a.elapsed_time(b) * 1e3 / 5 / 32
        del pbuf, g

        stream_us = c["loop_end_p50"] - c["prologue_p50"]
        terms = [
            ("launch skew + prologue (metadata round trip, scan; no K/V bytes in flight yet)", c["prologue_p50"]),
            ("stream: prologue end -> median workgroup's last tile", stream_us),
            ("tail: median -> slowest workgroup's last tile", c["loop_end_max"] - c["loop_end_p50"]),
            ("fold after the slowest last tile (waves -> output or record)", c["wg_end_max"] - c["loop_end_max"]),
            ("gap: split kernel end -> combine start", c["combine_start"] - c["wg_end_max"]),
            ("combine kernel", c["combine_end"] - c["combine_start"]),
            ("gap: combine end -> next call's first workgroup", c["next_start"] - c["combine_end"]),
        ]
        lines = [f"## {name}" + (f" at {budget:.0%} retained" if budget else "") +
                 f": {L} layer(s) x batch {B} x {Hq}q/{Hkv}kv, d {dim}, T {T}; {nbytes / 1e6:.1f} MB of K/V per call",
                 f"# graph-replayed decode steps; means over {len(calls)} calls of {n_graphs - n_warm} replays; "
                 "times in us from the call's first workgroup start",
                 f"product library, same graphs: {prod_us:.2f} us per call = {nbytes / (prod_us * 1e-6) / 1e9:.0f} GB/s "
                 f"({nbytes / (prod_us * 1e-6) / 1e9 / PEAK_HBM_GBPS:.1%} of 8 TB/s); stamped library "
                 f"{np.mean(stamped_us):.2f} us per call",
                 f"streaming-read probe over the same bytes (8 KiB per workgroup, graph-replayed): {probe_us:.2f} us per "
                 f"launch = {per / (probe_us * 1e-6) / 1e9:.0f} GB/s",
                 f"{'term':78s} {'us':>7s}"]
        for nm, val in terms:
            lines.append(f"{nm:78s} {val:7.2f}")
        lines += [f"{'call period (sum)':78s} {c['next_start']:7.2f}",
                  f"stream rate over the stream term: {nbytes / (stream_us * 1e-6) / 1e9:.0f} GB/s; workgroups "
                  f"{c['workgroups']:.0f}; last start {c['last_start']:.2f}; first tile reached (wave 0, median) "
                  f"{c['first_tile_p50']:.2f}; per-workgroup fold median {c['fold_p50']:.2f}",
                  f"workgroup end p10 / p50 / max: {c['wg_end_p10']:.2f} / {c['wg_end_p50']:.2f} / "
                  f"{c['wg_end_max']:.2f}; median end by XCD (id mod 8): " + ", ".join(f"{x:.2f}" for x in xcd),
                  f"workgroups' last tiles within a call: std {within:.2f}; of which persistent (std over workgroups "
                  f"of their mean over calls of the same layer): {persist:.2f}", ""]
        return lines

    lines = ["# per-phase time budget of decode calls (dkv_append_decode_attn: split kernel + combine kernel)",
             "# command: python paper_2609_32663_amd/build.py --phase-stamps && python bench.py --phase-budget",
             f"# sources measured: decode kernel sha256/16 {kernel_hash()} (stamps compiled in with "
             "DKV_PHASE_STAMPS=1; the product library has none); 100 MHz chip clock", ""]
    lines += case(WORKLOAD)
    lines += case("llama70b_layer_bs16_32k", 0.2)
    lines += case("qwen7b_stack_bs4_128k")
    with open(PHASE_FILE, "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def main():
    global SUSTAIN_ON
    args = parse()
    SUSTAIN_ON = not args.no_sustain
    if args.phase_budget:
        phase_budget(args)
        return
    if args.pmc_summary:
        pmc_summary(*args.pmc_summary, args.pmc_command)
        return
    if args.query_counters:
        query_counters(*args.query_counters, args.pmc_command)
        return
    if args.power_sample:
        power_sample()
        return
    if args.trace_summary:
        trace_summary(*args.trace_summary, args.pmc_command)
        return
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
    d.dkv_map_pattern(lay, pat_d, kv_mask, kv_len)  # first launch loads the code object
    torch.cuda.synchronize()
    e0.record(stream)
    d.dkv_map_pattern(lay, pat_d, kv_mask, kv_len)
    e1.record(stream)
    torch.cuda.synchronize()
    map_us = e0.elapsed_time(e1) * 1e3
    # kernel time: 20 calls back to back (no synchronisation between them)
    e0.record(stream)
    for _ in range(20):
        d.dkv_map_pattern(lay, pat_d, kv_mask, kv_len)
    e1.record(stream)
    torch.cuda.synchronize()
    map_b2b_us = e0.elapsed_time(e1) * 1e3 / 20
    lens = kv_len.cpu().to(torch.int64)
    rows = int((lens + cap).sum())
    # zeroed, so the two packs' buffers agree on the free rows neither writes
    k_c = torch.zeros((rows, dim), dtype=torch.bfloat16, device=dev)
    v_c = torch.zeros_like(k_c)
    seg_off = torch.empty(N * Hkv, dtype=torch.int64, device=dev)
    seg_len = torch.empty(N * Hkv, dtype=torch.int32, device=dev)
    cws = torch.empty(d.dkv_compact_workspace_bytes(lay), dtype=torch.uint8, device=dev)
    d.dkv_compact(lay, k, v, kv_mask, cap, k_c, v_c, seg_off, seg_len, cws)  # loads the code objects
    torch.cuda.synchronize()
    compact_ms = []
    for _ in range(3):  # best of three single calls (as for dkv_compact_bins below)
        e1.record(stream)
        d.dkv_compact(lay, k, v, kv_mask, cap, k_c, v_c, seg_off, seg_len, cws)
        e2.record(stream)
        torch.cuda.synchronize()
        compact_ms.append(e1.elapsed_time(e2))
    compact_us = min(compact_ms) * 1e3
    retained = int(lens.sum())
    compact_bytes = 2 * 2 * retained * dim * elem + N * Hkv * T  # K,V read+write + mask
    phys_frac = retained / float(N * Hkv * T)
    log(f"map {map_us:.0f} us, compact {compact_us:.0f} us, retained {phys_frac:.4f}")
    # the same pack straight from the pattern (block gather: no mask), into a
    # second buffer, checked bit for bit against dkv_compact's
    k_b, v_b = torch.zeros_like(k_c), torch.zeros_like(v_c)
    seg_off_b, seg_len_b = torch.empty_like(seg_off), torch.empty_like(seg_len)
    bws = torch.empty(d.dkv_compact_bins_workspace_bytes(lay), dtype=torch.uint8, device=dev)
    d.dkv_compact_bins(lay, k, v, pat_d, cap, k_b, v_b, seg_off_b, seg_len_b, bws)
    torch.cuda.synchronize()
    bins_ms = []
    for _ in range(3):
        e1.record(stream)
        d.dkv_compact_bins(lay, k, v, pat_d, cap, k_b, v_b, seg_off_b, seg_len_b, bws)
        e2.record(stream)
        torch.cuda.synchronize()
        bins_ms.append(e1.elapsed_time(e2))
    bins_us = min(bins_ms) * 1e3
    bins_equal = bool(torch.equal(seg_off_b, seg_off) and torch.equal(seg_len_b, seg_len)
                      and torch.equal(k_b.view(torch.int16), k_c.view(torch.int16))
                      and torch.equal(v_b.view(torch.int16), v_c.view(torch.int16)))
    del k_b, v_b, bws
    torch.cuda.empty_cache()
    bins_bytes = 2 * 2 * retained * dim * elem
    log(f"compact_bins {bins_us:.0f} us ({bins_bytes / (bins_us * 1e-6) / 1e9:.0f} GB/s), "
        f"equal to compact: {bins_equal}")
    # what a plain copy of the same bytes reaches: dkv_probe_copy of the
    # retained K and V bytes (one block of 4, 8 or 16 KiB per workgroup,
    # 16-byte non-temporal loads and stores)
    copy_bytes = 2 * retained * dim * elem
    csrc = torch.ones(copy_bytes // 2, dtype=torch.int16, device=dev)
    cdst = torch.empty_like(csrc)
    copy_gbps = {}
    for g in (1, 2, 4):
        d.dkv_probe_copy(csrc, cdst, g)
        torch.cuda.synchronize()
        e1.record(stream)
        for _ in range(3):
            d.dkv_probe_copy(csrc, cdst, g)
        e2.record(stream)
        torch.cuda.synchronize()
        copy_gbps[f"{4 * g}KiB"] = round(2 * copy_bytes / (e1.elapsed_time(e2) / 3 * 1e-3) / 1e9, 1)
    del csrc, cdst
    torch.cuda.empty_cache()
    log(f"copy probe over the packed bytes (read + write GB/s): {copy_gbps}")

    # ---------------- query block: a second pack with room for it ----------
    # The tokens after the context (the paper reserves 256 for query and
    # answer) are appended to every segment and attend to the packed context
    # and causally to themselves.
    NQ = QUERY_TOKENS
    cap_q = NQ + MT_STEPS  # room for the block and the tokens generated after it
    rows_q = int((lens + cap_q).sum())
    k_q = torch.empty((rows_q, dim), dtype=torch.bfloat16, device=dev)
    v_q = torch.empty_like(k_q)
    seg_off_q = torch.empty(N * Hkv, dtype=torch.int64, device=dev)
    seg_len_q = torch.empty(N * Hkv, dtype=torch.int32, device=dev)
    d.dkv_compact(lay, k, v, kv_mask, cap_q, k_q, v_q, seg_off_q, seg_len_q, cws)
    q_blocks, kv_blocks = [], []
    for layer in range(L):
        qb, kb, vb = di.query_block(w, layer, NQ, device=dev)
        segs = slice(layer * nseg_layer, (layer + 1) * nseg_layer)
        kb, vb = kb.reshape(nseg_layer, NQ, dim).contiguous(), vb.reshape(nseg_layer, NQ, dim).contiguous()
        d.dkv_append(kb, vb, 0, cap_q, k_q, v_q, seg_off_q[segs], seg_len_q[segs])
        q_blocks.append(qb.contiguous())
        kv_blocks.append((kb, vb))
    torch.cuda.synchronize()

    # ---------------- CPU oracle baseline + parity sample (layer 0) --------
    cpu = None
    cpu_all = None
    cpu_pack = None
    parity = None
    dws = torch.zeros(d.dkv_decode_workspace_bytes(B, Hq, Hkv, dim), dtype=torch.uint8, device=dev)
    out = torch.empty((B, Hq, dim), dtype=torch.float32, device=dev)
    if not args.no_cpu_baseline:
        import oracle as o
        from threadpoolctl import threadpool_limits
        log("oracle baseline: two decode steps over all layers")

        def bits_of(t):
            return t.cpu().view(torch.int16).numpy().view(np.uint16)
        cpu_s, sample_bytes, worst, same_pack = 0.0, 0, 0.0, True
        all_cores = len(os.sched_getaffinity(0))
        all_s, all_bytes, all_layers = 0.0, 0, min(4, L)
        pack_s, pack_bytes = 0.0, 0
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
            if layer == 0:  # kept for the query-block oracle sample
                k0_bits, v0_bits, okm0 = kb, vb, okm
            with threadpool_limits(1):
                t0 = time.perf_counter()
                ref = o.compact(kb, vb, okm, cap)
                pack_s += time.perf_counter() - t0
            pack_bytes += 2 * 2 * int(okm.sum()) * dim * elem + int(okm.size)
            with threadpool_limits(1):
                t0 = time.perf_counter()
                want = o.decode_attn(qb, ref["k_c"], ref["v_c"], ref["seg_off"], ref["seg_len"], 0,
                                     w.sm_scale, Hkv, o.BF16)
                cpu_s += time.perf_counter() - t0
            sample_bytes += int(ref["seg_len"].sum()) * dim * elem * 2 + B * Hq * dim * (elem + 4)
            if layer < all_layers:  # the same step with every host core the process may use
                with threadpool_limits(all_cores):
                    t0 = time.perf_counter()
                    o.decode_attn(qb, ref["k_c"], ref["v_c"], ref["seg_off"], ref["seg_len"], 0, w.sm_scale, Hkv,
                                  o.BF16)
                    all_s += time.perf_counter() - t0
                all_bytes += int(ref["seg_len"].sum()) * dim * elem * 2 + B * Hq * dim * (elem + 4)
            # second step of the sample: the step's token appended, then attend
            kn, vn = (bits_of(t).reshape(B, Hkv, 1, dim) for t in new_kv[layer])
            k1, v1 = o.append(ref["k_c"], ref["v_c"], ref["seg_off"], ref["seg_len"], kn, vn, 0)
            with threadpool_limits(1):
                t0 = time.perf_counter()
                o.decode_attn(qb, k1, v1, ref["seg_off"], ref["seg_len"], 1, w.sm_scale, Hkv, o.BF16)
                cpu_s += time.perf_counter() - t0
            sample_bytes += (int(ref["seg_len"].sum()) + nseg_layer) * dim * elem * 2 + B * Hq * dim * (elem + 4)
            del k1, v1
            err = float((np.abs(got - want).max(-1) / np.maximum(np.abs(want).max(-1), 1e-30)).max())
            worst = max(worst, err)
            same_pack &= bool(np.array_equal(seg_len[segs].cpu().numpy(), ref["seg_len"]))
            del kb, vb, ref
        cpu = {"value": round(sample_bytes / cpu_s / 1e9, 4), "unit": "GB/s", "cores": 1,
               "kind": "oracle",
               "sample": f"two decode steps over all {L} layers (the packed context alone, then "
                         f"with the step's appended token) by the fp64 NumPy oracle with 1 BLAS "
                         f"thread: {cpu_s:.2f} s for {sample_bytes / 1e9:.2f} GB of packed K/V"}
        parity = {"layers": L, "max_rel_err": worst, "seg_len_equal": same_pack}
        cpu_all = {"value": round(all_bytes / all_s / 1e9, 4), "unit": "GB/s", "cores": all_cores, "kind": "oracle",
                   "sample": f"the first decode step of layers 0-{all_layers - 1} by the same oracle with "
                             f"{all_cores} BLAS threads: {all_s:.2f} s for {all_bytes / 1e9:.2f} GB"}
        cpu_pack = {"value": round(pack_bytes / pack_s / 1e9, 4), "unit": "GB/s", "cores": 1, "kind": "oracle",
                    "sample": f"the oracle's compaction of all {L} layers (retained K/V read + written, mask "
                              f"read) with 1 BLAS thread: {pack_s:.2f} s for {pack_bytes / 1e9:.2f} GB"}
        log(f"oracle {cpu_s:.2f} s, worst parity err {worst:.2e}; all {all_cores} cores {all_s:.2f} s; "
            f"pack {pack_s:.2f} s")

    # ---------------- dense comparator cache [L][B*Hkv][T+cap][d] ----------
    t_cap = T + cap
    kd = torch.zeros((N, Hkv, t_cap, dim), dtype=torch.bfloat16, device=dev)
    vd = torch.zeros_like(kd)
    kd[:, :, :T].copy_(k)
    vd[:, :, :T].copy_(v)
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

    def step_args(step, mode, sh):
        """One decode step: per layer, one call that appends the step's token
        and attends over the cache."""
        slot = step % cap
        acts = []
        for layer in range(L):
            if mode == "dense":
                acts.append((lib.dkv_dense_append_decode_attn, dense_args(layer, T + slot, sh)))
            elif mode == "paged":
                acts.append((lib.dkv_paged_append_decode_attn, paged_args(layer, slot, sh)))
            else:
                acts.append((lib.dkv_append_decode_attn, packed_args(layer, slot, sh)))
        return acts

    def run(acts):
        for fn, a in acts:
            st = fn(*a)
            if st != 0:
                raise d.DkvError(fn.__name__, st)

    def decode_bytes(step, mode):
        n_tail = step % cap + 1
        rows_step = (N * Hkv * (T + n_tail)) if mode == "dense" else (retained + N * Hkv * n_tail)
        return rows_step * dim * elem * 2 + L * B * Hq * dim * (elem + 4) + L * nseg_layer * 12

    cap_stream = torch.cuda.Stream()

    timed_spread = {}

    def timed(mode, steps, warmup):
        """Step time as HIP-graph replays (one graph per step: each keeps its
        own append slot), plus the same steps launched eagerly."""
        run(step_args(0, mode, sh))  # warm: first launches load code objects
        torch.cuda.synchronize()
        graphs = []
        for s in range(warmup + steps):
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g, stream=cap_stream):
                run(step_args(s, mode, cap_stream.cuda_stream))
            graphs.append(g)
        rot = [0]

        def one():  # the step graphs in turn (each rewrites its own append slot)
            graphs[rot[0] % len(graphs)].replay()
            rot[0] += 1
        sustain(one)
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
        # the spread of single steps: the timed step graphs again, in turn, at
        # least SPREAD_REPS replays with one event pair each (a pass of its
        # own, so the timed region above is untouched; a graph replayed again
        # rewrites its append slot with the same token)
        reps = max(SPREAD_REPS, steps)
        evs = [ev() for _ in range(reps + 1)]
        evs[0].record(stream)
        for i in range(reps):
            graphs[warmup + i % steps].replay()
            evs[i + 1].record(stream)
        torch.cuda.synchronize()
        per_step = [evs[i].elapsed_time(evs[i + 1]) for i in range(reps)]
        spread = {"median": round(float(np.median(per_step)), 4), "p10": round(float(np.percentile(per_step, 10)), 4),
                  "p90": round(float(np.percentile(per_step, 90)), 4), "reps": reps}
        plans = [step_args(s, mode, sh) for s in range(warmup + steps)]
        for s in range(warmup):
            run(plans[s])
        torch.cuda.synchronize()
        a.record(stream)
        for s in range(warmup, warmup + steps):
            run(plans[s])
        b.record(stream)
        torch.cuda.synchronize()
        eager_ms = a.elapsed_time(b) / steps
        nbytes = sum(decode_bytes(s, mode) for s in range(warmup, warmup + steps)) / steps
        timed_spread[mode] = spread
        return ms, eager_ms, nbytes

    paged_state = {}

    def paged_args(layer, n_tail, sh):
        """dkv_paged_append_decode_attn: write the token at position T + n_tail
        of its page, attend through the layer's entries."""
        ps = paged_state
        off = layer * nseg_layer
        kn, vn = new_kv[layer]
        return (d.DKV_BF16, B, Hq, Hkv, dim, P(q_layers[layer].data_ptr()), P(kn.data_ptr()),
                P(vn.data_ptr()), 1, n_tail, cap, P(ps["k_pool"].data_ptr()), P(ps["v_pool"].data_ptr()),
                ps["n_pages"], PAGE_ROWS, P(ps["entries"].data_ptr() + off * ps["max_e"] * 16),
                P(ps["n_ent"].data_ptr() + 4 * off), ps["max_e"], T, w.sm_scale, ps["rows"][layer],
                P(out.data_ptr()), P(dws.data_ptr()), ws_bytes, P(sh))

    log("timing packed decode")
    ms, eager_ms, nbytes = timed("packed", args.steps, args.warmup)
    log("timing dense decode")
    dms, deager_ms, dbytes = timed("dense", args.steps, args.warmup)
    # the whole generation of the workload: every one of its decode steps
    # (tails 0 .. decode_steps - 1), one graph per step, replayed in order
    def full_generation(mode):
        graphs = []
        for s_ in range(w.decode_steps):
            g_ = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g_, stream=cap_stream):
                run(step_args(s_, mode, cap_stream.cuda_stream))
            graphs.append(g_)
        rot = [0]

        def one():
            graphs[rot[0] % len(graphs)].replay()
            rot[0] += 1
        sustain(one)
        for g_ in graphs:
            g_.replay()
        torch.cuda.synchronize()
        a_, b_ = ev(), ev()
        a_.record(stream)
        for g_ in graphs:
            g_.replay()
        b_.record(stream)
        torch.cuda.synchronize()
        n_bytes = sum(decode_bytes(s_, mode) for s_ in range(w.decode_steps))
        return a_.elapsed_time(b_) / w.decode_steps, n_bytes / w.decode_steps

    full_gen = None
    if not args.no_full_generation:
        log("timing the full generation")
        fg_ms, fg_bytes = full_generation("packed")
        fgd_ms, fgd_bytes = full_generation("dense")
        full_gen = {"steps": w.decode_steps, "ms_per_step": round(fg_ms, 4),
                    "gb_per_s": round(fg_bytes / (fg_ms * 1e-3) / 1e9, 2),
                    "dense_ms_per_step": round(fgd_ms, 4), "speedup_vs_dense": round(fgd_ms / fg_ms, 3),
                    "step": f"all {w.decode_steps} steps of the generation (tails 0-{w.decode_steps - 1}), one "
                            "graph per step, replayed once in order"}
        log(f"full generation: {fg_ms:.4f} ms/step packed, {fgd_ms:.4f} dense")
    # A step is exactly one attention call per layer on one stream, so the
    # average duration of a call (split + combine kernel, with the gaps
    # between them) is the timed region's event interval over L calls.
    launch_ms = ms / L
    dlaunch_ms = dms / L

    # ---------------- zero-copy paged variant -----------------------------
    # The stack kept in 128-row pages of one pool (context plus append region
    # per segment; each layer's pages shuffled within the layer's range, as an
    # allocator would leave them).  dkv_page_select lists every segment's
    # retained runs in place -- no K/V byte moves -- and a step runs one
    # dkv_paged_append_decode_attn per layer.
    log("paged variant: pools, selection")
    PR = PAGE_ROWS
    pps = -(-t_cap // PR)
    n_pages = N * Hkv * pps
    tables = []
    for layer in range(L):
        t_l, _ = di.page_table(nseg_layer, pps, seed=layer)
        tables.append(t_l + layer * nseg_layer * pps)
    k_pool = torch.empty((n_pages, PR, dim), dtype=torch.bfloat16, device=dev)
    v_pool = torch.empty_like(k_pool)
    for layer in range(L):
        u = slice(layer * B, (layer + 1) * B)
        di.fill_pages(k_pool, kd[u].reshape(nseg_layer, t_cap, dim), tables[layer], PR)
        di.fill_pages(v_pool, vd[u].reshape(nseg_layer, t_cap, dim), tables[layer], PR)
    del kd, vd  # the dense comparator is done
    torch.cuda.empty_cache()
    table_d = torch.from_numpy(np.concatenate(tables)).to(dev)
    max_e = int(d.dkv_page_entries_bound(lay, cap, PR))
    entries = torch.empty((N * Hkv, max_e, 4), dtype=torch.int32, device=dev)
    n_ent = torch.empty(N * Hkv, dtype=torch.int32, device=dev)
    p_len = torch.empty(N * Hkv, dtype=torch.int32, device=dev)
    used = torch.empty((N * Hkv, pps), dtype=torch.uint8, device=dev)
    sws = torch.empty(d.dkv_page_select_workspace_bytes(N * Hkv, T), dtype=torch.uint8, device=dev)
    kvm = kv_mask.view(N * Hkv, T)
    d.dkv_page_select(kvm, table_d, PR, cap, entries, n_ent, p_len, sws, page_used=used)
    torch.cuda.synchronize()
    a, b = ev(), ev()
    a.record(stream)
    for _ in range(5):
        d.dkv_page_select(kvm, table_d, PR, cap, entries, n_ent, p_len, sws, page_used=used)
    b.record(stream)
    torch.cuda.synchronize()
    select_us = a.elapsed_time(b) * 1e3 / 5
    n_ent_h = n_ent.cpu().to(torch.int64)
    assert int(n_ent_h.max()) <= max_e and torch.equal(p_len.cpu(), kv_len.cpu().view(-1))
    paged_state.update(k_pool=k_pool, v_pool=v_pool, n_pages=n_pages, entries=entries, n_ent=n_ent,
                       max_e=max_e,
                       rows=[int(n_ent_h[layer * nseg_layer:(layer + 1) * nseg_layer].sum()) * PR
                             for layer in range(L)])
    pages_used = int(used.to(torch.int64).sum())
    page_bytes = PR * dim * elem * 2
    paged_parity = None
    if not args.no_cpu_baseline:
        # layer 0, one step: the token appended at position T, then attention
        st_ = lib.dkv_paged_append_decode_attn(*paged_args(0, 0, sh))
        if st_ != 0:
            raise d.DkvError("dkv_paged_append_decode_attn", st_)
        torch.cuda.synchronize()
        got = out.cpu().numpy()
        n0 = nseg_layer * pps  # layer 0 owns pages [0, n0)
        kp0 = k_pool[:n0].cpu().view(torch.int16).numpy().view(np.uint16)
        vp0 = v_pool[:n0].cpu().view(torch.int16).numpy().view(np.uint16)
        sel0 = o.page_select(okm0.reshape(nseg_layer, T), tables[0], PR, cap)
        ent0 = entries[:nseg_layer].cpu().numpy()
        same = all(np.array_equal(ent0[s_, :sel0["n_entries"][s_]], sel0["entries"][s_])
                   for s_ in range(nseg_layer))
        same &= bool(np.array_equal(n_ent[:nseg_layer].cpu().numpy(), sel0["n_entries"]))
        qb0 = q_layers[0].cpu().view(torch.int16).numpy().view(np.uint16)
        want = o.paged_decode_attn(qb0, kp0, vp0, sel0["entries"], PR, T, 1, w.sm_scale, Hkv, o.BF16)
        err = float((np.abs(got - want).max(-1) / np.maximum(np.abs(want).max(-1), 1e-30)).max())
        paged_parity = {"layers": 1, "max_rel_err": err, "entries_equal": bool(same)}
        del kp0, vp0
        log(f"paged parity layer 0: err {err:.2e}, entries equal {same}")
    log("timing paged decode")
    pms, peager_ms, pbytes = timed("paged", args.steps, args.warmup)
    paged_res = {
        "page_rows": PR, "ms_per_step": round(pms, 4), "eager_ms_per_step": round(peager_ms, 4),
        "us_per_layer": round(pms * 1e3 / L, 2), "avg_launch_us": round(pms * 1e3 / L, 2),
        "gb_per_s": round(pbytes / (pms * 1e-3) / 1e9, 2),
        "launch_frac_of_peak": round(pbytes / L / (pms / L * 1e-3) / 1e9 / PEAK_HBM_GBPS, 4),
        "vs_packed": round(ms / pms, 3), "speedup_vs_dense": round(dms / pms, 3),
        "select_us": round(select_us, 1), "compact_us": round(compact_us, 1),
        "entries_per_segment": {"mean": round(float(n_ent_h.float().mean()), 1), "max": int(n_ent_h.max()),
                                "bound": max_e},
        "slots_per_retained_row": round(float(n_ent_h.sum()) * PR / retained, 4),
        "kv_cache_gib": {"pool": round(n_pages * page_bytes / 2 ** 30, 3),
                         "pages_used": round(pages_used * page_bytes / 2 ** 30, 3)},
        "kernel": "dkv_paged_append_decode_attn call: decode_kernel<bf16,128,4,paged> + decode_merge_kernel",
        "bytes_per_launch": int(pbytes / L), "traffic": None,
        "parity_layer0": paged_parity,
    }
    log(f"paged: {pms:.3f} ms/step ({pms * 1e3 / L:.1f} us/layer), select {select_us:.0f} us, "
        f"pages used {paged_res['kv_cache_gib']['pages_used']} GiB")

    # ---------------- exact-budget export and the ablation families -------
    # The paper's own bin layout (128-token bins: 1,015 at 131,072 tokens) on
    # the same 8B-shaped stack and the same K/V: the pattern is the
    # exact-budget export (K = round(0.2 L H D)) of stand-in retention
    # probabilities, then each ablation family of it; every pattern is mapped,
    # packed and decoded (32 layers, attend only) like the headline.
    log("exact-budget export and pattern families")
    wp = di.workload("llama8b_stack_128k_paper_bins")
    Lp, Hp, Dp = wp.num_layers, wp.num_q_heads, wp.num_bins
    probs = di.retention_probs(Lp, Hp, wp.num_kv_heads, Dp, seed=wp.cfg_id)
    k_budget = d.dkv_budget_entries(wp.rho, Lp, Hp, Dp)
    probs_d = torch.from_numpy(probs).to(dev)
    pat_x = torch.empty((Lp, Hp, Dp), dtype=torch.uint8, device=dev)
    tk_ws = torch.empty(d.dkv_topk_workspace_bytes(Lp, Hp, Dp), dtype=torch.uint8, device=dev)
    d.dkv_topk_pattern(probs_d, k_budget, pat_x, tk_ws)
    torch.cuda.synchronize()
    a, b = ev(), ev()
    a.record(stream)
    for _ in range(20):
        d.dkv_topk_pattern(probs_d, k_budget, pat_x, tk_ws)
    b.record(stream)
    torch.cuda.synchronize()
    topk_us = a.elapsed_time(b) * 1e3 / 20
    exported = pat_x.cpu().numpy()
    n_entries = Lp * Hp * Dp
    # bytes one export reads and writes: four passes over the probabilities
    # (three digit rounds, write) and the pattern
    topk_bytes = 4 * 4 * n_entries + n_entries
    topk_res = {"entries": n_entries, "k": int(k_budget), "rho": wp.rho, "us": round(topk_us, 1),
                "gb_per_s": round(topk_bytes / (topk_us * 1e-6) / 1e9, 1),
                "launches": 5, "ones": int(exported.sum()), "cpu_baseline": None, "equal_to_oracle": None}
    if not args.no_cpu_baseline:
        t0 = time.perf_counter()
        want_pat = o.topk_mask(probs, o.budget_entries(wp.rho, Lp, Hp, Dp))
        topk_cpu = time.perf_counter() - t0
        topk_res["equal_to_oracle"] = bool(np.array_equal(exported, want_pat))
        topk_res["cpu_baseline"] = {"value": round(topk_cpu * 1e3, 2), "unit": "ms", "cores": 1, "kind": "oracle",
                                    "sample": "the whole export (NumPy lexsort, one thread)"}
    log(f"topk export {topk_us:.1f} us for {n_entries} entries")
    lay_p = d.make_layout(N, Hq, Hkv, dim, T, wp.sink, wp.recent, list(wp.bin_edges))
    fam_res = {}
    fam_ws = torch.zeros(d.dkv_decode_workspace_bytes(B, Hq, Hkv, dim), dtype=torch.uint8, device=dev)
    fam_out = torch.empty((B, Hq, dim), dtype=torch.float32, device=dev)
    fam_stream = torch.cuda.Stream()
    Pv = ctypes.c_void_p
    for kind in ("exported",) + di.PATTERN_FAMILIES:
        pat_f = exported if kind == "exported" else di.pattern_family(exported, kind, Hkv, seed=wp.cfg_id)
        km_f = torch.empty((N, Hkv, T), dtype=torch.uint8, device=dev)
        kl_f = torch.empty((N, Hkv), dtype=torch.int32, device=dev)
        d.dkv_map_pattern(lay_p, torch.from_numpy(np.ascontiguousarray(pat_f)).to(dev), km_f, kl_f)
        lens_f = kl_f.cpu().to(torch.int64)
        rows_f = int(lens_f.sum())
        kc_f = torch.empty((rows_f, dim), dtype=torch.bfloat16, device=dev)
        vc_f = torch.empty_like(kc_f)
        so_f = torch.empty(N * Hkv, dtype=torch.int64, device=dev)
        sl_f = torch.empty(N * Hkv, dtype=torch.int32, device=dev)
        cws_f = torch.empty(d.dkv_compact_workspace_bytes(lay_p), dtype=torch.uint8, device=dev)
        d.dkv_compact(lay_p, k, v, km_f, 0, kc_f, vc_f, so_f, sl_f, cws_f)
        del km_f
        hints = [int(lens_f[layer * B:(layer + 1) * B].sum()) for layer in range(L)]

        def fam_calls(shp):
            for layer in range(L):
                off = layer * nseg_layer
                st_ = lib.dkv_decode_attn(d.DKV_BF16, B, Hq, Hkv, dim, Pv(q_layers[layer].data_ptr()),
                                          Pv(kc_f.data_ptr()), Pv(vc_f.data_ptr()), Pv(so_f.data_ptr() + 8 * off),
                                          Pv(sl_f.data_ptr() + 4 * off), 0, w.sm_scale, hints[layer],
                                          Pv(fam_out.data_ptr()), Pv(fam_ws.data_ptr()), fam_ws.numel(), Pv(shp))
                if st_ != 0:
                    raise d.DkvError("dkv_decode_attn", st_)
        fam_calls(sh)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=fam_stream):
            fam_calls(fam_stream.cuda_stream)
        sustain(g.replay)
        for _ in range(args.warmup):
            g.replay()
        torch.cuda.synchronize()
        a.record(stream)
        for _ in range(args.steps):
            g.replay()
        b.record(stream)
        torch.cuda.synchronize()
        f_ms = a.elapsed_time(b) / args.steps
        f_bytes = rows_f * dim * elem * 2 + L * B * Hq * dim * (elem + 4) + L * nseg_layer * 12
        per_head = lens_f.view(-1).to(torch.float64)
        fam_res[kind] = {"logical": round(float(pat_f.mean()), 4),
                         "physical": round(rows_f / float(N * Hkv * T), 4),
                         "ms_per_step": round(f_ms, 4), "us_per_layer": round(f_ms * 1e3 / L, 2),
                         "gb_per_s": round(f_bytes / (f_ms * 1e-3) / 1e9, 1),
                         "segment_rows": {"min": int(per_head.min()), "max": int(per_head.max()),
                                          "cv": round(float(per_head.std() / per_head.mean()), 3)},
                         "lengths_equal_oracle": None}
        if not args.no_cpu_baseline:
            olen = o.closed_form_lengths(pat_f, T, wp.sink, wp.recent, wp.bin_edges, Hkv)
            fam_res[kind]["lengths_equal_oracle"] = bool(np.array_equal(lens_f.numpy(), olen))
        log(f"pattern {kind}: physical {fam_res[kind]['physical']}, {f_ms * 1e3 / L:.1f} us/layer")
        del kc_f, vc_f, g
        torch.cuda.empty_cache()

    del k, v  # the dense input is no longer needed
    torch.cuda.empty_cache()

    # ---------------- ragged batch: contexts of different lengths ----------
    # The 70B-shaped batch (16 sequences x 64q/8kv, 20% physical budget) once
    # with every context 32K long and once with per-sequence contexts of
    # 4K-32K (dkv_map_pattern_ragged); then its 16 decode steps, one fused
    # append + decode call each, graph-replayed.
    log("ragged batch")
    wr = di.workload("llama70b_layer_bs16_32k")
    Br, Hqr, Hkvr, Tr, capr = wr.batch, wr.num_q_heads, wr.num_kv_heads, wr.context_len, wr.append_cap
    pat_r, _ = di.make_pattern(wr)
    kr = torch.empty((Br, Hkvr, Tr, dim), dtype=torch.bfloat16, device=dev)
    vr = torch.empty_like(kr)
    for b_ in range(Br):
        kb_, vb_ = di.kv_unit(wr, b_, device=dev)
        kr[b_].copy_(kb_)
        vr[b_].copy_(vb_)
    del kb_, vb_
    lay_r = d.make_layout(Br, Hqr, Hkvr, dim, Tr, wr.sink, wr.recent, list(wr.bin_edges))
    lens_r = di.sequence_lengths(wr, seed=1)
    q_r = [di.q_step(wr, 0, s_, device=dev) for s_ in range(wr.decode_steps)]
    new_r = [tuple(t.reshape(Br * Hkvr, 1, dim).contiguous() for t in di.kv_new_step(wr, 0, s_, device=dev))
             for s_ in range(wr.decode_steps)]
    ws_r = torch.zeros(d.dkv_decode_workspace_bytes(Br, Hqr, Hkvr, dim), dtype=torch.uint8, device=dev)
    out_r = torch.empty((Br, Hqr, dim), dtype=torch.float32, device=dev)
    ragged_res = {"workload": wr.name, "batch": Br, "steps": wr.decode_steps,
                  "context_lens": {"min": int(lens_r.min()), "max": int(lens_r.max()),
                                   "mean": round(float(lens_r.mean()), 1)}}
    for mode in ("uniform", "ragged"):
        km_r = torch.empty((Br, Hkvr, Tr), dtype=torch.uint8, device=dev)
        kl_r = torch.empty((Br, Hkvr), dtype=torch.int32, device=dev)
        pat_rd = torch.from_numpy(pat_r).to(dev)
        if mode == "ragged":
            d.dkv_map_pattern_ragged(lay_r, torch.from_numpy(lens_r).to(dev), pat_rd, km_r, kl_r)
        else:
            d.dkv_map_pattern(lay_r, pat_rd, km_r, kl_r)
        kept_r = int(kl_r.sum())
        rows_r = kept_r + Br * Hkvr * capr
        kc_r = torch.zeros((rows_r, dim), dtype=torch.bfloat16, device=dev)
        vc_r = torch.zeros_like(kc_r)
        so_r = torch.empty(Br * Hkvr, dtype=torch.int64, device=dev)
        sl_r = torch.empty(Br * Hkvr, dtype=torch.int32, device=dev)
        cws_r = torch.empty(d.dkv_compact_workspace_bytes(lay_r), dtype=torch.uint8, device=dev)
        pack_mask = lambda: d.dkv_compact(lay_r, kr, vr, km_r, capr, kc_r, vc_r, so_r, sl_r, cws_r)
        pack_mask()
        # the same pack straight from the pattern (the ragged block gather for
        # the ragged batch), into zeroed buffers of its own, checked against it
        kb_r, vb_r = torch.zeros_like(kc_r), torch.zeros_like(vc_r)
        sob_r, slb_r = torch.empty_like(so_r), torch.empty_like(sl_r)
        bws_r = torch.empty(d.dkv_compact_bins_workspace_bytes(lay_r), dtype=torch.uint8, device=dev)
        ulen_r = torch.from_numpy(lens_r).to(dev)
        if mode == "ragged":
            pack_bins = lambda: d.dkv_compact_bins_ragged(lay_r, ulen_r, kr, vr, pat_rd, capr, kb_r, vb_r, sob_r,
                                                          slb_r, bws_r)
        else:
            pack_bins = lambda: d.dkv_compact_bins(lay_r, kr, vr, pat_rd, capr, kb_r, vb_r, sob_r, slb_r, bws_r)
        pack_bins()
        torch.cuda.synchronize()
        pack_equal = bool(torch.equal(sob_r, so_r) and torch.equal(slb_r, sl_r)
                          and torch.equal(kb_r.view(torch.int16), kc_r.view(torch.int16))
                          and torch.equal(vb_r.view(torch.int16), vc_r.view(torch.int16)))
        pack_us = {}
        for name_, fn_ in (("compact", pack_mask), ("compact_bins", pack_bins)):
            t_ = []
            for _ in range(3):
                a, b = ev(), ev()
                a.record(stream)
                fn_()
                b.record(stream)
                torch.cuda.synchronize()
                t_.append(a.elapsed_time(b) * 1e3)
            pack_us[name_] = round(min(t_), 1)
        del km_r, kb_r, vb_r, bws_r

        def step_call(s_, shp):
            kn_, vn_ = new_r[s_]
            st_ = lib.dkv_append_decode_attn(d.DKV_BF16, Br, Hqr, Hkvr, dim, Pv(q_r[s_].data_ptr()),
                                             Pv(kn_.data_ptr()), Pv(vn_.data_ptr()), 1, s_, capr, Pv(kc_r.data_ptr()),
                                             Pv(vc_r.data_ptr()), Pv(so_r.data_ptr()), Pv(sl_r.data_ptr()),
                                             wr.sm_scale, kept_r + Br * Hkvr * (s_ + 1), Pv(out_r.data_ptr()),
                                             Pv(ws_r.data_ptr()), ws_r.numel(), Pv(shp))
            if st_ != 0:
                raise d.DkvError("dkv_append_decode_attn", st_)
        step_call(0, sh)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=fam_stream):
            for s_ in range(wr.decode_steps):
                step_call(s_, fam_stream.cuda_stream)
        sustain(g.replay)
        for _ in range(args.warmup):
            g.replay()
        torch.cuda.synchronize()
        a.record(stream)
        for _ in range(args.steps):
            g.replay()
        b.record(stream)
        torch.cuda.synchronize()
        r_us = a.elapsed_time(b) * 1e3 / args.steps / wr.decode_steps
        r_bytes = (kept_r + Br * Hkvr * (wr.decode_steps + 1) / 2) * dim * elem * 2 + Br * Hqr * dim * (elem + 4)
        seg = kl_r.view(-1).to(torch.float64)
        ragged_res[mode] = {"pack_us": pack_us, "packs_equal": pack_equal,
                            "retained_rows": kept_r, "us_per_step": round(r_us, 2),
                            "gb_per_s": round(r_bytes / (r_us * 1e-6) / 1e9, 1),
                            "segment_rows": {"min": int(seg.min()), "max": int(seg.max()),
                                             "cv": round(float(seg.std() / seg.mean()), 3)}}
        log(f"{mode} batch: {r_us:.1f} us/step, {ragged_res[mode]['gb_per_s']} GB/s; pack {pack_us}, "
            f"equal {pack_equal}")
        del kc_r, vc_r, g
        torch.cuda.empty_cache()
    del kr, vr

    # ---------------- query-block attention, all layers ------------------
    log("timing query-block attention")
    q_hints = [layer_rows[layer] + nseg_layer * NQ for layer in range(L)]
    q_wsb = max(d.dkv_query_workspace_bytes(B, Hq, Hkv, dim, NQ, h) for h in q_hints)
    q_ws = torch.empty(max(q_wsb, 16), dtype=torch.uint8, device=dev)
    q_out = torch.empty((B, NQ, Hq, dim), dtype=torch.float32, device=dev)

    def query_call(layer, shp):
        off = layer * nseg_layer
        st_ = lib.dkv_query_attn(d.DKV_BF16, B, Hq, Hkv, dim, NQ, P(q_blocks[layer].data_ptr()), 0, cap_q,
                                 P(k_q.data_ptr()), P(v_q.data_ptr()), P(seg_off_q.data_ptr() + 8 * off),
                                 P(seg_len_q.data_ptr() + 4 * off), w.sm_scale, q_hints[layer],
                                 P(q_out.data_ptr()), P(q_ws.data_ptr()), q_ws.numel(), P(shp))
        if st_ != 0:
            raise d.DkvError("dkv_query_attn", st_)

    for layer in range(L):
        query_call(layer, sh)
    torch.cuda.synchronize()
    gq = torch.cuda.CUDAGraph()
    with torch.cuda.graph(gq, stream=cap_stream):
        for layer in range(L):
            query_call(layer, cap_stream.cuda_stream)
    sustain(gq.replay)
    for _ in range(args.warmup):
        gq.replay()
    torch.cuda.synchronize()
    a, b = ev(), ev()
    a.record(stream)
    for _ in range(args.steps):
        gq.replay()
    b.record(stream)
    torch.cuda.synchronize()
    q_ms = a.elapsed_time(b) / args.steps
    # algorithmic flops: 4 d per visible (query row, key) pair; query token i
    # of a segment with n retained rows sees n + i + 1 keys, for G heads
    lens_np = lens.numpy().reshape(L, nseg_layer)
    q_flops = float(sum(4.0 * dim * w.group * (NQ * lens_np[layer].sum() + nseg_layer * NQ * (NQ + 1) / 2)
                        for layer in range(L)))
    q_tflops = q_flops / (q_ms * 1e-3) / 1e12
    query_res = {"n_q": NQ, "ms_per_step": round(q_ms, 4), "us_per_layer": round(q_ms * 1e3 / L, 1),
                 "tflop_per_step": round(q_flops / 1e12, 3),
                 # K/V rows a call attends (every row once), next to the counters' traffic
                 "kv_bytes_per_call": int(np.mean([(layer_rows[layer] + nseg_layer * NQ) * dim * elem * 2
                                                   for layer in range(L)])),
                 "roofline": {"bound": "mfma", "achieved": round(q_tflops, 1), "peak": PEAK_BF16_TFLOPS,
                              "unit": "TFLOP/s", "frac": round(q_tflops / PEAK_BF16_TFLOPS, 4),
                              "traffic": None,
                              "kernel": "dkv_query_attn call: query_plan_kernel + query_attn_kernel<128> + "
                                        "query_merge_kernel"},
                 "cpu_baseline": None, "parity_layer0": None}
    if not args.no_cpu_baseline:
        import oracle as o
        from threadpoolctl import threadpool_limits
        nqs = 32  # oracle sample: the block's first 32 tokens of layer 0
        qb0, kb0, vb0 = di.query_block(w, 0, NQ, device=dev)
        query_call(0, sh)
        torch.cuda.synchronize()
        got = q_out[:, :nqs].cpu().numpy()
        ref = o.compact(k0_bits, v0_bits, okm0, NQ)
        kc, vc = o.append(ref["k_c"], ref["v_c"], ref["seg_off"], ref["seg_len"],
                          kb0.cpu().view(torch.int16).numpy().view(np.uint16),
                          vb0.cpu().view(torch.int16).numpy().view(np.uint16), 0)
        qs = qb0[:, :nqs].contiguous().cpu().view(torch.int16).numpy().view(np.uint16)
        with threadpool_limits(1):
            t0 = time.perf_counter()
            want = o.query_attn(qs, kc, vc, ref["seg_off"], ref["seg_len"], 0, w.sm_scale, Hkv, o.BF16)
            cpu_q = time.perf_counter() - t0
        flops_s = 4.0 * dim * w.group * (nqs * lens_np[0].sum() + nseg_layer * nqs * (nqs + 1) / 2)
        err = float((np.abs(got - want).max(-1) / np.maximum(np.abs(want).max(-1), 1e-30)).max())
        query_res["cpu_baseline"] = {"value": round(flops_s / cpu_q / 1e9, 3), "unit": "GFLOP/s", "cores": 1,
                                     "kind": "oracle",
                                     "sample": f"the first {nqs} of the {NQ} block tokens of layer 0 by the fp64 "
                                               f"NumPy oracle with 1 BLAS thread: {cpu_q:.2f} s for "
                                               f"{flops_s / 1e9:.1f} GFLOP"}
        query_res["parity_layer0"] = {"tokens": nqs, "max_rel_err": err}
        log(f"query oracle {cpu_q:.2f} s, parity err {err:.2e}")
    log(f"query block {q_ms * 1e3 / L:.1f} us/layer, {q_tflops:.1f} TFLOP/s")

    # ---------------- multi-turn reuse of one compaction ------------------
    # Several query rounds over one packed cache: each turn writes a new
    # 256-token block into the append region (n_tail back to 0), attends it
    # over every layer (append + query attention per layer), then generates
    # MT_STEPS tokens (one fused append + decode per layer and token).  The
    # turn is captured once and replayed; contents do not change the cost.
    log("timing multi-turn reuse")
    mt_q = [di.q_step(w, layer, 0, device=dev).contiguous() for layer in range(L)]
    mt_new = []
    for layer in range(L):
        kn_, vn_ = di.kv_new_step(w, layer, 0, device=dev)
        mt_new.append((kn_.reshape(nseg_layer, 1, dim).contiguous(), vn_.reshape(nseg_layer, 1, dim).contiguous()))
    mt_out = torch.empty((L, B, Hq, dim), dtype=torch.float32, device=dev)

    def mt_prefill(shp):
        for layer in range(L):
            off = layer * nseg_layer
            kb_, vb_ = kv_blocks[layer]
            st_ = lib.dkv_append(d.DKV_BF16, nseg_layer, dim, P(kb_.data_ptr()), P(vb_.data_ptr()), NQ, 0, cap_q,
                                 P(k_q.data_ptr()), P(v_q.data_ptr()), P(seg_off_q.data_ptr() + 8 * off),
                                 P(seg_len_q.data_ptr() + 4 * off), P(shp))
            if st_ != 0:
                raise d.DkvError("dkv_append", st_)
            query_call(layer, shp)

    def mt_decode(shp):
        for s_ in range(MT_STEPS):
            for layer in range(L):
                off = layer * nseg_layer
                kn_, vn_ = mt_new[layer]
                st_ = lib.dkv_append_decode_attn(
                    d.DKV_BF16, B, Hq, Hkv, dim, P(mt_q[layer].data_ptr()), P(kn_.data_ptr()), P(vn_.data_ptr()), 1,
                    NQ + s_, cap_q, P(k_q.data_ptr()), P(v_q.data_ptr()), P(seg_off_q.data_ptr() + 8 * off),
                    P(seg_len_q.data_ptr() + 4 * off), w.sm_scale, q_hints[layer] + nseg_layer * (s_ + 1),
                    P(mt_out[layer].data_ptr()), P(dws.data_ptr()), dws.numel(), P(shp))
                if st_ != 0:
                    raise d.DkvError("dkv_append_decode_attn", st_)

    mt_prefill(sh)
    mt_decode(sh)
    torch.cuda.synchronize()
    gp, gd = torch.cuda.CUDAGraph(), torch.cuda.CUDAGraph()
    with torch.cuda.graph(gp, stream=cap_stream):
        mt_prefill(cap_stream.cuda_stream)
    with torch.cuda.graph(gd, stream=cap_stream):
        mt_decode(cap_stream.cuda_stream)
    def mt_turn():
        gp.replay()
        gd.replay()
    sustain(mt_turn)
    for _ in range(max(1, args.warmup)):
        gp.replay()
        gd.replay()
    torch.cuda.synchronize()
    ev3 = [ev() for _ in range(2 * MT_TURNS + 1)]
    ev3[0].record(stream)
    for t_ in range(MT_TURNS):
        gp.replay()
        ev3[2 * t_ + 1].record(stream)
        gd.replay()
        ev3[2 * t_ + 2].record(stream)
    torch.cuda.synchronize()
    pre_ms = [ev3[2 * t_].elapsed_time(ev3[2 * t_ + 1]) for t_ in range(MT_TURNS)]
    dec_ms = [ev3[2 * t_ + 1].elapsed_time(ev3[2 * t_ + 2]) for t_ in range(MT_TURNS)]
    turn_ms = ev3[0].elapsed_time(ev3[-1]) / MT_TURNS
    mt_res = {"turns": MT_TURNS, "block_tokens": NQ, "tokens_generated_per_turn": MT_STEPS,
              "ms_per_turn": round(turn_ms, 3), "prefill_ms": round(float(np.median(pre_ms)), 3),
              "decode_ms_per_token": round(float(np.median(dec_ms)) / MT_STEPS, 4),
              "compaction_ms": round(bins_us / 1e3, 3),
              "compaction_share": round(bins_us / 1e3 / (bins_us / 1e3 + MT_TURNS * turn_ms), 4),
              "compaction_call": "dkv_compact_bins",
              "step": "turn = per layer (append 256-token block + dkv_query_attn), then 16 x per layer "
                      "dkv_append_decode_attn; HIP-graph replays", "parity_layer0_last_token": None}
    if not args.no_cpu_baseline:
        import oracle as o
        # the last token of the last turn on layer 0: packed context, the block and 16 generated tokens
        ref = o.compact(k0_bits, v0_bits, okm0, cap_q)
        kb0_, vb0_ = kv_blocks[0]
        to_bits = lambda t_: t_.cpu().view(torch.int16).numpy().view(np.uint16)
        kc, vc = o.append(ref["k_c"], ref["v_c"], ref["seg_off"], ref["seg_len"],
                          to_bits(kb0_).reshape(B, Hkv, NQ, dim), to_bits(vb0_).reshape(B, Hkv, NQ, dim), 0)
        kn0 = np.repeat(to_bits(mt_new[0][0]).reshape(B, Hkv, 1, dim), MT_STEPS, axis=2)
        vn0 = np.repeat(to_bits(mt_new[0][1]).reshape(B, Hkv, 1, dim), MT_STEPS, axis=2)
        kc, vc = o.append(kc, vc, ref["seg_off"], ref["seg_len"], kn0, vn0, NQ)
        want = o.decode_attn(to_bits(mt_q[0]), kc, vc, ref["seg_off"], ref["seg_len"], NQ + MT_STEPS, w.sm_scale,
                             Hkv, o.BF16)
        got = mt_out[0].cpu().numpy().astype(np.float64)
        mt_res["parity_layer0_last_token"] = float(
            (np.abs(got - want).max(-1) / np.maximum(np.abs(want).max(-1), 1e-30)).max())
    log(f"multi-turn {turn_ms:.2f} ms/turn (prefill {mt_res['prefill_ms']} ms, "
        f"{mt_res['decode_ms_per_token']} ms/token), parity {mt_res['parity_layer0_last_token']}")
    del gp, gd

    # ---------------- the other configurations ---------------------------
    cfg_rows, cfg_calls = {}, []
    if not args.no_configs:
        log("other configurations: 8B layer at 32K, 70B-shaped batch, Qwen-shaped stack")
        cfg_rows, cfg_calls = bench_configs({"d": d, "lib": lib, "dev": dev, "stream": stream, "args": args,
                                             "oracle": None if args.no_cpu_baseline else __import__("oracle"),
                                             "peak_hbm": PEAK_HBM_GBPS})
    shown = ("us_per_step", "gb_per_s", "speedup_vs_dense")
    for name_, r_ in cfg_rows.items():
        row_ = {k_: r_[k_] for k_ in r_ if k_ in shown}
        row_.update({k_: {j_: v_[j_] for j_ in v_ if j_ in shown} for k_, v_ in r_.items()
                     if k_.startswith("budget_") and isinstance(v_, dict)})
        log(f"{name_}: " + json.dumps(row_))

    # ---------------- achievable read bandwidth at this launch size -------
    # The streaming-read probe (same 16-byte non-temporal buffer loads as the
    # decode kernel's K/V stream; one block of 4-32 KiB per workgroup) over L
    # slices of one decode launch's size, one launch per slice, captured and
    # replayed like a decode step.
    per = (int(nbytes / L) + 15) // 16 * 16
    pbuf = torch.ones(L * per // 2, dtype=torch.int16, device=dev)
    psink = torch.zeros(4, dtype=torch.int32, device=dev)
    probe_gbps = {}
    for gpt in (1, 2, 4, 8):
        def probe_step(shp, gpt=gpt):
            for layer in range(L):
                st_ = lib.dkv_probe_stream_read(P(pbuf.data_ptr() + layer * per), per,
                                                P(psink.data_ptr()), gpt, P(shp))
                if st_ != 0:
                    raise d.DkvError("dkv_probe_stream_read", st_)
        probe_step(sh)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=cap_stream):
            probe_step(cap_stream.cuda_stream)
        sustain(g.replay)
        for _ in range(args.warmup):
            g.replay()
        torch.cuda.synchronize()
        a, b = ev(), ev()
        a.record(stream)
        for _ in range(args.steps):
            g.replay()
        b.record(stream)
        torch.cuda.synchronize()
        probe_gbps[f"{4 * gpt}KiB"] = round(L * per / (a.elapsed_time(b) / args.steps * 1e-3) / 1e9, 1)
    del pbuf
    # the same probe over one 4 GiB buffer (a read of the whole device's scale)
    big = torch.ones(1 << 31, dtype=torch.int16, device=dev)
    big_gbps = {}
    for gpt in (1, 2, 4, 8):
        sustain(lambda gpt=gpt: d.dkv_probe_stream_read(big, psink, gpt), 0.5)
        torch.cuda.synchronize()
        a, b = ev(), ev()
        a.record(stream)
        for _ in range(3):
            d.dkv_probe_stream_read(big, psink, gpt)
        b.record(stream)
        torch.cuda.synchronize()
        big_gbps[f"{4 * gpt}KiB"] = round((1 << 32) / (a.elapsed_time(b) / 3 * 1e-3) / 1e9, 1)
    del big
    torch.cuda.empty_cache()
    achievable = {"kind": "dkv_probe_stream_read: streaming read, one launch per layer-sized slice, one block "
                          "per workgroup, HIP-graph replays", "bytes_per_launch": per,
                  "gb_per_s_by_block": probe_gbps, "best_gb_per_s": max(probe_gbps.values()),
                  "one_4GiB_launch": {"gb_per_s_by_block": big_gbps, "best_gb_per_s": max(big_gbps.values())}}
    log(f"probe {probe_gbps}; over 4 GiB {big_gbps}")

    if args.copy_probe:
        # an elementwise kernel (not a DMA/blit copy) that reads and writes 1 GiB
        src = torch.ones(1 << 29, dtype=torch.int16, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            torch.mul(src, 1, out=dst)
        torch.cuda.synchronize()

    per_launch_bytes = nbytes / L
    achieved = per_launch_bytes / (launch_ms * 1e-3) / 1e9
    traffic = compact_traffic = bins_traffic = None
    if os.path.exists(PMC_FILE):
        with open(PMC_FILE) as f:
            pmc = json.load(f)
        if pmc.get("kernel_sha256_16") == kernel_hash():
            traffic = pmc.get("traffic_bytes_per_launch")
            paged_res["traffic"] = pmc.get("paged_traffic_bytes_per_launch")
        if pmc.get("query_kernel_sha256_16") == kernel_hash(QUERY_SRCS):
            query_res["roofline"]["traffic"] = pmc.get("query_traffic_bytes_per_call")
        if pmc.get("compact_kernel_sha256_16") == kernel_hash(COMPACT_SRCS):
            compact_traffic = pmc.get("compact_traffic_bytes")
        if pmc.get("compact_bins_kernel_sha256_16") == kernel_hash(BINS_SRCS):
            bins_traffic = pmc.get("compact_bins_traffic_bytes")

    res = {
        "metric": METRIC,
        "value": round(nbytes / (ms * 1e-3) / 1e9, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "eager_ms_per_step": round(eager_ms, 4),
        "step_ms_spread": timed_spread.get("packed"),
        "untimed_load_s_before_each_timing": SUSTAIN_S if SUSTAIN_ON else 0,
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
        "cpu_baseline_all_cores": cpu_all,
        "cpu_baseline_compaction": cpu_pack,
        "host": host_info(),
        "achievable_read": achievable,
        "query_block": query_res,
        "multi_turn": mt_res,
        "us_per_step": round(ms * 1e3, 1),
        "dense": {"ms_per_step": round(dms, 4), "eager_ms_per_step": round(deager_ms, 4),
                  "step_ms_spread": timed_spread.get("dense"),
                  "gb_per_s": round(dbytes / (dms * 1e-3) / 1e9, 2),
                  "avg_launch_us": round(dlaunch_ms * 1e3, 2),
                  "launch_frac_of_peak": round(dbytes / L / (dlaunch_ms * 1e-3) / 1e9 / PEAK_HBM_GBPS, 4)},
        "speedup_vs_dense": round(dms / ms, 3),
        "full_generation": full_gen,
        "configs": cfg_rows,
        "configs_decode_calls": cfg_calls,
        "paged": paged_res,
        "topk_export": topk_res,
        "ragged_batch": ragged_res,
        "pattern_families": {"workload": "llama8b_stack_128k_paper_bins: the same stack with 128-token bins "
                                         "(1,015), pattern = exact-budget export at rho 0.2, then each family",
                             "step": "per layer: dkv_decode_attn (attend only); HIP-graph replays",
                             **fam_res},
        "one_time": {"map_us": round(map_us, 1),
                     "map_back_to_back_us": round(map_b2b_us, 2),
                     # the masks written (1 byte per position), over the back-to-back time
                     "map_write_gb_per_s": round(N * Hkv * T / (map_b2b_us * 1e-6) / 1e9, 1),
                     "compact_us": round(compact_us, 1),
                     "compact_timing": "best of 3 single calls, each between synchronisations",
                     "compact_bytes": int(compact_bytes),
                     "compact_gb_per_s": round(compact_bytes / (compact_us * 1e-6) / 1e9, 1),
                     "compact_bins_us": round(bins_us, 1), "compact_bins_bytes": int(bins_bytes),
                     "compact_bins_gb_per_s": round(bins_bytes / (bins_us * 1e-6) / 1e9, 1),
                     "compact_bins_equal_to_compact": bins_equal,
                     # HBM bytes from FETCH_SIZE + WRITE_SIZE (calibrated) of the same sources, else null
                     "compact_traffic": compact_traffic, "compact_bins_traffic": bins_traffic,
                     "copy_probe": {"kind": "dkv_probe_copy of the retained K and V bytes (read + write)",
                                    "bytes": int(2 * copy_bytes), "gb_per_s_by_block": copy_gbps,
                                    "best_gb_per_s": max(copy_gbps.values())},
                     "compact_frac_of_copy": round(compact_bytes / (compact_us * 1e-6) / 1e9
                                                   / max(copy_gbps.values()), 4),
                     "compact_bins_frac_of_copy": round(bins_bytes / (bins_us * 1e-6) / 1e9
                                                        / max(copy_gbps.values()), 4),
                     # the same time priced as a pass that reads the whole dense cache and
                     # writes the retained rows (what a non-gathering pack would move)
                     "compact_dense_read_gb_per_s": round(
                         (2 * N * Hkv * T * dim * elem + 2 * retained * dim * elem + N * Hkv * T)
                         / (compact_us * 1e-6) / 1e9, 1)},
        "kv_cache_gib": {"dense": round(N * Hkv * T * dim * elem * 2 / 2 ** 30, 3),
                         "packed": round(retained * dim * elem * 2 / 2 ** 30, 3)},
        "parity_layer0": parity,
        "pattern": pinfo,
    }
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
