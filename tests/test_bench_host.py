"""Host logic of bench.py's profile summaries (CPU only): which dispatches a
counter run attributes to the packed, paged and query-block calls and to the
two packs, and how the counters are scaled.  Synthetic counter files stand in for rocprofv3's."""

import csv
import importlib.util
import json
import os

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def bench():
    spec = importlib.util.spec_from_file_location("bench_under_test", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


PACKED = "void dkv::(anonymous namespace)::decode_kernel<true, 128, 4, false>(dkv::DecodeParams)"
PAGED = "void dkv::(anonymous namespace)::decode_kernel<true, 128, 4, true>(dkv::DecodeParams)"
MERGE = "void dkv::(anonymous namespace)::decode_merge_kernel<128, 4>(dkv::DecodeParams)"
PLAN = "dkv::(anonymous namespace)::query_plan_kernel(dkv::QueryParams)"
QATT = "void dkv::(anonymous namespace)::query_attn_kernel<128>(dkv::QueryParams)"
QMRG = "void dkv::(anonymous namespace)::query_merge_kernel<128>(dkv::QueryParams)"
COPY = "void at::native::elementwise_kernel<128, 2>(int, Lambda)"
CCOUNT = "dkv::(anonymous namespace)::compact_count_kernel(dkv::CompactParams)"
CSCAN = "dkv::(anonymous namespace)::compact_scan_kernel(dkv::CompactParams)"
CLIST = "dkv::(anonymous namespace)::compact_list_kernel(dkv::CompactParams)"
CCOPY = "void dkv::(anonymous namespace)::compact_copy_kernel<16>(dkv::CompactParams)"
BPLAN = "dkv::(anonymous namespace)::bins_plan_kernel(dkv::BinsParams)"
BSCAN = "dkv::(anonymous namespace)::bins_scan_kernel(dkv::BinsParams)"
BCOPY = "void dkv::(anonymous namespace)::bins_copy_kernel<16>(dkv::BinsParams)"
PCOPY = "void (anonymous namespace)::copy_kernel<1>(u32x4 const*, u32x4*, long)"


def test_helpers(bench):
    assert bench.is_paged_kernel(PAGED) and not bench.is_paged_kernel(PACKED)
    assert not bench.is_paged_kernel(MERGE)
    line = {"config": {"layers": 2}, "steps": 2, "warmup": 1}
    # warm step + graph warmup and timed replays + eager warmup and timed steps, per layer
    assert bench.timed_calls_per_mode(line) == 2 * (1 + 2 * 3)
    line["step_ms_spread"] = {"median": 1.0}
    assert bench.timed_calls_per_mode(line) == 2 * (1 + 2 * 3 + 2)
    line["step_ms_spread"] = {"median": 1.0, "reps": 50}  # the spread pass's own replay count
    assert bench.timed_calls_per_mode(line) == 2 * (1 + 2 * 3 + 50)


def _counter_csv(path, counter, dispatches):
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"])
        w.writeheader()
        for i, (name, kib) in enumerate(dispatches):
            # two rows per dispatch (one per counter instance): the summary adds them
            for part in (0.25, 0.75):
                w.writerow({"Dispatch_Id": i + 1, "Kernel_Name": name, "Counter_Name": counter,
                            "Counter_Value": kib * part})


@pytest.mark.parametrize("parity", [False, True])
def test_pmc_summary_attribution(bench, tmp_path, monkeypatch, parity):
    layers, steps, warmup = 2, 2, 1
    line = {"config": {"layers": layers}, "steps": steps, "warmup": warmup, "step_ms_spread": {"median": 1.0},
            "parity_layer0": {"layers": layers} if parity else None,
            "one_time": {"compact_bytes": 2 * 1024 * 1024, "compact_bins_bytes": 1024 * 1024}}
    m = bench.timed_calls_per_mode(line)
    log = tmp_path / "bench.log"
    log.write_text("[bench] noise\n" + json.dumps(line) + "\n")
    copy_kib = (1 << 30) / 1024.0  # a copy of exactly 1 GiB

    def run(scale):
        d = []
        # the one-time section: a warm and a timed mask pack, a warm and a timed
        # block gather (the second of each is counted), then the copy probe
        d += [(CCOUNT, 9.0), (CSCAN, 9.0), (CLIST, 9.0), (CCOPY, 9.0)]
        d += [(CCOUNT, 8.0 * scale), (CSCAN, 2.0 * scale), (CLIST, 30.0 * scale), (CCOPY, 2008.0 * scale)]
        d += [(BPLAN, 9.0), (BSCAN, 9.0), (BCOPY, 9.0)]
        d += [(BPLAN, 4.0 * scale), (BSCAN, 1.0 * scale), (BCOPY, 1019.0 * scale)]
        d += [(PCOPY, 5.0)] * 3
        d += [(PACKED, 999.0), (MERGE, 1.0)] * (layers if parity else 0)  # parity calls: not counted
        d += [(PACKED, 100.0 * scale), (MERGE, 2.0 * scale)] * m             # the packed calls
        d += [(PACKED, 300.0 * scale), (MERGE, 4.0 * scale)] * m             # the dense calls
        d += [(PAGED, 110.0 * scale), (MERGE, 2.0 * scale)] * 5              # paged, by template flag
        d += [(PLAN, 1.0 * scale), (QATT, 500.0 * scale), (QMRG, 50.0 * scale)] * 3
        d += [(PACKED, 7.0), (MERGE, 7.0)] * 4                               # later sections
        d += [(COPY, copy_kib * scale)]
        return d

    fetch, write = tmp_path / "fetch.csv", tmp_path / "write.csv"
    _counter_csv(fetch, "FETCH_SIZE", run(0.5))   # counter reads half the bytes: factor 2
    _counter_csv(write, "WRITE_SIZE", run(1.0))
    out = tmp_path / "pmc.json"
    monkeypatch.setattr(bench, "PMC_FILE", str(out))
    bench.pmc_summary(str(fetch), str(write), str(log), "cmd")
    res = json.loads(out.read_text())
    assert res["fetch_calibration"] == pytest.approx(2.0) and res["write_calibration"] == pytest.approx(1.0)
    assert res["fetch_calls_counted"] == m
    # every counter value is scaled back to bytes: 0.5 * 102 KiB * 2 = 102 KiB per packed call
    assert res["fetch_bytes_per_call"] == int(102 * 1024) and res["write_bytes_per_call"] == int(102 * 1024)
    assert res["traffic_bytes_per_launch"] == 2 * 102 * 1024
    assert res["paged_traffic_bytes_per_launch"] == 2 * 112 * 1024
    assert res["query_calls_counted"] == 3
    assert res["query_traffic_bytes_per_call"] == 2 * 551 * 1024
    assert res["kernel_sha256_16"] == bench.kernel_hash()
    assert res["query_kernel_sha256_16"] == bench.kernel_hash(bench.QUERY_SRCS)
    # the packs: the timed (second) call of each, scaled like the rest
    assert res["compact_traffic_bytes"] == 2 * 2048 * 1024
    assert res["compact_traffic_over_algorithmic"] == pytest.approx(2.0)
    assert res["compact_bins_traffic_bytes"] == 2 * 1024 * 1024
    assert res["compact_bins_traffic_over_algorithmic"] == pytest.approx(2.0)
    assert res["compact_kernel_sha256_16"] == bench.kernel_hash(bench.COMPACT_SRCS)
    assert res["compact_bins_kernel_sha256_16"] == bench.kernel_hash(bench.BINS_SRCS)


@pytest.mark.parametrize("argv,text", [(["--gpus", "2"], "one GPU only"), (["--steps", "0"], "--steps")])
def test_refusals_exit_before_any_gpu_work(argv, text):
    """More than one GPU, or no timed step, is refused with exit status 2
    before torch or the library is loaded."""
    import subprocess
    import sys
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *argv], capture_output=True, text=True,
                       timeout=120)
    assert r.returncode == 2
    assert text in r.stderr and r.stdout == ""
