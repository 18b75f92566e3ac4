"""Host-side logic of bench.py (no GPU): the counter summary that scales
FETCH_SIZE / WRITE_SIZE by the calibration copy, the decode kernel a default
launch runs, and the statistic of the headline."""
import csv
import json
import os
import sys

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
import bench  # noqa: E402

FIELDS = ["Kernel_Name", "Counter_Value"]


def _write(path, rows):
    os.makedirs(os.path.dirname(path), exist_ok=True)
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=FIELDS)
        w.writeheader()
        for name, v in rows:
            w.writerow({"Kernel_Name": name, "Counter_Value": v})


def test_traffic_summary_scales_by_calibration(tmp_path):
    d = str(tmp_path)
    copy_kib = (1 << 30) / 1024
    # the copy reads half its bytes in FETCH_SIZE units and all of them in WRITE_SIZE units
    _write(f"{d}/cal_FETCH_SIZE/p_counter_collection.csv",
           [("__amd_rocclr_copyBuffer", copy_kib / 2)] * 3)
    _write(f"{d}/cal_WRITE_SIZE/p_counter_collection.csv",
           [("__amd_rocclr_copyBuffer", copy_kib)] * 3)
    dec = "void rag::paged_decode_balanced_kernel<128, false>(rag::PagedKernelArgs)"
    pf = "void rag::prefill_varlen_kernel<128>(unsigned short const*)"
    _write(f"{d}/pmc_FETCH_SIZE/p_counter_collection.csv",
           [(dec, 100.0), (dec, 300.0), (pf, 1000.0), ("void other(int)", 5.0)])
    _write(f"{d}/pmc_WRITE_SIZE/p_counter_collection.csv",
           [(dec, 1.0), (dec, 3.0), (pf, 400.0), ("void other(int)", 5.0)])
    out = os.path.join(d, "traffic.json")
    t = bench.traffic_summary(d, out)
    assert json.load(open(out)) == t
    assert t["calibration"]["fetch_factor"] == 2.0 and t["calibration"]["write_factor"] == 1.0
    k = t["kernels"]["paged_decode_balanced_kernel<128, false>"]
    assert k["dispatches"] == 2
    assert k["fetch_bytes_per_launch"] == 200 * 1024 * 2
    assert k["write_bytes_per_launch"] == 2 * 1024
    assert k["bytes_per_launch"] == 200 * 1024 * 2 + 2 * 1024
    assert t["kernels"]["prefill_varlen_kernel<128>"]["bytes_per_launch"] == (2000 + 400) * 1024
    assert set(t["kernels"]) == {"paged_decode_balanced_kernel<128, false>",
                                 "prefill_varlen_kernel<128>"}
    assert t["source_hash"] == bench.kernel_source_hash()
    assert all(d in c for c in t["commands"][:4])


def test_stored_traffic_matches_current_sources():
    """The committed counters are keyed by the kernel names bench.py reports,
    or are null because the sources changed since they were taken."""
    with open(os.path.join(bench.PROFILES, "traffic.json")) as f:
        t = json.load(f)
    if t["source_hash"] != bench.kernel_source_hash():
        assert bench.stored_traffic("prefill_varlen_kernel<128>") is None
        return
    assert bench.stored_traffic("prefill_varlen_kernel<128>") > 0
    assert bench.stored_traffic(bench.decode_kernel_name(16, 8)) > 0


def test_decode_kernel_name():
    assert bench.decode_kernel_name(16, 8).startswith("paged_decode_balanced_kernel")
    assert bench.decode_kernel_name(31, 8).startswith("paged_decode_balanced_kernel")
    assert bench.decode_kernel_name(32, 8).startswith("paged_decode_kernel")
    assert bench.decode_kernel_name(320, 8).startswith("paged_decode_kernel")


def test_median():
    assert bench.median([3.0, 1.0, 2.0]) == 2.0
    assert bench.median([4.0, 1.0, 2.0, 3.0]) == 2.5
