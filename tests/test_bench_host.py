"""bench.py host logic without a GPU: the one-GPU guard, argument checks, the
algorithmic byte and flop counts (closed forms on tiny cases) and the
rocprofv3 summary's counter scaling."""
import csv
import json
import os
import subprocess
import sys


ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench as B  # noqa: E402


def _run(*args):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args],
                          capture_output=True, text=True, timeout=120)


def test_more_than_one_gpu_is_refused():
    r = _run("--gpus", "2")
    assert r.returncode == 2 and "one GPU" in r.stderr


def test_fp8_kv_only_for_decode_and_prefill_workloads():
    r = _run("--kv", "fp8", "--workload", "mixed")
    assert r.returncode == 2 and "--kv fp8" in r.stderr


def test_decode_bytes_closed_form():
    # K and V: 2 * Hkv * d * ctx * s; q and out: B * Hq * d * 2 * s; one int32
    # page id per page; one int32 length per request.
    assert B.decode_bytes([16], hq=2, hkv=1, d=4) == 2 * 1 * 4 * 16 * 2 + 2 * 4 * 2 * 2 + 4 + 4
    assert B.decode_bytes([16], hq=2, hkv=1, d=4, kv_s=1) == 2 * 4 * 16 + 2 * 4 * 2 * 2 + 4 + 4
    assert B.decode_bytes([1, 17], 8, 2, 64) == (2 * 2 * 64 * 18 * 2 + 2 * 8 * 64 * 4
                                                 + 4 * (1 + 2) + 8)


def test_prefill_flops_closed_form():
    # causal: row i sees i + 1 keys; 4 d flops per (row, key, head)
    assert B.prefill_flops([3], hq=1, d=2) == 4 * 2 * (1 + 2 + 3)
    assert B.prefill_flops([1, 4], hq=3, d=8) == 4 * 8 * 3 * (1 + 10)


def test_write_pack_bytes_closed_form():
    # K and V read once and written twice (pages and handoff buffer), page ids, lengths, offsets
    assert B.write_pack_bytes([17], hkv=1, d=4) == 2 * 17 * 4 * 3 * 2 + 4 * 2 + 8 + 8


def test_write_and_pack_bytes_closed_form():
    assert B.write_bytes([17], hkv=1, d=4) == 2 * 17 * 4 * 4 + 4 * 2 + 8
    assert B.write_bytes([17], hkv=1, d=4, out_s=1) == 2 * 17 * 4 * 3 + 4 * 2 + 8
    assert B.pack_bytes([5, 7], layers=2, hkv=3, d=8) == 2 * 2 * 2 * 3 * 12 * 8 * 2


def _write_csv(path, rows):
    os.makedirs(os.path.dirname(path), exist_ok=True)
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=list(rows[0]))
        w.writeheader()
        w.writerows(rows)


def test_summarize_scales_counters_by_the_calibration_kernel(tmp_path):
    d = tmp_path / "prof"
    _write_csv(str(d / "trace" / "t_kernel_stats.csv"), [
        {"Name": "void dopd::decode_split_kernel<128, false>(dopd::DecodeArgs)", "Calls": 5,
         "AverageNs": 200000, "MinNs": 190000, "MaxNs": 210000, "Percentage": 90.0}])
    rows = []
    # calibration: 1 MiB read and written, counters read half of it for FETCH
    for ctr, kib_calib, kib_dec in (("FETCH_SIZE", 512.0, 1000.0), ("WRITE_SIZE", 1024.0, 10.0)):
        rows.append({"Dispatch_Id": f"{ctr}1", "Counter_Name": ctr, "Counter_Value": kib_calib,
                     "Kernel_Name": "void at::native::vectorized_elementwise_kernel<4, at::native::neg_kernel_cuda>"})
        for i in range(3):  # per-dispatch values split over two counter rows (summed)
            rows.append({"Dispatch_Id": f"{ctr}d{i}", "Counter_Name": ctr,
                         "Counter_Value": kib_dec / 2,
                         "Kernel_Name": "void dopd::decode_split_kernel<128, false>(dopd::DecodeArgs)"})
            rows.append({"Dispatch_Id": f"{ctr}d{i}", "Counter_Name": ctr,
                         "Counter_Value": kib_dec / 2,
                         "Kernel_Name": "void dopd::decode_split_kernel<128, false>(dopd::DecodeArgs)"})
    _write_csv(str(d / "pmc" / "p_counter_collection.csv"), rows)
    out = tmp_path / "summary.md"
    r = _run("--summarize", str(d), "--label", "unit", "--copy-calib-mib", "1",
             "--summary-out", str(out), "--traffic-dir", str(tmp_path), "--command", "x")
    assert r.returncode == 0, r.stderr
    t = json.load(open(tmp_path / "traffic_unit.json"))
    assert t["copy_factors"] == {"FETCH_SIZE": 2.0, "WRITE_SIZE": 1.0}
    # 1000 KiB fetched x 2 + 10 KiB written x 1, per dispatch
    assert t["calls"]["decode"]["hbm_bytes_per_call"] == 1024 * (1000 * 2 + 10)
    assert t["source_hash"] == B.source_hash()
    text = out.read_text()
    assert "decode_split_kernel" in text and "200.00" in text


def test_repeat_timed_covers_the_requested_time():
    calls = []
    res, n, dt = B.repeat_timed(lambda: calls.append(1) or len(calls), 0.05)
    assert res == 1 and n == len(calls) and n >= 2 and dt >= 0.05
    res, n, _ = B.repeat_timed(lambda: 7, 0.0)
    assert res == 7 and n == 1


def test_bench_line_is_strict_json():
    import json
    line = {"value": 1.5, "calls": {"a": {"step_mean_us": B.mean_or_none([])}},
            "parity": [float("nan"), float("inf"), 2.0]}
    text = json.dumps(B.json_safe(line), allow_nan=False)
    assert json.loads(text) == {"value": 1.5, "calls": {"a": {"step_mean_us": None}},
                                "parity": [None, None, 2.0]}
    assert B.mean_or_none([1.0, 2.0]) == 1.5
