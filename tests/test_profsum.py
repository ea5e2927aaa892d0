"""The measurement chain on the CPU: rocprofv3 CSV -> profile summary ->
bench.py's `roofline.traffic`.  Synthetic CSV fixtures with known counter
values: the copy-kernel calibration scales FETCH_SIZE and WRITE_SIZE, the
summary states the kernel's HBM bytes per launch and the hash of the kernel
source, and the bench takes the bytes only while that source is unchanged."""
import csv
import hashlib
import importlib.util
import os

from paper_2607_24787_amd import profsum

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
KERNEL = "void spp::(anonymous namespace)::ffn_slices_kernel<unsigned short, 4, true, 3, 1>(spp::FfnArgs)"
COPY = "__amd_rocclr_copyBuffer"


def _counters(d, rows):
    os.makedirs(d, exist_ok=True)
    with open(os.path.join(d, "run_counter_collection.csv"), "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Kernel_Name", "Counter_Value"])
        w.writeheader()
        for name, v in rows:
            w.writerow({"Kernel_Name": name, "Counter_Value": v})


def _bench_module():
    spec = importlib.util.spec_from_file_location("bench_under_test", os.path.join(ROOT, "bench.py"))
    m = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(m)
    return m


def _fixture(tmp_path):
    # calibration: a 256 MiB copy whose FETCH_SIZE reads back half its bytes and WRITE_SIZE all of them
    _counters(tmp_path / "cal_f", [(COPY, 131072.0)])
    _counters(tmp_path / "cal_w", [(COPY, 262144.0)])
    # the kernel: two dispatches, 90 and 110 KiB fetched (mean 100), 10 KiB written
    _counters(tmp_path / "f", [(KERNEL, 90.0), (KERNEL, 110.0), (COPY, 131072.0)])
    _counters(tmp_path / "w", [(KERNEL, 10.0), (KERNEL, 10.0), (COPY, 262144.0)])
    src = tmp_path / "kernels.hip"
    src.write_text("// kernel source stand-in\n")
    return src


def test_traffic_scales_the_counters_by_the_copy_calibration(tmp_path):
    src = _fixture(tmp_path)
    text = profsum.traffic(str(tmp_path / "f"), str(tmp_path / "w"), str(tmp_path / "cal_f"), str(tmp_path / "cal_w"),
                           "ffn_slices_kernel", algorithmic=102400, source=str(src))
    # read = 100 KiB x 2 (FETCH_SIZE scale) = 204,800 B; written = 10 KiB x 1 = 10,240 B
    assert "scale 2.000" in text and "scale 1.000" in text
    assert "204,800 B read + 10,240 B written per launch" in text
    assert "read / algorithmic = 2.000" in text
    fields = dict(line.split(": ", 1) for line in text.splitlines() if ": " in line)
    assert int(fields["traffic_bytes_per_launch"]) == 215040
    assert fields["kernel_source_sha256_16"] == hashlib.sha256(src.read_bytes()).hexdigest()[:16]


def test_the_bench_takes_the_traffic_only_while_the_kernel_source_is_unchanged(tmp_path):
    src = _fixture(tmp_path)
    text = profsum.traffic(str(tmp_path / "f"), str(tmp_path / "w"), str(tmp_path / "cal_f"), str(tmp_path / "cal_w"),
                           "ffn_slices_kernel", source=str(src))
    prof = tmp_path / "profile.md"
    prof.write_text("# summary\n\n" + text + "\n")
    bench = _bench_module()
    assert bench.measured_traffic(str(prof), str(src)) == 215040
    src.write_text("// kernel source stand-in, changed\n")
    assert bench.measured_traffic(str(prof), str(src)) is None
    assert bench.measured_traffic(str(tmp_path / "missing.md"), str(src)) is None


def _trace(d, kernels, copies):
    os.makedirs(d, exist_ok=True)
    with open(os.path.join(d, "run_kernel_trace.csv"), "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Kernel_Name", "Start_Timestamp", "End_Timestamp"])
        w.writeheader()
        for name, s, e in kernels:
            w.writerow({"Kernel_Name": name, "Start_Timestamp": s, "End_Timestamp": e})
    with open(os.path.join(d, "run_memory_copy_trace.csv"), "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Direction", "Start_Timestamp", "End_Timestamp"])
        w.writeheader()
        for s, e in copies:
            w.writerow({"Direction": "MEMORY_COPY_HOST_TO_DEVICE", "Start_Timestamp": s, "End_Timestamp": e})


def test_overlap_splits_launches_by_a_concurrent_host_copy(tmp_path):
    # two FFN launches overlap the copy [1000, 5000] ns, one does not; medians 3.0 / 2.0 us
    _trace(tmp_path, [(KERNEL, 0, 2000), (KERNEL, 4000, 8000), (KERNEL, 10000, 12000)], [(1000, 5000)])
    text = profsum.overlap(str(tmp_path), ["ffn_slices_kernel"])
    assert "| `ffn_slices_kernel` | 2 | 3.00 | 1 | 2.00 |" in text


def test_copies_rates_and_link_sharing(tmp_path):
    blob = 9_437_184
    # an FFN launch marks the decode's start; two prefetches after it, 170 us alone and
    # 340 us half of which shares the link with an on-demand copy kernel
    ks = [(KERNEL, 1_000, 2_000), ("h2d_copy_kernel", 300_000, 470_000)]
    cps = [(-200_000, -30_000), (3_000, 173_000), (300_000, 640_000)]
    _trace(tmp_path, ks, cps)
    text = profsum.copies(str(tmp_path), blob)
    assert "3 host-to-device (1 before the decode" in text and "2 during the decode" in text
    assert f"median 170.0 µs per copy -> {blob / 170_000:.2f} GB/s" in text
    assert f"<5% shared): 1, median {blob / 170_000:.2f} GB/s" in text
    assert f"at least half their time: 1, median {blob / 340_000:.2f} GB/s" in text
    assert "mean 0.250" in text  # (0 + 0.5) / 2 of each prefetch's time shared
    assert "80.1% of the decode span (510 of 637 µs)" in text
