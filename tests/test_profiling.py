"""Host logic of the profile summaries: the traffic figure bench.py reports
is read back only for the kernel and the sources that were profiled."""
import os

from paper_2606_04238_amd import profiling


def _write(path, kernel, digest, traffic="1234"):
    with open(path, "w") as fh:
        fh.write("# x\n\n| a | b |\n\ntraffic_bytes_per_launch: %s\nkernel: %s\nsource_digest: %s\n"
                 % (traffic, kernel, digest))


def test_read_traffic_matches_digest_and_kernel(tmp_path):
    p = os.path.join(tmp_path, "k.md")
    _write(p, "fused_layer_kernel", profiling.source_digest())
    assert profiling.read_traffic(p, "fused_layer_kernel") == 1234.0
    assert profiling.read_traffic(p, "down_w4_kernel") is None


def test_read_traffic_stale_sources(tmp_path):
    p = os.path.join(tmp_path, "k.md")
    _write(p, "fused_layer_kernel", "0" * 16)
    assert profiling.read_traffic(p, "fused_layer_kernel") is None
    assert profiling.read_traffic(os.path.join(tmp_path, "missing.md"), "fused_layer_kernel") is None


def test_digest_is_stable():
    assert profiling.source_digest() == profiling.source_digest()
    assert len(profiling.source_digest()) == 16


def _csv(path, header, rows):
    import csv
    with open(path, "w", newline="") as fh:
        w = csv.writer(fh)
        w.writerow(header)
        w.writerows(rows)


def test_summary_sums_a_steps_kernels_and_uses_the_nontemporal_calibration(tmp_path):
    """A step of two kernels: the duration and bytes are the sums of the
    kernels' means; FETCH_SIZE is scaled by the non-temporal probe's factor
    (known / counted), WRITE_SIZE by the copy's."""
    kt, pf, pw = (tmp_path / n for n in ("kt", "pf", "pw"))
    for d in (kt, pf, pw):
        d.mkdir()
    _csv(kt / "x_kernel_stats.csv", ["Name", "Calls", "AverageNs", "MinNs", "MaxNs", "Percentage"],
         [["void a_kernel<1>()", 10, 1000.0, 900, 1100, 50], ["void b_kernel<2>()", 10, 3000.0, 2900, 3100, 50]])
    hdr = ["Kernel_Name", "Counter_Name", "Counter_Value"]
    _csv(pf / "x_counter_collection.csv", hdr,
         [["void a_kernel<1>()", "FETCH_SIZE", 100.0], ["void b_kernel<2>()", "FETCH_SIZE", 300.0],
          ["void a_kernel<1>()", "FETCH_SIZE", 100.0], ["void b_kernel<2>()", "FETCH_SIZE", 300.0],
          ["void stream_read_kernel<true>(x)", "FETCH_SIZE", 512.0],
          ["void stream_read_kernel<false>(x)", "FETCH_SIZE", 600.0],
          ["void at::native::vectorized_elementwise_kernel<8>", "FETCH_SIZE", 64.0]])
    _csv(pw / "x_counter_collection.csv", hdr,
         [["void a_kernel<1>()", "WRITE_SIZE", 10.0], ["void b_kernel<2>()", "WRITE_SIZE", 20.0],
          ["void at::native::vectorized_elementwise_kernel<8>", "WRITE_SIZE", 128.0]])
    out = tmp_path / "s.md"
    total = profiling.summarize(str(kt), str(pf), str(pw), "a_kernel|b_kernel", 128 / 1024, str(out),
                                ["cmd"], stream_mib=1)
    # fetch: (100 + 300) KiB * (1024 / 512); write: (10 + 20) KiB * (128 / 128)
    assert total == (400 * 2 + 30) * 1024
    text = out.read_text()
    assert "kernel_avg_us: 4.000" in text and "kernel: a_kernel|b_kernel" in text
    assert profiling.read_traffic(str(out), "a_kernel|b_kernel") == total


def test_step_dispatches_follow_the_launch_order():
    """Only runs of consecutive dispatches in the step's order count: a stray
    dispatch of one of the step's kernels (another call of it between steps)
    is left out."""
    names = ["a_kernel", "b_kernel", "a_kernel", "c_kernel", "a_kernel", "b_kernel", "b_kernel"]
    rows = [{"Dispatch_Id": str(i + 1), "Kernel_Name": n} for i, n in enumerate(names)]
    assert profiling.step_dispatches(rows, ["a_kernel", "b_kernel"], "Kernel_Name") == [[1, 5], [2, 6]]
    assert profiling.step_dispatches(rows, ["c_kernel", "b_kernel"], "Kernel_Name") is None
    assert profiling.step_dispatches([{"Kernel_Name": "a"}], ["a"], "Kernel_Name") is None


def test_summary_takes_the_step_dispatches_from_the_trace_and_counters(tmp_path):
    """With dispatch ids the summary averages the step's own dispatches; a
    stray a_kernel launch with other durations and byte counts is ignored."""
    kt, pf, pw = (tmp_path / n for n in ("kt", "pf", "pw"))
    for d in (kt, pf, pw):
        d.mkdir()
    _csv(kt / "x_kernel_stats.csv", ["Name", "Calls", "AverageNs", "MinNs", "MaxNs", "Percentage"],
         [["void a_kernel<1>()", 3, 700.0, 100, 1000, 50], ["void b_kernel<2>()", 2, 3000.0, 3000, 3000, 50]])
    seq = [("void a_kernel<1>()", 1000), ("void b_kernel<2>()", 3000), ("void a_kernel<1>()", 100),
           ("void a_kernel<1>()", 1000), ("void b_kernel<2>()", 3000)]
    _csv(kt / "x_kernel_trace.csv", ["Dispatch_Id", "Kernel_Name", "Start_Timestamp", "End_Timestamp"],
         [[i + 1, n, 10000 * i, 10000 * i + t] for i, (n, t) in enumerate(seq)])
    hdr = ["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"]
    vals = {"void a_kernel<1>()": 100.0, "void b_kernel<2>()": 300.0}
    _csv(pf / "x_counter_collection.csv", hdr,
         [[i + 1, n, "FETCH_SIZE", 7.0 if (i == 2) else vals[n]] for i, (n, _) in enumerate(seq)]
         + [[9, "void at::native::vectorized_elementwise_kernel<8>", "FETCH_SIZE", 64.0]])
    _csv(pw / "x_counter_collection.csv", hdr,
         [[i + 1, n, "WRITE_SIZE", 1.0 if (i == 2) else 10.0] for i, (n, _) in enumerate(seq)]
         + [[9, "void at::native::vectorized_elementwise_kernel<8>", "WRITE_SIZE", 128.0]])
    out = tmp_path / "s.md"
    total = profiling.summarize(str(kt), str(pf), str(pw), "a_kernel|b_kernel", 128 / 1024, str(out),
                                ["cmd"])
    # copy calibration: fetch 128 KiB known / 64 counted = 2; write 1
    assert total == ((100 + 300) * 2 + (10 + 10)) * 1024
    assert "kernel_avg_us: 4.000" in out.read_text()
