"""Host logic of bench.py that needs no GPU: interval algebra and the
overlap figures of a hand-built timeline, the FFN and copy rooflines, and
the rocprofv3 summaries (PMC scaling by the calibration copy, kernel
statistics) on small hand-written CSV files."""
import csv
import json
import os

import pytest

import bench


def _rec(kind, t0, t1, nbytes=0):
    return dict(kind=kind, layer=0, t0_ms=t0, t1_ms=t1, bytes=nbytes)


def test_interval_union_and_intersection():
    u = bench._union([(0, 2), (1, 3), (5, 6), (6, 7), (9, 9)])
    assert u == [[0, 3], [5, 7]]
    assert bench._length(u) == 5
    assert bench._intersect(u, bench._union([(2, 6)])) == 2


def test_analyse_overlap_figures():
    # one step: router 0-1, resident FFN 1-3, copies 2-6 and 6-8, streamed FFN 6-7, combine 8-9
    G = 10 ** 9
    tl = [_rec("router", 0, 1), _rec("ffn_resident", 1, 3, 300 * G), _rec("copy_miss", 2, 6, 400 * G),
          _rec("copy_miss", 6, 8, 200 * G), _rec("ffn_streamed", 6, 7, 100 * G), _rec("combine", 8, 9)]
    an = bench.analyse(tl, 1, 9.0)
    assert an["copy_ms"] == 6 and an["kernel_ms"] == 5
    # copies under kernels: 2-3 and 6-7 -> 2 ms of 6
    assert an["hidden_frac"] == pytest.approx(2 / 6)
    assert an["compute_hidden_frac"] == pytest.approx(2 / 5)
    assert an["overlap_eta"] == pytest.approx((5 + 6 - 9) / 5)
    assert an["miss_bytes"] == 600 * G and an["step_us"]["p50"] == pytest.approx(9000.0)
    roof = bench.ffn_roofline(an)
    assert roof["bytes_per_launch"] == 200 * G and roof["avg_launch_us"] == pytest.approx(1500.0)
    assert roof["achieved"] == pytest.approx(400 * G / 3e-3 / 1e9, rel=1e-3)
    assert roof["frac"] == pytest.approx(roof["achieved"] / 8000.0, rel=1e-3)
    cr = bench.copy_roofline(tl)
    assert cr["bound"] == "pcie" and cr["launches"] == 2
    assert cr["achieved"] == pytest.approx(600 * G / 6e-3 / 1e9, rel=1e-6)
    assert cr["peak"] == pytest.approx(63.02, abs=0.01)


def _write(path, header, rows):
    os.makedirs(os.path.dirname(path), exist_ok=True)
    with open(path, "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(header)
        w.writerows(rows)


def test_pmc_summary_scales_by_the_calibration_copy(tmp_path):
    cal_kib = bench.CALIB_BYTES / 1024
    hdr = ["Dispatch_Id", "Kernel_Name", "Counter_Value"]
    # FETCH_SIZE reads half of what moves (factor 0.5), WRITE_SIZE all of it
    _write(str(tmp_path / "f" / "x" / "f_counter_collection.csv"), hdr,
           [[1, "msk::ffn_chunk_kernel<1>(a)", 999.0], [2, "__amd_rocclr_copyBuffer", cal_kib * 0.5],
            [3, "void msk::ffn_chunk_kernel<unsigned short, 1, 1, 64, 4>(msk::FfnArgs)", 1000.0],
            [4, "void msk::ffn_chunk_kernel<unsigned short, 1, 1, 64, 4>(msk::FfnArgs)", 3000.0],
            [5, "msk::combine_planes_kernel(msk::CombineArgs)", 10.0]])
    _write(str(tmp_path / "w" / "x" / "w_counter_collection.csv"), hdr,
           [[2, "__amd_rocclr_copyBuffer", cal_kib],
            [3, "void msk::ffn_chunk_kernel<unsigned short, 1, 1, 64, 4>(msk::FfnArgs)", 4.0],
            [4, "void msk::ffn_chunk_kernel<unsigned short, 1, 1, 64, 4>(msk::FfnArgs)", 4.0]])
    out = str(tmp_path / "pmc.md")
    log = tmp_path / "pass.log"
    log.write_text("[bench] noise\n" + json.dumps({"pmc_pass": "wl", "ffn_launches": 2,
                                                   "ffn_algorithmic_bytes": 2 * 4000 * 1024}) + "\n")
    bench.pmc_summary(str(tmp_path / "f"), str(tmp_path / "w"), "wl", out, "cmd f", "cmd w", pass_log=str(log))
    text = open(out).read()
    vals = dict(line.strip("- ").split(": ") for line in text.splitlines() if line.startswith("- `"))
    # dispatches after the calibration copy only; fetch (1000 + 3000) / 2 / 0.5 KiB, write 4 KiB each
    assert vals["`ffn_dispatches`"] == "`2`"
    assert vals["`ffn_traffic_bytes_per_launch`"] == "`%d`" % int((2000 * 2 + 4) * 1024)
    assert vals["`ffn_algorithmic_bytes_per_launch`"] == "`%d`" % (4000 * 1024)
    assert vals["`ffn_traffic_ratio`"] == "`%.4f`" % ((4000 + 4) / 4000)
    assert "cmd f" in text and "cmd w" in text
    # bench reads (traffic, algorithmic bytes) back while the sources hash the same
    monkey = bench.PROFILES
    try:
        bench.PROFILES = str(tmp_path)
        import shutil
        shutil.copy(out, bench.pmc_profile_path("wl"))
        assert bench.traffic_from_profile("wl") == ((4000 + 4) * 1024, 4000 * 1024)
        assert bench.traffic_from_profile("other") is None
    finally:
        bench.PROFILES = monkey


def test_trace_summary_orders_kernels_by_time(tmp_path):
    hdr = ["Name", "Calls", "TotalDurationNs", "AverageNs", "Percentage", "MinNs", "MaxNs", "StdDev"]
    _write(str(tmp_path / "t" / "k_kernel_stats.csv"), hdr,
           [["void a(int)", 2, 1000, 500, 10.0, 400, 600, 1], ["b(x)", 1, 9000, 9000, 90.0, 9000, 9000, 0]])
    out = str(tmp_path / "k.md")
    bench.trace_summary(str(tmp_path / "t"), out, "the command")
    rows = [line for line in open(out).read().splitlines() if line.startswith("| `")]
    assert rows[0].startswith("| `b` | 1 | 0.009") and rows[1].startswith("| `a` | 2 |")


def test_more_than_one_gpu_is_refused(monkeypatch, capsys):
    monkeypatch.setattr("sys.argv", ["bench.py", "--gpus", "2"])
    with pytest.raises(SystemExit) as ei:
        bench.main()
    assert ei.value.code == 2
    assert "one GPU" in capsys.readouterr().err


def test_mfma_roofline_of_prefill_launches():
    import synth
    shape = synth.DEEPSEEK  # d 2048, F 1408, K 6, two shared experts of 1408
    T, steps = 512, 2
    # two steps: gate/up 0-1 ms and down 1-1.5 ms per step, 1 GB of weights per step
    tl = [_rec("router", 0, 0.1), _rec("ffn_resident", 0.1, 1.1, 2 * 10 ** 9 // 3),
          _rec("ffn_down", 1.1, 1.6, 10 ** 9 // 3),
          _rec("router", 2, 2.1), _rec("ffn_resident", 2.1, 3.1, 2 * 10 ** 9 // 3),
          _rec("ffn_down", 3.1, 3.6, 10 ** 9 // 3)]
    an = bench.analyse(tl, steps, 2.0)
    m = bench.mfma_roofline(an, shape, T, steps)
    flops_step = 6.0 * 2048 * (1408 * T * 6 + 1408 * T * 2)
    assert m["flops_per_step"] == pytest.approx(flops_step)
    assert m["achieved"] == pytest.approx(flops_step * steps / 3e-3 / 1e12, rel=1e-3)
    assert m["frac"] == pytest.approx(m["achieved"] / 2500.0, abs=1e-4)
    intensity = flops_step * steps / (2 * (2 * 10 ** 9 // 3 + 10 ** 9 // 3))
    assert m["flop_per_weight_byte"] == pytest.approx(intensity, rel=1e-3)
    # 70 GFLOP over 1 GB: 70 flop per byte x 8 TB/s = 560 TFLOP/s < 2500, so HBM bounds it
    assert m["bound"] == "hbm" and m["attainable"] == pytest.approx(intensity * 8.0, rel=1e-3)
    assert m["attainable_frac"] == pytest.approx(m["achieved"] / m["attainable"], abs=1e-4)
    # decode forwards (no down launches) report none
    assert bench.mfma_roofline(bench.analyse(tl[:2], 1, 1.0), shape, 1, 1) is None


def test_platform_info_never_fails():
    """The platform record is reporting only: without a GPU (this test runs
    on the CPU) it returns the host CPU fields and an error note instead of
    raising."""
    info = bench.platform_info()
    assert info["cpu"]["logical_cpus"] >= 1
    assert info["cpu"]["usable_cpus"] is None or info["cpu"]["usable_cpus"] >= 1
    assert "gpu" in info or "error" in info
