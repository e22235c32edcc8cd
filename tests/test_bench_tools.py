"""CPU checks of bench.py's measurement plumbing: the rocprofv3 counter
summaries, the copy calibration of the traffic counters, the kernel-source gate
on stored traffic, and the one-GPU guard."""
import csv
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402

FIELDS = ["Correlation_Id", "Dispatch_Id", "Agent_Id", "Queue_Id", "Process_Id", "Thread_Id",
          "Grid_Size", "Kernel_Id", "Kernel_Name", "Workgroup_Size", "LDS_Block_Size",
          "Scratch_Size", "VGPR_Count", "Accum_VGPR_Count", "SGPR_Count", "Counter_Name",
          "Counter_Value", "Start_Timestamp", "End_Timestamp"]


def _csv(path, rows):
    """rows: (dispatch id, kernel name, counter, value)"""
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=FIELDS)
        w.writeheader()
        for d, name, counter, value in rows:
            r = {k: 0 for k in FIELDS}
            r.update(Dispatch_Id=d, Correlation_Id=d, Kernel_Name=name, Counter_Name=counter,
                     Counter_Value=value, Agent_Id="Agent 1")
            w.writerow(r)
    return str(path)


FWD = "void ffk::(anonymous namespace)::k_fwd<false, 128, 128, 4, 2, 2, true>(...)"
DW = "void ffk::(anonymous namespace)::k_dw_adam_f32<64, 128, 32, 2, 4, 3, true>(...)"
COPY = "__amd_rocclr_copyBuffer"


def test_counter_per_dispatch_and_largest(tmp_path):
    p = _csv(tmp_path / "c.csv", [(1, FWD, "FETCH_SIZE", 100.0), (2, FWD, "FETCH_SIZE", 200.0),
                                  (3, DW, "FETCH_SIZE", 50.0), (4, COPY, "FETCH_SIZE", 7.0),
                                  (5, COPY, "FETCH_SIZE", 3000.0), (5, FWD, "WRITE_SIZE", 9.0)])
    per, n = bench._counter_per_dispatch(p, "FETCH_SIZE")
    assert per["forward"] == pytest.approx(150.0) and n["forward"] == 2
    assert per["dw_adam"] == pytest.approx(50.0) and n["dw_adam"] == 1
    assert bench._largest_dispatch(p, "FETCH_SIZE") == 3000.0


def test_traffic_summary_scales_by_the_copy(tmp_path, monkeypatch):
    """A 1 GiB copy that reads FETCH_SIZE = 0.5 GiB and WRITE_SIZE = 1 GiB
    scales fetches by 2 and writes by 1."""
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    monkeypatch.setattr(bench, "kernel_source_hash", lambda: "feedc0de01234567")
    os.makedirs(tmp_path / "profiles")
    gib_kib = float(1 << 20)
    f = _csv(tmp_path / "f.csv", [(1, FWD, "FETCH_SIZE", 1000.0), (2, FWD, "FETCH_SIZE", 3000.0)])
    w = _csv(tmp_path / "w.csv", [(1, FWD, "WRITE_SIZE", 500.0), (2, FWD, "WRITE_SIZE", 500.0)])
    cf = _csv(tmp_path / "cf.csv", [(1, COPY, "FETCH_SIZE", gib_kib / 2)])
    cw = _csv(tmp_path / "cw.csv", [(1, COPY, "WRITE_SIZE", gib_kib)])
    bench.traffic_summary(f, w, cf, cw, "wl", 1 << 30)
    t = json.load(open(tmp_path / "profiles" / "traffic.json"))
    assert t["fetch_factor"] == pytest.approx(2.0) and t["write_factor"] == pytest.approx(1.0)
    e = t["wl"]["forward"]
    assert e["fetch_bytes_per_launch"] == pytest.approx(2000.0 * 1024 * 2)
    assert e["write_bytes_per_launch"] == pytest.approx(500.0 * 1024)
    assert e["kernel_source_sha256_16"] == "feedc0de01234567"


def test_stored_traffic_only_for_the_same_kernel_source(tmp_path, monkeypatch):
    assert len(bench.kernel_source_hash()) == 16  # of the real kernel file
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    monkeypatch.setattr(bench, "kernel_source_hash", lambda: "feedc0de01234567")
    os.makedirs(tmp_path / "profiles")
    path = tmp_path / "profiles" / "traffic.json"
    entry = {"bytes_per_launch": 123.0, "kernel_source_sha256_16": bench.kernel_source_hash()}
    json.dump({"wl": {"forward": entry}}, open(path, "w"))
    assert bench.load_traffic("forward", "wl") == 123.0
    entry["kernel_source_sha256_16"] = "0" * 16
    json.dump({"wl": {"forward": entry}}, open(path, "w"))
    assert bench.load_traffic("forward", "wl") is None
    assert bench.load_traffic("dw_adam", "wl") is None


def test_counter_summary_mfma_busy(tmp_path, capsys):
    """Half of the 1024 SIMDs' cycles busy over a GPU-active time of 1000
    cycles per XCD (8 XCDs summed) reads as 50 % MFMA busy."""
    d = tmp_path / "focus_1_2_3_0"
    os.makedirs(d)
    p = _csv(d / "run_counter_collection.csv",
             [(1, FWD, "SQ_VALU_MFMA_BUSY_CYCLES", 1024 * 1000 * 0.5),
              (1, FWD, "GRBM_GUI_ACTIVE", 8 * 1000.0), (1, FWD, "SQ_WAVE_CYCLES", 200.0),
              (1, FWD, "SQ_WAIT_ANY", 50.0), (1, FWD, "SQ_WAIT_INST_LDS", 10.0),
              (1, FWD, "SQ_INSTS_LDS", 100.0), (1, FWD, "SQ_LDS_BANK_CONFLICT", 5.0)])
    bench.counter_summary([p])
    out = capsys.readouterr().out
    row = [ln for ln in out.splitlines() if "forward" in ln][0]
    cells = [c.strip() for c in row.strip("|").split("|")]
    assert cells[0] == "focus_1_2_3_0" and cells[2] == "1"
    assert cells[3] == "50.0 %" and cells[4] == "25.0 %" and cells[5] == "5.0 %"
    assert cells[6] == "0.050"


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


TRACE_FIELDS = ["Kind", "Agent_Id", "Queue_Id", "Stream_Id", "Thread_Id", "Dispatch_Id",
                "Kernel_Id", "Kernel_Name", "Correlation_Id", "Start_Timestamp", "End_Timestamp",
                "Grid_Size_X"]
LOSS = "void ffk::(anonymous namespace)::k_loss_rows(...)"


def _trace(path, rows):
    """rows: (dispatch id, kernel name, duration in ns)"""
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=TRACE_FIELDS)
        w.writeheader()
        t = 1000
        for d, name, ns in rows:
            r = {k: 0 for k in TRACE_FIELDS}
            r.update(Dispatch_Id=d, Kernel_Name=name, Start_Timestamp=t, End_Timestamp=t + ns)
            t += ns + 10
            w.writerow(r)
    return str(path)


def _rec(kind, m, n, k, flops, bytes_, ms, aux=0):
    return dict(kind=kind, m=m, n=n, k=k, aux=aux, ms=ms, flops=flops, bytes=bytes_)


def test_shape_labels_and_weighted_fraction():
    a = _rec("forward", 2048, 2000, 784, 2.0 * 2048 * 2000 * 784, 1e6, 0.1)
    b = _rec("forward", 2048, 2000, 2000, 2.0 * 2048 * 2000 * 2000, 1e6, 0.2)
    assert bench.shape_label(a) == "2048x784->2000"
    assert bench.shape_label(_rec("forward", 100, 2000, 784, 0, 0, 0, aux=10)) == \
        "100x784->2000 (x10 labels)"
    assert bench.shape_label(_rec("dw_adam", 2000, 784, 2048, 0, 0, 0)) == "784->2000 over 2048 rows"
    assert bench.shape_label(_rec("embed_norm", 4096, 3072, 0, 0, 0, 0, aux=1 | 16)) == \
        "4096x3072 (pairs, bf16 out)"
    recs = [a, b, b]
    shapes = bench.by_shape(recs, "f32")
    assert [s["launches"] for s in shapes] == [1, 2]
    assert shapes[1]["avg_us"] == pytest.approx(200.0)
    tot = bench.kind_totals(recs, "f32")["forward"]
    # shape-weighted: summed flops over summed time, not the mean of the per-shape fractions
    want = (a["flops"] + 2 * b["flops"]) / (0.5e-3) / 1e12
    assert tot["TFLOP/s"] == pytest.approx(want)
    assert tot["frac"] == pytest.approx(want / bench.PEAK["f32"][1])


def test_rocprof_shapes_matches_dispatches_in_order(tmp_path, capsys):
    recs = [_rec("forward", 64, 64, 64, 2.0 * 64 ** 3, 1.0, 0.005),
            _rec("loss", 64, 64, 1, 0.0, 4e6, 0.002),
            _rec("forward", 64, 64, 64, 2.0 * 64 ** 3, 1.0, 0.004),
            _rec("loss", 64, 64, 1, 0.0, 4e6, 0.001)]
    lst = tmp_path / "l.json"
    bench.write_launch_list(str(lst), recs, [False, False, True, True], "f32", "test")
    # a torch kernel between ours is skipped; durations come from the trace
    tr = _trace(tmp_path / "t.csv", [(1, FWD, 5000), (2, "at::native::copy", 99), (3, LOSS, 2000),
                                     (4, FWD, 8000), (5, LOSS, 1000)])
    bench.rocprof_shapes(tr, str(lst))
    out = capsys.readouterr().out
    assert "| forward | 64x64->64 | 1 | 8.0 | 4.0 |" in out
    assert "| loss | 64x64 | 1 | 1.0 | 1.0 | 4.00 MB | 4000 GB/s | 50.0 % |" in out
    bad = _trace(tmp_path / "b.csv", [(1, FWD, 5000), (3, FWD, 2000), (4, FWD, 8000),
                                      (5, LOSS, 1000)])
    with pytest.raises(SystemExit, match="launch 1"):
        bench.rocprof_shapes(bad, str(lst))
    short = _trace(tmp_path / "s.csv", [(1, FWD, 5000)])
    with pytest.raises(SystemExit, match="dispatches"):
        bench.rocprof_shapes(short, str(lst))
    # set-up dispatches before the recorded window are skipped
    pre = _trace(tmp_path / "p.csv", [(0, "k_bf16_shadow", 700), (1, FWD, 5000), (3, LOSS, 2000),
                                      (4, FWD, 6000), (5, LOSS, 1000)])
    bench.rocprof_shapes(pre, str(lst))
    out = capsys.readouterr().out
    assert "after 1 earlier ones" in out and "| forward | 64x64->64 | 1 | 6.0 | 4.0 |" in out


def test_copy_sweep_summary_reads_the_timed_copies(tmp_path, capsys):
    rows, d = [], 1
    for mb in bench.COPY_SWEEP_MB:
        for k in range(bench._copy_rotation(mb)):  # untimed pass
            rows.append((d, "__amd_rocclr_copyBuffer", 10 ** 9))
            d += 1
        for k in range(bench.COPY_SWEEP_REPS):
            rows.append((d, "__amd_rocclr_copyBuffer", 2 * mb * (1 << 20) // 4000))  # 4000 B/ns
            d += 1
            rows.append((d, "at::native::fill", 5))
            d += 1
    bench.copy_sweep_summary(_trace(tmp_path / "c.csv", rows))
    out = capsys.readouterr().out
    assert out.count("| 4000 GB/s | 50.0 % |") == len(bench.COPY_SWEEP_MB)
    with pytest.raises(SystemExit, match="copy dispatches"):
        bench.copy_sweep_summary(_trace(tmp_path / "s.csv", rows[:5]))


def test_traffic_by_shape_matches_dispatches_and_scales(tmp_path, monkeypatch, capsys):
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    monkeypatch.setattr(bench, "kernel_source_hash", lambda: "feedc0de01234567")
    os.makedirs(tmp_path / "profiles")
    recs = [_rec("forward", 64, 64, 64, 1.0, 3e6, 0.1), _rec("forward", 64, 64, 64, 1.0, 3e6, 0.1),
            _rec("loss", 64, 64, 1, 0.0, 1e6, 0.1)]
    lst = tmp_path / "l.json"
    bench.write_launch_list(str(lst), recs, [False, True, True], "f32", "test")
    kib = 1e6 / 1024.0
    # a torch kernel and a set-up dispatch before the list are skipped
    f = _csv(tmp_path / "f.csv", [(1, FWD, "FETCH_SIZE", 7.0), (2, FWD, "FETCH_SIZE", 1.0),
                                  (3, "at::native::x", "FETCH_SIZE", 9.0),
                                  (4, FWD, "FETCH_SIZE", 2 * kib), (5, LOSS, "FETCH_SIZE", kib)])
    w = _csv(tmp_path / "w.csv", [(1, FWD, "WRITE_SIZE", 7.0), (2, FWD, "WRITE_SIZE", 1.0),
                                  (4, FWD, "WRITE_SIZE", kib), (5, LOSS, "WRITE_SIZE", 0.0)])
    gib_kib = float(1 << 20)
    cf = _csv(tmp_path / "cf.csv", [(1, COPY, "FETCH_SIZE", gib_kib / 2)])
    cw = _csv(tmp_path / "cw.csv", [(1, COPY, "WRITE_SIZE", gib_kib)])
    bench.traffic_by_shape(f, w, cf, cw, str(lst), "wl", 1 << 30)
    out = capsys.readouterr().out
    assert "| forward | 64x64->64 | 1 | 4.0 | 1.0 | 3.0 | 1.67 |" in out
    t = json.load(open(tmp_path / "profiles" / "traffic.json"))["wl"]
    assert t["forward"]["bytes_per_launch"] == pytest.approx(5e6)
    assert t["loss"]["fetch_bytes_per_launch"] == pytest.approx(2e6)


def test_overlap_summary_of_the_second_epoch(tmp_path, capsys):
    def trace(path, rows):  # (dispatch id, kernel name, start us, end us)
        with open(path, "w", newline="") as f:
            w = csv.DictWriter(f, fieldnames=TRACE_FIELDS)
            w.writeheader()
            for d, name, s, e in rows:
                r = {k: 0 for k in TRACE_FIELDS}
                r.update(Dispatch_Id=d, Kernel_Name=name, Start_Timestamp=int(s * 1000),
                         End_Timestamp=int(e * 1000))
                w.writerow(r)
        return str(path)
    first = [(1, FWD, 0, 10), (2, LOSS, 10, 20), (3, FWD, 20, 30)]
    second = [(4, FWD, 1000, 1100), (5, LOSS, 1050, 1150), (6, FWD, 1200, 1300)]
    tr = trace(tmp_path / "t.csv", first + [(9, "at::native::copy", 0, 5000)] + second)
    bench.overlap_summary(tr)
    out = capsys.readouterr().out
    assert "3 dispatches of the library's kernels over 0.30 ms" in out
    assert "some kernel runs 83.3 %" in out and "(1.00 kernels at once" in out
    assert "| forward | 2 | 200.0 | 100.0 |" in out and "| loss | 1 | 100.0 | 100.0 |" in out
    assert "| forward | 150.0 | 50.0 % |" in out
    assert "| forward + loss | 50.0 | 16.7 % |" in out
    assert "| loss | 50.0 | 16.7 % |" in out and "| (none) | 50.0 | 16.7 % |" in out
    odd = trace(tmp_path / "o.csv", first + second[:2])
    with pytest.raises(SystemExit, match="not two equal epochs"):
        bench.overlap_summary(odd)
