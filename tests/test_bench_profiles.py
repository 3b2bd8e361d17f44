"""The benchmark's readers of rocprofv3 counter output (host only): a role's
launches are the kernels between a pair of role markers on the marker's own
hardware queue; counters are summed over their instances; FETCH_SIZE and
WRITE_SIZE (KiB per dispatch) are scaled by what they read for a copy of
known size; the kernel trace's role spans come from marker pairs on one
stream.  Checked on small synthetic counter files and trace databases."""
import csv
import json
import os

import pytest

import bench

FIELDS = ["Dispatch_Id", "Queue_Id", "Kernel_Name", "Counter_Name", "Counter_Value"]


def _write(d, rows):
    os.makedirs(d, exist_ok=True)
    with open(os.path.join(d, "run_counter_collection.csv"), "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=FIELDS)
        w.writeheader()
        for r in rows:
            w.writerow(dict(zip(FIELDS, r)))


def _role_rows(counter, values):
    """Queue 1 holds the role (two marked launches of two kernels each, one
    unmarked kernel between them); queue 2 runs other kernels interleaved.
    Each dispatch reports its value as two instances of half the value."""
    seq = [(1, "role_marker"), (1, "gemm_a"), (2, "other_x"), (1, "reduce_b"), (1, "role_marker"),
           (1, "outside"), (2, "other_y"),
           (1, "role_marker"), (1, "gemm_a"), (1, "reduce_b"), (1, "role_marker")]
    rows = []
    for i, (q, name) in enumerate(seq):
        v = values.get((i, name), 0.0 if name == "role_marker" else 1000.0)
        rows += [(i, q, name, counter, v / 2), (i, q, name, counter, v / 2)]
    return rows


def test_role_launches_are_the_kernels_between_marker_pairs_on_their_queue(tmp_path):
    vals = {(1, "gemm_a"): 10.0, (3, "reduce_b"): 2.0, (8, "gemm_a"): 30.0, (9, "reduce_b"): 4.0}
    _write(tmp_path / "c", _role_rows("SQ_INSTS_MFMA", vals))
    launches = bench._between_markers(bench._per_dispatch(bench._pmc_rows(str(tmp_path / "c")), "SQ_INSTS_MFMA"))
    assert [l[0] for l in launches] == [12.0, 34.0]  # instances summed; queue 2 and "outside" excluded
    assert all(l[1] == ["gemm_a", "reduce_b"] for l in launches)


def test_counter_summary_reports_the_median_launch(tmp_path, capsys):
    rows = _role_rows("SQ_WAVE_CYCLES", {(1, "gemm_a"): 5.0, (3, "reduce_b"): 1.0, (8, "gemm_a"): 7.0,
                                         (9, "reduce_b"): 1.0})
    rows += [(r[0], r[1], r[2], "GRBM_GUI_ACTIVE", 3.0) for r in rows[::2]]
    _write(tmp_path / "c", rows)
    bench.counter_summary(str(tmp_path / "c"), "ffn1.dw")
    out = json.loads(capsys.readouterr().out)
    assert out["role"] == "ffn1.dw" and out["launches"] == 2
    # median of two launches = the upper one (index len // 2)
    assert out["counters"]["SQ_WAVE_CYCLES"] == 8.0
    assert out["counters"]["GRBM_GUI_ACTIVE"] == 6.0
    assert out["kernels"] == ["gemm_a", "reduce_b"]


def test_traffic_is_scaled_by_the_copy_calibration(tmp_path, monkeypatch, capsys):
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(tmp_path / "traffic.json"))
    kib = bench.COPY_BYTES / 1024
    # the copy read (just over) half its bytes on FETCH_SIZE and all of them on
    # WRITE_SIZE; a small dispatch of the same kernel is not a calibration
    _write(tmp_path / "cal_f", [(0, 1, "elementwise_kernel", "FETCH_SIZE", kib * 0.5001),
                                (1, 1, "elementwise_kernel", "FETCH_SIZE", 4.0)])
    _write(tmp_path / "cal_w", [(0, 1, "elementwise_kernel", "WRITE_SIZE", kib)])
    _write(tmp_path / "f", _role_rows("FETCH_SIZE", {(1, "gemm_a"): 100.0, (3, "reduce_b"): 0.0,
                                                     (8, "gemm_a"): 100.0, (9, "reduce_b"): 0.0}))
    _write(tmp_path / "w", _role_rows("WRITE_SIZE", {(1, "gemm_a"): 40.0, (3, "reduce_b"): 10.0,
                                                     (8, "gemm_a"): 40.0, (9, "reduce_b"): 10.0}))
    bench.traffic_summary(str(tmp_path / "f"), str(tmp_path / "w"), str(tmp_path / "cal_f"),
                          str(tmp_path / "cal_w"), "qkv.dw", "synthetic workload")
    e = json.loads(capsys.readouterr().out)["qkv.dw"]
    assert e["fetch_scale"] == pytest.approx(1 / 0.5001) and e["write_scale"] == pytest.approx(1.0)
    assert e["fetch_bytes_per_launch"] == pytest.approx(100.0 * 1024 / 0.5001)
    assert e["write_bytes_per_launch"] == pytest.approx(50.0 * 1024)
    stored = json.load(open(tmp_path / "traffic.json"))
    assert stored["source_sha256"] == bench.source_digest() and stored["workload"] == "synthetic workload"
    assert stored["roles"]["qkv.dw"]["bytes_per_launch"] == pytest.approx(e["bytes_per_launch"])


def test_kernel_trace_roles_from_marker_pairs(tmp_path, capsys):
    """The kernel-trace summary attributes to a role the kernels that its
    start and end markers (role = grid_x / workgroup_x, edge = grid_y - 1)
    enclose on the same stream, in dispatch order."""
    import sqlite3
    from paper_1811_06965_amd import gp
    role = gp.KERNEL_ROLE["ffn1.fwd"]
    d = tmp_path / "trace"
    d.mkdir()
    db = sqlite3.connect(str(d / "run_results.db"))
    db.execute("create table kernels (name text, grid_x int, grid_y int, workgroup_x int, start int, end int, "
               "stream_id int, dispatch_id int)")
    ns = 1000
    rows = [("role_marker", role * 64, 1, 64, 0, 1, 1),
            ("gemm_dl<256>(gp::GemmArgs)", 256, 1, 256, 10 * ns, 40 * ns, 1),
            ("other_kernel", 64, 1, 64, 20 * ns, 60 * ns, 2),
            ("role_marker", role * 64, 2, 64, 41 * ns, 41 * ns + 1, 1),
            ("outside_kernel", 64, 1, 64, 60 * ns, 90 * ns, 1),
            ("role_marker", role * 64, 1, 64, 95 * ns, 95 * ns + 1, 1),
            ("gemm_dl<256>(gp::GemmArgs)", 256, 1, 256, 100 * ns, 140 * ns, 1),
            ("splitk_reduce(gp::GemmArgs, int)", 64, 1, 64, 145 * ns, 150 * ns, 1),
            ("role_marker", role * 64, 2, 64, 151 * ns, 151 * ns + 1, 1)]
    db.executemany("insert into kernels values (?, ?, ?, ?, ?, ?, ?, ?)",
                   [r + (i,) for i, r in enumerate(rows)])
    db.commit()
    db.close()
    roles_json = tmp_path / "roles.json"
    bench.kernel_summary(str(d), "cmd", roles_json=str(roles_json))
    out = capsys.readouterr().out
    assert "| ffn1.fwd | 2 | 37.5 | 40.0 |" in out  # kernel time 30 and 45 us; first start to last end 30 and 50
    rec = json.load(open(roles_json))["roles"]["ffn1.fwd"]
    assert rec["launches"] == 2 and rec["mean_kernel_us"] == pytest.approx(37.5)
    assert rec["mean_span_us"] == pytest.approx(40.0)
    assert "other_kernel" not in str(rec["kernels"]) and "outside_kernel" not in str(rec["kernels"])
