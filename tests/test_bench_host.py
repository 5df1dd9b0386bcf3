"""Host logic of bench.py on the CPU: the rocprofv3 summaries (kernel
trace, HBM traffic with the copy calibration, SQ counters) computed from
small synthetic result databases shaped like rocprofv3's, the traffic read
back only for a matching kernel-source digest, and the one-GPU guard."""
import os
import sqlite3
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402

FWD = "void mk::fwd_kernel<128, true, false, 1, true, false>(mk::FwdArgs)"
COPY = "void __amd_rocclr_copyBuffer(...)"


def _db(path, kernels=(), pmc=()):
    os.makedirs(path, exist_ok=True)
    con = sqlite3.connect(os.path.join(path, "x_results.db"))
    con.execute("create table kernels (name text, duration integer)")
    con.execute("create table pmc_events (dispatch_id integer, name text, counter_name text, "
                "counter_value real)")
    con.executemany("insert into kernels values (?, ?)", kernels)
    con.executemany("insert into pmc_events values (?, ?, ?, ?)", pmc)
    con.commit()
    con.close()
    return path


def test_summarize_trace_averages_per_kernel(tmp_path):
    d = _db(str(tmp_path / "t"), kernels=[(FWD, 80_000), (FWD, 90_000), (COPY, 10_000)])
    out = bench.summarize_trace(d, "cmd", ["fwd_kernel"])
    row = [l for l in out.splitlines() if "fwd_kernel" in l][0]
    cells = [c.strip() for c in row.split("|")]
    assert cells[2] == "2"              # calls
    assert cells[3] == "85.00"          # avg us
    assert cells[4] == "80.00" and cells[5] == "90.00"
    assert cells[6] == "94.4"           # share of all GPU time (170 of 180 us)
    assert "copyBuffer" not in out


def test_summarize_pmc_scales_by_the_copy(tmp_path):
    calib = 1 << 30
    # the copy reads half its bytes in FETCH_SIZE units (x2) and all in WRITE_SIZE
    fetch = _db(str(tmp_path / "f"), pmc=[(1, COPY, "FETCH_SIZE", calib / 1024 / 2),
                                          (2, FWD, "FETCH_SIZE", 1000.0),
                                          (3, FWD, "FETCH_SIZE", 3000.0)])
    write = _db(str(tmp_path / "w"), pmc=[(1, COPY, "WRITE_SIZE", calib / 1024),
                                          (2, FWD, "WRITE_SIZE", 500.0),
                                          (3, FWD, "WRITE_SIZE", 500.0)])
    out = bench.summarize_pmc(fetch, write, ["fwd_kernel"], calib, ["a", "b"])
    total = float(out.split("hbm_bytes_per_launch:")[1].split()[0])
    assert total == pytest.approx(2000.0 * 1024 * 2 + 500.0 * 1024)


def test_summarize_sq_ratios(tmp_path):
    a = _db(str(tmp_path / "a"), pmc=[(1, FWD, "GRBM_GUI_ACTIVE", 8.0e6),
                                      (1, FWD, "SQ_VALU_MFMA_BUSY_CYCLES", 0.5 * 1024 * 1.0e6),
                                      (1, FWD, "SQ_WAVE_CYCLES", 1.0e9),
                                      (1, FWD, "SQ_WAIT_ANY", 2.5e8)])
    b = _db(str(tmp_path / "b"), pmc=[(1, FWD, "SQ_INSTS_VALU", 5.0e6),
                                      (1, FWD, "SQ_INSTS_MFMA", 1.0e6)])
    out = bench.summarize_sq([a, b], "fwd_kernel<128", ["cmd"])
    assert "MFMA busy: 50.0 %" in out
    assert "SQ_WAIT_ANY / SQ_WAVE_CYCLES: 25.0 %" in out
    assert "vector instructions per MFMA (SQ_INSTS_VALU less MFMA): 4.00" in out


def test_traffic_needs_matching_digest(tmp_path, monkeypatch):
    prof = tmp_path / "profiles"
    prof.mkdir()
    (prof / "k_counters.md").write_text("kernel_source_digest: abc123\n\nhbm_bytes_per_launch: 1.5e+08\n")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    assert bench.read_traffic("k_counters.md", "abc123") == 1.5e8
    assert bench.read_traffic("k_counters.md", "ffff00") is None
    assert bench.read_traffic("missing.md", "abc123") is None


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_summarize_trace_splits_one_kernel_by_grid(tmp_path):
    d = str(tmp_path / "g")
    os.makedirs(d)
    con = sqlite3.connect(os.path.join(d, "x_results.db"))
    con.execute("create table kernels (name text, duration integer, grid_x integer, "
                "workgroup_x integer)")
    con.executemany("insert into kernels values (?, ?, ?, ?)",
                    [(FWD, 80_000, 1024 * 256, 256), (FWD, 7_000_000, 8192 * 256, 256),
                     (FWD, 82_000, 1024 * 256, 256)])
    con.commit()
    con.close()
    out = bench.summarize_trace(d, "cmd", ["fwd_kernel"])
    rows = {l.split("`")[1]: l for l in out.splitlines() if l.startswith("| `")}
    assert set(rows) == {"mk::fwd_kernel<128, true, false, 1, true, false> [1024 workgroups]",
                         "mk::fwd_kernel<128, true, false, 1, true, false> [8192 workgroups]"}
    small = [c.strip() for c in rows["mk::fwd_kernel<128, true, false, 1, true, false> "
                                     "[1024 workgroups]"].split("|")]
    assert small[2] == "2" and small[3] == "81.00"


def test_summarize_trace_tells_persistent_launches_by_their_copy(tmp_path):
    """The persistent forward launches 256 workgroups on every workload; its
    launches are told apart by the V^T copy made just before each."""
    pers = "void mk::fwd_kernel<128, true, false, 1, true, false, 8, false, true, true>(mk::FwdArgs)"
    pack = "void mk::vt_pack_kernel<128>(mk::VtPackArgs)"
    d = str(tmp_path / "p")
    os.makedirs(d)
    con = sqlite3.connect(os.path.join(d, "x_results.db"))
    con.execute("create table kernels (dispatch_id integer, name text, duration integer, "
                "grid_x integer, workgroup_x integer)")
    con.executemany("insert into kernels values (?, ?, ?, ?, ?)",
                    [(1, pack, 25_000, 4096 * 256, 256), (2, pers, 7_000_000, 256 * 512, 512),
                     (3, pack, 15_000, 2048 * 256, 256), (4, pers, 1_000_000, 256 * 512, 512),
                     (5, pack, 26_000, 4096 * 256, 256), (6, pers, 7_200_000, 256 * 512, 512)])
    con.commit()
    con.close()
    out = bench.summarize_trace(d, "cmd", ["fwd_kernel"])
    rows = {l.split("`")[1]: [c.strip() for c in l.split("|")]
            for l in out.splitlines() if l.startswith("| `")}
    name = "mk::fwd_kernel<128, true, false, 1, true, false, 8, false, true, true>"
    assert set(rows) == {f"{name} [after a V^T copy of 4096 tiles]",
                         f"{name} [after a V^T copy of 2048 tiles]"}
    assert rows[f"{name} [after a V^T copy of 4096 tiles]"][2:4] == ["2", "7100.00"]
    assert rows[f"{name} [after a V^T copy of 2048 tiles]"][2:4] == ["1", "1000.00"]


def test_summarize_pmc_splits_one_kernel_by_grid(tmp_path):
    """'name@N' selects the launches of a kernel with N workgroups, so one
    forward kernel timed on two workloads gets one traffic figure each."""
    calib = 1 << 30

    def db(path, counter, copy_val, vals):
        os.makedirs(path)
        con = sqlite3.connect(os.path.join(path, "x_results.db"))
        con.execute("create table kernels (dispatch_id integer, name text, duration integer, "
                    "grid_x integer, workgroup_x integer)")
        con.execute("create table pmc_events (dispatch_id integer, name text, "
                    "counter_name text, counter_value real)")
        con.executemany("insert into kernels values (?, ?, ?, ?, ?)",
                        [(1, COPY, 1, 4096 * 256, 256), (2, FWD, 1, 1024 * 256, 256),
                         (3, FWD, 1, 8192 * 256, 256), (4, FWD, 1, 1024 * 256, 256)])
        con.executemany("insert into pmc_events values (?, ?, ?, ?)",
                        [(1, COPY, counter, copy_val)] +
                        [(d, FWD, counter, v) for d, v in zip((2, 3, 4), vals)])
        con.commit()
        con.close()
        return path
    fetch = db(str(tmp_path / "f"), "FETCH_SIZE", calib / 1024 / 2, (100.0, 9000.0, 300.0))
    write = db(str(tmp_path / "w"), "WRITE_SIZE", calib / 1024, (50.0, 4000.0, 50.0))
    small = bench.summarize_pmc(fetch, write, ["fwd_kernel@1024"], calib, ["c"])
    big = bench.summarize_pmc(fetch, write, ["fwd_kernel@8192"], calib, ["c"])
    t_small = float(small.split("hbm_bytes_per_launch:")[1].split()[0])
    t_big = float(big.split("hbm_bytes_per_launch:")[1].split()[0])
    assert t_small == pytest.approx(200.0 * 1024 * 2 + 50.0 * 1024)
    assert t_big == pytest.approx(9000.0 * 1024 * 2 + 4000.0 * 1024)


def test_unknown_leg_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--legs", "c9"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode != 0
    assert "unknown legs" in r.stderr
