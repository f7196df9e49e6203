"""bench.py's command line on the host: a request for more than one GPU ends before any
device work, with exit status 2 and a message that names the one-GPU limit (no GPU needed)."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_bench_refuses_more_than_one_gpu():
    for n in (2, 8):
        r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", str(n),
                            "--steps", "1", "--warmup", "0"],
                           cwd=ROOT, capture_output=True, text=True, timeout=120)
        assert r.returncode == 2, (r.returncode, r.stdout, r.stderr)
        assert "one GPU" in r.stderr and f"--gpus {n}" in r.stderr
        assert r.stdout.strip() == ""        # no JSON line for a run that did not happen


def _counter_db(path, rows):
    import sqlite3
    con = sqlite3.connect(path)
    con.execute("create table counters_collection (kernel_name text, counter_name text, "
                "dispatch_id integer, value real)")
    con.executemany("insert into counters_collection values (?, ?, ?, ?)", rows)
    con.commit()
    con.close()


def test_pmc_summary_scales_by_the_copy_kernel_and_picks_the_timed_instance(tmp_path,
                                                                            monkeypatch):
    sys.path.insert(0, ROOT)
    import bench
    probe = "void fpsk::stream_kernel<0, false, 4, 4, 1, true, false>(fpsk::StreamArgs)"
    calib = "void fpsk::stream_kernel<0, false, 1, 4, 1, true, false>(fpsk::StreamArgs)"
    copy = "void fpsk::copy_kernel(float4 const*, float4*, long)"
    # two counter instances per dispatch (summed), 3 timed dispatches, 1 calibration dispatch;
    # the copy kernel reads 2x and writes 0.5x its 262144 KiB
    fetch = [(probe, "FETCH_SIZE", d, 600.0) for d in (1, 2, 3) for _ in range(2)]
    fetch += [(calib, "FETCH_SIZE", 9, 50.0), (copy, "FETCH_SIZE", 10, 524288.0)]
    write = [(probe, "WRITE_SIZE", d, 10.0) for d in (1, 2, 3)]
    write += [(calib, "WRITE_SIZE", 9, 5.0), (copy, "WRITE_SIZE", 10, 131072.0)]
    fdb, wdb = str(tmp_path / "f.db"), str(tmp_path / "w.db")
    _counter_db(fdb, fetch)
    _counter_db(wdb, write)
    out = tmp_path / "summary.txt"
    monkeypatch.setattr(bench, "pmc_summary_path", lambda workload: str(out))
    assert bench.write_pmc_summary("square16384_fp16", 2, fdb, wdb) == 0
    kv = dict(ln.split("=", 1) for ln in out.read_text().splitlines()
              if "=" in ln and not ln.startswith("#"))
    assert kv["kernel"] == probe and kv["stream_dispatches"] == "3"
    assert float(kv["fetch_scale"]) == 0.5 and float(kv["write_scale"]) == 2.0
    # 1200 KiB fetched x 0.5 + 10 KiB written x 2, in bytes
    assert float(kv["traffic_bytes_per_launch"]) == (600.0 + 20.0) * 1024
    assert "--workload square16384_fp16 --sets 2" in out.read_text()
