"""The HBM-traffic record built from rocprofv3 counter passes: per-launch
means of the kernel's working dispatches, each counter scaled by what it
reads for a copy of known size, the sources' digest and the probe budget."""
import argparse
import csv

from paper_2608_15438_amd import counters as CT


def _csv(path, rows):
    with open(path, "w", newline="") as fh:
        w = csv.DictWriter(fh, fieldnames=["Dispatch_Id", "Kernel_Name", "Counter_Name",
                                           "Counter_Value"])
        w.writeheader()
        for r in rows:
            w.writerow(r)


def test_traffic_record(tmp_path):
    k = "void nr::k_scan<1, 1, 1, 6>(nr::SharedArgs)"
    # two working launches and an empty one (skipped as not working)
    _csv(tmp_path / "f.csv", [
        dict(Dispatch_Id=1, Kernel_Name=k, Counter_Name="FETCH_SIZE", Counter_Value=1000.0),
        dict(Dispatch_Id=2, Kernel_Name=k, Counter_Name="FETCH_SIZE", Counter_Value=3000.0),
        dict(Dispatch_Id=3, Kernel_Name=k, Counter_Name="FETCH_SIZE", Counter_Value=1.0)])
    _csv(tmp_path / "w.csv", [
        dict(Dispatch_Id=1, Kernel_Name=k, Counter_Name="WRITE_SIZE", Counter_Value=10.0),
        dict(Dispatch_Id=2, Kernel_Name=k, Counter_Name="WRITE_SIZE", Counter_Value=30.0),
        dict(Dispatch_Id=3, Kernel_Name=k, Counter_Name="WRITE_SIZE", Counter_Value=0.0)])
    c = "copyBuffer"
    # the copy moves 4096 KiB each way: FETCH reads half of it, WRITE all of it
    _csv(tmp_path / "cf.csv", [dict(Dispatch_Id=9, Kernel_Name=c, Counter_Name="FETCH_SIZE",
                                    Counter_Value=2048.0)])
    _csv(tmp_path / "cw.csv", [dict(Dispatch_Id=9, Kernel_Name=c, Counter_Name="WRITE_SIZE",
                                    Counter_Value=4096.0)])
    a = argparse.Namespace(kernel="k_scan", workload="w", fetch=str(tmp_path / "f.csv"),
                           write=str(tmp_path / "w.csv"), copy_fetch=str(tmp_path / "cf.csv"),
                           copy_write=str(tmp_path / "cw.csv"), copy_bytes=4096 * 1024,
                           copy_kernel="copy", command="cmd", probe_budget=304)
    rec = CT.traffic(a)
    assert rec["dispatches"] == {"fetch": 2, "write": 2}
    assert rec["fetch_scale"] == 2.0 and rec["write_scale"] == 1.0
    assert rec["hbm_fetch_bytes_per_launch"] == 2000 * 1024 * 2
    assert rec["hbm_write_bytes_per_launch"] == 20 * 1024
    assert rec["hbm_bytes_per_launch"] == 2000 * 2048 + 20 * 1024
    assert rec["probe_budget"] == 304
    assert rec["source_sha256"] == CT.source_digest("k_scan")
