"""Host logic of bench.py that runs without a GPU: the HBM traffic record
built from rocprofv3 --pmc counter files (FETCH_SIZE and WRITE_SIZE in KiB per
dispatch, each scaled by what the counter reads for a plain copy of known
size, and checked against the read probe, which reads each token once)."""
import json
import os

import bench


def _counters(d, counter, rows):
    os.makedirs(d)
    with open(os.path.join(d, "p_counter_collection.csv"), "w") as f:
        f.write('"Kernel_Name","Counter_Name","Counter_Value"\n')
        for name, value in rows:
            f.write('"%s","%s","%r"\n' % (name, counter, value))


def test_traffic_summary(tmp_path, monkeypatch):
    d = str(tmp_path)
    gib4 = 4 << 30
    # the copy reads FETCH_SIZE = half its bytes and WRITE_SIZE = all of them
    _counters(os.path.join(d, "prof_copy_fetch"), "FETCH_SIZE", [("__amd_rocclr_copyBuffer", gib4 / 1024 / 2)] * 3)
    _counters(os.path.join(d, "prof_copy_write"), "WRITE_SIZE", [("__amd_rocclr_copyBuffer", gib4 / 1024)] * 3)
    scan = "void pk::scan_rows<0>(pk::ScanArgs)"
    # the read probe reads each of the run's 262,144 tokens once: 1 MiB, FETCH_SIZE 512 KiB
    _counters(os.path.join(d, "prof_fetch"), "FETCH_SIZE",
              [(scan, 1000.0), (scan, 1002.0), ("pk::rows_fast<false>(pk::RowArgs)", 10.0),
               ("pk::read_probe(HIP_vector_type<int, 4u> const*, long)", 512.0)])
    _counters(os.path.join(d, "prof_write"), "WRITE_SIZE", [(scan, 7.0), (scan, 9.0)])
    with open(os.path.join(d, "prof_fetch.log"), "w") as f:
        f.write("profiler noise\n")
        f.write(json.dumps({"config": {"workload": "large: 1 row", "tokens": 262144},
                            "roofline": {"algorithmic_bytes": 2_000_000.0}}) + "\n")
    out = tmp_path / "traffic.json"
    monkeypatch.setattr(bench, "PROFILE_TRAFFIC", str(out))
    bench.traffic_summary(d)
    rec = json.loads(out.read_text())
    # fetch 1001 KiB / 0.5 + write 8 KiB / 1.0
    assert rec["bytes_per_launch"] == 1001 * 1024 / 0.5 + 8 * 1024
    assert rec["launches"] == 2 and rec["workload"] == "large"
    assert rec["copy_calibration"]["fetch_factor"] == 0.5 and rec["copy_calibration"]["write_factor"] == 1.0
    assert rec["traffic_over_algorithmic"] == rec["bytes_per_launch"] / 2_000_000.0
    assert rec["kernel_source_sha"] == bench.kernel_sha()
    # the second calibration point: the probe's own factor, and the copy's factor applied to it
    assert rec["probe_check"]["fetch_factor"] == 0.5
    assert rec["probe_check"]["calibrated_over_read"] == 1.0
