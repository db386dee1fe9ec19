"""Host logic of bench.py (CPU only): the HBM-counter summary scales each
counter by what it reads for the reference conversion, takes the most
frequent (symbol, grid) group of each site among the step's dispatches
(those before the reference conversion), and the traffic it writes is used
only while the kernel sources it was taken on are unchanged."""
import csv
import json

import bench


def _write(d, counter, rows):
    d.mkdir(parents=True)
    with open(d / "x_counter_collection.csv", "w", newline="") as fh:
        w = csv.DictWriter(fh, fieldnames=["Dispatch_Id", "Kernel_Name", "Grid_Size", "Counter_Name", "Counter_Value"])
        w.writeheader()
        for i, (name, grid, kib) in enumerate(rows, 1):
            w.writerow({"Dispatch_Id": i, "Kernel_Name": name, "Grid_Size": grid, "Counter_Name": counter,
                        "Counter_Value": kib})


def test_counter_summary_scales_by_the_reference_and_picks_the_frequent_group(tmp_path):
    ref = ("o5::f32_to_bf16_kernel(unsigned long, float const*, unsigned short*)", bench.COPY_REF_N // 8)
    fwd = "void o5::gemm_kk<256, o5::EpiLstmCell<unsigned short>, unsigned short>(...)"
    # FETCH_SIZE counts half of the reference's bytes read; WRITE_SIZE all of them
    # the step's dispatches, then the reference, then other workloads (the
    # same symbol and grid as the step's, which must not count)
    fetch = [(fwd, 262144, 1000.0)] * 16 + [(fwd, 131072, 5.0)]      # the behaviour pass's other grid
    fetch += [(ref[0], ref[1], 4.0 * bench.COPY_REF_N / 1024 / 2)] + [(fwd, 262144, 7.0)] * 40
    write = [(fwd, 262144, 100.0)] * 16 + [(fwd, 131072, 1.0)]
    write += [(ref[0], ref[1], 2.0 * bench.COPY_REF_N / 1024)] + [(fwd, 262144, 3.0)] * 40
    _write(tmp_path / "f", "FETCH_SIZE", fetch)
    _write(tmp_path / "w", "WRITE_SIZE", write)
    out = bench.summarize_counters(str(tmp_path / "f"), str(tmp_path / "w"), str(tmp_path / "t.json"))
    assert abs(out["FETCH_SIZE"]["scale"] - 2.0) < 1e-12 and abs(out["WRITE_SIZE"]["scale"] - 1.0) < 1e-12
    k = out["kernels"]["lstm_fwd_gemm"]
    assert k["grid_threads"] == 262144 and k["dispatches_fetch_size"] == 16
    assert k["fetch_bytes_per_launch"] == round(2.0 * 1000.0 * 1024) and k["write_bytes_per_launch"] == 100 * 1024
    assert bench.measured_traffic("lstm_fwd_gemm", str(tmp_path / "t.json")) == 2000 * 1024 + 100 * 1024
    assert bench.measured_traffic("adam_step", str(tmp_path / "t.json")) is None


def test_traffic_taken_on_other_sources_is_not_used(tmp_path):
    t = {"source_digest": "0" * 64, "kernels": {"lstm_fwd_gemm": {"fetch_bytes_per_launch": 1,
                                                                   "write_bytes_per_launch": 2}}}
    p = tmp_path / "t.json"
    p.write_text(json.dumps(t))
    assert bench.measured_traffic("lstm_fwd_gemm", str(p)) is None
    t["source_digest"] = bench.source_digest()
    p.write_text(json.dumps(t))
    assert bench.measured_traffic("lstm_fwd_gemm", str(p)) == 3
    assert bench.measured_traffic("lstm_fwd_gemm", str(tmp_path / "missing.json")) is None
