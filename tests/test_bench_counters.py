"""bench.py's ingest of two rocprofv3 counter runs (FETCH_SIZE, WRITE_SIZE),
on synthetic counter CSVs: every op must be matched to its own kernel
(the pack's kernel is not the three-launch form's ``pack_rows``, nor is
that combine's ``unpack_rows``, although one name contains the other), and the counters are scaled by the 1 GiB calibration
copy."""

import csv
import json

import bench

NS = "void purlin::(anonymous namespace)::"
KERNELS = {
    "exec_reduce": NS + "exec_reduce<8, true, 2, true, false>(purlin::ExecArgs)",
    "exec_copy": NS + "exec_copy<4, false, true>(purlin::ExecArgs)",
    "pack_onepass": NS + "pack_onepass<true, true>(int, int, int, int, int, unsigned int, char const*)",
    "pack_rows": NS + "pack_rows<1, false, true>(int, int, int, int, int, char const*)",
    "unpack_rows": NS + "unpack_rows<1, true, true, true>(int, int, int, int, long)",
    "pack_scan": NS + "pack_scan(int, int, int, int*)",
    "copy": "void at::native::copy_kernel<short>(int)",
}


def _write(d, counter, values):
    d.mkdir()
    with open(d / "run_counter_collection.csv", "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Kernel_Name", "Counter_Name", "Counter_Value"])
        w.writeheader()
        for k, vs in values.items():
            for v in vs:
                w.writerow({"Kernel_Name": KERNELS[k], "Counter_Name": counter, "Counter_Value": v})


def test_each_op_gets_its_own_kernel_and_the_calibrated_scale(tmp_path):
    gib_kib = (1 << 30) / 1024
    # FETCH_SIZE reads half of the true bytes, WRITE_SIZE all of them
    fetch = {"copy": [1.0, gib_kib / 2], "exec_reduce": [1000.0, 1000.0], "exec_copy": [200.0],
             "pack_onepass": [300.0, 500.0], "pack_rows": [77.0], "unpack_rows": [9000.0], "pack_scan": [5.0]}
    write = {"copy": [3.0, gib_kib], "exec_reduce": [100.0], "exec_copy": [800.0],
             "pack_onepass": [4000.0], "pack_rows": [66.0], "unpack_rows": [700.0], "pack_scan": [1.0]}
    _write(tmp_path / "f", "FETCH_SIZE", fetch)
    _write(tmp_path / "w", "WRITE_SIZE", write)
    out = tmp_path / "traffic.json"
    assert bench.ingest_counters(str(tmp_path / "f"), str(tmp_path / "w"), path=str(out)) == 0
    t = json.loads(out.read_text())
    assert abs(t["calibration"]["fetch_scale"] - 2.0) < 1e-12
    assert abs(t["calibration"]["write_scale"] - 1.0) < 1e-12
    ops = t["ops"]
    assert set(ops) == set(bench.KERNEL_OF_OP)
    assert "::pack_onepass<" in ops["moe_pack"]["kernel"] and "unpack" not in ops["moe_pack"]["kernel"]
    assert "unpack_rows<" in ops["moe_combine"]["kernel"]
    assert "exec_reduce<" in ops["reduce_scatter"]["kernel"] and "exec_copy<" in ops["allgather"]["kernel"]
    # means over dispatches, scaled: pack fetch (300 + 500) / 2 KiB x 2, write 4000 KiB x 1
    assert ops["moe_pack"]["hbm_read_bytes"] == round(400.0 * 1024 * 2)
    assert ops["moe_pack"]["hbm_write_bytes"] == round(4000.0 * 1024)
    assert ops["moe_pack"]["hbm_bytes_per_launch"] == round(400.0 * 1024 * 2) + round(4000.0 * 1024)
    assert t["kernel_source_hash"] == bench.kernel_source_hash()
