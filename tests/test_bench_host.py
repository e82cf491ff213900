"""bench.py's host-side logic without a GPU: the refusal of more than one GPU and the
summaries it prints from rocprofv3 CSV folders (built here from known values)."""
import csv
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def write_csv(path, rows):
    os.makedirs(os.path.dirname(path), exist_ok=True)
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=list(rows[0]))
        w.writeheader()
        w.writerows(rows)


def test_more_than_one_gpu_exits_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=300)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and "--gpus must be 1" in r.stderr


def test_trace_summary_tables(tmp_path):
    name = "void samd::(anonymous namespace)::conv1d_kernel<3, 4>(unsigned int const*, int*, int)"
    write_csv(str(tmp_path / "h" / "1_kernel_stats.csv"), [
        {"Name": name, "Calls": "30", "AverageNs": "4000", "MinNs": "3000", "MaxNs": "9000", "Percentage": "60.5"},
        {"Name": "void rare_kernel()", "Calls": "2", "AverageNs": "1", "MinNs": "1", "MaxNs": "1",
         "Percentage": "0.1"}])
    # 30 dispatches of one shape: 10 of 5 us, then 20 of 3 us
    trace = [{"Kernel_Name": name, "Workgroup_Size_X": "256", "Workgroup_Size_Y": "1", "Workgroup_Size_Z": "1",
              "Grid_Size_X": "1024", "Grid_Size_Y": "2", "Grid_Size_Z": "1", "VGPR_Count": "40", "SGPR_Count": "96",
              "Start_Timestamp": str(1000 * i), "End_Timestamp": str(1000 * i + (5000 if i < 10 else 3000))}
             for i in range(30)]
    write_csv(str(tmp_path / "h" / "1_kernel_trace.csv"), trace)
    out = bench.trace_summary(str(tmp_path)).splitlines()
    assert "| conv1d_kernel<3, 4> | 30 | 4.00 | 3.00 | 9.00 | 60.50 |" in out
    assert not any("rare_kernel" in line for line in out)
    # per shape: 2048 threads, mean (10 x 5 + 20 x 3) / 30 us, min 3, the last 20 at 3
    assert "| conv1d_kernel<3, 4> | 256 | 2048 | 40 | 96 | 30 | 3.67 | 3.00 | 3.00 |" in out


def test_int8_summary_rows(tmp_path):
    """Two counter passes over --int8-counters on VGG-B layer 1: every candidate launched
    twice, the table keeps the second dispatch of each, names it by its launch, and prices
    its duration against the layer's MACs."""
    import paper_1809_10572_amd as samd
    shape = bench.int8_layer("vggb1")
    cands = samd.conv2d_int8_candidates(shape, samd.Fmt(4, False), samd.Fmt(4, True))
    assert cands and cands[0].halo == 3
    macs = shape.N * shape.M * shape.H * shape.W * shape.C * 9
    for folder, counters in (("a", {"SQ_WAVES": 800.0, "SQ_WAVE_CYCLES": 1000.0, "SQ_WAIT_INST_ANY": 250.0}),
                             ("b", {"TCP_TCC_READ_REQ_sum": 1200.0, "TCP_TCC_WRITE_REQ_sum": 2.0e5,
                                    "TCC_HIT_sum": 3.0, "TCC_MISS_sum": 1.0})):
        rows = []
        for k in range(2 * len(cands)):
            dur = 10000 if k % 2 == 0 else 7000   # ns: the second dispatch of each is 7 us
            for cname, v in counters.items():
                rows.append({"Dispatch_Id": str(k + 1), "Kernel_Name": "void samd::(anonymous namespace)::"
                             "conv2d_i8_packed_kernel<false>(unsigned char const*)", "Counter_Name": cname,
                             "Counter_Value": str(v), "Start_Timestamp": "0", "End_Timestamp": str(dur)})
        write_csv(str(tmp_path / folder / "p_counter_collection.csv"), rows)
    table = bench.int8_summary([str(tmp_path / "a"), str(tmp_path / "b")], "vggb1").splitlines()
    body = [line for line in table[2:] if line.startswith("|")]
    assert len(body) == len(cands)
    first = [c.strip() for c in body[0].strip("|").split("|")]
    assert first[0] == bench.int8_launch_name(cands[0]) and first[1] == "conv2d_i8_packed_kernel<false>"
    assert first[2] == "7.00"
    assert first[3] == f"{100 * macs / 7e-6 / bench.PEAK_I8_MACS:.1f}"
    assert first[5] == "25"                     # wait cycles / wave cycles
    assert first[9] == "75.0"                   # L2 hit %
    assert first[12] == "2e+05"                 # L1 -> L2 write requests


@pytest.mark.parametrize("layer", sorted(bench.INT8_LAYERS))
def test_int8_layers_resolve(layer):
    import samd_workloads as wl
    shape = bench.int8_layer(layer)
    assert shape == wl.MID or shape in wl.VGGB_LAYERS or shape in wl.ALEXNET_LAYERS
