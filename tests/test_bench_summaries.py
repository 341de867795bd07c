"""The rocprofv3 summarizers of bench.py on small synthetic CSVs (CPU only):
kernels named with their template arguments, the per-call HBM traffic of the
32K-layer decode picked by its variant (another decode variant with the same
grid must not leak in), the copy-window grouping, and the stored traffic
honoured only while the decode sources still hash to the recorded value."""
import csv

import pytest

import bench

DECODE_32K = "void lynx::(anonymous namespace)::anchor_decode_kernel<4, 0, 4>(lynx::DecodeArgs)"
DECODE_70B = "void lynx::(anonymous namespace)::anchor_decode_kernel<8, 0, 64>(lynx::DecodeArgs)"
COMBINE = ("void lynx::(anonymous namespace)::attn_combine_kernel<8>(lynx::(anonymous namespace)::AttnArgs, "
           "unsigned short*, float*)")
COPY = "__amd_rocclr_copyBuffer"


def write_csv(path, rows):
    path.parent.mkdir(parents=True, exist_ok=True)
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=list(rows[0]))
        w.writeheader()
        w.writerows(rows)


def test_variant_keeps_template_arguments():
    assert bench._variant(DECODE_32K) == "anchor_decode_kernel<4, 0, 4>"
    assert bench._variant(DECODE_70B) == "anchor_decode_kernel<8, 0, 64>"
    assert bench._variant(COMBINE) == "attn_combine_kernel<8>"
    assert bench._variant(COPY) == "copyBuffer"
    # the short name still groups every instance
    assert bench._short(DECODE_70B) == "anchor_decode_kernel"


def pmc_rows(counter, per_dispatch):
    """Counter rows: (dispatch id, kernel, grid, KiB) -> one row each."""
    return [{"Dispatch_Id": str(i), "Kernel_Name": k, "Grid_Size": str(g), "Queue_Id": "1",
             "Counter_Name": counter, "Counter_Value": str(v)} for i, k, g, v in per_dispatch]


def test_pmc_traffic_takes_only_the_32k_decode_calls(tmp_path, capsys):
    known_kib = bench.COPY_CALIBRATION_BYTES / 1024
    grid = bench.DECODE_32K_GRID
    # FETCH_SIZE counts half the bytes read, WRITE_SIZE all of them (as on the part)
    fetch = [(1, COPY, 4096, known_kib / 2),
             (2, DECODE_32K, grid, 1000.0), (3, DECODE_32K, grid, 1200.0),
             (4, DECODE_70B, grid, 300000.0),  # same grid, other variant
             (5, DECODE_32K, grid, 1100.0)]
    write = [(1, COPY, 4096, known_kib),
             (2, DECODE_32K, grid, 10.0), (3, DECODE_32K, grid, 30.0),
             (4, DECODE_70B, grid, 2000.0),
             (5, DECODE_32K, grid, 20.0)]
    write_csv(tmp_path / "f" / "run_counter_collection.csv", pmc_rows("FETCH_SIZE", fetch))
    write_csv(tmp_path / "w" / "run_counter_collection.csv", pmc_rows("WRITE_SIZE", write))
    bench.summarize_pmc(str(tmp_path / "f"), str(tmp_path / "w"))
    out = capsys.readouterr().out
    assert "32K-layer anchor-decode calls measured: 3" in out
    want = ((1000 + 1200 + 1100) * 2 + (10 + 30 + 20)) * 1024 / 3
    got = int(out.split("traffic_bytes_per_call:")[1].split()[0])
    assert got == pytest.approx(want, rel=1e-6)


def trace_row(i, name, grid, start, end):
    return {"Dispatch_Id": str(i), "Kernel_Name": name, "Grid_Size_X": str(grid), "Grid_Size_Y": "1",
            "Grid_Size_Z": "1", "Queue_Id": "1", "Start_Timestamp": str(start), "End_Timestamp": str(end)}


def test_copy_windows_group_by_the_kernels_inside(tmp_path, capsys):
    ms = 1_000_000  # ns
    kernels = [trace_row(1, DECODE_32K, 131072, 1 * ms, 1 * ms + 15_000),
               trace_row(2, DECODE_32K, 131072, 2 * ms, 2 * ms + 15_000),
               trace_row(3, DECODE_70B, 131072, 30 * ms, 30 * ms + 100_000)]
    copies = [{"Kind": "MEMORY_COPY", "Direction": "MEMORY_COPY_HOST_TO_DEVICE", "Start_Timestamp": str(s),
               "End_Timestamp": str(e)}
              for s, e in ((0, 5 * ms), (10 * ms, 15 * ms), (29 * ms, 34 * ms),
                           (40 * ms, 40 * ms + 500_000))]  # the last is under 1 ms: left out
    write_csv(tmp_path / "t" / "run_kernel_trace.csv", kernels)
    write_csv(tmp_path / "t" / "run_memory_copy_trace.csv", copies)
    bench.summarize_copies(str(tmp_path / "t"))
    lines = [l for l in capsys.readouterr().out.splitlines() if l.startswith("| ") and "---" not in l][1:]
    assert len(lines) == 3
    assert lines[0].startswith("| 1 | 5000.0 | anchor_decode_kernel<4, 0, 4> [131072] x2: 30.0")
    assert lines[1].startswith("| 1 | 5000.0 | none")
    assert lines[2].startswith("| 1 | 5000.0 | anchor_decode_kernel<8, 0, 64> [131072] x1: 100.0")


def test_stored_traffic_needs_the_recorded_sources(tmp_path, monkeypatch):
    summary = tmp_path / "traffic.md"
    summary.write_text(f"kernel_sources_sha256: {bench.decode_sources_hash()}\ntraffic_bytes_per_call: 123\n")
    monkeypatch.setattr(bench, "TRAFFIC_SUMMARY", summary)
    assert bench.stored_traffic() == 123
    summary.write_text("kernel_sources_sha256: " + "0" * 64 + "\ntraffic_bytes_per_call: 123\n")
    assert bench.stored_traffic() is None
