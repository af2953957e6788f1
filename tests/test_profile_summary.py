"""Host logic of the rocprofv3 summaries that the committed profiles and
bench.py's measured-traffic fields rest on: per-kernel averages of counters
(with the full-size-dispatch filter), the counted window after a marker
kernel, and the trace grouping.  Synthetic CSVs in rocprofv3's column layout."""
import csv

from paper_2504_18583_amd import profile_summary as ps

COLS = ["Correlation_Id", "Dispatch_Id", "Grid_Size", "Workgroup_Size", "Kernel_Name", "Counter_Name",
        "Counter_Value"]


def _write(path, rows):
    with open(path, "w", newline="") as fh:
        w = csv.writer(fh)
        w.writerow(COLS)
        w.writerows(rows)


def _pmc_rows():
    rows = []
    # k_gemm_rows<2> with 224 workgroups: full passes (MOPS 132) and shorter ones (MOPS 66)
    for d, mops, fetch in [(1, 66, 10.0), (2, 132, 20.0), (3, 132, 22.0), (4, 66, 12.0), (5, 132, 24.0)]:
        rows.append([d, d, 224 * 256, 256, "k_gemm_rows<2>(args)", "MOPS", mops])
        rows.append([d, d, 224 * 256, 256, "k_gemm_rows<2>(args)", "FETCH_SIZE", fetch])
    # the same kernel on another grid, and another kernel: never mixed in
    rows.append([6, 6, 448 * 256, 256, "k_gemm_rows<2>(args)", "FETCH_SIZE", 1000.0])
    rows.append([7, 7, 224 * 256, 256, "k_gemm_rows<1>(args)", "FETCH_SIZE", 2000.0])
    return rows


def test_pmc_mean_over_kernel_and_grid(tmp_path):
    p = tmp_path / "c.csv"
    _write(p, _pmc_rows())
    out = ps.pmc(str(p), "k_gemm_rows<2>", 224, 0)
    assert "FETCH_SIZE: dispatches 5, mean 17.6, min 10.0, max 24.0" in out


def test_pmc_skip_drops_first_dispatches(tmp_path):
    p = tmp_path / "c.csv"
    _write(p, _pmc_rows())
    out = ps.pmc(str(p), "k_gemm_rows<2>", 224, 2)
    assert "FETCH_SIZE: dispatches 3, mean 19.3, min 12.0, max 24.0" in out


def test_pmc_at_max_keeps_full_size_dispatches(tmp_path):
    p = tmp_path / "c.csv"
    _write(p, _pmc_rows())
    out = ps.pmc(str(p), "k_gemm_rows<2>", 224, 0, "MOPS")
    assert "FETCH_SIZE: dispatches 3, mean 22.0, min 20.0, max 24.0" in out
    assert "MOPS: dispatches 3, mean 132.0, min 132.0, max 132.0" in out


def test_window_sums_after_last_marker(tmp_path):
    p = tmp_path / "w.csv"
    rows = [
        [1, 1, 64, 64, "k_step_marker(int*)", "FETCH_SIZE", 1.0],
        [2, 2, 256, 256, "k_a(x)", "FETCH_SIZE", 100.0],     # before the last marker: not counted
        [3, 3, 64, 64, "k_step_marker(int*)", "FETCH_SIZE", 1.0],
        [4, 4, 256, 256, "k_a(x)", "FETCH_SIZE", 10.0],
        [5, 5, 256, 256, "k_b(x)", "FETCH_SIZE", 5.0],
        [6, 6, 256, 256, "k_a(x)", "FETCH_SIZE", 7.5],
    ]
    _write(p, rows)
    out = ps.window(str(p), "k_step_marker")
    assert "dispatches after the last 'k_step_marker': 3" in out
    assert "FETCH_SIZE: total 22.5" in out
