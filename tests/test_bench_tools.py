"""Host-side tools of bench.py: the kernel-only summary of a sweep trace (CPU only, synthetic
trace files)."""
import csv
import io
import contextlib

import pytest

import bench


def _write_trace(path, steps, drop_last=False):
    cases = [(n, m) for n in bench.SWEEP_N for m in bench.SWEEP_M]
    per_case = 3 + steps + 1
    rows, t = [], 1000
    for ci in range(len(cases)):
        for s in range(per_case):
            if drop_last and ci == len(cases) - 1 and s == per_case - 1:
                continue
            launches = [("void lapattn::pool_kernel<0>(float const*)", 1000),
                        ("void at::native::vectorized_elementwise_kernel<4>(int)", 7000),   # not the library's
                        ("void lapattn::key_summary_kernel<32>(float const*)", 2000),
                        ("void lapattn::ns_solve_kernel<64, 32>(float const*)", (ci + 1) * 10000 + s * 1000),
                        ("_ZN7lapattn13bwd_ns_kernelILi64ELi32EEEvPKf", 3000),
                        ("void lapattn::kll_bwd_kernel<32, 64>(float const*)", 500)]
            for name, dur in launches:
                rows.append({"Kind": "KERNEL_DISPATCH", "Kernel_Name": name, "Start_Timestamp": t,
                             "End_Timestamp": t + dur})
                t += dur + 100
    with open(path / "run_kernel_trace.csv", "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Kind", "Kernel_Name", "Start_Timestamp", "End_Timestamp"])
        w.writeheader()
        # the summary orders launches by start time, not by file order
        w.writerows(reversed(rows))


def test_sweep_trace_summary_takes_the_timed_steps(tmp_path):
    steps = 3
    _write_trace(tmp_path, steps)
    out = io.StringIO()
    with contextlib.redirect_stdout(out):
        bench.summarize_sweep_trace(str(tmp_path), steps)
    lines = [ln for ln in out.getvalue().splitlines() if ln.startswith("| ") and ln[2].isdigit()]
    cases = [(n, m) for n in bench.SWEEP_N for m in bench.SWEEP_M]
    assert len(lines) == len(cases)
    header = out.getvalue().splitlines()[0]
    cols = [c.strip() for c in header.strip("|").split("|")]
    assert cols == ["n", "m", "lap_fwd", "lap_bwd", "ns_fwd", "ns_bwd", "ns_bwd_kll"]
    for ci, (ln, (n, m)) in enumerate(zip(lines, cases)):
        cells = [c.strip() for c in ln.strip("|").split("|")]
        assert (int(cells[0]), int(cells[1])) == (n, m)
        got = dict(zip(cols[2:], map(float, cells[2:])))
        # the timed steps are 3, 4, 5 of each case (after 3 warmup steps, before the comparison
        # step): their median solve is step 4's
        assert got["ns_fwd"] == pytest.approx((ci + 1) * 10 + 4.0)
        assert got["lap_fwd"] == pytest.approx(2.0)
        assert got["lap_bwd"] == 0.0
        assert got["ns_bwd"] == pytest.approx(3.0)
        assert got["ns_bwd_kll"] == pytest.approx(3.5)


def test_sweep_trace_summary_rejects_a_wrong_step_count(tmp_path):
    _write_trace(tmp_path, 3, drop_last=True)
    with pytest.raises(SystemExit):
        bench.summarize_sweep_trace(str(tmp_path), 3)
