"""Host-side parts of bench.py: the confidence interval of the median call
time and the naming of profiled kernels (CPU only)."""
import math

import numpy as np
import pytest

import bench


def _coverage(n, j):
    # P(x_(j) <= median <= x_(n-j+1)) for a continuous distribution
    return 1.0 - 2.0 * sum(math.comb(n, k) for k in range(j)) / 2.0 ** n


@pytest.mark.parametrize("n", [6, 10, 11, 20, 30])
def test_median_interval_has_at_least_95_percent_coverage(n):
    xs = list(np.arange(n, dtype=float))
    med, (lo, hi) = bench.median_ci95(xs)
    assert med == float(np.median(xs))
    j = int(lo) + 1  # rank of the lower bound (xs holds 0 .. n-1)
    assert hi == n - j
    assert _coverage(n, j) >= 0.95
    # one rank further in would fall below 95%
    assert _coverage(n, j + 1) < 0.95


def test_median_interval_small_samples_span_the_range():
    med, (lo, hi) = bench.median_ci95([3.0, 1.0, 2.0])
    assert med == 2.0 and (lo, hi) == (1.0, 3.0)


def test_median_interval_empirical_coverage():
    rng = np.random.Generator(np.random.PCG64(5))
    hits = 0
    for _ in range(2000):
        xs = rng.standard_normal(20)
        _, (lo, hi) = bench.median_ci95(xs)
        hits += lo <= 0.0 <= hi
    assert hits / 2000 >= 0.94


@pytest.mark.parametrize("name,label", [
    ("void adst::(anonymous namespace)::adj_allencahn3d7<double, false, true>(double const*, "
     "double const*, double*, int)", "adj_allencahn3d7"),
    ("void adst::(anonymous namespace)::adj_allencahn3d7<double, true, false>(double const*)",
     "adj_allencahn3d7<dp>"),
    ("void adst::(anonymous namespace)::fwd_allencahn3d7_n<double, 3, 4, 64, true, false>(x)",
     "fwd_allencahn3d7_n<3>"),
    ("void adst::(anonymous namespace)::fwd_allencahn3d7_n<double, 2, 4, 32, false, true>(x)",
     "fwd_allencahn3d7_n<2,store>"),
    ("void adst::(anonymous namespace)::jacobi_march<double, 6, true, true>(double const*)",
     "jacobi_march<adj,6>"),
    ("void adst::(anonymous namespace)::jacobi_march<float, 4, false, true>(float const*)",
     "jacobi_march<fwd,4>"),
    ("void adst::(anonymous namespace)::adj_vardiff2d9<float, true, 4, false, true>(float)",
     "adj_vardiff2d9<dK>"),
    ("void adst::(anonymous namespace)::fwd_vardiff2d9_x2<float, 8, true, true>(float)",
     "fwd_vardiff2d9_x2<store>"),
    ("void adst::(anonymous namespace)::gs_wave<double, true, true>(double*)", "gs_wave<adj>"),
    ("void adst::(anonymous namespace)::seed_loss<double, 1>(double const*)", "seed_loss"),
    ("__amd_rocclr_copyBuffer", "hipMemcpyAsync copy"),
    ("void adst::(anonymous namespace)::ac_march<double, 3, false, 4, 64, 0, true, false>(adst::("
     "anonymous namespace)::AcMarchArgs<double>)", "ac_march<fwd,3,store>"),
    ("void adst::(anonymous namespace)::ac_march<double, 0, true, 4, 64, 1, false, true>(x)",
     "ac_march<adj>"),
    ("void adst::(anonymous namespace)::ac_march<double, 1, true, 4, 64, 1, false, true>(x)",
     "ac_march<fwd1+adj>"),
    ("void adst::(anonymous namespace)::ac_march<double, 1, false, 4, 64, 0, false, true>(x)",
     "ac_march<fwd,1>"),
])
def test_rocprof_names_map_to_library_labels(name, label):
    assert bench.rocprof_label(name) == label


def test_kernel_rows_from_rocpd_database(tmp_path):
    # rocprofv3 writes SQLite when no CSV format is asked for: the summary
    # aggregates its kernel dispatches per name
    import sqlite3
    d = tmp_path / "kt" / "host"
    d.mkdir(parents=True)
    con = sqlite3.connect(str(d / "run_results.db"))
    con.execute("CREATE TABLE kernels (name TEXT, duration INTEGER)")
    con.executemany("INSERT INTO kernels VALUES (?, ?)",
                    [("a", 10), ("a", 30), ("b", 60)])
    con.commit()
    con.close()
    rows = {r["Name"]: r for r in bench._kernel_rows(str(tmp_path / "kt"))}
    assert rows["a"]["Calls"] == 2 and rows["a"]["TotalDurationNs"] == 40
    assert rows["a"]["MinNs"] == 10 and rows["a"]["MaxNs"] == 30
    assert abs(rows["b"]["Percentage"] - 60.0) < 1e-12


def test_sweep_lists_known_workloads_and_schedules():
    from paper_2509_02197_amd.workloads import WORKLOADS
    for name, sched, budget in bench.SWEEP:
        assert name in WORKLOADS and sched in bench.SCHED_NAMES.values() and budget > 0
