"""Host-side helpers of bench.py (no GPU): the oracle process pool returns results in
order and is closed and joined (not terminated), and the baseline states both the
processes it used and the host's cores."""
import os

import bench


def _square(x):
    return x * x


def test_pool_map_returns_results_in_order():
    assert bench.pool_map(_square, list(range(20)), 3) == [x * x for x in range(20)]


def test_oracle_pool_size_and_core_fields():
    host = len(os.sched_getaffinity(0))
    p = bench.oracle_procs()
    assert 1 <= p <= min(host, bench.BOX_CPU_SHARE)
    assert bench.oracle_procs(2) <= 2
    f = bench.cores_fields(p)
    assert f["cores"] == p and f["host_cores"] == host and str(host) in f["cores_note"]
