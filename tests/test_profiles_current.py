"""The committed rocprofv3 summaries under profiles/ still describe the
committed kernels: every counter, traffic and kernel-trace summary that the
bench line reads carries the hash of its kernel's sources, and the bench
reports a figure only while that hash matches. A kernel changed without
re-profiling fails here (host only, no GPU)."""
import os

import pytest

import bench

PROFILES = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "profiles")


@pytest.mark.parametrize("op", ["conv_fwd", "conv_wgrad"])
@pytest.mark.parametrize("workload", ["c2", "c3", "c4", "c5"])
def test_counter_summary_current(op, workload):
    assert os.path.exists(os.path.join(PROFILES, f"{op}_{workload}_counters.txt"))
    ctr = bench.measured_counters(op, workload)
    assert ctr is not None, f"profiles/{op}_{workload}_counters.txt is stale: re-profile"
    assert 0.0 < ctr["mfma_busy_frac"] < 1.0
    assert 1000.0 < ctr["clock_mhz"] < 2500.0


@pytest.mark.parametrize("op", ["conv_fwd", "conv_wgrad"])
def test_traffic_summary_current(op):
    t = bench.measured_traffic(op, "c3")
    assert t is not None, f"profiles/{op}_c3_traffic.txt is stale: re-profile"
    # at least the algorithmic bytes of a launch (tile + output or dy), at most 2x
    assert 4.3e9 < t < 8.7e9


def test_halo_trace_current():
    hk = bench.measured_halo_kernel("c3")
    assert hk is not None, "profiles/halo_c3_kernel_trace.txt is stale: re-profile"
    # a 64 MiB pair can take no less than 64 MiB / 8 TB/s = 8.4 us
    assert 8.4 < hk["pack"] < 30.0 and 8.4 < hk["unpack"] < 30.0
