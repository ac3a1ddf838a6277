"""The committed rocprofv3 summaries that bench.py reads (conv_last's HBM
traffic per launch and its kernel-trace average) belong to the current conv
kernel sources and to the headline workload, so a kernel change without a new
profile shows up here instead of as a silent null in the bench line; every
summary under profiles/ states the rocprofv3 command that made it.  CPU only."""
import glob
import os

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADLINE = "hdl64_b14"


def test_conv_last_traffic_profile_matches_the_kernel_sources():
    traffic = bench.read_traffic(HEADLINE)
    assert traffic is not None, (f"{bench.TRAFFIC_FILE} was taken on other kernel sources "
                                 f"(current sha256 prefix {bench.model_source_hash()})")
    # between the algorithmic bytes of one launch and a few times them
    assert 1e6 < traffic < 1e9


def test_conv_last_trace_profile_matches_the_kernel_sources():
    trace = bench.read_trace(HEADLINE)
    assert trace is not None, (f"{bench.TRACE_FILE} was taken on other kernel sources "
                               f"(current sha256 prefix {bench.model_source_hash()})")
    avg_us, dispatches = trace
    assert avg_us > 0 and dispatches > 0


def test_every_profile_states_its_command():
    files = sorted(glob.glob(os.path.join(ROOT, "profiles", "*.md")) +
                   glob.glob(os.path.join(ROOT, "profiles", "*.txt")))
    assert files
    for f in files:
        text = open(f).read()
        assert "rocprofv3" in text, f"{os.path.basename(f)} does not give the rocprofv3 command"
        assert len(text) < 64 * 1024, f"{os.path.basename(f)} is not a short summary"
