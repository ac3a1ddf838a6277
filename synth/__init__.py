"""Seeded synthetic inputs (LiDAR scans and model weights) shared by the oracle
tests, the GPU parity tests and the benchmark.  Holds none of the codec's
arithmetic."""
from .configs import CONFIGS, BY_NAME, HEADLINE, ScanConfig
from .lidar import gen_scan, gen_frames
from .weights import gen_weights

__all__ = ["CONFIGS", "BY_NAME", "HEADLINE", "ScanConfig", "gen_scan", "gen_frames",
           "gen_weights"]
