"""The five synthetic LiDAR workloads: scan geometry, grid and model shape.

The paper measures on KITTI (Velodyne HDL-64E) and Ford scans (Sec. 4.1.1);
none of those datasets is used here.  These seeded scenes stand in for them:
a spinning multi-beam sensor over a ground plane with boxes and poles.
"""
from __future__ import annotations

from dataclasses import dataclass


@dataclass(frozen=True)
class ScanConfig:
    name: str
    beams: int
    elev_min_deg: float
    elev_max_deg: float
    azimuth_steps: int
    boxes: int
    cylinders: int
    extent_m: float          # object centres uniform in [-extent, extent]^2
    max_range_m: float
    sigma_m: float           # Gaussian range noise
    bit_depth: int           # B: the finest grid has 2^B cells per axis
    range_m: float           # R: the grid spans [-R, R) on each axis
    min_bit_depth: int       # b0: the coarsest scale of the pyramid
    channels: int            # C
    layers: int              # L sparse 3x3x3 conv layers
    frames: int = 1
    frame_step_m: float = 0.0  # sensor translation per frame along +x
    box_side: tuple = (1.0, 5.0)
    box_height: tuple = (1.0, 3.0)
    cyl_radius: tuple = (0.1, 0.5)
    cyl_height: tuple = (2.0, 8.0)
    ground_z: float = -1.7
    scene_seed: int = 0
    noise_seed: int = 1
    weight_seed: int = 2


CONFIGS = [
    ScanConfig("tiny16_b10", beams=16, elev_min_deg=-15.0, elev_max_deg=15.0,
               azimuth_steps=512, boxes=20, cylinders=0, extent_m=30.0,
               max_range_m=50.0, sigma_m=0.02, bit_depth=10, range_m=51.2,
               min_bit_depth=4, channels=16, layers=2),
    ScanConfig("hdl64_b12", beams=64, elev_min_deg=-24.8, elev_max_deg=2.0,
               azimuth_steps=2048, boxes=150, cylinders=60, extent_m=80.0,
               max_range_m=80.0, sigma_m=0.02, bit_depth=12, range_m=131.0,
               min_bit_depth=4, channels=32, layers=2),
    ScanConfig("hdl64_b14", beams=64, elev_min_deg=-24.8, elev_max_deg=2.0,
               azimuth_steps=2048, boxes=150, cylinders=60, extent_m=80.0,
               max_range_m=80.0, sigma_m=0.02, bit_depth=14, range_m=131.0,
               min_bit_depth=4, channels=32, layers=3),
    ScanConfig("dense128_b16", beams=128, elev_min_deg=-22.5, elev_max_deg=22.5,
               azimuth_steps=2048, boxes=300, cylinders=150, extent_m=100.0,
               max_range_m=100.0, sigma_m=0.01, bit_depth=16, range_m=131.0,
               min_bit_depth=4, channels=32, layers=3),
    ScanConfig("stream10_hdl64_b14", beams=64, elev_min_deg=-24.8, elev_max_deg=2.0,
               azimuth_steps=2048, boxes=150, cylinders=60, extent_m=80.0,
               max_range_m=80.0, sigma_m=0.02, bit_depth=14, range_m=131.0,
               min_bit_depth=4, channels=32, layers=3, frames=10, frame_step_m=1.0),
]

BY_NAME = {c.name: c for c in CONFIGS}
HEADLINE = CONFIGS[2]
