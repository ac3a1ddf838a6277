"""Seeded synthetic spinning-LiDAR scans (fp32 xyz in the sensor frame).

Scene: a ground plane, axis-aligned boxes standing on it and vertical poles
(cylinders).  The sensor casts ``beams x azimuth_steps`` rays; each ray keeps its
nearest positive hit within the maximum range, and the range gets Gaussian
noise.  Objects whose footprint comes within 2 m of any sensor position are
redrawn, so the sensor never sits inside an object.

Randomness: scene stream ``scene_seed``, range noise stream ``noise_seed``
(draw index = ray index, drawn for every ray so that indices never shift).
"""
from __future__ import annotations

import numpy as np

from . import rng
from .configs import ScanConfig

_SCENE_STREAM = 11
_NOISE_STREAM = 12


def _scene(cfg: ScanConfig):
    """Boxes [nb][6] = (cx, cy, sx, sy, h, 0) and cylinders [nc][4] = (cx, cy, r, h)."""
    path_x = np.array([f * cfg.frame_step_m for f in range(cfg.frames)])
    draw = [0]

    def u(n):
        out = rng.uniform(cfg.scene_seed, _SCENE_STREAM, draw[0], n)
        draw[0] += n
        return out

    def clear_of_path(cx, cy, half):
        # footprint (centre +/- half on each axis) at least 2 m from the path
        dx = np.maximum(np.abs(cx - np.clip(cx, path_x.min(), path_x.max())) - half, 0.0)
        dy = np.maximum(np.abs(cy) - half, 0.0)
        return np.hypot(dx, dy) >= 2.0

    boxes = []
    while len(boxes) < cfg.boxes:
        a = u(5)
        cx = (2.0 * a[0] - 1.0) * cfg.extent_m
        cy = (2.0 * a[1] - 1.0) * cfg.extent_m
        sx = cfg.box_side[0] + a[2] * (cfg.box_side[1] - cfg.box_side[0])
        sy = cfg.box_side[0] + a[3] * (cfg.box_side[1] - cfg.box_side[0])
        h = cfg.box_height[0] + a[4] * (cfg.box_height[1] - cfg.box_height[0])
        if clear_of_path(cx, cy, max(sx, sy) / 2.0):
            boxes.append((cx, cy, sx, sy, h, 0.0))
    cyls = []
    while len(cyls) < cfg.cylinders:
        a = u(4)
        cx = (2.0 * a[0] - 1.0) * cfg.extent_m
        cy = (2.0 * a[1] - 1.0) * cfg.extent_m
        r = cfg.cyl_radius[0] + a[2] * (cfg.cyl_radius[1] - cfg.cyl_radius[0])
        h = cfg.cyl_height[0] + a[3] * (cfg.cyl_height[1] - cfg.cyl_height[0])
        if clear_of_path(cx, cy, r):
            cyls.append((cx, cy, r, h))
    return (np.array(boxes, dtype=np.float64).reshape(-1, 6),
            np.array(cyls, dtype=np.float64).reshape(-1, 4))


def _ray_dirs(cfg: ScanConfig) -> np.ndarray:
    el = np.deg2rad(np.linspace(cfg.elev_min_deg, cfg.elev_max_deg, cfg.beams))
    az = 2.0 * np.pi * np.arange(cfg.azimuth_steps) / cfg.azimuth_steps
    el, az = np.meshgrid(el, az, indexing="ij")          # ray index = beam * steps + az
    d = np.stack([np.cos(el) * np.cos(az), np.cos(el) * np.sin(az), np.sin(el)], axis=-1)
    return d.reshape(-1, 3)


def _cast(origin, d, boxes, cyls, cfg: ScanConfig, chunk=8192):
    n = d.shape[0]
    t_best = np.full(n, np.inf)
    gz = cfg.ground_z
    with np.errstate(divide="ignore", invalid="ignore"):
        tg = np.where(d[:, 2] < 0.0, (gz - origin[2]) / d[:, 2], np.inf)
    t_best = np.minimum(t_best, np.where(tg > 0.0, tg, np.inf))
    for s in range(0, n, chunk):
        dd = d[s:s + chunk]
        best = t_best[s:s + chunk]
        if boxes.shape[0]:
            lo = (boxes[:, 0] - boxes[:, 2] / 2, boxes[:, 1] - boxes[:, 3] / 2,
                  np.full(boxes.shape[0], gz))
            hi = (boxes[:, 0] + boxes[:, 2] / 2, boxes[:, 1] + boxes[:, 3] / 2,
                  gz + boxes[:, 4])
            tmin = np.full((dd.shape[0], boxes.shape[0]), -np.inf)
            tmax = np.full((dd.shape[0], boxes.shape[0]), np.inf)
            with np.errstate(divide="ignore", invalid="ignore"):
                for ax in range(3):
                    inv = (1.0 / dd[:, ax])[:, None]                       # [r][1]
                    t1 = (lo[ax] - origin[ax])[None] * inv                 # [r][nb]
                    t2 = (hi[ax] - origin[ax])[None] * inv
                    tmin = np.fmax(tmin, np.fmin(t1, t2))
                    tmax = np.fmin(tmax, np.fmax(t1, t2))
            hit = (tmin <= tmax) & (tmin > 0.0)
            best = np.minimum(best, np.where(hit, tmin, np.inf).min(axis=1))
        if cyls.shape[0]:
            ox = origin[0] - cyls[:, 0]
            oy = origin[1] - cyls[:, 1]
            a = dd[:, 0:1] ** 2 + dd[:, 1:2] ** 2                          # [r][1]
            b = 2.0 * (dd[:, 0:1] * ox[None] + dd[:, 1:2] * oy[None])     # [r][nc]
            c = (ox ** 2 + oy ** 2 - cyls[:, 2] ** 2)[None]
            disc = b * b - 4.0 * a * c
            with np.errstate(divide="ignore", invalid="ignore"):
                t = (-b - np.sqrt(np.maximum(disc, 0.0))) / (2.0 * a)
            z = origin[2] + t * dd[:, 2:3]
            hit = (disc >= 0.0) & (t > 0.0) & (z >= gz) & (z <= gz + cyls[:, 3][None])
            best = np.minimum(best, np.where(hit, t, np.inf).min(axis=1))
        t_best[s:s + chunk] = best
    return t_best


def gen_scan(cfg: ScanConfig, frame: int = 0) -> np.ndarray:
    """fp32 points [M][3] of frame ``frame`` (sensor at (frame*step, 0, 0)),
    expressed relative to the sensor."""
    boxes, cyls = _scene(cfg)
    origin = np.array([frame * cfg.frame_step_m, 0.0, 0.0])
    d = _ray_dirs(cfg)
    t = _cast(origin, d, boxes, cyls, cfg)
    nrays = d.shape[0]
    noise = rng.normal(cfg.noise_seed, _NOISE_STREAM, frame * nrays, nrays) * cfg.sigma_m
    keep = np.isfinite(t) & (t <= cfg.max_range_m)
    r = t[keep] + noise[keep]
    return (d[keep] * r[:, None]).astype(np.float32)


def gen_frames(cfg: ScanConfig):
    return [gen_scan(cfg, f) for f in range(cfg.frames)]
