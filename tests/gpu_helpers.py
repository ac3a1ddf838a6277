"""Shared drivers for the GPU tests: run the HIP path through the C ABI on the
seeded inputs the tests also hand to the oracle, and compare levels with it.
Every GPU step prints what it runs first."""
from __future__ import annotations

import sys

import numpy as np

import paper_2503_12382_amd as reno

LOGIT_TOL = 1e-3         # absolute, fp32 path vs fp64 oracle
BITS_REL_TOL = 1e-3      # total bits per frame, relative
# per-voxel bits = (lse - z_o)/ln 2: two logit-sized errors
BITS_ABS_TOL = 2 * LOGIT_TOL / np.log(2.0)


def say(*a):
    print("[gpu]", *a, flush=True)
    sys.stdout.flush()


def torch():
    import torch as t
    return t


def make_ctx(cfg_like, max_points, max_model_voxels=0):
    return reno.Context(max_points=max(int(max_points), 1), max_bit_depth=cfg_like["B"],
                        min_bit_depth=cfg_like["b0"], range_m=cfg_like["R"],
                        channels=cfg_like["C"], layers=cfg_like["L"],
                        max_model_voxels=max_model_voxels)


def cfg_dict(cfg):
    return {"B": cfg.bit_depth, "b0": cfg.min_bit_depth, "R": cfg.range_m, "C": cfg.channels,
            "L": cfg.layers}


def to_dev(a):
    t = torch()
    return t.from_numpy(np.ascontiguousarray(a)).to("cuda")


def encode(ctx, pts, B):
    say("build_pyramid", pts.shape, "B", B)
    ctx.build_pyramid(to_dev(pts), B)
    ctx.sync()


def levels_from_gpu(ctx, b0, B):
    out = {}
    for b in range(b0, B + 1):
        xyz, keys = ctx.coords(b)
        lv = {"xyz": xyz.cpu().numpy().astype(np.int64), "keys": keys.cpu().numpy().view(np.uint64),
              "parent": ctx.parent_rows(b).cpu().numpy()}
        if b < B:
            lv["codes"] = ctx.occupancy_codes(b).cpu().numpy()
        out[b] = lv
    return out


def assert_levels_equal(gpu, P, b0, B):
    for b in range(b0, B + 1):
        g = gpu[b]
        assert g["xyz"].shape[0] == P.num(b), (b, g["xyz"].shape[0], P.num(b))
        np.testing.assert_array_equal(g["keys"], P.keys(b), err_msg=f"keys b={b}")
        np.testing.assert_array_equal(g["xyz"], P.xyz(b), err_msg=f"xyz b={b}")
        np.testing.assert_array_equal(g["parent"], P.parent(b), err_msg=f"parent b={b}")
        if b < B:
            np.testing.assert_array_equal(g["codes"], P.codes(b), err_msg=f"codes b={b}")
