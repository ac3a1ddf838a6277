"""GPU edge cases against the oracle: empty and degenerate frames, ragged
sizes around every tile boundary, grid-edge clamping, the extreme bit depths,
dense occupancy, other model shapes, and every error path the device latches."""
import numpy as np
import pytest
import torch  # noqa: F401  (slow first import on a fresh box: at collection)

import oracle
import paper_2503_12382_amd as reno
from gpu_helpers import (BITS_ABS_TOL, LOGIT_TOL, assert_levels_equal, encode, levels_from_gpu,
                         make_ctx, say, to_dev)
from synth import gen_weights

pytestmark = pytest.mark.gpu


def _cfg(B, b0, C=16, L=2, R=10.0):
    return {"B": B, "b0": b0, "R": R, "C": C, "L": L}


def _points_from_voxels(xyz, B, R):
    """fp32 points at the centres of the given integer cells."""
    step = 2.0 * R / (1 << B)
    return (-R + (np.asarray(xyz, np.float64) + 0.5) * step).astype(np.float32)


def _check_frame(pts, cfg, weights=None, max_model_voxels=0):
    B, b0 = cfg["B"], cfg["b0"]
    ctx = make_ctx(cfg, max(len(pts), 1), max_model_voxels)
    encode(ctx, pts, B)
    P = oracle.Pyramid.from_points(pts, B, b0, cfg["R"]) if len(pts) else None
    if P is not None:
        assert_levels_equal(levels_from_gpu(ctx, b0, B), P, b0, B)
    if weights is not None:
        ctx.set_weights(reno.weights_to_device(weights))
        lg = ctx.predict_probs(reno.RENO_ALL_SCALES, logits=True)
        bits, total = ctx.code_length(reno.RENO_ALL_SCALES)
        if P is not None:
            off = 0
            lg = lg.cpu().numpy()
            bits = bits.cpu().numpy()
            for b in range(b0 + 1, B):
                n = P.num(b)
                olg, _, obits = P.model(b, weights)
                assert np.abs(lg[off:off + n] - olg).max() <= LOGIT_TOL
                assert np.abs(bits[off:off + n] - obits).max() <= BITS_ABS_TOL
                np.testing.assert_array_equal(ctx.neighbor_map(b).cpu().numpy(), P.neighbors(b))
                off += n
            T, _ = P.totals(weights)
            assert abs(total - T) <= 1e-3 * T
    ctx.close()


def test_empty_frame():
    cfg = _cfg(10, 4)
    ctx = make_ctx(cfg, 16)
    ctx.build_pyramid(torch.zeros((0, 3), dtype=torch.float32, device="cuda"), 10)
    for b in range(4, 11):
        assert ctx.num_voxels(b) == 0
    ctx.set_weights(reno.weights_to_device(gen_weights(16, 2, seed=3)))
    ctx.predict_probs(reno.RENO_ALL_SCALES)
    _, total = ctx.code_length(reno.RENO_ALL_SCALES, per_voxel=False)
    assert total == 32.0                       # raw count of an empty initial state
    ctx.close()


@pytest.mark.parametrize("copies", [1, 1000])
def test_single_voxel_and_all_duplicates(copies):
    cfg = _cfg(9, 3)
    pts = np.repeat(_points_from_voxels([[200, 17, 511]], 9, 10.0), copies, axis=0)
    say("single voxel x", copies)
    _check_frame(pts, cfg, gen_weights(16, 2, seed=4, bias_std=0.2))


@pytest.mark.parametrize("n", [2, 63, 64, 65, 1023, 1024, 1025, 2049, 4097])
def test_ragged_sizes(n):
    rs = np.random.default_rng(n)
    B = 8 + n % 5
    cfg = _cfg(B, 3)
    xyz = rs.integers(0, 1 << B, size=(n, 3))
    if n % 2:                                     # clustered: deep pyramids, dense neighbourhoods
        xyz = (xyz // 8) + (1 << (B - 2))
    pts = _points_from_voxels(xyz, B, 10.0)
    say("ragged", n, "B", B)
    _check_frame(pts, cfg, gen_weights(16, 2, seed=n, bias_std=0.1))


def test_grid_edges_and_clamping():
    R, B = 10.0, 8
    cfg = _cfg(B, 3, R=R)
    vals = np.array([-R, -R + 1e-6, -1e-7, 0.0, 1e-7, R - 1e-4, R, R + 5, -R - 5, 1e6, -1e6],
                    np.float32)
    g = np.stack(np.meshgrid(vals, vals, vals, indexing="ij"), -1).reshape(-1, 3)
    say("edges", g.shape)
    _check_frame(g, cfg, gen_weights(16, 2, seed=5, bias_std=0.1))


def test_no_model_scales():
    cfg = _cfg(5, 4)
    rs = np.random.default_rng(1)
    pts = _points_from_voxels(rs.integers(0, 32, size=(300, 3)), 5, 10.0)
    ctx = make_ctx(cfg, len(pts))
    encode(ctx, pts, 5)
    P = oracle.Pyramid.from_points(pts, 5, 4, 10.0)
    assert_levels_equal(levels_from_gpu(ctx, 4, 5), P, 4, 5)
    ctx.set_weights(reno.weights_to_device(gen_weights(16, 2, seed=3)))
    ctx.predict_probs(reno.RENO_ALL_SCALES)             # nothing to do
    _, total = ctx.code_length(reno.RENO_ALL_SCALES, per_voxel=False)
    assert total == 32 + P.num(4) * (3 * 4 + 8)
    ctx.close()


def test_root_base_scale():
    cfg = _cfg(6, 0)
    rs = np.random.default_rng(2)
    pts = _points_from_voxels(rs.integers(0, 64, size=(700, 3)), 6, 10.0)
    _check_frame(pts, cfg, gen_weights(16, 2, seed=6, bias_std=0.1))


def test_max_bit_depth_21():
    """63-bit keys, 8 sort passes, scales 4..21 (pyramid only: 17 model scales)."""
    B, b0, R = 21, 4, 131.0
    rs = np.random.default_rng(21)
    pts = rs.uniform(-R, R, size=(20000, 3)).astype(np.float32)
    pts[:5000] = pts[:5000] * 1e-3                       # a dense cluster near the centre
    cfg = _cfg(B, b0, R=R)
    ctx = make_ctx(cfg, len(pts))
    encode(ctx, pts, B)
    P = oracle.Pyramid.from_points(pts, B, b0, R)
    assert_levels_equal(levels_from_gpu(ctx, b0, B), P, b0, B)
    ctx.close()


def test_dense_cube_neighbourhoods():
    """Full occupancy of a 24^3 block: every voxel has 27 neighbours, heavy hash load."""
    B = 6
    g = np.stack(np.meshgrid(*[np.arange(20, 44)] * 3, indexing="ij"), -1).reshape(-1, 3)
    cfg = _cfg(B, 2, C=32, L=3)
    _check_frame(_points_from_voxels(g, B, 10.0), cfg,
                 gen_weights(32, 3, seed=7, bias_std=0.1))


@pytest.mark.parametrize("C,L", [(16, 1), (32, 1), (32, 4), (16, 8), (32, 8)])  # L = 8: the most layers a context takes
def test_other_model_shapes(C, L):
    rs = np.random.default_rng(C + L)
    B = 9
    xyz = rs.integers(0, 1 << B, size=(3000, 3)) // 4 + 100
    cfg = _cfg(B, 3, C=C, L=L)
    _check_frame(_points_from_voxels(xyz, B, 10.0), cfg,
                 gen_weights(C, L, seed=11, bias_std=0.1, head_scale=10.0))


# ---- errors latched on the device and call-order errors ----------------------------------

def test_nonfinite_point_reported():
    cfg = _cfg(8, 3)
    pts = np.zeros((100, 3), np.float32)
    pts[37, 1] = np.nan
    ctx = make_ctx(cfg, 100)
    ctx.build_pyramid(to_dev(pts), 8)
    with pytest.raises(reno.RenoError) as e:
        ctx.sync()
    assert e.value.status == reno.RENO_E_INPUT
    # the next frame starts clean
    ctx.build_pyramid(to_dev(np.zeros((4, 3), np.float32)), 8)
    ctx.sync()
    ctx.close()


def test_decoder_input_errors():
    cfg = _cfg(8, 3)
    ctx = make_ctx(cfg, 100)
    xyz = torch.tensor([[0, 0, 0], [1, 0, 0]], dtype=torch.int32, device="cuda")
    ctx.set_base(8, xyz, torch.tensor([1, 0], dtype=torch.uint8, device="cuda"))   # zero code
    with pytest.raises(reno.RenoError) as e:
        ctx.sync()
    assert e.value.status == reno.RENO_E_INPUT
    xyz_bad = torch.tensor([[1, 0, 0], [0, 0, 0]], dtype=torch.int32, device="cuda")  # unsorted
    ctx.set_base(8, xyz_bad, torch.tensor([1, 2], dtype=torch.uint8, device="cuda"))
    with pytest.raises(reno.RenoError):
        ctx.sync()
    xyz_out = torch.tensor([[0, 0, 9]], dtype=torch.int32, device="cuda")            # off grid
    ctx.set_base(8, xyz_out, torch.tensor([1], dtype=torch.uint8, device="cuda"))
    with pytest.raises(reno.RenoError):
        ctx.sync()
    # a zero code met during expansion
    ctx.set_base(8, xyz[:1].contiguous(), torch.tensor([3], dtype=torch.uint8, device="cuda"))
    ctx.expand(3)
    ctx.expand(4, torch.tensor([0, 1], dtype=torch.uint8, device="cuda"))
    with pytest.raises(reno.RenoError) as e:
        ctx.sync()
    assert e.value.status == reno.RENO_E_INPUT
    ctx.close()


def test_call_order_and_argument_errors():
    cfg = _cfg(8, 3)
    ctx = make_ctx(cfg, 100)
    with pytest.raises(reno.RenoError) as e:
        ctx.predict_probs(5)                             # no frame
    assert e.value.status == reno.RENO_E_STATE
    pts = _points_from_voxels(np.random.default_rng(0).integers(0, 256, (50, 3)), 8, 10.0)
    encode(ctx, pts, 8)
    with pytest.raises(reno.RenoError) as e:
        ctx.predict_probs(5)                             # no weights yet
    assert e.value.status == reno.RENO_E_STATE
    ctx.set_weights(reno.weights_to_device(gen_weights(16, 2, seed=1)))
    with pytest.raises(reno.RenoError) as e:
        ctx.code_length(5)                               # not predicted yet
    assert e.value.status == reno.RENO_E_STATE
    with pytest.raises(reno.RenoError) as e:
        ctx.predict_probs(3)                             # the base scale is not modelled
    assert e.value.status == reno.RENO_E_INVALID
    with pytest.raises(reno.RenoError) as e:
        ctx.predict_probs(8)                             # nor is the finest
    assert e.value.status == reno.RENO_E_INVALID
    with pytest.raises(reno.RenoError) as e:
        ctx.expand(5)                                    # encoder context holds every scale
    assert e.value.status == reno.RENO_E_STATE
    with pytest.raises(reno.RenoError) as e:
        ctx.build_pyramid(to_dev(np.zeros((101, 3), np.float32)), 8)   # over capacity
    assert e.value.status == reno.RENO_E_INVALID
    with pytest.raises(reno.RenoError) as e:
        ctx.build_pyramid(to_dev(pts), 9)                # above max_bit_depth
    assert e.value.status == reno.RENO_E_INVALID
    ctx.close()


def test_model_capacity_overflow_reported():
    cfg = _cfg(9, 3)
    rs = np.random.default_rng(9)
    pts = _points_from_voxels(rs.integers(0, 512, size=(2000, 3)), 9, 10.0)
    ctx = make_ctx(cfg, len(pts), max_model_voxels=100)
    ctx.build_pyramid(to_dev(pts), 9)
    with pytest.raises(reno.RenoError) as e:
        ctx.sync()
    assert e.value.status == reno.RENO_E_CAPACITY
    ctx.close()


@pytest.mark.parametrize("extra", [0, 1])
def test_quad_split_boundary(extra):
    """A model scale of exactly 1024 tiles (16384 voxels: a 32 x 32 x 16 block)
    runs with a quad of waves per tile when launched alone; one voxel more
    (1025 tiles) runs one wave per tile.  Either way the per-scale launches of
    the encoder and of the decoder reproduce the all-scale launch (one wave per
    tile) bit for bit, and match the oracle."""
    B, b0, R, C, L = 8, 4, 10.0, 32, 3
    g = np.stack(np.meshgrid(np.arange(32), np.arange(32), np.arange(16), indexing="ij"), -1).reshape(-1, 3)
    cells7 = g + np.array([40, 50, 60])
    if extra:
        cells7 = np.concatenate([cells7, [[3, 120, 7]]])
    pts = _points_from_voxels(2 * cells7, B, R)  # one finest-scale child per scale-7 voxel
    w = gen_weights(C, L, seed=61, bias_std=0.1)
    cfg = _cfg(B, b0, C, L, R)
    say("quad split boundary, scale-7 voxels", len(cells7))
    enc = make_ctx(cfg, len(pts))
    encode(enc, pts, B)
    assert enc.num_voxels(7) == 16384 + extra
    enc.set_weights(reno.weights_to_device(w))
    lg = enc.predict_probs(reno.RENO_ALL_SCALES, logits=True).cpu().numpy()
    bits, total = enc.code_length(reno.RENO_ALL_SCALES)
    P = oracle.Pyramid.from_points(pts, B, b0, R)
    off = {}
    o = 0
    for b in range(b0 + 1, B):
        off[b] = o
        n = P.num(b)
        olg, _, obits = P.model(b, w)
        assert np.abs(lg[o:o + n] - olg).max() <= LOGIT_TOL, b
        assert np.abs(bits.cpu().numpy()[o:o + n] - obits).max() <= BITS_ABS_TOL, b
        o += n
    # encoder, one scale per launch
    for b in range(b0 + 1, B):
        n = P.num(b)
        np.testing.assert_array_equal(enc.predict_probs(b, logits=True).cpu().numpy(), lg[off[b]:off[b] + n])
    # decoder
    codes = {b: enc.occupancy_codes(b).clone() for b in range(b0, B)}
    base, _ = enc.coords(b0)
    dec = make_ctx(cfg, len(pts))
    dec.set_weights(reno.weights_to_device(w))
    dec.set_base(B, base.clone(), codes[b0])
    for b in range(b0 + 1, B):
        dec.expand(b - 1, None if b - 1 == b0 else codes[b - 1])
        n = P.num(b)
        np.testing.assert_array_equal(dec.predict_probs(b, logits=True).cpu().numpy(), lg[off[b]:off[b] + n])
    dec.expand(B - 1, codes[B - 1])
    dbits, dtotal = dec.code_length(reno.RENO_ALL_SCALES)
    np.testing.assert_array_equal(dbits.cpu().numpy(), bits.cpu().numpy())
    assert dtotal == total
    enc.close()
    dec.close()
