"""Full target occupancy predictor (Sec. 3.2, Eqs. 6-9) on the GPU against the
oracle: logits, per-voxel bits and frame totals with the one-stage and the
two-stage head; the decoder's per-scale calls bit-identical to the encoder's
all-scale call (and earlier scales' features left intact by later calls);
edge cases: the root as base scale, a single voxel, an empty frame."""
import numpy as np
import pytest
import torch

import oracle
import paper_2503_12382_amd as reno
from gpu_helpers import BITS_ABS_TOL, BITS_REL_TOL, LOGIT_TOL, say, to_dev
from synth import CONFIGS, gen_weights

pytestmark = pytest.mark.gpu

# two stages: four logit-sized errors per voxel
BITS2_ABS_TOL = 4 * LOGIT_TOL / np.log(2.0)


def _weights(C, seed, two=False, head_scale=1.0):
    return gen_weights(C, 2, seed=seed, bias_std=0.1, head_scale=head_scale, two_stage=two, top=True)


def _ctx(B, b0, R, C, M, two=False):
    return reno.Context(max(M, 1), B, b0, R, C, 2, two_stage=two, top=True)


def _encode(B, b0, R, C, pts, w, two=False):
    ctx = _ctx(B, b0, R, C, len(pts), two)
    ctx.set_weights(reno.weights_to_device(w))
    ctx.build_pyramid(to_dev(pts), B)
    lg = ctx.predict_probs(reno.RENO_ALL_SCALES, logits=True)
    bits, total = ctx.code_length(reno.RENO_ALL_SCALES)
    return ctx, lg.cpu().numpy(), bits.cpu().numpy(), total


def _check_against_oracle(pts, B, b0, R, C, w, two):
    ctx, lg, bits, total = _encode(B, b0, R, C, pts, w, two)
    P = oracle.Pyramid.from_points(pts, B, b0, R)
    off = 0
    for b in range(b0 + 1, B):
        n = P.num(b)
        if two:
            l1, l2, _, _, obits = P.model2(b, w)
            assert np.abs(lg[off:off + n, :16] - l1).max() <= LOGIT_TOL, b
            assert np.abs(lg[off:off + n, 16:] - l2).max() <= LOGIT_TOL, b
            assert np.abs(bits[off:off + n] - obits).max() <= BITS2_ABS_TOL, b
        else:
            olg, _, obits = P.model(b, w)
            assert np.abs(lg[off:off + n] - olg).max() <= LOGIT_TOL, b
            assert np.abs(bits[off:off + n] - obits).max() <= BITS_ABS_TOL, b
        np.testing.assert_array_equal(ctx.neighbor_map(b).cpu().numpy(), P.neighbors(b))
        off += n
    assert off == len(bits)
    T, _ = P.totals(w)
    assert abs(total - T) <= BITS_REL_TOL * T
    ctx.close()


@pytest.mark.parametrize("ci,two", [(0, False), (0, True), (1, False), (1, True), (2, False), (2, True),
                                    (3, False), (3, True)])
def test_top_encoder_matches_oracle(ci, two, scan_cache):
    cfg = CONFIGS[ci]
    pts = scan_cache(ci)
    w = _weights(cfg.channels, cfg.weight_seed + 17, two)
    say("full predictor encoder", cfg.name, "two-stage", two)
    _check_against_oracle(pts, cfg.bit_depth, cfg.min_bit_depth, cfg.range_m, cfg.channels, w, two)


@pytest.mark.parametrize("C", [16, 32])
def test_top_other_channels_and_peaked_head(C, scan_cache):
    cfg = CONFIGS[0]
    w = _weights(C, 23, head_scale=8.0)
    say("full predictor C", C)
    _check_against_oracle(scan_cache(0), cfg.bit_depth, cfg.min_bit_depth, cfg.range_m, C, w, False)


def _cells(xyz, B, R):
    step = 2.0 * R / (1 << B)
    return (-R + (np.asarray(xyz, np.float64) + 0.5) * step).astype(np.float32)


def test_top_root_base_and_dense_block():
    """b0 = 0 (a one-voxel base scale) and a fully occupied block (27 neighbours)."""
    B, R = 7, 10.0
    rs = np.random.default_rng(4)
    g = np.stack(np.meshgrid(*[np.arange(40, 56)] * 3, indexing="ij"), -1).reshape(-1, 3)
    xyz = np.concatenate([g, rs.integers(0, 1 << B, size=(500, 3))])
    w = _weights(32, 29)
    say("full predictor root base + dense block")
    _check_against_oracle(_cells(xyz, B, R), B, 0, R, 32, w, False)


@pytest.mark.parametrize("copies", [1, 50])
def test_top_single_voxel(copies):
    B, R = 9, 10.0
    pts = np.repeat(_cells([[300, 7, 511]], B, R), copies, axis=0)
    say("full predictor single voxel x", copies)
    _check_against_oracle(pts, B, 3, R, 16, _weights(16, 31), False)


def test_top_empty_frame():
    ctx = _ctx(10, 4, 10.0, 16, 16)
    ctx.set_weights(reno.weights_to_device(_weights(16, 3)))
    ctx.build_pyramid(torch.zeros((0, 3), dtype=torch.float32, device="cuda"), 10)
    ctx.predict_probs(reno.RENO_ALL_SCALES)
    _, total = ctx.code_length(reno.RENO_ALL_SCALES, per_voxel=False)
    assert total == 32.0
    ctx.close()


@pytest.mark.parametrize("ci,two", [(1, False), (2, True)])
def test_top_decoder_bit_identical(ci, two, scan_cache):
    """Per-scale calls (decoder order: predict b, then expand b) give exactly the
    encoder's all-scale logits; code lengths read after every later scale has
    run still equal the encoder's."""
    cfg = CONFIGS[ci]
    B, b0, C = cfg.bit_depth, cfg.min_bit_depth, cfg.channels
    pts = scan_cache(ci)
    w = _weights(C, cfg.weight_seed + 5, two)
    say("full predictor decoder", cfg.name, "two-stage", two)
    enc, lg, bits, total = _encode(B, b0, cfg.range_m, C, pts, w, two)
    codes = {b: enc.occupancy_codes(b).clone() for b in range(b0, B)}
    base, _ = enc.coords(b0)
    counts = {b: enc.num_voxels(b) for b in range(b0, B + 1)}
    dec = _ctx(B, b0, cfg.range_m, C, len(pts), two)
    dec.set_weights(reno.weights_to_device(w))
    dec.set_base(B, base.clone(), codes[b0])
    off = 0
    for b in range(b0 + 1, B):
        dec.expand(b - 1, None if b - 1 == b0 else codes[b - 1])
        n = counts[b]
        if two:
            l1 = dec.predict_probs(b, logits=True).cpu().numpy()[:, :16]
            l2 = dec.predict_second(b, (codes[b] & 15).to(torch.uint8), logits=True).cpu().numpy()
            np.testing.assert_array_equal(l1, lg[off:off + n, :16])
            np.testing.assert_array_equal(l2, lg[off:off + n, 16:])
        else:
            np.testing.assert_array_equal(dec.predict_probs(b, logits=True).cpu().numpy(), lg[off:off + n])
        off += n
    dec.expand(B - 1, codes[B - 1])
    dbits, dtotal = dec.code_length(reno.RENO_ALL_SCALES)
    np.testing.assert_array_equal(dbits.cpu().numpy(), bits)
    assert dtotal == total
    enc.close()
    dec.close()


def test_top_single_scale_encoder_calls(scan_cache):
    """predict_probs(b) one scale at a time on the encoder equals the all-scale call."""
    cfg = CONFIGS[0]
    B, b0, C = cfg.bit_depth, cfg.min_bit_depth, cfg.channels
    pts = scan_cache(0)
    w = _weights(C, 41)
    enc, lg, bits, _ = _encode(B, b0, cfg.range_m, C, pts, w)
    ctx = _ctx(B, b0, cfg.range_m, C, len(pts))
    ctx.set_weights(reno.weights_to_device(w))
    ctx.build_pyramid(to_dev(pts), B)
    off = 0
    for b in range(B - 1, b0, -1):                       # any order
        got = ctx.predict_probs(b, logits=True).cpu().numpy()
        start = sum(enc.num_voxels(s) for s in range(b0 + 1, b))
        np.testing.assert_array_equal(got, lg[start:start + got.shape[0]])
        off += got.shape[0]
    assert off == lg.shape[0]
    enc.close()
    ctx.close()
