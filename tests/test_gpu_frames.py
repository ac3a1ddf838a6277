"""Frame batches (several frames in one key space, frame id above the Morton
bits) on the GPU: each frame's pyramid, codes, logits and bits equal the
oracle's for that frame alone and, bit for bit, a single-frame run of the
same context shape; the batched decoder reproduces the batched encoder; the
full predictor and the two-stage head work on batches; malformed frame ranges
and frame ids are reported."""
import numpy as np
import pytest
import torch

import oracle
import paper_2503_12382_amd as reno
from gpu_helpers import BITS_ABS_TOL, BITS_REL_TOL, LOGIT_TOL, say, to_dev
from synth import CONFIGS, gen_weights

pytestmark = pytest.mark.gpu


def _frames(scan):
    """Four frames of different sizes: the scan, the scan moved 3.3 m along x,
    an empty frame, and the first 1000 points."""
    f1 = scan.copy()
    f1[:, 0] += np.float32(3.3)
    return [scan, f1, scan[:0], scan[:1000]]


def _batch(frames):
    pts = np.concatenate(frames).astype(np.float32)
    start = np.cumsum([0] + [len(f) for f in frames]).astype(np.int64)
    return pts, start


def _ctx(cfg, M, **kw):
    return reno.Context(max(M, 1), cfg.bit_depth, cfg.min_bit_depth, cfg.range_m, cfg.channels, cfg.layers, **kw)


def _split(keys, b, nframes):
    """Row ranges of each frame in a scale of the batch (keys sorted by frame)."""
    fr = (keys >> np.uint64(3 * b)).astype(np.int64)
    return [np.searchsorted(fr, f, "left") for f in range(nframes + 1)]


@pytest.mark.parametrize("ci", [0, 1])
def test_frame_batch_encoder_matches_oracle_per_frame(ci, scan_cache):
    cfg = CONFIGS[ci]
    B, b0 = cfg.bit_depth, cfg.min_bit_depth
    frames = _frames(scan_cache(ci))
    pts, start = _batch(frames)
    w = gen_weights(cfg.channels, cfg.layers, seed=cfg.weight_seed + 3, bias_std=0.1)
    say("frame batch encoder", cfg.name, [len(f) for f in frames])
    ctx = _ctx(cfg, len(pts))
    ctx.set_weights(reno.weights_to_device(w))
    ctx.build_pyramid_frames(to_dev(pts), to_dev(start), B)
    lg = ctx.predict_probs(reno.RENO_ALL_SCALES, logits=True).cpu().numpy()
    bits, total = ctx.code_length(reno.RENO_ALL_SCALES)
    bits = bits.cpu().numpy()
    Ps = [oracle.Pyramid.from_points(f, B, b0, cfg.range_m) if len(f) else None for f in frames]
    off = 0
    for b in range(b0, B + 1):
        xyz, keys = ctx.coords(b)
        xyz, keys = xyz.cpu().numpy(), keys.cpu().numpy().view(np.uint64)
        cut = _split(keys, b, len(frames))
        codes = ctx.occupancy_codes(b).cpu().numpy() if b < B else None
        for f, P in enumerate(Ps):
            lo, hi = cut[f], cut[f + 1]
            if P is None:
                assert hi == lo
                continue
            np.testing.assert_array_equal(xyz[lo:hi], P.xyz(b), err_msg=f"xyz b={b} f={f}")
            np.testing.assert_array_equal(keys[lo:hi] & np.uint64((1 << (3 * b)) - 1), P.keys(b))
            if codes is not None:
                np.testing.assert_array_equal(codes[lo:hi], P.codes(b), err_msg=f"codes b={b} f={f}")
            if b0 < b < B:
                olg, _, obits = P.model(b, w)
                assert np.abs(lg[off + lo:off + hi] - olg).max() <= LOGIT_TOL, (b, f)
                assert np.abs(bits[off + lo:off + hi] - obits).max() <= BITS_ABS_TOL, (b, f)
        if b0 < b < B:
            off += len(keys)
    assert off == len(bits)
    T = sum(P.totals(w)[0] for P in Ps if P is not None) + 32.0   # the empty frame's raw count
    assert abs(total - T) <= BITS_REL_TOL * T
    # bit-identical to single-frame runs of each frame
    off = 0
    single = []
    for f in frames:
        if len(f) == 0:
            single.append(None)
            continue
        c1 = _ctx(cfg, len(pts))
        c1.set_weights(reno.weights_to_device(w))
        c1.build_pyramid(to_dev(f), B)
        single.append(c1.predict_probs(reno.RENO_ALL_SCALES, logits=True).cpu().numpy())
        c1.close()
    for b in range(b0 + 1, B):
        _, keys = ctx.coords(b)
        cut = _split(keys.cpu().numpy().view(np.uint64), b, len(frames))
        for f, P in enumerate(Ps):
            if P is None:
                continue
            s_off = sum(P.num(s) for s in range(b0 + 1, b))
            np.testing.assert_array_equal(lg[off + cut[f]:off + cut[f + 1]],
                                          single[f][s_off:s_off + P.num(b)])
        off += cut[-1]
    ctx.close()


def _decoder_round(cfg, frames, two, top):
    """Batched encoder, then the batched decoder from its base scale and codes:
    every logit, bit, total and scale identical.  Returns the base-scale count."""
    B, b0 = cfg.bit_depth, cfg.min_bit_depth
    pts, start = _batch(frames)
    w = gen_weights(cfg.channels, cfg.layers, seed=cfg.weight_seed + 9, bias_std=0.1, two_stage=two, top=top)
    enc = _ctx(cfg, len(pts), two_stage=two, top=top)
    enc.set_weights(reno.weights_to_device(w))
    enc.build_pyramid_frames(to_dev(pts), to_dev(start), B)
    lg = enc.predict_probs(reno.RENO_ALL_SCALES, logits=True).cpu().numpy()
    bits, total = enc.code_length(reno.RENO_ALL_SCALES)
    codes = {b: enc.occupancy_codes(b).clone() for b in range(b0, B)}
    base, keys = enc.coords(b0)
    fid = (keys.cpu().numpy().view(np.uint64) >> np.uint64(3 * b0)).astype(np.int32)
    counts = {b: enc.num_voxels(b) for b in range(b0, B + 1)}
    dec = _ctx(cfg, len(pts), two_stage=two, top=top)
    dec.set_weights(reno.weights_to_device(w))
    dec.set_base_frames(B, base.clone(), to_dev(fid), codes[b0], len(frames))
    off = 0
    for b in range(b0 + 1, B):
        dec.expand(b - 1, None if b - 1 == b0 else codes[b - 1])
        n = counts[b]
        got = dec.predict_probs(b, logits=True).cpu().numpy()
        if two:
            l2 = dec.predict_second(b, (codes[b] & 15).to(torch.uint8), logits=True).cpu().numpy()
            np.testing.assert_array_equal(got[:, :16], lg[off:off + n, :16])
            np.testing.assert_array_equal(l2, lg[off:off + n, 16:])
        else:
            np.testing.assert_array_equal(got, lg[off:off + n])
        off += n
    dec.expand(B - 1, codes[B - 1])
    dbits, dtotal = dec.code_length(reno.RENO_ALL_SCALES)
    np.testing.assert_array_equal(dbits.cpu().numpy(), bits.cpu().numpy())
    assert dtotal == total
    for b in range(b0, B + 1):
        np.testing.assert_array_equal(dec.coords(b)[1].cpu().numpy(), enc.coords(b)[1].cpu().numpy())
    enc.close()
    dec.close()
    return counts[b0]


@pytest.mark.parametrize("two,top", [(False, False), (True, False), (False, True)])
def test_frame_batch_decoder_bit_identical(two, top, scan_cache):
    say("frame batch decoder two-stage", two, "full predictor", top)
    _decoder_round(CONFIGS[1], _frames(scan_cache(1)), two, top)


@pytest.mark.parametrize("small", [True, False])
def test_frame_batch_decoder_base_paths(small, scan_cache):
    """A batch whose base scale has fewer than 256 voxels in all (the decoder
    clears its frame and writes the base scale, hash regions included, in one
    launch) and one with more (a clear, then the base-scale kernel)."""
    scan = scan_cache(0)
    if small:
        f1 = scan[:300].copy()
        f1[:, 1] += np.float32(2.0)
        frames = [scan[:300], f1, scan[:0], scan[:40]]
    else:
        frames = []
        for k in range(4):
            f = scan.copy()
            f[:, 0] += np.float32(0.7 * k)
            frames.append(f)
    say("frame batch decoder, base scale", "small" if small else "large")
    n0 = _decoder_round(CONFIGS[0], frames, False, False)
    assert (0 < n0 < 256) if small else n0 >= 256, n0


def test_frame_batch_errors(scan_cache):
    cfg = CONFIGS[0]
    frames = _frames(scan_cache(0))
    pts, start = _batch(frames)
    ctx = _ctx(cfg, len(pts))
    bad = start.copy()
    bad[2] = bad[1] - 1                                   # ranges not ascending
    say("frame batch errors")
    ctx.build_pyramid_frames(to_dev(pts), to_dev(bad), cfg.bit_depth)
    with pytest.raises(reno.RenoError) as e:
        ctx.sync()
    assert e.value.status == reno.RENO_E_INPUT
    bad = start.copy()
    bad[-1] -= 1                                          # does not end at n
    ctx.build_pyramid_frames(to_dev(pts), to_dev(bad), cfg.bit_depth)
    with pytest.raises(reno.RenoError):
        ctx.sync()
    with pytest.raises(reno.RenoError) as e:              # too many frames
        ctx.build_pyramid_frames(to_dev(pts), to_dev(np.zeros(1026, np.int64)), cfg.bit_depth)
    assert e.value.status == reno.RENO_E_INVALID
    ctx.build_pyramid_frames(to_dev(pts), to_dev(start), cfg.bit_depth)
    ctx.sync()                                            # a good batch after the errors
    xyz, keys = ctx.coords(cfg.min_bit_depth)
    fid = (keys.cpu().numpy().view(np.uint64) >> np.uint64(3 * cfg.min_bit_depth)).astype(np.int32)
    fid[0] = 7                                            # outside [0, frames)
    codes = ctx.occupancy_codes(cfg.min_bit_depth)
    ctx.set_base_frames(cfg.bit_depth, xyz.clone(), to_dev(fid), codes, len(frames))
    with pytest.raises(reno.RenoError) as e:
        ctx.sync()
    assert e.value.status == reno.RENO_E_INPUT
    ctx.close()


def test_large_batch_pyramid_matches_oracle(scan_cache):
    """36 copies of the 12-bit scan as one batch (4.6M points: the large-tile
    sort path): every frame's scales, codes and parents equal the oracle's."""
    cfg = CONFIGS[1]
    B, b0 = cfg.bit_depth, cfg.min_bit_depth
    scan = scan_cache(1)
    K = 36
    pts = np.concatenate([scan] * K)
    start = (np.arange(K + 1) * len(scan)).astype(np.int64)
    assert len(pts) >= 1 << 22
    say("large frame batch", len(pts), "points")
    ctx = _ctx(cfg, len(pts))
    ctx.build_pyramid_frames(to_dev(pts), to_dev(start), B)
    ctx.sync()
    P = oracle.Pyramid.from_points(scan, B, b0, cfg.range_m)
    for b in range(b0, B + 1):
        n = P.num(b)
        assert ctx.num_voxels(b) == K * n
        xyz, keys = ctx.coords(b)
        keys = keys.cpu().numpy().view(np.uint64)
        want = np.concatenate([P.keys(b) | (np.uint64(f) << np.uint64(3 * b)) for f in range(K)])
        np.testing.assert_array_equal(keys, want, err_msg=f"keys b={b}")
        np.testing.assert_array_equal(xyz.cpu().numpy(), np.concatenate([P.xyz(b)] * K))
        par = ctx.parent_rows(b).cpu().numpy()
        if b > b0:
            np.testing.assert_array_equal(
                par, np.concatenate([P.parent(b) + f * P.num(b - 1) for f in range(K)]))
        if b < B:
            np.testing.assert_array_equal(ctx.occupancy_codes(b).cpu().numpy(), np.concatenate([P.codes(b)] * K))
    ctx.close()
