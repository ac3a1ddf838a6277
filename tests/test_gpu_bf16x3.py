"""Split-bf16 precision (RENO_PREC_BF16X3) against the oracle, with its own
tolerance study: every fp32 operand is carried as bf16 hi + lo and each
product as hi*hi + hi*lo + lo*hi on bf16 MFMA (fp32 accumulation), so a
product is exact to about 2^-16 relative instead of fp32's 2^-24.  The bar
stays the fp32 path's: logits within 1e-3 absolute of the fp64 oracle, total
bits within 0.1 %; the measured worst logit error is printed next to the
fp32 path's on the same inputs.  Integer outputs (neighbour maps) and the
encoder/decoder identity are unchanged."""
import numpy as np
import pytest
import torch  # noqa: F401  (slow first import on a fresh box: at collection)

import oracle
import paper_2503_12382_amd as reno
from gpu_helpers import BITS_REL_TOL, LOGIT_TOL, say, to_dev
from synth import CONFIGS, gen_weights

pytestmark = pytest.mark.gpu


def _ctx(cfg, M, precision, two=False):
    return reno.Context(max(M, 1), cfg.bit_depth, cfg.min_bit_depth, cfg.range_m, cfg.channels,
                        cfg.layers, two_stage=two, precision=precision)


def _logit_errors(ci, w, scan_cache, two=False):
    cfg = CONFIGS[ci]
    B, b0 = cfg.bit_depth, cfg.min_bit_depth
    pts = scan_cache(ci)
    P = oracle.Pyramid.from_points(pts, B, b0, cfg.range_m)
    ref = []
    for b in range(b0 + 1, B):
        if two:
            l1, l2, _, _, _ = P.model2(b, w)
            ref.append(np.concatenate([l1, l2], 1))
        else:
            ref.append(P.model(b, w)[0])
    ref = np.concatenate(ref)
    T, _ = P.totals(w)
    out = {}
    for prec in (reno.RENO_PREC_FP32, reno.RENO_PREC_BF16X3):
        ctx = _ctx(cfg, len(pts), prec, two)
        ctx.set_weights(reno.weights_to_device(w))
        ctx.build_pyramid(to_dev(pts), B)
        lg = ctx.predict_probs(reno.RENO_ALL_SCALES, logits=True).cpu().numpy()
        _, total = ctx.code_length(reno.RENO_ALL_SCALES, per_voxel=False)
        maps = {b: ctx.neighbor_map(b).cpu().numpy() for b in range(b0 + 1, B)}
        out[prec] = (float(np.abs(lg - ref).max()), total, maps)
        ctx.close()
    for b in range(b0 + 1, B):
        np.testing.assert_array_equal(out[reno.RENO_PREC_BF16X3][2][b], P.neighbors(b))
    return out, T, float(np.abs(ref).max())


@pytest.mark.parametrize("ci,head_scale", [(0, 1.0), (0, 10.0), (1, 1.0), (1, 10.0), (2, 1.0), (3, 1.0)])
def test_bf16x3_tolerance_one_stage(ci, head_scale, scan_cache):
    cfg = CONFIGS[ci]
    w = gen_weights(cfg.channels, cfg.layers, seed=cfg.weight_seed, bias_std=0.1, head_scale=head_scale)
    say("bf16x3 one-stage", cfg.name, "head scale", head_scale)
    out, T, lmax = _logit_errors(ci, w, scan_cache)
    e32, t32, _ = out[reno.RENO_PREC_FP32]
    ebf, tbf, _ = out[reno.RENO_PREC_BF16X3]
    say(f"  max |logit| {lmax:.2f}; worst logit error fp32 {e32:.2e}, bf16x3 {ebf:.2e}; "
        f"total bits rel. error fp32 {abs(t32 - T) / T:.1e}, bf16x3 {abs(tbf - T) / T:.1e}")
    assert ebf <= LOGIT_TOL
    assert abs(tbf - T) <= BITS_REL_TOL * T


@pytest.mark.parametrize("ci", [0, 1, 2])
def test_bf16x3_tolerance_two_stage(ci, scan_cache):
    cfg = CONFIGS[ci]
    w = gen_weights(cfg.channels, cfg.layers, seed=cfg.weight_seed + 7, bias_std=0.1, two_stage=True)
    say("bf16x3 two-stage", cfg.name)
    out, T, _ = _logit_errors(ci, w, scan_cache, two=True)
    ebf, tbf, _ = out[reno.RENO_PREC_BF16X3]
    say(f"  worst logit error fp32 {out[reno.RENO_PREC_FP32][0]:.2e}, bf16x3 {ebf:.2e}")
    assert ebf <= LOGIT_TOL
    assert abs(tbf - T) <= BITS_REL_TOL * T


def test_bf16x3_decoder_bit_identical(scan_cache):
    cfg = CONFIGS[1]
    B, b0 = cfg.bit_depth, cfg.min_bit_depth
    pts = scan_cache(1)
    w = reno.weights_to_device(gen_weights(cfg.channels, cfg.layers, seed=cfg.weight_seed, bias_std=0.1))
    say("bf16x3 decoder", cfg.name)
    enc = _ctx(cfg, len(pts), reno.RENO_PREC_BF16X3)
    enc.set_weights(w)
    enc.build_pyramid(to_dev(pts), B)
    lg = enc.predict_probs(reno.RENO_ALL_SCALES, logits=True).cpu().numpy()
    _, total = enc.code_length(reno.RENO_ALL_SCALES, per_voxel=False)
    codes = {b: enc.occupancy_codes(b).clone() for b in range(b0, B)}
    base, _ = enc.coords(b0)
    dec = _ctx(cfg, len(pts), reno.RENO_PREC_BF16X3)
    dec.set_weights(w)
    dec.set_base(B, base.clone(), codes[b0])
    off = 0
    for b in range(b0 + 1, B):
        dec.expand(b - 1, None if b - 1 == b0 else codes[b - 1])
        l = dec.predict_probs(b, logits=True).cpu().numpy()
        np.testing.assert_array_equal(l, lg[off:off + l.shape[0]])
        off += l.shape[0]
    dec.expand(B - 1, codes[B - 1])
    _, dtotal = dec.code_length(reno.RENO_ALL_SCALES, per_voxel=False)
    assert dtotal == total
    enc.close()
    dec.close()
