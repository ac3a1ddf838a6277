"""GPU parity: the HIP path (through the C ABI) against the CPU oracle on the
same seeded inputs.  Integer results bit-exact; logits within 1e-3 absolute;
total bits within 0.1 %."""
import numpy as np
import pytest
import torch  # noqa: F401  (the first import on a fresh box is slow: do it at collection)

import oracle
import paper_2503_12382_amd as reno
from gpu_helpers import (BITS_ABS_TOL, BITS_REL_TOL, LOGIT_TOL, assert_levels_equal, cfg_dict,
                         encode, levels_from_gpu, make_ctx, say, to_dev, torch)
from synth import CONFIGS, gen_weights

pytestmark = pytest.mark.gpu


def _weights(cfg, **kw):
    kw.setdefault("bias_std", 0.1)
    return gen_weights(cfg.channels, cfg.layers, seed=cfg.weight_seed, **kw)


@pytest.mark.parametrize("ci", [0, 1, 2, 3])
def test_pyramid_codes_parents(ci, scan_cache):
    cfg = CONFIGS[ci]
    pts = scan_cache(ci)
    say("pyramid parity", cfg.name, "M", len(pts))
    ctx = make_ctx(cfg_dict(cfg), len(pts))
    encode(ctx, pts, cfg.bit_depth)
    gpu = levels_from_gpu(ctx, cfg.min_bit_depth, cfg.bit_depth)
    P = oracle.Pyramid.from_points(pts, cfg.bit_depth, cfg.min_bit_depth, cfg.range_m)
    assert_levels_equal(gpu, P, cfg.min_bit_depth, cfg.bit_depth)
    ctx.close()


@pytest.mark.parametrize("ci", [0, 1, 2, 3])
def test_model_full_parity(ci, scan_cache):
    """Every logit and per-voxel bit of every model scale against the oracle
    (1e-3 absolute), every neighbour map bit-exact, and the frame's total bits
    (0.1 %), on all four single-frame scans up to the full 14- and 16-bit
    frames; the oracle runs scale by scale to bound host memory."""
    cfg = CONFIGS[ci]
    pts = scan_cache(ci)
    w = _weights(cfg)
    say("model parity", cfg.name, "M", len(pts))
    ctx = make_ctx(cfg_dict(cfg), len(pts))
    encode(ctx, pts, cfg.bit_depth)
    ctx.set_weights(reno.weights_to_device(w))
    logits = ctx.predict_probs(reno.RENO_ALL_SCALES, logits=True).cpu().numpy()
    bits, total = ctx.code_length(reno.RENO_ALL_SCALES)
    bits = bits.cpu().numpy()
    P = oracle.Pyramid.from_points(pts, cfg.bit_depth, cfg.min_bit_depth, cfg.range_m)
    b0 = cfg.min_bit_depth
    T = 32.0 + P.num(b0) * (3 * b0 + 8)          # the raw initial state
    off = 0
    for b in range(b0 + 1, cfg.bit_depth):
        n = P.num(b)
        lg, lse, bt = P.model(b, w)
        err = np.abs(logits[off:off + n] - lg).max()
        berr = np.abs(bits[off:off + n] - bt).max()
        say(f"b={b} n={n} max|dlogit|={err:.2e} max|dbits|={berr:.2e}")
        assert err <= LOGIT_TOL, (b, err)
        assert berr <= BITS_ABS_TOL, (b, berr)
        del lg, lse
        nb = ctx.neighbor_map(b).cpu().numpy()
        np.testing.assert_array_equal(nb, P.neighbors(b), err_msg=f"neighbours b={b}")
        T += float(bt.sum())
        off += n
    assert off == len(bits)
    say(f"total bits gpu={total:.3f} oracle={T:.3f}")
    assert abs(total - T) <= BITS_REL_TOL * T
    if ci <= 1:   # the oracle's own total is the same sum
        assert P.totals(w)[0] == pytest.approx(T, rel=1e-12)
    ctx.close()


@pytest.mark.parametrize("ci", [0, 1, 2, 3])
def test_decoder_expansion_and_determinism(ci, scan_cache):
    """Decoder: initial state + codes -> every scale bit-exact (Eq. 2), and the
    decoder's distributions bit-identical to the encoder's."""
    cfg = CONFIGS[ci]
    pts = scan_cache(ci)
    w = _weights(cfg)
    wd = reno.weights_to_device(w)
    b0, B = cfg.min_bit_depth, cfg.bit_depth
    P = oracle.Pyramid.from_points(pts, B, b0, cfg.range_m)
    say("encoder", cfg.name)
    enc = make_ctx(cfg_dict(cfg), len(pts))
    encode(enc, pts, B)
    enc.set_weights(wd)
    enc_logits = enc.predict_probs(reno.RENO_ALL_SCALES, logits=True).cpu().numpy()
    enc_bits, enc_total = enc.code_length(reno.RENO_ALL_SCALES)
    say("decoder", cfg.name)
    dec = make_ctx(cfg_dict(cfg), len(pts))
    dec.set_weights(wd)
    dec.set_base(B, to_dev(P.xyz(b0).astype(np.int32)), to_dev(P.codes(b0)))
    dec_logits = []
    for b in range(b0 + 1, B):
        dec.expand(b - 1, None if b - 1 == b0 else to_dev(P.codes(b - 1)))
        dec_logits.append(dec.predict_probs(b, logits=True).cpu().numpy())
    dec.expand(B - 1, to_dev(P.codes(B - 1)))
    dec_bits, dec_total = dec.code_length(reno.RENO_ALL_SCALES)
    gpu = levels_from_gpu(dec, b0, B)
    assert_levels_equal(gpu, P, b0, B)
    dl = np.concatenate(dec_logits)
    assert np.array_equal(dl.view(np.uint32), enc_logits.view(np.uint32)), "decoder logits differ"
    assert np.array_equal(dec_bits.cpu().numpy().view(np.uint32), enc_bits.cpu().numpy().view(np.uint32))
    assert dec_total == enc_total
    # run the encoder model again: bitwise identical
    again = enc.predict_probs(reno.RENO_ALL_SCALES, logits=True).cpu().numpy()
    assert np.array_equal(again.view(np.uint32), enc_logits.view(np.uint32))
    enc.close()
    dec.close()


@pytest.mark.parametrize("ci", [0, 1])
def test_round_trip_through_host_rans(ci, scan_cache):
    """Encoder codes -> host rANS with the encoder's tables; decoder predicts
    each scale before its codes are known, decodes them with its own tables
    and expands; the decoded frame equals the encoder's."""
    cfg = CONFIGS[ci]
    pts = scan_cache(ci)
    wd = reno.weights_to_device(_weights(cfg, head_scale=4.0))
    b0, B = cfg.min_bit_depth, cfg.bit_depth
    enc = make_ctx(cfg_dict(cfg), len(pts))
    encode(enc, pts, B)
    enc.set_weights(wd)
    enc.predict_probs(reno.RENO_ALL_SCALES)
    streams = {}
    for b in range(b0 + 1, B):
        f = enc.symbol_freqs(b).cpu().numpy().view(np.uint16)
        codes = enc.occupancy_codes(b).cpu().numpy()
        streams[b] = (reno.rans_encode(codes, f), codes.size, codes)
    base_xyz, _ = enc.coords(b0)
    base_codes = enc.occupancy_codes(b0)
    _, total = enc.code_length(reno.RENO_ALL_SCALES)
    coded = sum(32 * s[0].size for s in streams.values())
    base = 32 + base_codes.numel() * (3 * b0 + 8)
    say(f"ideal {total:.0f} bits, coded {coded + base} bits")
    assert coded + base >= total - 64 and coded + base <= total * 1.001 + 64 * len(streams)

    dec = make_ctx(cfg_dict(cfg), len(pts))
    dec.set_weights(wd)
    dec.set_base(B, base_xyz.contiguous(), base_codes.contiguous())
    prev = None                        # decoded codes of the previous scale (b0: given)
    for b in range(b0 + 1, B):
        dec.expand(b - 1, prev)        # builds V_b and records O_{b-1}
        dec.predict_probs(b)           # O_b is not known yet
        f = dec.symbol_freqs(b).cpu().numpy().view(np.uint16)
        words, n, truth = streams[b]
        codes = reno.rans_decode(words, f, n)
        assert np.array_equal(codes, truth), f"scale {b}"
        prev = to_dev(codes)
    dec.expand(B - 1, prev)
    xyz, _ = dec.coords(B)
    exyz, _ = enc.coords(B)
    assert torch().equal(xyz, exyz)
    enc.close()
    dec.close()
