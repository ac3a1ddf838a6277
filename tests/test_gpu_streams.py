"""Frames in flight on several streams (multi-frame throughput mode): two
frames, each with its own encoder and decoder context on its own stream,
interleaved call by call and replayed as HIP graphs, give bit-identical totals
to running them one after the other, and the decoders match the encoders."""
import pytest
import torch

import paper_2503_12382_amd as reno
from gpu_helpers import say
from synth import BY_NAME, gen_scan, gen_weights

pytestmark = pytest.mark.gpu


def _codec(cfg, M, stream, wd):
    mk = lambda: reno.Context(M, cfg.bit_depth, cfg.min_bit_depth, cfg.range_m, cfg.channels,
                              cfg.layers, stream=stream)
    with torch.cuda.stream(stream):
        enc, dec = mk(), mk()
        enc.set_weights(wd)
        dec.set_weights(wd)
    return enc, dec


def _inputs(enc, pts, cfg):
    B, b0 = cfg.bit_depth, cfg.min_bit_depth
    enc.build_pyramid(pts, B)
    codes = {b: enc.occupancy_codes(b).clone() for b in range(b0, B)}
    base, _ = enc.coords(b0)
    return base.clone(), codes


def _step(enc, dec, pts, base, codes, cfg):
    B, b0 = cfg.bit_depth, cfg.min_bit_depth
    enc.build_pyramid(pts, B)
    enc.predict_probs(reno.RENO_ALL_SCALES)
    dec.set_base(B, base, codes[b0])
    for b in range(b0 + 1, B):
        dec.expand(b - 1, None if b - 1 == b0 else codes[b - 1])
        dec.predict_probs(b)
    dec.expand(B - 1, codes[B - 1])


def _totals(enc, dec):
    _, e = enc.code_length(reno.RENO_ALL_SCALES, per_voxel=False)
    _, d = dec.code_length(reno.RENO_ALL_SCALES, per_voxel=False)
    return e, d


def test_two_frames_on_two_streams():
    cfg = BY_NAME["stream10_hdl64_b14"]
    w = reno.weights_to_device(gen_weights(cfg.channels, cfg.layers, seed=cfg.weight_seed))
    frames = [torch.from_numpy(gen_scan(cfg, f)).cuda() for f in (0, 3)]
    M = max(int(f.shape[0]) for f in frames)
    s = [torch.cuda.Stream(), torch.cuda.Stream()]
    # reference: one after the other on one stream
    say("streams: sequential reference")
    ref = []
    enc, dec = _codec(cfg, M, s[0], w)
    with torch.cuda.stream(s[0]):
        for f in frames:
            base, codes = _inputs(enc, f, cfg)
            _step(enc, dec, f, base, codes, cfg)
            ref.append(_totals(enc, dec))
    enc.close()
    dec.close()
    assert ref[0][0] == ref[0][1] and ref[1][0] == ref[1][1] and ref[0][0] != ref[1][0]
    # concurrent: one codec per frame and stream, calls interleaved
    say("streams: interleaved eager, then graph replays")
    cs = [_codec(cfg, M, s[i], w) for i in range(2)]
    ins = []
    for i, f in enumerate(frames):
        with torch.cuda.stream(s[i]):
            ins.append(_inputs(cs[i][0], f, cfg))
    for rep in range(2):
        for i, f in enumerate(frames):
            with torch.cuda.stream(s[i]):
                _step(*cs[i], f, *ins[i], cfg)
    torch.cuda.synchronize()
    for i in range(2):
        with torch.cuda.stream(s[i]):
            assert _totals(*cs[i]) == ref[i]
    graphs = []
    for i, f in enumerate(frames):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=s[i]):
            _step(*cs[i], f, *ins[i], cfg)
        graphs.append(g)
    for rep in range(3):
        for i in range(2):
            with torch.cuda.stream(s[i]):
                graphs[i].replay()
        torch.cuda.synchronize()
        for i in range(2):
            with torch.cuda.stream(s[i]):
                assert _totals(*cs[i]) == ref[i], (rep, i)
    for enc, dec in cs:
        enc.close()
        dec.close()
