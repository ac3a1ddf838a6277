"""Kernel timing through the C ABI (reno_profile / reno_profile_read): the
conv launches of the plain model are timed by events bound to their dispatch,
one interval per launch; other kinds by events recorded around the launch.
Timing changes no result."""
import numpy as np
import pytest
import torch

import paper_2503_12382_amd as reno
from gpu_helpers import cfg_dict, encode, make_ctx, say
from synth import CONFIGS, gen_weights

pytestmark = pytest.mark.gpu


def test_profile_counts_and_intervals(scan_cache):
    cfg = CONFIGS[1]
    B, b0 = cfg.bit_depth, cfg.min_bit_depth
    pts = scan_cache(1)
    w = reno.weights_to_device(gen_weights(cfg.channels, cfg.layers, seed=cfg.weight_seed, bias_std=0.1))
    say("profile", cfg.name)
    ctx = make_ctx(cfg_dict(cfg), len(pts))
    ctx.set_weights(w)
    encode(ctx, pts, B)
    ref = ctx.predict_probs(reno.RENO_ALL_SCALES, logits=True).cpu().numpy()
    ctx.profile(["conv_first", "conv_last", "sort", "codes"])
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    t0.record()
    reps = 5
    for _ in range(reps):
        ctx.build_pyramid(ctx._points, B)
        got = ctx.predict_probs(reno.RENO_ALL_SCALES, logits=True)
        for b in range(b0 + 1, B):
            ctx.predict_probs(b)                     # one launch per layer and scale
    t1.record()
    prof = ctx.profile_read()
    wall = t0.elapsed_time(t1)
    ctx.profile([])
    nscales = B - b0 - 1
    assert prof["conv_last"][1] == reps * (1 + nscales)
    assert prof["conv_first"][1] == reps * (1 + nscales)
    assert prof["codes"][1] == reps
    for k, (ms, n) in prof.items():
        say(f"  {k}: {n} launches, {1000 * ms / n:.1f} us avg")
        assert 0.0 < ms < wall, (k, ms, wall)
    assert np.array_equal(got.cpu().numpy().view(np.uint32), ref.view(np.uint32))
    ctx.close()
