"""The allocation-free FCG expansion (reno_expand_noalloc) against the
context entry point reno_expand on the same parents: children keys and parent
rows bit-exact, on two calls in a row sharing the device scratch, the second
with a smaller input; first-child rows, capacity and zero-code errors, an
empty input, and a good call after each error."""
import numpy as np
import pytest
import torch

import oracle
import paper_2503_12382_amd as reno
from gpu_helpers import cfg_dict, encode, make_ctx, say, to_dev
from synth import CONFIGS

pytestmark = pytest.mark.gpu


def _buffers(cap, n):
    dev = "cuda"
    return (torch.full((cap,), -1, dtype=torch.int64, device=dev),
            torch.full((cap,), -7, dtype=torch.int32, device=dev),
            torch.full((n,), -3, dtype=torch.int32, device=dev),
            torch.full((2,), 99, dtype=torch.int64, device=dev))


def _call(keys, codes, ck, cp, res, fc=None):
    reno.expand_noalloc(keys, codes, ck, cp, res, first_child=fc)
    torch.cuda.synchronize()
    return int(res[0].item()), int(res[1].item())


def test_expand_noalloc_matches_expand(scan_cache):
    cfg = CONFIGS[2]
    B, b0 = cfg.bit_depth, cfg.min_bit_depth
    pts = scan_cache(2)
    say("noalloc expand: encoder", cfg.name)
    enc = make_ctx(cfg_dict(cfg), len(pts))
    encode(enc, pts, B)
    keys = {b: enc.coords(b)[1].clone() for b in range(b0, B + 1)}
    codes = {b: enc.occupancy_codes(b).clone() for b in range(b0, B)}
    say("noalloc expand: decoder through reno_expand")
    dec = make_ctx(cfg_dict(cfg), len(pts))
    base, _ = enc.coords(b0)
    dec.set_base(B, base.clone(), codes[b0])
    ref = {}
    for b in range(b0, B):
        dec.expand(b, None if b == b0 else codes[b])
        ref[b + 1] = (dec.coords(b + 1)[1].cpu().numpy(), dec.parent_rows(b + 1).cpu().numpy())
    P = oracle.Pyramid.from_points(pts, B, b0, cfg.range_m)

    # two calls in a row on the same output buffers, the second smaller
    cap = int(keys[B].shape[0]) + 100
    ck, cp, fc, res = _buffers(cap, int(keys[B - 1].shape[0]))
    for b in (B - 1, 9):
        n = int(keys[b].shape[0])
        say(f"noalloc expand: scale {b} -> {b + 1}, {n} parents")
        nc, st = _call(keys[b], codes[b], ck, cp, res, fc[:n])
        rk, rp = ref[b + 1]
        assert st == reno.RENO_OK and nc == rk.size, (b, nc, st, rk.size)
        got_k = ck[:nc].cpu().numpy().view(np.uint64)
        np.testing.assert_array_equal(got_k, rk.view(np.uint64), err_msg=f"child keys b={b}")
        np.testing.assert_array_equal(got_k, P.keys(b + 1), err_msg=f"oracle keys b={b}")
        np.testing.assert_array_equal(cp[:nc].cpu().numpy(), rp, err_msg=f"parent rows b={b}")
        np.testing.assert_array_equal(fc[:n].cpu().numpy(),
                                      np.searchsorted(rp, np.arange(n)).astype(np.int32))
        if b == B - 1:   # nothing written past the children
            assert bool((ck[nc:] == -1).all()) and bool((cp[nc:] == -7).all())

    # capacity too small: the children are clamped and the error reported
    b = B - 1
    n = int(keys[b].shape[0])
    small = 1000
    ck2, cp2, _, res2 = _buffers(small, 1)
    nc, st = _call(keys[b], codes[b], ck2, cp2, res2)
    assert st == reno.RENO_E_CAPACITY and nc == small
    np.testing.assert_array_equal(ck2.cpu().numpy().view(np.uint64), ref[b + 1][0][:small].view(np.uint64))
    # a zero code
    bad = codes[b].clone()
    bad[n // 2] = 0
    nc, st = _call(keys[b], bad, ck, cp, res)
    assert st == reno.RENO_E_INPUT
    # an empty input
    nc, st = _call(keys[b][:0], codes[b][:0], ck, cp, res)
    assert (nc, st) == (0, reno.RENO_OK)
    # a good call after the errors: bit-exact again
    nc, st = _call(keys[b], codes[b], ck, cp, res)
    assert st == reno.RENO_OK
    np.testing.assert_array_equal(ck[:nc].cpu().numpy().view(np.uint64), ref[b + 1][0].view(np.uint64))
    enc.close()
    dec.close()


def test_expand_noalloc_frame_batch_keys(scan_cache):
    """Keys carrying frame ids above the Morton bits expand per frame exactly
    as the context's batched decoder does."""
    cfg = CONFIGS[1]
    B, b0 = cfg.bit_depth, cfg.min_bit_depth
    scan = scan_cache(1)
    frames = [scan, scan[: len(scan) // 3]]
    pts = np.concatenate(frames).astype(np.float32)
    start = np.cumsum([0] + [len(f) for f in frames]).astype(np.int64)
    say("noalloc expand: frame batch", [len(f) for f in frames])
    ctx = make_ctx(cfg_dict(cfg), len(pts))
    ctx.build_pyramid_frames(to_dev(pts), to_dev(start), B)
    ctx.sync()
    b = B - 2
    keys, codes = ctx.coords(b)[1].clone(), ctx.occupancy_codes(b).clone()
    want_k = ctx.coords(b + 1)[1].cpu().numpy()
    want_p = ctx.parent_rows(b + 1).cpu().numpy()
    ck, cp, _, res = _buffers(want_k.size, 1)
    nc, st = _call(keys, codes, ck, cp, res)
    assert st == reno.RENO_OK and nc == want_k.size
    np.testing.assert_array_equal(ck.cpu().numpy(), want_k)
    np.testing.assert_array_equal(cp.cpu().numpy(), want_p)
    ctx.close()
