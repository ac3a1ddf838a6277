"""A 64-frame batch of the streaming workload (the 14-bit 64-beam generator,
sensor moving 1 m per frame; its ten distinct scans cycled) in one key space:
about 8M points and 15M model voxels, so the conv launches run in their
chunk-capped tile mode (more than 256 x 256 tiles per launch) and the sort in
its large-tile mode.  Against the oracle, frame by frame: every scale's keys,
coordinates and codes bit-exact (hence exact per-frame counts), neighbour
maps, logits and per-voxel bits on sampled rows of every frame of every model
scale, and the batch's total bits; then the batched decoder from the frames'
initial states and the encoder's codes, bit-identical to the encoder on every
scale (keys, logits, bits, total)."""
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest
import torch

import oracle
import paper_2503_12382_amd as reno
from gpu_helpers import BITS_ABS_TOL, BITS_REL_TOL, LOGIT_TOL, say, to_dev
from synth import CONFIGS, gen_weights

pytestmark = pytest.mark.gpu

K = 64
ROWS_PER_FRAME = 24       # sampled rows per frame and model scale


def test_frame_batch_64_matches_oracle_per_frame(scan_cache):
    cfg = CONFIGS[4]
    B, b0 = cfg.bit_depth, cfg.min_bit_depth
    say("stress batch: generating", cfg.frames, "distinct scans")
    scans = [scan_cache(4, f) for f in range(cfg.frames)]
    w = gen_weights(cfg.channels, cfg.layers, seed=cfg.weight_seed + 5, bias_std=0.1)
    # the oracle of each distinct scan (the library calls release the GIL)
    oracle.lib()
    with ThreadPoolExecutor(max_workers=len(scans)) as ex:
        Ps = list(ex.map(lambda s: oracle.Pyramid.from_points(s, B, b0, cfg.range_m), scans))
        Ts = list(ex.map(lambda P: P.totals(w)[0], Ps))
    src = [f % len(scans) for f in range(K)]
    pts = np.concatenate([scans[s] for s in src]).astype(np.float32)
    start = np.cumsum([0] + [len(scans[s]) for s in src]).astype(np.int64)
    model = sum(Ps[s].num(b) for s in src for b in range(b0 + 1, B))
    cap = (model + model // 8 + 4095) // 4096 * 4096
    tiles = -(-max(sum(Ps[s].num(b) for s in src) for b in range(b0 + 1, B)) // 16)
    say(f"stress batch: K={K} points={len(pts)} model voxels={model} "
        f"largest scale {tiles} tiles of 16")
    assert tiles > 256 * 256          # the chunk-capped tile mode of the conv launches
    ctx = reno.Context(len(pts), B, b0, cfg.range_m, cfg.channels, cfg.layers, max_model_voxels=cap)
    ctx.set_weights(reno.weights_to_device(w))
    ctx.build_pyramid_frames(to_dev(pts), to_dev(start), B)
    lg = ctx.predict_probs(reno.RENO_ALL_SCALES, logits=True)
    bits, total = ctx.code_length(reno.RENO_ALL_SCALES)
    ctx.sync()
    rs = np.random.default_rng(64)
    off = 0
    for b in range(b0, B + 1):
        _, keys = ctx.coords(b)
        keys = keys.cpu().numpy().view(np.uint64)
        counts = [Ps[s].num(b) for s in src]
        assert keys.size == sum(counts), (b, keys.size, sum(counts))
        lo = np.cumsum([0] + counts)
        want = np.concatenate([Ps[s].keys(b) | (np.uint64(f) << np.uint64(3 * b))
                               for f, s in enumerate(src)])
        np.testing.assert_array_equal(keys, want, err_msg=f"keys b={b}")
        if b < B:
            codes = ctx.occupancy_codes(b).cpu().numpy()
            np.testing.assert_array_equal(codes, np.concatenate([Ps[s].codes(b) for s in src]),
                                          err_msg=f"codes b={b}")
        if not b0 < b < B:
            continue
        # sampled rows of every frame; the oracle evaluates each distinct
        # scan's union of sampled rows once
        pick = [np.unique(rs.choice(c, size=min(c, ROWS_PER_FRAME), replace=False)) for c in counts]
        ref = {}
        for s in range(len(scans)):
            rows = np.unique(np.concatenate([pick[f] for f in range(K) if src[f] == s]))
            olg, _, obt = Ps[s].model(b, w, rows=rows)
            ref[s] = (rows, olg, obt, Ps[s].neighbors(b)[rows])
        grow = np.concatenate([lo[f] + pick[f] for f in range(K)])
        idx = torch.from_numpy(grow).to("cuda")
        glg = lg[off:off + lo[-1]].index_select(0, idx).cpu().numpy()
        gbt = bits[off:off + lo[-1]].index_select(0, idx).cpu().numpy()
        gnb = ctx.neighbor_map(b).index_select(0, idx).cpu().numpy()
        at, worst = 0, 0.0
        for f in range(K):
            rows, olg, obt, onb = ref[src[f]]
            j = np.searchsorted(rows, pick[f])
            n = pick[f].size
            e = np.abs(glg[at:at + n] - olg[j]).max()
            worst = max(worst, e)
            assert e <= LOGIT_TOL, (b, f, e)
            assert np.abs(gbt[at:at + n] - obt[j]).max() <= BITS_ABS_TOL, (b, f)
            want_nb = np.where(onb[j] >= 0, onb[j] + lo[f], -1)
            np.testing.assert_array_equal(gnb[at:at + n], want_nb, err_msg=f"neighbours b={b} f={f}")
            at += n
        say(f"b={b} rows={lo[-1]} sampled={grow.size} max|dlogit|={worst:.2e}")
        off += lo[-1]
    T = sum(Ts[s] for s in src)
    say(f"total bits gpu={total:.1f} oracle={T:.1f}")
    assert abs(total - T) <= BITS_REL_TOL * T

    # the batched decoder: initial state of every frame plus the encoder's
    # codes -> every scale's keys, every logit and every bit identical to the
    # encoder's (compared on the device)
    say("stress batch: decoder")
    codes = {b: ctx.occupancy_codes(b).clone() for b in range(b0, B)}
    base, bkeys = ctx.coords(b0)
    fid = (bkeys >> (3 * b0)).to(torch.int32).contiguous()
    dec = reno.Context(len(pts), B, b0, cfg.range_m, cfg.channels, cfg.layers, max_model_voxels=cap)
    dec.set_weights(reno.weights_to_device(w))
    dec.set_base_frames(B, base.clone(), fid, codes[b0], K)
    off = 0
    for b in range(b0 + 1, B):
        dec.expand(b - 1, None if b - 1 == b0 else codes[b - 1])
        assert torch.equal(dec.coords(b)[1], ctx.coords(b)[1]), f"decoder keys b={b}"
        dl = dec.predict_probs(b, logits=True)
        n = dl.shape[0]
        assert torch.equal(dl.view(torch.int32), lg[off:off + n].view(torch.int32)), f"decoder logits b={b}"
        off += n
        del dl
    dec.expand(B - 1, codes[B - 1])
    assert torch.equal(dec.coords(B)[1], ctx.coords(B)[1])
    dbits, dtotal = dec.code_length(reno.RENO_ALL_SCALES)
    assert torch.equal(dbits.view(torch.int32), bits.view(torch.int32))
    assert dtotal == total
    dec.close()
    ctx.close()
    del lg, bits, dbits
    torch.cuda.empty_cache()
