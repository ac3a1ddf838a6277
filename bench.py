#!/usr/bin/env python3
"""Throughput of the RENO codec hot path on one MI355X.

One step = one frame encoded and decoded through the C ABI:
  encode: build_pyramid (quantise, sort, all scales, FOG codes)
          -> predict_probs on every model scale in one batch -> code_length
  decode: set_base (initial state) -> for each scale: expand, predict_probs
          -> final expand -> code_length
The decoder's symbols are injected from the encoder (a stand-in for an
instant entropy decoder; the host rANS round trip is covered by the tests).
Inputs are resident in device memory before the timed region.  The default
timed region replays the step as one HIP graph; --mode eager launches it
call by call.

Prints ONE JSON line (rank 0, N=1).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_FP32_MFMA_TFLOPS = 157.3
PEAK_BF16_MFMA_TFLOPS = 2500.0
PEAK_HBM_GBS = 8000.0
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "conv_last_traffic_hdl64_b14.txt")
TRACE_FILE = os.path.join(ROOT, "profiles", "conv_last_headline_trace_hdl64_b14.txt")
MODEL_SRCS = [os.path.join(ROOT, "paper_2503_12382_amd", "csrc", f) for f in ("k_model.hip", "dev.h", "ctx.h")]
# a neighbour-map row as the method defines it: 27 int32 entries (the stored
# rows are padded to 32 for alignment; the padding is not algorithmic traffic)
MAP_ROW_BYTES = 4 * 27
# interleaved rANS streams per scale (and stage) in the end-to-end coder
STREAM_SYMBOLS = 1024  # whole-frame coding: symbols per rANS stream


def alg_bytes_per_frame(counts, b0, B, M, C, hash_slots, status_words):
    """Minimum HBM bytes per frame (encoder + decoder) of each kernel kind:
    every input read once, every output written once.  Gathers of
    neighbour rows and hash probes that hit cached lines are not counted, so
    these are lower bounds on the traffic."""
    N = {b0 + i: n for i, n in enumerate(counts)}
    model = [b for b in range(b0 + 1, B)]
    nm = sum(N[b] for b in model)
    parents_hashed = sum(N[b] for b in range(b0, B - 1))
    passes = (3 * B + 7) // 8
    row = 4 * C
    out = {}
    clear = 16 * hash_slots + 4 * status_words
    # the decoder clears its frame in the launch that writes a base scale of
    # fewer than 256 voxels (one block), else in a launch of its own
    dec_clear_in_base = N[b0] < 256
    out["zero"] = clear * (1 if dec_clear_in_base else 2)
    out["quantize"] = M * (12 + 8)
    out["sort"] = passes * M * 16
    out["pyramid"] = M * 8 + sum(N[b] * 12 for b in range(b0, B + 1)) + sum(N[b] * 4 for b in range(b0, B))
    # codes: child keys read, codes + child feature words written, parents hashed
    out["codes"] = sum(N[b + 1] * (8 + 2) + N[b] for b in range(b0, B)) + 16 * parents_hashed
    out["set_base"] = N[b0] * (12 + 1 + 8) + (clear if dec_clear_in_base else 0)
    # expand: parent key + code read; child key, parent row, feature word and the
    # parent's first-child row written; parents hashed
    out["expand"] = sum(N[b] * (8 + 1 + 4) + N[b + 1] * (8 + 4 + 2) for b in range(b0, B)) + \
        16 * parents_hashed
    # conv layers (encoder + decoder): first reads keys, parent slots and feature
    # words, writes the neighbour map and h; later layers read map + h, write h
    first = sum(N[b] * (8 + 2 + MAP_ROW_BYTES + row) + 16 * N[b - 1] for b in model)
    mid = nm * (MAP_ROW_BYTES + 2 * row)
    out["conv_first"] = 2 * first
    out["conv_mid"] = 2 * mid
    out["conv_last"] = 2 * (mid + nm * 4)
    out["code_length"] = 2 * nm * (1 + 4 + row)
    return out


def alg_bytes_encoder(counts, b0, B, M, C, hash_slots, status_words, fb):
    """Minimum HBM bytes of one encoder pass over a frame batch (every input
    read once, every output written once), per kernel kind.  The sort's
    minimum is one read and one write per key; its LSD passes (over the 3B
    Morton bits and the fb frame-id bits) each move that much, reported
    separately."""
    N = {b0 + i: n for i, n in enumerate(counts)}
    model = [b for b in range(b0 + 1, B)]
    nm = sum(N[b] for b in model)
    parents_hashed = sum(N[b] for b in range(b0, B - 1))
    row = 4 * C
    return {
        "zero": 16 * hash_slots + 4 * status_words,
        "quantize": M * (12 + 8),
        "sort": M * 16,
        "pyramid": M * 8 + sum(N[b] * 12 for b in range(b0, B + 1)) + sum(N[b] * 4 for b in range(b0, B)),
        "codes": sum(N[b + 1] * (8 + 2) + N[b] for b in range(b0, B)) + 16 * parents_hashed,
        "conv_first": sum(N[b] * (8 + 2 + MAP_ROW_BYTES + row) + 16 * N[b - 1] for b in model),
        "conv_mid": nm * (MAP_ROW_BYTES + 2 * row),
        "conv_last": nm * (MAP_ROW_BYTES + 2 * row) + nm * 4,
        "code_length": nm * (1 + 4 + row),
    }


def model_source_hash():
    """sha256 prefix of the sources the conv kernels are built from (the
    launcher declarations of ctx.h, which other files' changes add to, are
    left out)."""
    import hashlib
    h = hashlib.sha256()
    for f in MODEL_SRCS:
        text = open(f, "rb").read()
        if f.endswith("ctx.h"):
            text = text.split(b"\nhipError_t launch_", 1)[0]
        h.update(text)
    return h.hexdigest()[:16]


def read_profile_kv(path, workload):
    """key = value lines of a committed rocprofv3 summary, or None when the
    kernel sources changed since it was taken or it covers another workload."""
    if not os.path.exists(path):
        return None
    kv = {}
    for line in open(path):
        if "=" in line and not line.startswith("#"):
            k, v = line.split("=", 1)
            kv[k.strip()] = v.strip()
    if kv.get("model_sources_sha256_16") != model_source_hash() or kv.get("workload") != workload:
        return None
    return kv


def read_traffic(workload):
    """HBM traffic of conv_last per launch from the committed rocprofv3 PMC
    summary (FETCH_SIZE and WRITE_SIZE runs scaled by a copy kernel's counts),
    or None when it is stale."""
    kv = read_profile_kv(TRAFFIC_FILE, workload)
    return None if kv is None else float(kv["bytes_per_launch"])


def read_trace(workload):
    """conv_last's average dispatch duration (us) and dispatch count from the
    committed rocprofv3 kernel trace of this bench's headline run alone
    (--headline-only), or None when it is stale."""
    kv = read_profile_kv(TRACE_FILE, workload)
    return None if kv is None else (float(kv["avg_us"]), int(kv["dispatches"]))


def measure_copy_peak(torch, dev, stream, mib=2048, reps=20):
    """Device-to-device copy bandwidth (GB/s counting the bytes read and the
    bytes written), the measured stand-in for the HBM peak beside the nominal
    8 TB/s."""
    n = mib << 20
    src = torch.empty(n, dtype=torch.uint8, device=dev)
    dst = torch.empty(n, dtype=torch.uint8, device=dev)
    src.fill_(1)
    with torch.cuda.stream(stream):
        for _ in range(3):
            dst.copy_(src)
        t0 = torch.cuda.Event(enable_timing=True)
        t1 = torch.cuda.Event(enable_timing=True)
        t0.record(stream)
        for _ in range(reps):
            dst.copy_(src)
        t1.record(stream)
    stream.synchronize()
    gbs = 2.0 * n * reps / (t0.elapsed_time(t1) * 1e-3) / 1e9
    del src, dst
    torch.cuda.empty_cache()
    return gbs


def host_info():
    """Core count and CPU model of the host the oracle baseline runs on."""
    model = None
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return {"nproc": os.cpu_count(), "affinity_cpus": len(os.sched_getaffinity(0)), "cpu_model": model}


def oracle_frame(args):
    """One frame through the oracle (encode: pyramid, codes, model, bits;
    decode: FCG expansion, model, bits); returns (T, t_enc, t_dec)."""
    cfg_name, seed_shift = args
    import oracle
    from synth import BY_NAME, gen_scan, gen_weights
    cfg = BY_NAME[cfg_name]
    pts = gen_scan(cfg)
    w = gen_weights(cfg.channels, cfg.layers, seed=cfg.weight_seed)
    B, b0 = cfg.bit_depth, cfg.min_bit_depth
    t = time.perf_counter()
    P = oracle.Pyramid.from_points(pts, B, b0, cfg.range_m)
    T_enc, _ = P.totals(w)
    t_enc = time.perf_counter() - t
    t = time.perf_counter()
    D = oracle.Pyramid.from_codes(P.xyz(b0), b0, B, [P.codes(b) for b in range(b0, B)])
    T_dec, _ = D.totals(w)
    t_dec = time.perf_counter() - t
    return T_enc, T_dec, t_enc, t_dec


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


class Codec:
    """An encoder and a decoder context on one stream and one encode + decode
    step over a resident frame.  The decoder's symbols come from the encoder
    (a stand-in for an instant entropy decoder)."""

    def __init__(self, reno, torch, cfg, pts, M, cap_model, stream, w_np, two_stage, precision=0, top=False,
                 frame_start=None, channels=None, kernel_size=3):
        self.reno, self.torch, self.stream = reno, torch, stream
        B, b0, C, L = cfg.bit_depth, cfg.min_bit_depth, channels or cfg.channels, cfg.layers
        self.B, self.b0, self.C, self.two_stage = B, b0, C, two_stage
        self.frame_start = frame_start     # a frame batch (int64 device tensor [K + 1]) or None
        self.K = 1 if frame_start is None else int(frame_start.shape[0]) - 1
        wd = reno.weights_to_device(w_np)
        with torch.cuda.stream(stream):
            mk = lambda: reno.Context(M, B, b0, cfg.range_m, C, L, max_model_voxels=cap_model,
                                      stream=stream, two_stage=two_stage, precision=precision, top=top,
                                      kernel_size=kernel_size)
            self.enc, self.dec = mk(), mk()
            self.enc.set_weights(wd)
            self.dec.set_weights(wd)
            # decoder inputs (resident before timing): initial state and every scale's codes
            self.build(pts)
            base, keys = self.enc.coords(b0)
            self.base = base.clone()
            self.fid = (keys >> (3 * b0)).to(torch.int32).contiguous()  # frame ids of a batch
            self.codes = {b: self.enc.occupancy_codes(b).clone() for b in range(b0, B)}
            self.s1 = {b: (self.codes[b] & 15).contiguous() for b in range(b0, B)}
            self.enc.predict_probs(reno.RENO_ALL_SCALES)
            _, self.enc_total = self.enc.code_length(reno.RENO_ALL_SCALES, per_voxel=False)
            self.pairs = {b: int((self.enc.neighbor_map(b) >= 0).sum().item()) for b in range(b0 + 1, B)}
            stream.synchronize()
        self.pts = pts
        self.graph = None

    def build(self, pts):
        if self.frame_start is None:
            self.enc.build_pyramid(pts, self.B)
        else:
            self.enc.build_pyramid_frames(pts, self.frame_start, self.B)

    def step(self):
        self.enc_step()
        self.dec_step()

    def enc_step(self):
        reno, enc = self.reno, self.enc
        self.build(self.pts)
        enc.predict_probs(reno.RENO_ALL_SCALES)
        enc.code_length(reno.RENO_ALL_SCALES, per_voxel=False, total=False)

    def dec_step(self):
        reno, dec, B, b0 = self.reno, self.dec, self.B, self.b0
        if self.frame_start is None:
            dec.set_base(B, self.base, self.codes[b0])
        else:
            dec.set_base_frames(B, self.base, self.fid, self.codes[b0], self.K)
        for b in range(b0 + 1, B):
            dec.expand(b - 1, None if b - 1 == b0 else self.codes[b - 1])
            dec.predict_probs(b)
            if self.two_stage:
                dec.predict_second(b, self.s1[b])
        dec.expand(B - 1, self.codes[B - 1])
        dec.code_length(reno.RENO_ALL_SCALES, per_voxel=False, total=False)

    def check(self, what):
        reno = self.reno
        with self.torch.cuda.stream(self.stream):
            _, d = self.dec.code_length(reno.RENO_ALL_SCALES, per_voxel=False)
            _, e = self.enc.code_length(reno.RENO_ALL_SCALES, per_voxel=False)
        if not (d == e == self.enc_total):
            log(what, "decoder/encoder bit totals differ", d, e, self.enc_total)
            sys.exit(1)

    def time(self, steps, warmup, mode):
        """Milliseconds per step over `steps` steps (HIP events on the stream)."""
        torch, stream = self.torch, self.stream
        with torch.cuda.stream(stream):
            for _ in range(warmup):
                self.step()
            stream.synchronize()
        self.check("after warm-up:")
        if mode == "graph" and self.graph is None:
            self.graph = torch.cuda.CUDAGraph()
            with torch.cuda.graph(self.graph, stream=stream):
                self.step()
            with torch.cuda.stream(stream):
                for _ in range(warmup):
                    self.graph.replay()
            stream.synchronize()
        t0 = torch.cuda.Event(enable_timing=True)
        t1 = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        with torch.cuda.stream(stream):
            t0.record(stream)
            for _ in range(steps):
                if mode == "graph":
                    self.graph.replay()
                else:
                    self.step()
            t1.record(stream)
        torch.cuda.synchronize()
        self.check("after the timed steps:")  # the last replayed frame is consistent
        return t0.elapsed_time(t1) / steps

    def frame_times(self, frames):
        """Milliseconds of each of `frames` single graph replays (one frame
        encoded + decoded each), every replay bracketed by its own HIP events."""
        torch, stream = self.torch, self.stream
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(frames)]
        with torch.cuda.stream(stream):
            for a, b in ev:
                a.record(stream)
                self.graph.replay()
                b.record(stream)
        stream.synchronize()
        self.check("after the per-frame timing:")
        return [a.elapsed_time(b) for a, b in ev]

    def time_sides(self, steps):
        """(encoder ms, decoder ms) per frame, each side captured as its own
        HIP graph and replayed `steps` times."""
        torch, stream = self.torch, self.stream
        out = []
        for fn in (self.enc_step, self.dec_step):
            g = torch.cuda.CUDAGraph()
            with torch.cuda.stream(stream):
                fn()
                stream.synchronize()
            with torch.cuda.graph(g, stream=stream):
                fn()
            with torch.cuda.stream(stream):
                g.replay()
            stream.synchronize()
            t0 = torch.cuda.Event(enable_timing=True)
            t1 = torch.cuda.Event(enable_timing=True)
            with torch.cuda.stream(stream):
                t0.record(stream)
                for _ in range(steps):
                    g.replay()
                t1.record(stream)
            torch.cuda.synchronize()
            out.append(t0.elapsed_time(t1) / steps)
        self.check("after the per-side timing:")
        return tuple(out)

    def profile_conv_last(self, steps):
        """(total ms, launches) of conv_last over `steps` eager steps: the
        library launches each timed conv kernel with two HIP events bound to
        its dispatch (hipExtLaunchKernelGGL), so each interval is the kernel's
        execution on the context stream."""
        with self.torch.cuda.stream(self.stream):
            self.enc.profile(["conv_last"])
            self.dec.profile(["conv_last"])
            for _ in range(steps):
                self.step()
            pe, pd = self.enc.profile_read(), self.dec.profile_read()
            self.enc.profile([])
            self.dec.profile([])
        return pe["conv_last"][0] + pd["conv_last"][0], pe["conv_last"][1] + pd["conv_last"][1]

    def conv_last_flops(self, counts):
        """Algorithmic flops of the last conv layer + head per frame (encoder +
        decoder): 2*C*C per occupied neighbour and, per voxel, 2*C*256 (one-stage
        head) or 2*C*16*2 (two stages of 16)."""
        C = self.C
        head = 2 * C * 32 if self.two_stage else 2 * C * 256
        return 2 * sum(2 * C * C * self.pairs[b] + head * counts[b - self.b0] for b in self.pairs)

    def close(self):
        self.enc.close()
        self.dec.close()


class EndToEnd:
    """True end-to-end coding of one frame through the library's whole-frame
    calls: the points copied in from pinned host memory, then
    reno_encode_frame (GPU pyramid + model + symbol intervals + rANS streams)
    into a host bitstream, and reno_decode_frame from that bitstream alone
    (copied in once; per scale expand, predict, cumulative tables and stream
    decoding on the GPU, one synchronisation at the end)."""

    def __init__(self, reno, torch, cfg, pts, M, cap_model, stream, w_np, two_stage, L=STREAM_SYMBOLS):
        self.reno, self.torch, self.stream, self.two, self.L = reno, torch, stream, two_stage, L
        self.B, self.b0 = cfg.bit_depth, cfg.min_bit_depth
        wd = reno.weights_to_device(w_np)
        mk = lambda: reno.Context(M, self.B, self.b0, cfg.range_m, cfg.channels, cfg.layers,
                                  max_model_voxels=cap_model, stream=stream, two_stage=two_stage)
        with torch.cuda.stream(stream):
            self.enc, self.dec = mk(), mk()
            self.enc.set_weights(wd)
            self.dec.set_weights(wd)
        self.pts_host = torch.empty(tuple(pts.shape), dtype=pts.dtype, pin_memory=True)
        self.pts_host.copy_(pts.cpu())
        self.pts = torch.empty_like(pts)
        self.buf = np.empty(2 * M + 65536, np.uint32)

    def encode(self):
        with self.torch.cuda.stream(self.stream):
            self.pts.copy_(self.pts_host, non_blocking=True)
            return self.enc.encode_frame(self.pts, self.B, stream_symbols=self.L, out=self.buf)

    def decode(self, words):
        with self.torch.cuda.stream(self.stream):
            self.dec.decode_frame(words)

    def run(self, frames, check=True):
        """Mean seconds per frame of encode and of decode, coded bits."""
        torch = self.torch
        te = td = 0.0
        bits = None
        for i in range(frames + 1):                        # first pass: warm-up
            t = time.perf_counter()
            words = self.encode()
            t1 = time.perf_counter()
            self.decode(words)
            t2 = time.perf_counter()
            if i:
                te += t1 - t
                td += t2 - t1
            if check and i in (0, frames):
                with torch.cuda.stream(self.stream):
                    same = bool(torch.equal(self.dec.coords(self.B)[0], self.enc.coords(self.B)[0]))
                if not same:
                    log("end-to-end: decoded frame differs from the input")
                    sys.exit(1)
            bits = 32 * words.size
        return te / frames, td / frames, bits

    def close(self):
        self.enc.close()
        self.dec.close()


def e2e_in_flight(reno, torch, args, dev, workers=(1, 2, 3, 4, 8), per_worker=12):
    """Throughput of whole-frame coding with W frames in flight: W host
    threads (the library's calls release the interpreter), each encoding and
    decoding its share of the streaming workload's scans through its own pair
    of contexts on its own stream; every decoded frame is checked."""
    from concurrent.futures import ThreadPoolExecutor
    from synth import BY_NAME, gen_scan, gen_weights
    mcfg = BY_NAME[args.stream_config]
    scans = [gen_scan(mcfg, f) for f in range(mcfg.frames)]
    w = reno.weights_to_device(gen_weights(mcfg.channels, mcfg.layers, seed=mcfg.weight_seed))
    M = max(f.shape[0] for f in scans)
    out = {"workload": f"{mcfg.name}: its {mcfg.frames} distinct scans cycled, one-stage head, "
                       f"L = {STREAM_SYMBOLS}, each frame encoded to host memory and decoded from it", "runs": []}
    # the streams are created once, together, so that the first few land on
    # different hardware queues (the runtime hands queues out in turn)
    pool = [torch.cuda.Stream(device=dev) for _ in range(max(workers))]
    for W in workers:
        lanes = []
        for i in range(W):
            st = pool[i]
            with torch.cuda.stream(st):
                mk = lambda: reno.Context(M, mcfg.bit_depth, mcfg.min_bit_depth, mcfg.range_m, mcfg.channels,
                                          mcfg.layers, stream=st)
                enc, dec = mk(), mk()
                enc.set_weights(w)
                dec.set_weights(w)
                pts = [torch.from_numpy(scans[(i + k * W) % len(scans)]).to(dev) for k in range(per_worker)]
            lanes.append((st, enc, dec, pts, np.empty(2 * M + 65536, np.uint32)))
        torch.cuda.synchronize()

        def work(lane, check=False):
            st, enc, dec, pts, buf = lane
            with torch.cuda.stream(st):
                for p in pts:
                    words = enc.encode_frame(p, mcfg.bit_depth, stream_symbols=STREAM_SYMBOLS, out=buf)
                    dec.decode_frame(words)
                    if check and not torch.equal(dec.coords(mcfg.bit_depth)[0], enc.coords(mcfg.bit_depth)[0]):
                        return False
            return True

        with ThreadPoolExecutor(max_workers=W) as ex:
            if not all(ex.map(lambda l: work(l, True), lanes)):      # warm-up pass, every frame checked
                log("end-to-end in flight: decoded frame differs from the input")
                sys.exit(1)
            t = time.perf_counter()
            list(ex.map(work, lanes))
            dt = time.perf_counter() - t
        n = W * per_worker
        out["runs"].append({"frames_in_flight": W, "frames": n, "frames_per_s": round(n / dt, 1),
                            "ms_per_frame": round(1000 * dt / n, 3)})
        for _, enc, dec, _, _ in lanes:
            enc.close()
            dec.close()
    return out


def run_stress(args, reno, torch, dev, stream, copy_peak=None):
    """HBM stress: K frames of the streaming generator (its distinct frames,
    cycled) batched into one key space, frame id above the Morton bits; one
    encoder pass (pyramid, all model scales, code lengths) per batch, every
    launch bracketed with HIP events.  At K = 512 the keys, levels and
    feature rows far exceed the 256 MB Infinity Cache."""
    from synth import BY_NAME, gen_scan, gen_weights
    scfg = BY_NAME[args.stream_config]
    sframes = [gen_scan(scfg, f) for f in range(scfg.frames)]
    sB, sb0, sC, sL = scfg.bit_depth, scfg.min_bit_depth, scfg.channels, scfg.layers
    sw = reno.weights_to_device(gen_weights(sC, sL, seed=scfg.weight_seed))
    mv = []
    for f in sframes:
        with torch.cuda.stream(stream):
            pr = reno.Context(f.shape[0], sB, sb0, scfg.range_m, sC, sL, stream=stream)
            pr.build_pyramid(torch.from_numpy(f).to(dev), sB)
            mv.append(sum(pr.num_voxels(b) for b in range(sb0 + 1, sB)))
            pr.close()
    stress = {"workload": f"{scfg.name}: K frames (its {len(sframes)} distinct scans cycled) in one key "
                          f"space, {sB}-bit, encoder pass (pyramid, codes + hash, {sL} conv layers + head "
                          "on every model scale, code lengths)", "runs": []}
    skinds = ["zero", "quantize", "sort", "pyramid", "codes", "conv_first", "conv_mid", "conv_last",
              "code_length", "other"]
    ks = [int(x) for x in args.stress.split(",") if x]
    # every K in fp32, and the largest K again with the split-bf16 contraction
    # (about 5x less MFMA time per product than fp32), where the conv layers
    # are no longer bound by the contraction and the gather shows its own rate
    runs = [(K, reno.RENO_PREC_FP32) for K in ks] + ([(max(ks), reno.RENO_PREC_BF16X3)] if ks else [])
    for K, prec in runs:
        sel = [sframes[i % len(sframes)] for i in range(K)]
        start = np.cumsum([0] + [f.shape[0] for f in sel]).astype(np.int64)
        SM = int(start[-1])
        cap = sum(mv[i % len(mv)] for i in range(K))
        cap = (cap + cap // 8 + 4095) // 4096 * 4096
        pts_d = torch.from_numpy(np.concatenate(sel)).to(dev)
        st_d = torch.from_numpy(start).to(dev)
        del sel
        with torch.cuda.stream(stream):
            sc = reno.Context(SM, sB, sb0, scfg.range_m, sC, sL, max_model_voxels=cap, stream=stream,
                              precision=prec)
            sc.set_weights(sw)

            def enc():
                sc.build_pyramid_frames(pts_d, st_d, sB)
                sc.predict_probs(reno.RENO_ALL_SCALES)
                sc.code_length(reno.RENO_ALL_SCALES, per_voxel=False, total=False)

            enc()
            sc.sync()
            reps = max(1, min(20, 64 // K))
            t0 = torch.cuda.Event(enable_timing=True)
            t1 = torch.cuda.Event(enable_timing=True)
            t0.record(stream)
            for _ in range(reps):
                enc()
            t1.record(stream)
            stream.synchronize()
            ms = t0.elapsed_time(t1) / reps
            sc.profile(skinds)
            enc()
            prof = sc.profile_read()
            sc.profile([])
            sc.sync()
            cnt = sc.scale_counts()[sb0:sB + 1].tolist()
            smem = sc.memory_info()
        if sum(cnt[1:-1]) != sum(mv[i % len(mv)] for i in range(K)):
            log("stress K", K, "model voxels of the batch differ from the sum over its frames")
            sys.exit(1)
        fb = max(0, (K - 1).bit_length())
        alg = alg_bytes_encoder(cnt, sb0, sB, SM, sC, smem["hash_slots"], smem["status_words"], fb)
        kinds_out = {}
        for k in skinds:
            if k not in prof:
                continue
            us = 1000.0 * prof[k][0]
            e = {"us": round(us, 1), "launches": prof[k][1]}
            if k in alg:
                gbs = alg[k] / (us * 1e-6) / 1e9
                e.update({"alg_MB": round(alg[k] / 1e6, 2), "alg_GBs": round(gbs, 1),
                          "hbm_frac": round(gbs / PEAK_HBM_GBS, 4)})
                if copy_peak:
                    e["hbm_frac_of_copy"] = round(gbs / copy_peak, 4)
            if k == "sort":  # every LSD pass reads and writes each key once
                passes = (3 * sB + fb + 7) // 8
                pgbs = passes * alg[k] / (us * 1e-6) / 1e9
                e.update({"passes": passes, "pass_MB": round(passes * alg[k] / 1e6, 2),
                          "pass_GBs": round(pgbs, 1), "pass_hbm_frac": round(pgbs / PEAK_HBM_GBS, 4)})
                if copy_peak:
                    e["pass_hbm_frac_of_copy"] = round(pgbs / copy_peak, 4)
            kinds_out[k] = e
        run = {"K": K, "precision": "fp32" if prec == reno.RENO_PREC_FP32 else "bf16x3",
               "points": SM, "voxels": int(sum(cnt)), "model_rows_capacity": cap,
               "device_bytes": smem["device_bytes"], "encoder_ms_per_batch": round(ms, 4),
               "encoder_frames_per_s": round(K * 1000.0 / ms, 1), "kinds": kinds_out}
        stress["runs"].append(run)
        log("stress K", K, run["precision"],
            {k: (v["us"], v.get("pass_hbm_frac", v.get("hbm_frac"))) for k, v in kinds_out.items()},
            f"{ms:.3f} ms/batch")
        sc.close()
        del pts_d, st_d
        torch.cuda.empty_cache()
    stress["note"] = ("hbm_frac = algorithmic bytes (each input read once, each output written once) / "
                      "kernel time / 8 TB/s (hbm_frac_of_copy: / the measured device copy rate); sort = all LSD passes (pass_* count every pass's read + write), "
                      "codes = code words + hash build, conv_first = hash probes + first-layer gather, "
                      "conv_mid = neighbour-row gather")

    return stress


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawTextHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--config", default="hdl64_b14")
    ap.add_argument("--mode", choices=["graph", "eager"], default="graph")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-two-stage", action="store_true", help="skip the two-stage head measurement")
    ap.add_argument("--no-bf16x3", action="store_true", help="skip the split-bf16 precision measurement")
    ap.add_argument("--no-top", action="store_true", help="skip the full-predictor measurement")
    ap.add_argument("--stress-only", action="store_true",
                    help="run only the HBM stress pass and print its JSON (for counter runs)")
    ap.add_argument("--stress", default="1,8,64,512",
                    help="frame-batch sizes K of the HBM stress pass (encoder stages on K frames in one key "
                         "space); empty to skip")
    ap.add_argument("--e2e-frames", type=int, default=20,
                    help="frames for the end-to-end measurement through the whole-frame calls (0 to skip)")
    ap.add_argument("--in-flight", default="1,2,3,4,8",
                    help="frames in flight (host threads) for the end-to-end throughput measurement "
                         "('' to skip)")
    ap.add_argument("--stream-config", default="stream10_hdl64_b14",
                    help="multi-frame workload measured with frames in flight on several streams")
    ap.add_argument("--streams", default="1,2,4",
                    help="stream counts for the multi-frame measurement ('' to skip)")
    ap.add_argument("--cpu-workers", type=int, default=0,
                    help="processes for the all-cores oracle baseline (0: the CPUs this process may use, at most 16)")
    ap.add_argument("--headline-only", action="store_true",
                    help="only the headline timed region (warm-up, graph capture, timed replays): the run "
                         "whose rocprofv3 kernel trace gives conv_last's per-dispatch duration")
    ap.add_argument("--calib-copy", action="store_true",
                    help="run one 256 MiB device-to-device copy first (counter calibration for PMC runs)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}): frames are independent, "
              "so multi-GPU throughput is N independent copies of this line; no multi-GPU "
              "path is built.", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2503_12382_amd as reno
    from synth import BY_NAME, gen_scan, gen_weights

    cfg = BY_NAME[args.config]
    B, b0, C, L = cfg.bit_depth, cfg.min_bit_depth, cfg.channels, cfg.layers
    log("generating", cfg.name)
    pts_np = gen_scan(cfg)
    M = pts_np.shape[0]
    w_np = gen_weights(C, L, seed=cfg.weight_seed)
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    stream = torch.cuda.Stream(device=dev)
    pts = torch.from_numpy(pts_np).to(dev)
    if args.stress_only:
        if args.calib_copy:
            src = torch.ones(64 << 20, dtype=torch.float32, device=dev)
            dst = torch.empty_like(src)
            torch.mul(src, 1.0, out=dst)
            torch.cuda.synchronize()
            del src, dst
        cp = measure_copy_peak(torch, dev, stream)
        print(json.dumps({"hbm_copy_peak_GBs": round(cp, 1),
                          "hbm_stress": run_stress(args, reno, torch, dev, stream, cp)}), flush=True)
        return
    if args.calib_copy:
        # plain kernels of known traffic: a fill (256 MiB written), then an
        # elementwise copy (256 MiB read, 256 MiB written)
        src = torch.ones(64 << 20, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.mul(src, 1.0, out=dst)
        torch.cuda.synchronize()
        log("calibration: fill writes 268435456 bytes; copy reads and writes 268435456 bytes")
        del src, dst

    # probe pass with the always-sufficient capacity to learn this sensor's
    # model-voxel count; the timed contexts are sized to it (+12.5 %)
    with torch.cuda.stream(stream):
        probe = reno.Context(M, B, b0, cfg.range_m, C, L, stream=stream)
        probe.build_pyramid(pts, B)
        counts = [probe.num_voxels(b) for b in range(b0, B + 1)]
        probe.close()
    model_vox = sum(counts[1:-1])
    cap_model = (model_vox + model_vox // 8 + 4095) // 4096 * 4096
    log("N_b", counts, "model voxels", model_vox, "capacity", cap_model)

    one = Codec(reno, torch, cfg, pts, M, cap_model, stream, w_np, two_stage=False)
    enc, dec, step = one.enc, one.dec, one.step
    pairs, enc_total = one.pairs, one.enc_total
    ms_step = one.time(args.steps, args.warmup, args.mode)
    fps = 1000.0 / ms_step
    log(f"{args.mode}: {ms_step * 1000:.1f} us/frame, {fps:.1f} frames/s")
    if args.headline_only:
        print(json.dumps({"metric": "frames/s (headline timed region only)", "value": round(fps, 2),
                          "unit": "frames/s", "ms_per_step": round(ms_step, 5), "steps": args.steps,
                          "warmup": args.warmup, "mode": args.mode, "workload": cfg.name,
                          "conv_last_launches_per_frame": 1 + (B - b0 - 1)}), flush=True)
        one.close()
        return
    per_frame = one.frame_times(50) if args.mode == "graph" else None
    if per_frame:
        med = float(np.median(per_frame))
        log(f"per-frame graph replays: median {med * 1000:.1f} us over {len(per_frame)} frames")
    enc_ms, dec_ms = one.time_sides(args.steps) if args.mode == "graph" else (None, None)
    if enc_ms is not None:
        log(f"encode {enc_ms * 1000:.1f} us, decode {dec_ms * 1000:.1f} us per frame")
    cl_ms, cl_launches = one.profile_conv_last(args.steps)
    achieved_tflops = one.conv_last_flops(counts) * args.steps / (cl_ms * 1e-3) / 1e12
    log(f"conv_last: {cl_launches} launches, {1000 * cl_ms / cl_launches:.1f} us avg, "
        f"{achieved_tflops:.2f} TFLOP/s algorithmic")

    # per-kind breakdown over 20 eager frames (all kernels bracketed)
    kinds = reno.KERNELS
    nb = 20
    with torch.cuda.stream(stream):
        enc.profile(kinds)
        dec.profile(kinds)
        for _ in range(nb):
            step()
        be, bd = enc.profile_read(), dec.profile_read()
        enc.profile([])
        dec.profile([])
    mem = enc.memory_info()
    alg = alg_bytes_per_frame(counts, b0, B, M, C, mem["hash_slots"], mem["status_words"])
    copy_peak = measure_copy_peak(torch, dev, stream)
    log(f"measured device copy: {copy_peak:.0f} GB/s (read + write)")
    breakdown = {}
    for k in kinds:
        ms = be.get(k, (0.0, 0))[0] + bd.get(k, (0.0, 0))[0]
        n = be.get(k, (0.0, 0))[1] + bd.get(k, (0.0, 0))[1]
        if n:
            us = 1000.0 * ms / nb
            breakdown[k] = {"us_per_frame": round(us, 2), "launches_per_frame": n // nb}
            if k in alg:
                gbs = alg[k] / (us * 1e-6) / 1e9
                breakdown[k].update({"alg_bytes_per_frame": alg[k], "alg_GBs": round(gbs, 1),
                                     "hbm_frac": round(gbs / PEAK_HBM_GBS, 4),
                                     "hbm_frac_of_copy": round(gbs / copy_peak, 4)})

    # ---- the bitwise two-stage head (the paper's default head), same frame ----
    two = None
    if not args.no_two_stage:
        w2_np = gen_weights(C, L, seed=cfg.weight_seed, two_stage=True)
        ts = Codec(reno, torch, cfg, pts, M, cap_model, stream, w2_np, two_stage=True)
        st = max(args.steps // 2, 1)
        ms2 = ts.time(st, args.warmup, args.mode)
        cl2_ms, cl2_n = ts.profile_conv_last(st)
        tf2 = ts.conv_last_flops(counts) * st / (cl2_ms * 1e-3) / 1e12
        two = {"value": round(1000.0 / ms2, 2), "unit": "frames/s", "ms_per_step": round(ms2, 5),
               "steps": st, "bits_per_point": round(ts.enc_total / M, 4),
               "conv_last_avg_launch_us": round(1000 * cl2_ms / cl2_n, 2),
               "conv_last_achieved_tflops": round(tf2, 3),
               "conv_last_frac": round(tf2 / PEAK_FP32_MFMA_TFLOPS, 4)}
        log("two-stage head", two)
        ts.close()

    # ---- split-bf16 precision (bf16 hi + lo operands, three bf16 MFMA products
    # per fp32 product), same frame and weights ----
    bfx = None
    if not args.no_bf16x3:
        bc = Codec(reno, torch, cfg, pts, M, cap_model, stream, w_np, two_stage=False,
                   precision=reno.RENO_PREC_BF16X3)
        st = max(args.steps // 2, 1)
        msb = bc.time(st, args.warmup, args.mode)
        clb_ms, clb_n = bc.profile_conv_last(st)
        tfb = bc.conv_last_flops(counts) * st / (clb_ms * 1e-3) / 1e12
        bfx = {"value": round(1000.0 / msb, 2), "unit": "frames/s", "ms_per_step": round(msb, 5),
               "steps": st, "dtype": "bf16x3 (fp32 accumulate)",
               "bits_per_point": round(bc.enc_total / M, 4),
               "bits_rel_diff_vs_fp32": abs(bc.enc_total - enc_total) / enc_total,
               "conv_last_avg_launch_us": round(1000 * clb_ms / clb_n, 2),
               "conv_last_achieved_tflops": round(tfb, 3),
               "conv_last_frac_of_bf16_peak": round(tfb / PEAK_BF16_MFMA_TFLOPS, 4)}
        log("bf16x3", bfx)
        bc.close()

    # ---- the full target occupancy predictor (occupancy embedding and a
    # residual block on the parent scale, replication + octant embedding and a
    # residual block on the target scale), both heads, same frame ----
    topm = None
    if not args.no_top:
        topm = {}
        for name, is_two in (("one_stage", False), ("two_stage", True)):
            wt = gen_weights(C, L, seed=cfg.weight_seed, two_stage=is_two, top=True)
            tc = Codec(reno, torch, cfg, pts, M, cap_model, stream, wt, two_stage=is_two, top=True)
            st = max(args.steps // 2, 1)
            mst = tc.time(st, args.warmup, args.mode)
            clt_ms, clt_n = tc.profile_conv_last(st)
            tft = tc.conv_last_flops(counts) * st / (clt_ms * 1e-3) / 1e12
            with torch.cuda.stream(stream):
                tc.enc.profile(kinds)
                tc.dec.profile(kinds)
                for _ in range(nb):
                    tc.step()
                pe, pd = tc.enc.profile_read(), tc.dec.profile_read()
                tc.enc.profile([])
                tc.dec.profile([])
            kinds_us = {k: round(1000.0 * (pe.get(k, (0.0, 0))[0] + pd.get(k, (0.0, 0))[0]) / nb, 2)
                        for k in kinds if k in pe or k in pd}
            topm[name] = {"value": round(1000.0 / mst, 2), "unit": "frames/s", "ms_per_step": round(mst, 5),
                          "steps": st, "bits_per_point": round(tc.enc_total / M, 4),
                          "conv_last_avg_launch_us": round(1000 * clt_ms / clt_n, 2),
                          "conv_last_achieved_tflops": round(tft, 3),
                          "conv_last_frac": round(tft / PEAK_FP32_MFMA_TFLOPS, 4),
                          "us_per_frame_by_kind": kinds_us}
            log("full predictor", name, topm[name])
            tc.close()
        # the large variant (c128, k5; the paper's RENO-L) with the two-stage
        # head: streamed-weight conv kernels and a separate head launch
        LC, LK = 128, 5
        wl = gen_weights(LC, L, seed=cfg.weight_seed, two_stage=True, top=True, kernel_size=LK)
        lc = Codec(reno, torch, cfg, pts, M, cap_model, stream, wl, two_stage=True, top=True, channels=LC,
                   kernel_size=LK)
        st = max(args.steps // 10, 5)
        msl = lc.time(st, max(args.warmup // 2, 2), args.mode)
        with torch.cuda.stream(stream):
            lc.enc.profile(kinds)
            lc.dec.profile(kinds)
            for _ in range(5):
                lc.step()
            pe, pd = lc.enc.profile_read(), lc.dec.profile_read()
            lc.enc.profile([])
            lc.dec.profile([])
        lk_us = {k: round(1000.0 * (pe.get(k, (0.0, 0))[0] + pd.get(k, (0.0, 0))[0]) / 5, 1)
                 for k in kinds if k in pe or k in pd}
        # algorithmic conv flops per frame (encoder + decoder): block B's two
        # convs on every model scale, block A's on every scale below one
        # (the base scale's map is not exposed: left out, a lower bound)
        pl = lc.pairs
        conv_flops = 2 * 2 * 2 * LC * LC * (sum(pl.values()) + sum(v for b, v in pl.items() if b < B - 1))
        conv_us = lk_us.get("conv_mid", 0.0)
        topm["large_c128_k5_two_stage"] = {
            "value": round(1000.0 / msl, 2), "unit": "frames/s", "ms_per_step": round(msl, 4), "steps": st,
            "bits_per_point": round(lc.enc_total / M, 4), "us_per_frame_by_kind": lk_us,
            "conv_alg_gflop_per_frame": round(conv_flops / 1e9, 2),
            "conv_achieved_tflops": round(conv_flops / (conv_us * 1e-6) / 1e12, 2) if conv_us else None,
            "conv_frac": round(conv_flops / (conv_us * 1e-6) / 1e12 / PEAK_FP32_MFMA_TFLOPS, 4) if conv_us else None,
            "paper_context_s": "RENO-L NN 0.184 s per 14-bit frame, encoder, RTX 4090 (Table S2)"}
        log("full predictor large", topm["large_c128_k5_two_stage"])
        lc.close()

    # ---- end to end: GPU model + host rANS per scale, both heads ----
    e2e = None
    if args.e2e_frames > 0:
        e2e = {}
        for name, is_two, wts in (("one_stage", False, w_np),
                                  ("two_stage", True, gen_weights(C, L, seed=cfg.weight_seed, two_stage=True))):
            ee = EndToEnd(reno, torch, cfg, pts, M, cap_model, stream, wts, is_two)
            te, td, bits = ee.run(args.e2e_frames)
            e2e[name] = {"encode_frames_per_s": round(1.0 / te, 2), "decode_frames_per_s": round(1.0 / td, 2),
                         "encode_ms": round(1000 * te, 3), "decode_ms": round(1000 * td, 3),
                         "coded_bits_per_point": round(bits / M, 4), "stream_symbols": STREAM_SYMBOLS}
            log("end-to-end", name, e2e[name])
            # shorter streams: more of them decode in parallel, each costs its
            # final state and length (80 bits)
            trade = []
            for L in (256, 512, 2048):
                ee.L = L
                te2, td2, bits2 = ee.run(max(args.e2e_frames // 2, 2))
                trade.append({"stream_symbols": L, "encode_ms": round(1000 * te2, 3),
                              "decode_ms": round(1000 * td2, 3), "coded_bits_per_point": round(bits2 / M, 4)})
            e2e[name]["stream_length_tradeoff"] = trade
            log("end-to-end", name, "stream lengths", trade)
            ee.close()
        # frames in flight: W host threads, each with its own encoder and
        # decoder context on its own HIP stream, coding the streaming
        # workload's distinct scans; a frame's coder kernels occupy few CUs,
        # so frames overlap
        workers = tuple(int(x) for x in args.in_flight.split(",") if x.strip())
        if workers:
            e2e["frames_in_flight"] = e2e_in_flight(reno, torch, args, dev, workers=workers)
            log("end-to-end frames in flight", e2e["frames_in_flight"])
        e2e["note"] = ("wall-clock per frame through reno_encode_frame / reno_decode_frame: points copied in "
                       "from pinned host memory; GPU pyramid + model + symbol intervals + rANS streams "
                       f"(ceil(N_b / {STREAM_SYMBOLS}) streams per scale and stage, one wavefront each), bitstream "
                       "copied out; the decoder starts from the host bitstream alone, copies it in once and runs "
                       "expand, predict, cumulative tables and stream decoding (one wavefront per stream) scale "
                       "by scale on the GPU; coded bits = the whole bitstream (header, bit-packed base voxels, "
                       "16-bit stream lengths, streams)")

    # ---- multi-frame throughput: F different frames, each with its own encoder
    # and decoder context and captured step, replayed round-robin over S
    # streams so that frames are in flight together ----
    multi = None
    if args.streams and args.mode == "graph":
        mcfg = BY_NAME[args.stream_config]
        frames = [gen_scan(mcfg, f) for f in range(mcfg.frames)]
        mw = gen_weights(mcfg.channels, mcfg.layers, seed=mcfg.weight_seed)
        ns = [int(x) for x in args.streams.split(",")]
        streams = [torch.cuda.Stream(device=dev) for _ in range(max(ns))]
        mM = max(f.shape[0] for f in frames)
        codecs = []
        for i, f in enumerate(frames):
            fp = torch.from_numpy(f).to(dev)
            with torch.cuda.stream(streams[0]):
                pr = reno.Context(mM, mcfg.bit_depth, mcfg.min_bit_depth, mcfg.range_m, mcfg.channels,
                                  mcfg.layers, stream=streams[0])
                pr.build_pyramid(fp, mcfg.bit_depth)
                mv = sum(pr.num_voxels(b) for b in range(mcfg.min_bit_depth + 1, mcfg.bit_depth))
                pr.close()
            cap = (mv + mv // 8 + 4095) // 4096 * 4096
            codecs.append((fp, cap))
        cap_all = max(c[1] for c in codecs)
        vox = 0
        multi = {"workload": f"{mcfg.name}: {mcfg.frames} consecutive synthetic {mcfg.beams}-beam scans "
                             f"(sensor moving {mcfg.frame_step_m} m per frame), {mcfg.bit_depth}-bit, "
                             "each frame encoded + decoded", "frames": mcfg.frames, "runs": []}
        for S in ns:
            cs = [Codec(reno, torch, mcfg, fp, mM, cap_all, streams[i % S], mw, two_stage=False)
                  for i, (fp, _) in enumerate(codecs)]
            for c in cs:
                c.time(1, 2, "graph")              # warm-up, capture, self-check
            reps = max(args.steps // 10, 2)
            torch.cuda.synchronize()
            t = time.perf_counter()
            for _ in range(reps):
                for c in cs:
                    with torch.cuda.stream(c.stream):
                        c.graph.replay()
            torch.cuda.synchronize()
            ms = (time.perf_counter() - t) * 1000.0 / reps
            for c in cs:
                c.check("multi-frame:")
            multi["runs"].append({"streams": S, "frames_per_s": round(len(cs) * 1000.0 / ms, 2),
                                  "ms_per_batch": round(ms, 4)})
            log(f"multi-frame {len(cs)} frames on {S} streams: {ms:.3f} ms, {len(cs) * 1000.0 / ms:.1f} frames/s")
            for c in cs:
                c.close()
        # frame batches: the frames split into S batches (one key space each,
        # frame id above the Morton bits), one encoder + decoder context pair
        # and captured step per batch, batches replayed on S streams
        for S in [x for x in (1, 2) if x <= len(codecs) and x <= len(streams)]:
            groups = [list(range(len(codecs)))[g::S] for g in range(S)]
            cs = []
            for g, idx in enumerate(groups):
                bp = torch.cat([codecs[i][0] for i in idx])
                st = torch.tensor(np.cumsum([0] + [codecs[i][0].shape[0] for i in idx]), dtype=torch.int64,
                                  device=dev)
                bcap = sum(codecs[i][1] for i in idx)
                cs.append(Codec(reno, torch, mcfg, bp, int(bp.shape[0]), bcap, streams[g], mw, two_stage=False,
                                frame_start=st))
            for c in cs:
                c.time(1, 2, "graph")
            reps = max(args.steps // 10, 2)
            torch.cuda.synchronize()
            t = time.perf_counter()
            for _ in range(reps):
                for c in cs:
                    with torch.cuda.stream(c.stream):
                        c.graph.replay()
            torch.cuda.synchronize()
            ms = (time.perf_counter() - t) * 1000.0 / reps
            for c in cs:
                c.check("frame batch:")
            multi["runs"].append({"frame_batches": S, "frames_per_batch": [len(x) for x in groups],
                                  "streams": S, "frames_per_s": round(len(codecs) * 1000.0 / ms, 2),
                                  "ms_per_batch": round(ms, 4)})
            log(f"multi-frame {len(codecs)} frames as {S} frame batch(es) on {S} streams: {ms:.3f} ms, "
                f"{len(codecs) * 1000.0 / ms:.1f} frames/s")
            for c in cs:
                c.close()
        del codecs

    # ---- HBM stress: K frames of the streaming generator in one key space ----
    stress = run_stress(args, reno, torch, dev, stream, copy_peak) if args.stress else None

    # ---- CPU baseline: the oracle (single-threaded C++, fp64), one frame per
    # process, first alone, then one process per available core at once ----
    cpu = None
    oracle_bpp = None
    if not args.no_cpu_baseline:
        import multiprocessing as mp
        T_enc, T_dec, t_enc, t_dec = oracle_frame((cfg.name, 0))
        oracle_bpp = T_enc / M
        single = 1.0 / (t_enc + t_dec)
        workers = args.cpu_workers or min(16, len(os.sched_getaffinity(0)))
        t = time.perf_counter()
        with mp.get_context("spawn").Pool(workers) as pool:
            res = pool.map(oracle_frame, [(cfg.name, i) for i in range(workers)])
        wall = time.perf_counter() - t
        if any(r[0] != T_enc for r in res):
            log("oracle runs disagree")
            sys.exit(1)
        cpu = {"value": round(workers / wall, 4), "unit": "frames/s", "cores": workers,
               "kind": "oracle", "host": host_info(),
               "sample": f"{workers} copies of one {cfg.name} frame ({M} points), one process per core, "
                         f"{wall:.1f} s wall; each: oracle encode (pyramid, codes, model, bits) + decode "
                         f"(FCG expansion, model, bits) in single-threaded C++ fp64",
               "single_thread_value": round(single, 4),
               "single_thread_sample": f"one frame alone: encode {t_enc:.1f} s + decode {t_dec:.1f} s"}
        log("cpu baseline", cpu)

    voxels_frame = sum(counts)
    traffic = read_traffic(cfg.name)
    trace = read_trace(cfg.name)
    flops_launch = one.conv_last_flops(counts) / (cl_launches / args.steps)
    frac_trace = None
    if trace is not None:
        frac_trace = round(flops_launch / (trace[0] * 1e-6) / 1e12 / PEAK_FP32_MFMA_TFLOPS, 4)
    out = {
        "metric": "frames/s + Mvoxels/s, encode+decode model path, 14-bit 64-beam scan; bits/pt",
        "value": round(fps, 2),
        "unit": "frames/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "mvoxels_per_s": round(fps * voxels_frame / 1e6, 2),
        "model_mvoxels_per_s": round(fps * model_vox / 1e6, 2),
        "encode_ms": None if enc_ms is None else round(enc_ms, 5),
        "decode_ms": None if dec_ms is None else round(dec_ms, 5),
        "bits_per_point": round(enc_total / M, 4),
        "oracle_bits_per_point": None if oracle_bpp is None else round(oracle_bpp, 4),
        "config": {"workload": f"{cfg.name}: synthetic {cfg.beams}-beam x {cfg.azimuth_steps}-azimuth "
                               f"LiDAR scan, {B}-bit grid over +-{cfg.range_m} m, pyramid {B}->{b0}, "
                               f"random-init predictor C={C} L={L}, one frame encoded + decoded "
                               "per step",
                   "points": M, "voxels_per_frame": voxels_frame, "model_voxels": model_vox,
                   "device_bytes_per_context": mem["device_bytes"],
                   "mode": args.mode},
        "roofline": {"bound": "mfma", "kernel": "conv_last (last sparse conv + 256-way head)",
                     "achieved": round(achieved_tflops, 3), "peak": PEAK_FP32_MFMA_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(achieved_tflops / PEAK_FP32_MFMA_TFLOPS, 4),
                     "traffic": traffic,
                     "avg_launch_us": round(1000 * cl_ms / cl_launches, 2),
                     "launches": cl_launches,
                     "flops_per_launch": round(flops_launch),
                     "timing": "HIP events bound to each conv_last dispatch (hipExtLaunchKernelGGL), eager steps",
                     "trace_avg_launch_us": None if trace is None else trace[0],
                     "trace_dispatches": None if trace is None else trace[1],
                     "frac_trace": frac_trace},
        "hbm_copy_peak_GBs": round(copy_peak, 1),
        "median_ms_per_frame": None if not per_frame else round(float(np.median(per_frame)), 5),
        "median_frames_per_s": None if not per_frame else round(1000.0 / float(np.median(per_frame)), 2),
        "cpu_baseline": cpu,
        "kernels": breakdown,
        "two_stage_head": two,
        "precision_bf16x3": bfx,
        "full_predictor": topm,
        "hbm_stress": stress,
        "end_to_end": e2e,
        "multi_frame": multi,
    }
    print(json.dumps(out), flush=True)
    one.close()


if __name__ == "__main__":
    main()
