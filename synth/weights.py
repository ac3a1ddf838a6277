"""Seeded random-init weights for the probability model.

Layout (fp32, row-major, shared by every consumer):
  conv_w[l]  [27][C_in][C_out]   offset k = (dx+1) + 3(dy+1) + 9(dz+1)
  conv_b[l]  [C_out]
  head_w     [C][256]
  head_b     [256]
and, with ``two_stage=True``, the bitwise two-stage head (Sec. 3.2,
Eqs. 11-13): S1 = O & 15 first, then S2 = O >> 4 given S1:
  head1_w    [C][16]    head1_b [16]     stage 1: z1 = head1_w^T h + head1_b
  emb_s1     [16][C]                     Emb(S1), added to h before stage 2
  head2_w    [C][16]    head2_b [16]     stage 2: z2 = head2_w^T (h + emb_s1[S1]) + head2_b
and, with ``top=True``, the full target occupancy predictor (Sec. 3.2,
Eqs. 6-9), which replaces the L plain layers:
  emb_o      [256][C]   Emb(O^{d-1}) of the parent-scale codes
  emb_d      [8][C]     Emb(delta) of the octant
  top_w[i]   [27][C][C], top_b[i] [C], i = A1, A2 (residual block at scale
             d-1), B1, B2 (residual block at scale d)
with C_in = 11 for the first layer and C for the rest.  Kaiming-normal:
std = sqrt(2 / fan_in), fan_in = 27 * C_in for a conv and C for the head.
Biases are zero unless ``bias_std`` is given (tests use non-zero biases so
that the bias path is exercised).
"""
from __future__ import annotations

import numpy as np

from . import rng

IN_FEATURES = 11
SYMBOLS = 256
KVOL = 27
_W_STREAM = 21


def gen_weights(channels: int, layers: int, seed: int = 2, bias_std: float = 0.0,
                head_scale: float = 1.0, in_features: int = IN_FEATURES,
                two_stage: bool = False, emb_std: float = 1.0, top: bool = False,
                kernel_size: int = 3) -> dict:
    draw = [0]

    def normals(n):
        out = rng.normal(seed, _W_STREAM, draw[0], n)
        draw[0] += n
        return out

    conv_w, conv_b = [], []
    c_in = in_features
    for _ in range(layers):
        fan_in = KVOL * c_in
        w = normals(KVOL * c_in * channels) * np.sqrt(2.0 / fan_in)
        conv_w.append(w.reshape(KVOL, c_in, channels).astype(np.float32))
        b = normals(channels) * bias_std
        conv_b.append(b.astype(np.float32))
        c_in = channels
    hw = normals(channels * SYMBOLS) * np.sqrt(2.0 / channels) * head_scale
    hb = normals(SYMBOLS) * bias_std * head_scale
    out = {
        "c_in": in_features, "channels": channels, "layers": layers,
        "conv_w": conv_w, "conv_b": conv_b,
        "head_w": hw.reshape(channels, SYMBOLS).astype(np.float32),
        "head_b": hb.astype(np.float32),
    }
    if two_stage:  # drawn after the one-stage weights, which stay unchanged
        std = np.sqrt(2.0 / channels) * head_scale
        out["head1_w"] = (normals(channels * 16) * std).reshape(channels, 16).astype(np.float32)
        out["head1_b"] = (normals(16) * bias_std * head_scale).astype(np.float32)
        out["emb_s1"] = (normals(16 * channels) * emb_std).reshape(16, channels).astype(np.float32)
        out["head2_w"] = (normals(channels * 16) * std).reshape(channels, 16).astype(np.float32)
        out["head2_b"] = (normals(16) * bias_std * head_scale).astype(np.float32)
    if top:  # drawn after everything above, which stays unchanged
        out["emb_o"] = (normals(256 * channels) * emb_std).reshape(256, channels).astype(np.float32)
        out["emb_d"] = (normals(8 * channels) * emb_std).reshape(8, channels).astype(np.float32)
        out["top_w"], out["top_b"] = [], []
        kv = kernel_size ** 3   # the full predictor's convs: ks^3 offsets
        for _ in range(4):
            w_ = normals(kv * channels * channels) * np.sqrt(2.0 / (kv * channels))
            out["top_w"].append(w_.reshape(kv, channels, channels).astype(np.float32))
            out["top_b"].append((normals(channels) * bias_std).astype(np.float32))
    return out
