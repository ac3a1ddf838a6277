"""ctypes wrapper of the CPU oracle (oracle.cpp).

TEST INFRASTRUCTURE ONLY: the tests, ``__graft_entry__.smoke()`` and the
benchmark's CPU-baseline leg are the only callers.  The GPU library never
imports this package and this package never imports the GPU library.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.cpp")
_LIB = os.path.join(_HERE, "liboracle.so")
_lib = None

SYMBOLS = 256


def build(verbose: bool = False) -> str:
    """Compiles liboracle.so in place (plain g++, no SIMD flags, no fp contraction)."""
    cmd = ["g++", "-O2", "-std=c++17", "-ffp-contract=off", "-fno-fast-math", "-Wall",
           "-fPIC", "-shared", _SRC, "-o", _LIB + ".tmp"]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    os.replace(_LIB + ".tmp", _LIB)
    return _LIB


class OrcWeights(ctypes.Structure):
    _fields_ = [("c_in", ctypes.c_int), ("channels", ctypes.c_int), ("layers", ctypes.c_int),
                ("pad", ctypes.c_int),
                ("conv_w", ctypes.c_void_p * 8), ("conv_b", ctypes.c_void_p * 8),
                ("head_w", ctypes.c_void_p), ("head_b", ctypes.c_void_p),
                ("head_mode", ctypes.c_int), ("pad2", ctypes.c_int),
                ("head1_w", ctypes.c_void_p), ("head1_b", ctypes.c_void_p),
                ("emb_s1", ctypes.c_void_p), ("head2_w", ctypes.c_void_p),
                ("head2_b", ctypes.c_void_p),
                ("model_mode", ctypes.c_int), ("pad3", ctypes.c_int),
                ("emb_o", ctypes.c_void_p), ("emb_d", ctypes.c_void_p),
                ("top_w", ctypes.c_void_p * 4), ("top_b", ctypes.c_void_p * 4),
                ("kernel_size", ctypes.c_int), ("pad4", ctypes.c_int)]


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
            build()
        L = ctypes.CDLL(_LIB)
        vp, i64, i32, c_int, dbl = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_int, ctypes.c_double
        sig = {
            "orc_morton": (ctypes.c_uint64, [i64, i64, i64, c_int]),
            "orc_quantize": (c_int, [vp, i64, c_int, dbl, vp]),
            "orc_pyramid_from_points": (vp, [vp, i64, c_int, c_int, dbl]),
            "orc_pyramid_from_voxels": (vp, [vp, i64, c_int, c_int]),
            "orc_pyramid_from_codes": (vp, [vp, i64, c_int, c_int, vp, i64]),
            "orc_free": (None, [vp]),
            "orc_num": (i64, [vp, c_int]),
            "orc_raw_points": (i64, [vp]),
            "orc_xyz": (None, [vp, c_int, vp]),
            "orc_keys": (None, [vp, c_int, vp]),
            "orc_codes": (c_int, [vp, c_int, vp]),
            "orc_parent": (None, [vp, c_int, vp]),
            "orc_expand": (i64, [vp, c_int, vp, vp]),
            "orc_neighbors": (None, [vp, c_int, c_int, vp]),
            "orc_features": (None, [vp, c_int, vp]),
            "orc_sparse_conv": (c_int, [vp, i64, c_int, vp, c_int, vp, vp, c_int, c_int, c_int, vp]),
            "orc_model": (c_int, [vp, c_int, ctypes.POINTER(OrcWeights), vp, i64, vp, vp, vp]),
            "orc_model2": (c_int, [vp, c_int, ctypes.POINTER(OrcWeights), vp, i64, vp, vp, vp, vp,
                                   vp, vp]),
            "orc_totals": (dbl, [vp, ctypes.POINTER(OrcWeights), vp]),
            "orc_freqs_from_probs": (None, [vp, vp]),
            "orc_freqs_from_probs_k": (None, [vp, c_int, vp]),
            "orc_rans_encode": (i64, [vp, vp, i64, vp, i64]),
            "orc_rans_decode": (c_int, [vp, i64, vp, i64, vp]),
        }
        for name, (res, args) in sig.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def _p(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def morton(x: int, y: int, z: int, bits: int) -> int:
    return int(lib().orc_morton(x, y, z, bits))


def quantize(points: np.ndarray, B: int, R: float) -> np.ndarray:
    pts = np.ascontiguousarray(points, dtype=np.float32)
    q = np.empty((pts.shape[0], 3), dtype=np.int64)
    if lib().orc_quantize(_p(pts), pts.shape[0], B, R, _p(q)) != 0:
        raise ValueError("non-finite point")
    return q


def kernel_size_of(w: np.ndarray) -> int:
    """Kernel size ks of a conv weight array [ks^3][C_in][C_out]."""
    kv = int(np.asarray(w).shape[0])
    ks = int(round(kv ** (1.0 / 3.0)))
    if ks ** 3 != kv or ks % 2 == 0:
        raise ValueError(f"{kv} offsets is not an odd cube")
    return ks


class _W:
    """Keeps the fp32 weight arrays alive while the oracle holds pointers."""

    def __init__(self, w: dict, two_stage=None):
        self.arrays = []
        s = OrcWeights()
        s.c_in = w["c_in"]
        s.channels = w["channels"]
        s.layers = w["layers"]
        for l in range(w["layers"]):
            cw = np.ascontiguousarray(w["conv_w"][l], dtype=np.float32)
            cb = np.ascontiguousarray(w["conv_b"][l], dtype=np.float32)
            self.arrays += [cw, cb]
            s.conv_w[l] = cw.ctypes.data
            s.conv_b[l] = cb.ctypes.data
        hw = np.ascontiguousarray(w["head_w"], dtype=np.float32)
        hb = np.ascontiguousarray(w["head_b"], dtype=np.float32)
        self.arrays += [hw, hb]
        s.head_w = hw.ctypes.data
        s.head_b = hb.ctypes.data
        if two_stage is None:
            two_stage = "head1_w" in w
        s.head_mode = 1 if two_stage else 0
        if two_stage:
            for name in ("head1_w", "head1_b", "emb_s1", "head2_w", "head2_b"):
                a = np.ascontiguousarray(w[name], dtype=np.float32)
                self.arrays.append(a)
                setattr(s, name, a.ctypes.data)
        if "top_w" in w:  # the full predictor
            s.model_mode = 1
            for name in ("emb_o", "emb_d"):
                a = np.ascontiguousarray(w[name], dtype=np.float32)
                self.arrays.append(a)
                setattr(s, name, a.ctypes.data)
            s.kernel_size = kernel_size_of(w["top_w"][0])
            for i in range(4):
                tw = np.ascontiguousarray(w["top_w"][i], dtype=np.float32)
                tb = np.ascontiguousarray(w["top_b"][i], dtype=np.float32)
                self.arrays += [tw, tb]
                s.top_w[i] = tw.ctypes.data
                s.top_b[i] = tb.ctypes.data
        self.s = s


class Pyramid:
    """The oracle's multiscale sparse tensor: V_b, O_b and parent rows per scale."""

    def __init__(self, handle, B: int, b0: int):
        if not handle:
            raise ValueError("oracle rejected the input")
        self._h = handle
        self.B = B
        self.b0 = b0

    def __del__(self):
        if getattr(self, "_h", None):
            lib().orc_free(self._h)
            self._h = None

    @classmethod
    def from_points(cls, points: np.ndarray, B: int, b0: int, R: float) -> "Pyramid":
        pts = np.ascontiguousarray(points, dtype=np.float32).reshape(-1, 3)
        return cls(lib().orc_pyramid_from_points(_p(pts), pts.shape[0], B, b0, R), B, b0)

    @classmethod
    def from_voxels(cls, xyz: np.ndarray, B: int, b0: int) -> "Pyramid":
        v = np.ascontiguousarray(xyz, dtype=np.int64).reshape(-1, 3)
        return cls(lib().orc_pyramid_from_voxels(_p(v), v.shape[0], B, b0), B, b0)

    @classmethod
    def from_codes(cls, base_xyz: np.ndarray, b0: int, B: int, codes: list) -> "Pyramid":
        v = np.ascontiguousarray(base_xyz, dtype=np.int64).reshape(-1, 3)
        c = np.ascontiguousarray(np.concatenate([np.asarray(x, np.uint8) for x in codes])
                                 if codes else np.zeros(0, np.uint8))
        return cls(lib().orc_pyramid_from_codes(_p(v), v.shape[0], b0, B, _p(c), c.size), B, b0)

    def num(self, b: int) -> int:
        return int(lib().orc_num(self._h, b))

    @property
    def raw_points(self) -> int:
        return int(lib().orc_raw_points(self._h))

    def xyz(self, b: int) -> np.ndarray:
        out = np.empty((self.num(b), 3), dtype=np.int64)
        lib().orc_xyz(self._h, b, _p(out))
        return out

    def keys(self, b: int) -> np.ndarray:
        out = np.empty(self.num(b), dtype=np.uint64)
        lib().orc_keys(self._h, b, _p(out))
        return out

    def codes(self, b: int) -> np.ndarray:
        out = np.empty(self.num(b), dtype=np.uint8)
        if lib().orc_codes(self._h, b, _p(out)) != 0:
            raise ValueError(f"scale {b} has no codes")
        return out

    def parent(self, b: int) -> np.ndarray:
        out = np.empty(self.num(b), dtype=np.int32)
        lib().orc_parent(self._h, b, _p(out))
        return out

    def expand(self, b: int, codes: np.ndarray) -> np.ndarray:
        c = np.ascontiguousarray(codes, dtype=np.uint8)
        assert c.size == self.num(b)
        n = lib().orc_expand(self._h, b, _p(c), None)
        out = np.empty((n, 3), dtype=np.int64)
        lib().orc_expand(self._h, b, _p(c), _p(out))
        return out

    def neighbors(self, b: int, ks: int = 3) -> np.ndarray:
        """Neighbour rows [N_b][ks^3] (-1: absent or off-grid)."""
        out = np.empty((self.num(b), ks ** 3), dtype=np.int32)
        lib().orc_neighbors(self._h, b, ks, _p(out))
        return out

    def features(self, b: int) -> np.ndarray:
        out = np.empty((self.num(b), 11), dtype=np.float64)
        lib().orc_features(self._h, b, _p(out))
        return out

    def model(self, b: int, weights: dict, rows=None, logits=True, bits=True):
        """Logits [n][256], lse [n] and bits [n] (bits only for b < B) of the
        requested rows of scale b (all rows when ``rows`` is None)."""
        if rows is None:
            rows = np.arange(self.num(b), dtype=np.int64)
        rows = np.ascontiguousarray(rows, dtype=np.int64)
        n = rows.size
        lg = np.empty((n, SYMBOLS), dtype=np.float64) if logits else None
        lse = np.empty(n, dtype=np.float64)
        bt = np.empty(n, dtype=np.float64) if (bits and b < self.B) else None
        W = _W(weights)
        rc = lib().orc_model(self._h, b, ctypes.byref(W.s), _p(rows), n,
                             _p(lg) if lg is not None else None, _p(lse),
                             _p(bt) if bt is not None else None)
        if rc != 0:
            raise ValueError("oracle model rejected the arguments")
        return lg, lse, bt

    def model2(self, b: int, weights: dict, rows=None, s1=None, logits=True, bits=True):
        """Bitwise two-stage head: (logits1 [n][16], logits2 [n][16], lse1 [n],
        lse2 [n], bits [n]) for the requested rows.  S1 (the low nibble) comes
        from ``s1`` when given, else from the codes of scale b (then bits are
        returned for b < B)."""
        if rows is None:
            rows = np.arange(self.num(b), dtype=np.int64)
        rows = np.ascontiguousarray(rows, dtype=np.int64)
        n = rows.size
        s1a = None if s1 is None else np.ascontiguousarray(s1, dtype=np.uint8)
        l1 = np.empty((n, 16)) if logits else None
        l2 = np.empty((n, 16)) if logits else None
        lse1, lse2 = np.empty(n), np.empty(n)
        bt = np.empty(n) if (bits and s1 is None and b < self.B) else None
        W = _W(weights, two_stage=True)
        rc = lib().orc_model2(self._h, b, ctypes.byref(W.s), _p(rows), n,
                              _p(s1a) if s1a is not None else None,
                              _p(l1) if l1 is not None else None, _p(l2) if l2 is not None else None,
                              _p(lse1), _p(lse2), _p(bt) if bt is not None else None)
        if rc != 0:
            raise ValueError("oracle two-stage model rejected the arguments")
        return l1, l2, lse1, lse2, bt

    def totals(self, weights: dict, two_stage=None):
        """(T, per_scale[B+1]): total ideal bits and its split per scale
        (two-stage head when the weights carry one, unless told otherwise)."""
        per = np.zeros(self.B + 1, dtype=np.float64)
        W = _W(weights, two_stage)
        T = lib().orc_totals(self._h, ctypes.byref(W.s), _p(per))
        if T < 0:
            raise ValueError("oracle totals failed")
        return float(T), per


def sparse_conv(xyz: np.ndarray, bits: int, feats: np.ndarray, W: np.ndarray, bias: np.ndarray,
                relu: bool) -> np.ndarray:
    v = np.ascontiguousarray(xyz, dtype=np.int64).reshape(-1, 3)
    f = np.ascontiguousarray(feats, dtype=np.float64)
    Wf = np.ascontiguousarray(W, dtype=np.float32)
    bf = np.ascontiguousarray(bias, dtype=np.float32)
    c_in, c_out = Wf.shape[1], Wf.shape[2]
    ks = kernel_size_of(Wf)
    out = np.empty((v.shape[0], c_out), dtype=np.float64)
    if lib().orc_sparse_conv(_p(v), v.shape[0], bits, _p(f), c_in, _p(Wf), _p(bf), c_out,
                             int(relu), ks, _p(out)) != 0:
        raise ValueError("duplicate voxel")
    return out


def freqs_from_probs(p: np.ndarray, k: int = SYMBOLS) -> np.ndarray:
    """Quantised tables [n][k] from probabilities [n][k] (k = 256 or 16)."""
    p = np.ascontiguousarray(p, dtype=np.float64).reshape(-1, k)
    out = np.empty(p.shape, dtype=np.uint32)
    for i in range(p.shape[0]):
        lib().orc_freqs_from_probs_k(_p(p[i]), k, _p(out[i]))
    return out


def rans_encode(sym: np.ndarray, freq: np.ndarray) -> np.ndarray:
    s = np.ascontiguousarray(sym, dtype=np.uint8)
    f = np.ascontiguousarray(freq, dtype=np.uint32)
    cap = 2 * s.size + 16
    out = np.empty(cap, dtype=np.uint32)
    n = lib().orc_rans_encode(_p(s), _p(f), s.size, _p(out), cap)
    if n < 0:
        raise ValueError("rANS encode failed")
    return out[:n].copy()


def rans_decode(words: np.ndarray, freq: np.ndarray, n: int) -> np.ndarray:
    w = np.ascontiguousarray(words, dtype=np.uint32)
    f = np.ascontiguousarray(freq, dtype=np.uint32)
    out = np.empty(n, dtype=np.uint8)
    if lib().orc_rans_decode(_p(w), w.size, _p(f), n, _p(out)) != 0:
        raise ValueError("rANS decode failed")
    return out


def encode_frame_bits(points: np.ndarray, B: int, b0: int, R: float, weights: dict):
    """Oracle encode of one frame: pyramid, codes, model and total ideal bits."""
    P = Pyramid.from_points(points, B, b0, R)
    T, per = P.totals(weights)
    return P, T, per


def decode_frame(base_xyz: np.ndarray, b0: int, B: int, codes: list, weights: dict):
    """Oracle decode of one frame: FCG expansion from the initial state and the
    model on every decoded scale (the decoder needs the same distributions)."""
    P = Pyramid.from_codes(base_xyz, b0, B, codes)
    T, per = P.totals(weights)
    return P, T, per
