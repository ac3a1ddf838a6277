"""MI355X (gfx950) hot path of the RENO LiDAR geometry codec.

Thin ctypes binding over the C ABI of libreno.so (declared in include/reno.h):
argument marshalling only.  Device memory and streams come from PyTorch; every
step of the codec runs in the library's HIP kernels.  Importing works without
a GPU; creating a context needs one, and the library must have been built
(``python -m paper_2503_12382_amd.build``) -- there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libreno.so")

RENO_OK = 0
RENO_E_INVALID = -1
RENO_E_STATE = -2
RENO_E_NOMEM = -3
RENO_E_HIP = -4
RENO_E_CAPACITY = -5
RENO_E_INPUT = -6
RENO_MAX_LAYERS = 8
RENO_MAX_BIT_DEPTH = 21
RENO_ALL_SCALES = -1
RENO_MAX_FRAMES = 1024
RENO_HEAD_ONE_STAGE = 0
RENO_HEAD_TWO_STAGE = 1
RENO_PREC_FP32 = 0
RENO_PREC_BF16X3 = 1
RENO_MODEL_PLAIN = 0
RENO_MODEL_TOP = 1
SYMBOLS = 256

_STATUS = {0: "RENO_OK", -1: "RENO_E_INVALID", -2: "RENO_E_STATE", -3: "RENO_E_NOMEM",
           -4: "RENO_E_HIP", -5: "RENO_E_CAPACITY", -6: "RENO_E_INPUT"}


class RenoError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{_STATUS.get(status, status)}: {msg}")
        self.status = status


class reno_params(ctypes.Structure):
    _fields_ = [("max_points", ctypes.c_int64), ("max_model_voxels", ctypes.c_int64),
                ("max_bit_depth", ctypes.c_int), ("min_bit_depth", ctypes.c_int),
                ("range_m", ctypes.c_double), ("in_features", ctypes.c_int),
                ("channels", ctypes.c_int), ("layers", ctypes.c_int),
                ("head_mode", ctypes.c_int), ("precision", ctypes.c_int),
                ("model_mode", ctypes.c_int), ("kernel_size", ctypes.c_int)]


class reno_weights(ctypes.Structure):
    _fields_ = [("conv_w", ctypes.c_void_p * RENO_MAX_LAYERS),
                ("conv_b", ctypes.c_void_p * RENO_MAX_LAYERS),
                ("head_w", ctypes.c_void_p), ("head_b", ctypes.c_void_p),
                ("head1_w", ctypes.c_void_p), ("head1_b", ctypes.c_void_p),
                ("emb_s1", ctypes.c_void_p), ("head2_w", ctypes.c_void_p),
                ("head2_b", ctypes.c_void_p), ("emb_o", ctypes.c_void_p),
                ("emb_d", ctypes.c_void_p), ("top_w", ctypes.c_void_p * 4),
                ("top_b", ctypes.c_void_p * 4)]


# exported symbol -> (restype, argtypes); exactly the functions of include/reno.h
_vp, _i64, _int = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int
_SIGS = {
    "reno_create": (_int, [ctypes.POINTER(reno_params), _vp, ctypes.POINTER(_vp)]),
    "reno_destroy": (_int, [_vp]),
    "reno_last_error": (ctypes.c_char_p, [_vp]),
    "reno_sync": (_int, [_vp]),
    "reno_memory_info": (_int, [_vp, _vp]),
    "reno_set_weights": (_int, [_vp, ctypes.POINTER(reno_weights)]),
    "reno_build_pyramid": (_int, [_vp, _vp, _i64, _int]),
    "reno_set_base": (_int, [_vp, _int, _vp, _vp, _i64]),
    "reno_build_pyramid_frames": (_int, [_vp, _vp, _i64, _vp, _int, _int]),
    "reno_set_base_frames": (_int, [_vp, _int, _vp, _vp, _vp, _i64, _int]),
    "reno_expand": (_int, [_vp, _int, _vp]),
    "reno_expand_noalloc": (_int, [_vp, _vp, _i64, _vp, _vp, _i64, _vp, _vp, _vp]),
    "reno_num_voxels": (_int, [_vp, _int, ctypes.POINTER(_i64)]),
    "reno_scale_counts": (_int, [_vp, _vp]),
    "reno_coords": (_int, [_vp, _int, _vp, _vp]),
    "reno_occupancy_codes": (_int, [_vp, _int, _vp]),
    "reno_parent_rows": (_int, [_vp, _int, _vp]),
    "reno_predict_probs": (_int, [_vp, _int, ctypes.POINTER(reno_weights), _vp]),
    "reno_predict_second": (_int, [_vp, _int, _vp, _vp]),
    "reno_code_length": (_int, [_vp, _int, _vp, ctypes.POINTER(ctypes.c_double)]),
    "reno_neighbor_map": (_int, [_vp, _int, _vp]),
    "reno_symbol_freqs": (_int, [_vp, _int, _vp]),
    "reno_symbol_freqs16": (_int, [_vp, _int, _int, _vp]),
    "reno_symbol_intervals": (_int, [_vp, _int, _vp]),
    "reno_symbol_cdf": (_int, [_vp, _int, _int, _vp]),
    "reno_rans_encode_intervals": (_int, [_vp, _i64, _i64, _vp, _i64, ctypes.POINTER(_i64)]),
    "reno_rans_decode16": (_int, [_vp, _i64, _vp, _i64, _vp]),
    "reno_rans_encode": (_int, [_vp, _vp, _i64, _vp, _i64, ctypes.POINTER(_i64)]),
    "reno_rans_decode": (_int, [_vp, _i64, _vp, _i64, _vp]),
    "reno_rans_encode_streams": (_int, [_vp, _i64, _i64, _int, _int, _vp, _i64, _vp]),
    "reno_rans_decode_streams": (_int, [_vp, _vp, _int, _int, _vp, _int, _i64, _vp]),
    "reno_encode_frame": (_int, [_vp, _vp, _i64, _int, _int, _vp, _i64, ctypes.POINTER(_i64)]),
    "reno_decode_frame": (_int, [_vp, _vp, _i64]),
    "reno_profile": (_int, [_vp, ctypes.c_uint32]),
    "reno_profile_read": (_int, [_vp, _vp, _vp]),
}

KERNELS = ["zero", "quantize", "sort", "pyramid", "codes", "set_base", "expand", "conv_first",
           "conv_mid", "conv_last", "code_length", "other", "top_input", "entropy"]

_lib = None


def lib():
    """The loaded C library; raises if it has not been built."""
    global _lib
    if _lib is None:
        try:                      # load torch's HIP runtime first so that both share it
            import torch  # noqa: F401
        except ImportError:
            pass
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2503_12382_amd.build` (no CPU fallback exists)")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


class Context:
    """One codec context (reno_ctx) bound to a torch device and stream."""

    def __init__(self, max_points: int, max_bit_depth: int, min_bit_depth: int, range_m: float,
                 channels: int, layers: int, max_model_voxels: int = 0, stream=None,
                 two_stage: bool = False, precision: int = RENO_PREC_FP32, top: bool = False,
                 kernel_size: int = 3):
        import torch
        self.torch = torch
        self.device = torch.device("cuda", torch.cuda.current_device())
        self.stream = stream if stream is not None else torch.cuda.current_stream()
        p = reno_params(max_points, max_model_voxels, max_bit_depth, min_bit_depth, range_m, 11,
                        channels, layers, RENO_HEAD_TWO_STAGE if two_stage else RENO_HEAD_ONE_STAGE,
                        precision, RENO_MODEL_TOP if top else RENO_MODEL_PLAIN, kernel_size)
        h = ctypes.c_void_p()
        rc = lib().reno_create(ctypes.byref(p), ctypes.c_void_p(self.stream.cuda_stream),
                               ctypes.byref(h))
        if rc != RENO_OK:
            raise RenoError(rc, lib().reno_last_error(None).decode())
        self._h = h
        self.params = p
        self.b0 = min_bit_depth
        self.channels = channels
        self.layers = layers
        self.two_stage = two_stage
        self.top = top
        self.kernel_size = kernel_size
        self.B = 0
        self._keep = []

    def close(self):
        if getattr(self, "_h", None):
            lib().reno_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def _check(self, rc):
        if rc != RENO_OK:
            raise RenoError(rc, lib().reno_last_error(self._h).decode())

    def _empty(self, shape, dtype):
        return self.torch.empty(shape, dtype=dtype, device=self.device)

    # ---- C ABI calls -------------------------------------------------------------------------
    def sync(self):
        self._check(lib().reno_sync(self._h))

    def set_weights(self, weights: dict):
        """weights: dict of fp32 device tensors conv_w[l], conv_b[l] (full predictor:
        emb_o, emb_d, top_w[4], top_b[4]) and the head of the context's head mode."""
        w = reno_weights()
        keep = []
        if self.top:
            for i in range(4):
                tw = weights["top_w"][i].contiguous()
                tb = weights["top_b"][i].contiguous()
                keep += [tw, tb]
                w.top_w[i] = tw.data_ptr()
                w.top_b[i] = tb.data_ptr()
        else:
            for l in range(self.layers):
                cw = weights["conv_w"][l].contiguous()
                cb = weights["conv_b"][l].contiguous()
                keep += [cw, cb]
                w.conv_w[l] = cw.data_ptr()
                w.conv_b[l] = cb.data_ptr()
        names = (("head1_w", "head1_b", "emb_s1", "head2_w", "head2_b") if self.two_stage
                 else ("head_w", "head_b"))
        if self.top:
            names = names + ("emb_o", "emb_d")
        for name in names:
            t = weights[name].contiguous()
            keep.append(t)
            setattr(w, name, t.data_ptr())
        self._check(lib().reno_set_weights(self._h, ctypes.byref(w)))
        self._keep = keep        # alive until the next set_weights (stream-ordered)

    def build_pyramid(self, points, bit_depth: int):
        n = int(points.shape[0])
        pts = points.contiguous()
        self._check(lib().reno_build_pyramid(self._h, _ptr(pts) if n else None, n, bit_depth))
        self._points = pts
        self.B = bit_depth

    def build_pyramid_frames(self, points, frame_start, bit_depth: int):
        """Frame batch: points [n][3] of all frames back to back; frame_start int64
        device tensor [frames + 1] (frame f = points[frame_start[f]:frame_start[f+1]])."""
        n = int(points.shape[0])
        pts = points.contiguous()
        fs = frame_start.contiguous()
        frames = int(fs.shape[0]) - 1
        self._check(lib().reno_build_pyramid_frames(self._h, _ptr(pts) if n else None, n, _ptr(fs), frames,
                                                    bit_depth))
        self._points = (pts, fs)
        self.B = bit_depth

    def set_base_frames(self, bit_depth: int, xyz, frame_of, codes, frames: int):
        """Frame batch decoder start: base voxels xyz [n][3] with their frame ids
        (int32 [n]), strictly ascending in (frame, Morton) order."""
        n = int(xyz.shape[0])
        x, f, c = xyz.contiguous(), frame_of.contiguous(), codes.contiguous()
        self._check(lib().reno_set_base_frames(self._h, bit_depth, _ptr(x) if n else None,
                                               _ptr(f) if n else None, _ptr(c) if n else None, n, frames))
        self._base = (x, f, c)
        self.B = bit_depth

    def set_base(self, bit_depth: int, xyz, codes):
        n = int(xyz.shape[0])
        x = xyz.contiguous()
        c = codes.contiguous()
        self._check(lib().reno_set_base(self._h, bit_depth, _ptr(x) if n else None,
                                        _ptr(c) if n else None, n))
        self._base = (x, c)
        self.B = bit_depth

    def expand(self, scale: int, codes=None):
        c = codes.contiguous() if codes is not None else None
        self._check(lib().reno_expand(self._h, scale, _ptr(c)))
        if c is not None:
            self._last_codes = c

    def num_voxels(self, scale: int) -> int:
        n = ctypes.c_int64()
        self._check(lib().reno_num_voxels(self._h, scale, ctypes.byref(n)))
        return n.value

    def coords(self, scale: int):
        n = self.num_voxels(scale)
        xyz = self._empty((max(n, 1), 3), self.torch.int32)
        keys = self._empty((max(n, 1),), self.torch.int64)
        self._check(lib().reno_coords(self._h, scale, _ptr(xyz), _ptr(keys)))
        return xyz[:n], keys[:n]

    def occupancy_codes(self, scale: int):
        n = self.num_voxels(scale)
        out = self._empty((max(n, 1),), self.torch.uint8)
        self._check(lib().reno_occupancy_codes(self._h, scale, _ptr(out)))
        return out[:n]

    def parent_rows(self, scale: int):
        n = self.num_voxels(scale)
        out = self._empty((max(n, 1),), self.torch.int32)
        self._check(lib().reno_parent_rows(self._h, scale, _ptr(out)))
        return out[:n]

    def predict_probs(self, scale: int, weights: dict | None = None, logits: bool = False):
        if weights is not None:
            self.set_weights(weights)
        out = None
        if logits:
            if scale == RENO_ALL_SCALES:
                n = sum(self.num_voxels(b) for b in range(self.b0 + 1, self.B))
            else:
                n = self.num_voxels(scale)
            out = self._empty((max(n, 1), 32 if self.two_stage else SYMBOLS), self.torch.float32)
        self._check(lib().reno_predict_probs(self._h, scale, None, _ptr(out)))
        if logits:
            return out[:n]
        return None

    def predict_second(self, scale: int, s1=None, logits: bool = False):
        """Stage 2 of the two-stage head given the first sub-codes S1 (uint8
        device tensor [N_scale]); None takes S1 from the known codes."""
        out = None
        n = self.num_voxels(scale) if logits else 0
        if logits:
            out = self._empty((max(n, 1), 16), self.torch.float32)
        s1c = None if s1 is None else s1.contiguous()
        self._check(lib().reno_predict_second(self._h, scale, _ptr(s1c) if s1c is not None else None,
                                              _ptr(out)))
        self._s1 = s1c
        return out[:n] if logits else None

    def code_length(self, scale: int, per_voxel: bool = True, total: bool = True):
        out = None
        if per_voxel:
            if scale == RENO_ALL_SCALES:
                n = sum(self.num_voxels(b) for b in range(self.b0 + 1, self.B))
            else:
                n = self.num_voxels(scale)
            out = self._empty((max(n, 1),), self.torch.float32)
        tot = ctypes.c_double()
        self._check(lib().reno_code_length(self._h, scale, _ptr(out),
                                           ctypes.byref(tot) if total else None))
        return (out[:n] if per_voxel else None), (tot.value if total else None)

    def neighbor_map(self, scale: int):
        n = self.num_voxels(scale)
        out = self._empty((max(n, 1), self.kernel_size ** 3 if self.top else 27), self.torch.int32)
        self._check(lib().reno_neighbor_map(self._h, scale, _ptr(out)))
        return out[:n]

    def scale_counts(self) -> np.ndarray:
        """N_b of every scale (index b), one synchronising copy."""
        out = np.zeros(RENO_MAX_BIT_DEPTH + 1, np.int64)
        self._check(lib().reno_scale_counts(self._h, out.ctypes.data_as(_vp)))
        return out

    def memory_info(self) -> dict:
        """Sizes fixed at create time: hash slots, look-back status words,
        model-row capacity and the device bytes the context allocated."""
        info = np.zeros(4, np.int64)
        self._check(lib().reno_memory_info(self._h, info.ctypes.data_as(_vp)))
        return {"hash_slots": int(info[0]), "status_words": int(info[1]),
                "model_rows": int(info[2]), "device_bytes": int(info[3])}

    def profile(self, kinds=()):
        """Time the launches of the named kernel kinds (see KERNELS) with HIP events."""
        mask = 0
        for k in kinds:
            mask |= 1 << KERNELS.index(k)
        self._check(lib().reno_profile(self._h, mask))

    def profile_read(self) -> dict:
        ms = np.zeros(len(KERNELS), np.float64)
        n = np.zeros(len(KERNELS), np.int64)
        self._check(lib().reno_profile_read(self._h, ms.ctypes.data_as(_vp), n.ctypes.data_as(_vp)))
        return {k: (float(ms[i]), int(n[i])) for i, k in enumerate(KERNELS) if n[i]}

    def symbol_freqs16(self, scale: int, stage: int):
        """Two-stage head: uint16 [N][16] table of stage 1 or 2 per voxel."""
        n = self.num_voxels(scale)
        out = self._empty((max(n, 1), 16), self.torch.int16)
        self._check(lib().reno_symbol_freqs16(self._h, scale, stage, _ptr(out)))
        return out[:n]

    def symbol_intervals(self, scale: int, out=None):
        """(start, freq) of each voxel's code in its table: int16-typed uint16
        [N][2] (one-stage) or [N][4] (two-stage); RENO_ALL_SCALES concatenates
        the model scales.  ``out`` may be a preallocated device tensor."""
        if scale == RENO_ALL_SCALES:
            n = sum(self.num_voxels(b) for b in range(self.b0 + 1, self.B))
        else:
            n = self.num_voxels(scale)
        per = 4 if self.two_stage else 2
        if out is None:
            out = self._empty((max(n, 1), per), self.torch.int16)
        self._check(lib().reno_symbol_intervals(self._h, scale, _ptr(out)))
        return out[:n]

    def symbol_cdf(self, scale: int, stage: int = 0, out=None):
        """Cumulative tables (start of every symbol): int16-typed uint16
        [N][256] (one-stage head, stage 0) or [N][16] (two-stage head, stage 1
        or 2).  ``out`` may be a preallocated device tensor."""
        n = self.num_voxels(scale)
        k = 16 if stage else SYMBOLS
        if out is None:
            out = self._empty((max(n, 1), k), self.torch.int16)
        self._check(lib().reno_symbol_cdf(self._h, scale, stage, _ptr(out)))
        return out[:n]

    def encode_frame(self, points, bit_depth: int, stream_symbols: int = 1024, out: np.ndarray | None = None):
        """Whole frame to bitstream (reno_encode_frame): points device float
        [n][3]; each scale's symbols go to ceil(N / stream_symbols)
        interleaved rANS streams.  Returns the bitstream as a host uint32
        array (a view of ``out`` when given and large enough)."""
        n = int(points.shape[0])
        pts = points.contiguous()
        nw = ctypes.c_int64()
        buf = out if out is not None else np.empty(2 * n + 4096, np.uint32)
        cap = int(buf.size)
        for _ in range(2):              # a second try with the size the first one reported
            rc = lib().reno_encode_frame(self._h, _ptr(pts) if n else None, n, bit_depth, stream_symbols,
                                         buf.ctypes.data_as(_vp) if buf.size else None, cap, ctypes.byref(nw))
            if rc != RENO_E_CAPACITY or nw.value <= cap:
                break
            cap = int(nw.value)
            buf = np.empty(cap, np.uint32)
        self._check(rc)
        self._points = pts
        self.B = bit_depth
        return buf[:nw.value]

    def decode_frame(self, words: np.ndarray):
        """Bitstream (host uint32 array) to frame (reno_decode_frame): every
        scale rebuilt on the device; coords(B) are the decoded voxels."""
        w = np.ascontiguousarray(words, dtype=np.uint32)
        self._check(lib().reno_decode_frame(self._h, w.ctypes.data_as(_vp), w.size))
        self.B = int(w[1])

    def symbol_freqs(self, scale: int):
        n = self.num_voxels(scale)
        out = self._empty((max(n, 1), SYMBOLS), self.torch.int16)
        self._check(lib().reno_symbol_freqs(self._h, scale, _ptr(out)))
        return out[:n]


RENO_NOALLOC_MAX_PARENTS = 1 << 25


def expand_noalloc(keys, codes, child_keys, child_parent, result, first_child=None, stream=None):
    """FCG expansion without a context and without device allocation
    (reno_expand_noalloc): every argument is a caller-owned device tensor --
    keys int64 [n], codes uint8 [n], child_keys int64 [cap], child_parent int32
    [cap], result int64 [2] (children written, status), first_child int32 [n]
    or None.  Enqueued on ``stream`` (default: torch's current stream)."""
    import torch
    n = int(keys.shape[0])
    if int(codes.shape[0]) != n or (first_child is not None and int(first_child.shape[0]) < n):
        raise ValueError("keys, codes and first_child must have n entries")
    cap = min(int(child_keys.shape[0]), int(child_parent.shape[0]))
    for t in (keys, codes, child_keys, child_parent, result) + ((first_child,) if first_child is not None else ()):
        if not t.is_contiguous():
            raise ValueError("arguments must be contiguous")
    st = stream if stream is not None else torch.cuda.current_stream()
    rc = lib().reno_expand_noalloc(_ptr(keys), _ptr(codes), n, _ptr(child_keys), _ptr(child_parent), cap,
                                   _ptr(first_child), _ptr(result), ctypes.c_void_p(st.cuda_stream))
    if rc != RENO_OK:
        raise RenoError(rc, lib().reno_last_error(None).decode())


def rans_encode(sym: np.ndarray, freq: np.ndarray) -> np.ndarray:
    """Host rANS encode of one scale's symbols with per-symbol frequency tables."""
    s = np.ascontiguousarray(sym, dtype=np.uint8)
    f = np.ascontiguousarray(freq, dtype=np.uint16).reshape(-1, SYMBOLS)
    cap = s.size + 16
    out = np.empty(cap, dtype=np.uint32)
    nw = ctypes.c_int64()
    rc = lib().reno_rans_encode(s.ctypes.data_as(_vp), f.ctypes.data_as(_vp), s.size,
                                out.ctypes.data_as(_vp), cap, ctypes.byref(nw))
    if rc != RENO_OK:
        raise RenoError(rc, "rANS encode failed")
    return out[:nw.value].copy()


def rans_decode(words: np.ndarray, freq: np.ndarray, n: int) -> np.ndarray:
    """Host rANS decode with per-symbol tables of 256 (or, [n][16], 16) entries."""
    w = np.ascontiguousarray(words, dtype=np.uint32)
    k = 16 if (np.asarray(freq).ndim == 2 and np.asarray(freq).shape[1] == 16) else SYMBOLS
    f = np.ascontiguousarray(freq, dtype=np.uint16).reshape(-1, k)
    out = np.empty(n, dtype=np.uint8)
    fn = lib().reno_rans_decode16 if k == 16 else lib().reno_rans_decode
    rc = fn(w.ctypes.data_as(_vp), w.size, f.ctypes.data_as(_vp), n, out.ctypes.data_as(_vp))
    if rc != RENO_OK:
        raise RenoError(rc, "rANS decode failed")
    return out


def rans_encode_intervals(iv: np.ndarray, stride: int = 2, offset: int = 0) -> np.ndarray:
    """Host rANS encode from (start, freq) intervals: symbol i uses
    iv.flat[offset + i * stride] and the entry after it (a contiguous uint16
    array, e.g. [n][2], or [n][4] with offset 0 / 2 for the two stages)."""
    a = np.ascontiguousarray(iv, dtype=np.uint16).reshape(-1)
    n = (a.size - offset - 2) // stride + 1 if a.size >= offset + 2 else 0
    cap = n + 16
    out = np.empty(cap, dtype=np.uint32)
    nw = ctypes.c_int64()
    rc = lib().reno_rans_encode_intervals(a[offset:].ctypes.data_as(_vp), n, stride,
                                          out.ctypes.data_as(_vp), cap, ctypes.byref(nw))
    if rc != RENO_OK:
        raise RenoError(rc, "rANS encode failed")
    return out[:nw.value].copy()


RENO_RANS_MAX_STREAMS = 256


def rans_encode_streams(iv: np.ndarray, nstreams: int, stride: int = 2, offset: int = 0, threads: int = 0):
    """Interleaved multi-stream rANS encode from (start, freq) intervals (host
    memory, layout as rans_encode_intervals): symbol i goes to stream i mod S.
    Returns (words of all streams back to back, word count of each stream)."""
    a = np.ascontiguousarray(iv, dtype=np.uint16).reshape(-1)
    n = (a.size - offset - 2) // stride + 1 if a.size >= offset + 2 else 0
    cap = n + 16 * nstreams
    out = np.empty(cap, dtype=np.uint32)
    counts = np.zeros(nstreams, dtype=np.int64)
    rc = lib().reno_rans_encode_streams(a[offset:].ctypes.data_as(_vp), n, stride, nstreams, threads,
                                        out.ctypes.data_as(_vp), cap, counts.ctypes.data_as(_vp))
    if rc != RENO_OK:
        raise RenoError(rc, "rANS multi-stream encode failed")
    return out[:int(counts.sum())].copy(), counts


def rans_decode_streams(words: np.ndarray, counts: np.ndarray, start: np.ndarray, n: int, threads: int = 0,
                        out: np.ndarray | None = None) -> np.ndarray:
    """Decodes S interleaved streams (words back to back, counts [S]) with
    cumulative tables start [n][k] (k = 256 or 16) into n symbols."""
    w = np.ascontiguousarray(words, dtype=np.uint32)
    c = np.ascontiguousarray(counts, dtype=np.int64)
    st = np.ascontiguousarray(start, dtype=np.uint16)
    k = st.shape[1] if st.ndim == 2 else SYMBOLS
    sym = out if out is not None else np.empty(n, dtype=np.uint8)
    rc = lib().reno_rans_decode_streams(w.ctypes.data_as(_vp), c.ctypes.data_as(_vp), c.size, threads,
                                        st.ctypes.data_as(_vp), k, n, sym.ctypes.data_as(_vp))
    if rc != RENO_OK:
        raise RenoError(rc, "rANS multi-stream decode failed")
    return sym


def weights_to_device(w: dict, device="cuda") -> dict:
    """numpy weight dict (synth layout) -> fp32 device tensors."""
    import torch
    out = {"conv_w": [torch.from_numpy(np.ascontiguousarray(x)).to(device) for x in w["conv_w"]],
           "conv_b": [torch.from_numpy(np.ascontiguousarray(x)).to(device) for x in w["conv_b"]]}
    for name in ("head_w", "head_b", "head1_w", "head1_b", "emb_s1", "head2_w", "head2_b",
                 "emb_o", "emb_d"):
        if name in w:
            out[name] = torch.from_numpy(np.ascontiguousarray(w[name], dtype=np.float32)).to(device)
    for name in ("top_w", "top_b"):
        if name in w:
            out[name] = [torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(device)
                         for x in w[name]]
    return out
