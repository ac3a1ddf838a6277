"""C ABI: the library loads, exports every function include/reno.h declares,
rejects bad arguments before touching the GPU, and its host rANS coder round
trips.  Runs on the CPU (no kernel is launched)."""
import ctypes
import os
import re

import numpy as np
import pytest

import paper_2503_12382_amd as reno

HEADER = os.path.join(os.path.dirname(os.path.dirname(__file__)), "include", "reno.h")

pytestmark = pytest.mark.skipif(not os.path.exists(reno.LIB_PATH),
                                reason="libreno.so not built (run __graft_entry__.build())")


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return set(re.findall(r"\b(reno_[a-z_0-9]+)\s*\(", src))


def test_header_and_binding_agree():
    decl = declared_functions()
    assert decl == set(reno._SIGS), decl ^ set(reno._SIGS)
    assert len(decl) == 35


def _struct_fields(name):
    src = re.sub(r"/\*.*?\*/", "", open(HEADER).read(), flags=re.S)
    body = re.search(r"typedef struct \{([^{}]*)\}\s*" + name + r"\s*;", src).group(1)
    return [m.group(1) for m in re.finditer(r"(\w+)\s*(?:\[[^\]]*\])?\s*;", body)]


@pytest.mark.parametrize("name,cls", [("reno_params", reno.reno_params), ("reno_weights", reno.reno_weights)])
def test_struct_layouts_agree(name, cls):
    """The ctypes structures list the header's fields in the header's order."""
    assert _struct_fields(name) == [f[0] for f in cls._fields_]


def test_every_symbol_exported():
    L = ctypes.CDLL(reno.LIB_PATH)
    for name in declared_functions():
        assert hasattr(L, name), name


def test_create_rejects_bad_params_without_gpu():
    L = reno.lib()
    h = ctypes.c_void_p()
    assert L.reno_create(None, None, ctypes.byref(h)) == reno.RENO_E_INVALID
    good = dict(max_points=1000, max_model_voxels=0, max_bit_depth=12, min_bit_depth=4,
                range_m=131.0, in_features=11, channels=32, layers=3)
    bad_cases = [dict(max_points=0), dict(max_bit_depth=22), dict(min_bit_depth=12),
                 dict(range_m=-1.0), dict(range_m=float("inf")), dict(in_features=8),
                 dict(channels=24), dict(layers=0), dict(layers=9), dict(max_points=1 << 30),
                 dict(model_mode=2), dict(model_mode=reno.RENO_MODEL_TOP, precision=reno.RENO_PREC_BF16X3)]
    for bad in bad_cases:
        p = reno.reno_params(**{**good, **bad})
        rc = L.reno_create(ctypes.byref(p), None, ctypes.byref(h))
        assert rc == reno.RENO_E_INVALID, bad
        assert L.reno_last_error(None)                 # a message is set


def test_null_context_calls():
    L = reno.lib()
    assert L.reno_destroy(None) == reno.RENO_E_INVALID
    assert L.reno_sync(None) == reno.RENO_E_INVALID
    assert L.reno_build_pyramid(None, None, 0, 10) == reno.RENO_E_INVALID
    assert L.reno_expand(None, 4, None) == reno.RENO_E_INVALID
    assert L.reno_predict_probs(None, 5, None, None) == reno.RENO_E_INVALID
    assert L.reno_code_length(None, 5, None, None) == reno.RENO_E_INVALID


def _random_tables(rs, n, peaked):
    logits = rs.normal(size=(n, 256)) * (6.0 if peaked else 1.0)
    p = np.exp(logits - logits.max(1, keepdims=True))
    p /= p.sum(1, keepdims=True)
    f = 1 + np.floor(p.astype(np.float32) * np.float32(65024)).astype(np.int64)
    f[np.arange(n), f.argmax(1)] += 65536 - f.sum(1)
    assert np.all(f.sum(1) == 65536)
    return p, f.astype(np.uint16)


@pytest.mark.parametrize("peaked", [False, True])
def test_host_rans_round_trip(peaked):
    rs = np.random.default_rng(31 + peaked)
    n = 30000
    p, f = _random_tables(rs, n, peaked)
    sym = np.array([rs.choice(256, p=pi) for pi in p], dtype=np.uint8)
    words = reno.rans_encode(sym, f)
    assert np.array_equal(reno.rans_decode(words, f, n), sym)
    ideal = -np.log2(f[np.arange(n), sym].astype(np.float64) / 65536.0).sum()
    coded = 32.0 * words.size
    assert abs(coded - ideal) <= n * np.log2(1 + 2.0 ** -15) + 96


def test_host_rans_errors():
    rs = np.random.default_rng(5)
    n = 100
    _, f = _random_tables(rs, n, False)
    sym = rs.integers(0, 256, n).astype(np.uint8)
    words = reno.rans_encode(sym, f)
    with pytest.raises(reno.RenoError):
        reno.rans_decode(words[:-1], f, n)            # truncated
    bad = f.copy()
    bad[3, 0] += 1                                     # table no longer sums to 2^16
    with pytest.raises(reno.RenoError):
        reno.rans_encode(sym, bad)


def test_host_rans_empty_stream():
    f = np.zeros((0, 256), np.uint16)
    words = reno.rans_encode(np.zeros(0, np.uint8), f)
    assert words.size == 2
    assert reno.rans_decode(words, f, 0).size == 0


def test_expand_noalloc_rejects_bad_arguments_without_gpu():
    """Argument checks of the allocation-free expansion come before any HIP call."""
    L = reno.lib()
    res = ctypes.c_void_p(16)            # never dereferenced: every case fails its checks first
    one = ctypes.c_void_p(8)
    cases = [
        (one, one, reno.RENO_NOALLOC_MAX_PARENTS + 1, one, one, 8, None, res),   # too many parents
        (one, one, -1, one, one, 8, None, res),                                  # negative count
        (one, one, 4, one, one, 1 << 31, None, res),                             # capacity too large
        (one, one, 4, one, one, -1, None, res),                                  # negative capacity
        (one, one, 4, one, one, 8, None, None),                                  # no result array
        (None, one, 4, one, one, 8, None, res),                                  # no keys
        (one, None, 4, one, one, 8, None, res),                                  # no codes
        (one, one, 4, None, one, 8, None, res),                                  # no child keys
        (one, one, 4, one, None, 8, None, res),                                  # no child parents
    ]
    for args in cases:
        assert L.reno_expand_noalloc(*args, None) == reno.RENO_E_INVALID, args
        assert L.reno_last_error(None)


def test_frame_coding_rejects_bad_arguments_without_gpu():
    """Whole-frame calls check their arguments before any HIP call."""
    L = reno.lib()
    nw = ctypes.c_int64()
    buf = (ctypes.c_uint32 * 8)()
    assert L.reno_encode_frame(None, None, 0, 10, 16, buf, 8, ctypes.byref(nw)) == reno.RENO_E_INVALID
    assert L.reno_decode_frame(None, buf, 8) == reno.RENO_E_INVALID


def _intervals_and_starts(f, sym):
    """(start, freq) of each symbol and the cumulative tables of f."""
    start = np.zeros_like(f, dtype=np.int64)
    start[:, 1:] = np.cumsum(f[:, :-1].astype(np.int64), axis=1)
    n = len(sym)
    iv = np.stack([start[np.arange(n), sym], f[np.arange(n), sym].astype(np.int64)], 1).astype(np.uint16)
    return iv, start.astype(np.uint16)


@pytest.mark.parametrize("nstreams,threads", [(1, 1), (7, 3), (16, 0), (64, 16)])
def test_host_rans_streams_are_single_streams_and_round_trip(nstreams, threads):
    """Stream j of the interleaved coder is exactly the single-stream coding of
    symbols j, j + S, ...: word for word equal to the CPU oracle's independent
    rANS write-up of that subsequence; the threaded decoder with cumulative
    tables restores every symbol."""
    import oracle
    rs = np.random.default_rng(40 + nstreams)
    n = 5000
    p, f = _random_tables(rs, n, peaked=True)
    sym = np.array([rs.choice(256, p=pi) for pi in p], dtype=np.uint8)
    iv, start = _intervals_and_starts(f, sym)
    words, counts = reno.rans_encode_streams(iv, nstreams, threads=threads)
    assert counts.size == nstreams and words.size == counts.sum()
    off = np.concatenate([[0], np.cumsum(counts)])
    for j in range(nstreams):
        ref = oracle.rans_encode(sym[j::nstreams], f[j::nstreams].astype(np.uint32))
        np.testing.assert_array_equal(words[off[j]:off[j + 1]], ref, err_msg=f"stream {j}")
    dec = reno.rans_decode_streams(words, counts, start, n, threads=threads)
    np.testing.assert_array_equal(dec, sym)


def test_host_rans_streams_16_symbol_tables_and_errors():
    rs = np.random.default_rng(44)
    n, S = 3001, 8
    logits = rs.normal(size=(n, 16)) * 3
    pr = np.exp(logits - logits.max(1, keepdims=True))
    pr /= pr.sum(1, keepdims=True)
    f = 1 + np.floor(pr.astype(np.float32) * np.float32(65504)).astype(np.int64)
    f[np.arange(n), f.argmax(1)] += 65536 - f.sum(1)
    f = f.astype(np.uint16)
    sym = np.array([rs.choice(16, p=pi) for pi in pr], dtype=np.uint8)
    iv, start = _intervals_and_starts(f, sym)
    words, counts = reno.rans_encode_streams(iv, S)
    assert np.array_equal(reno.rans_decode_streams(words, counts, start, n), sym)
    single = reno.rans_decode(reno.rans_encode_intervals(iv), f, n)     # the single-stream coder agrees
    assert np.array_equal(single, sym)
    with pytest.raises(reno.RenoError):                                   # a stream cut short
        bad = counts.copy()
        bad[3] -= 1
        reno.rans_decode_streams(np.delete(words, counts[:3].sum()), bad, start, n)
    with pytest.raises(reno.RenoError):                                   # a table that does not start at 0
        s2 = start.copy()
        s2[10, 0] = 1
        reno.rans_decode_streams(words, counts, s2, n)
    with pytest.raises(reno.RenoError):                                   # an empty interval
        iv2 = iv.copy()
        iv2[5, 1] = 0
        reno.rans_encode_streams(iv2, S)
    # fewer symbols than streams: the empty streams hold the two flush words
    w2, c2 = reno.rans_encode_streams(iv[:3], S)
    assert list(c2[3:]) == [2] * (S - 3)
    assert np.array_equal(reno.rans_decode_streams(w2, c2, start[:3], 3), sym[:3])
