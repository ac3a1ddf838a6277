"""Pins of the CPU oracle against what the paper and the mathematics fix.

Nothing here compares the oracle with itself: every check is a hand-worked
fixture, a closed form, an invariant implied by the equations, a library
routine (torch conv3d) or brute force on tiny inputs.
"""
import itertools
import json
import math
import os

import numpy as np
import pytest

import oracle
from synth import CONFIGS, gen_weights

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _load(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


# ---- P6: ordering -----------------------------------------------------------------------

def test_morton_worked_values():
    g = _load("morton_worked.json")
    for (x, y, z), key in g["cases"]:
        assert oracle.morton(x, y, z, g["bits"]) == key


def test_morton_child_relation():
    rs = np.random.default_rng(5)
    for _ in range(200):
        b = int(rs.integers(1, 20))
        v = rs.integers(0, 1 << b, size=3)
        k = oracle.morton(int(v[0]), int(v[1]), int(v[2]), b)
        for d in range(8):
            c = 2 * v + np.array([d & 1, (d >> 1) & 1, (d >> 2) & 1])
            assert oracle.morton(int(c[0]), int(c[1]), int(c[2]), b + 1) == 8 * k + d


# ---- P5: quantisation -------------------------------------------------------------------

def test_quantize_edges():
    g = _load("quantize_edges.json")
    pts = np.array([[p, p, p] for p, _ in g["cases"]], dtype=np.float32)
    q = oracle.quantize(pts, g["B"], g["R"])
    for (p, expect), row in zip(g["cases"], q):
        assert list(row) == [expect] * 3, p


def test_quantize_error_bound():
    # reconstruction at the cell centre is within half a step of the input
    # (the paper's "+-8 mm at 14 bits" statement of precision)
    rs = np.random.default_rng(1)
    for B, R in [(10, 51.2), (12, 131.0), (14, 131.0), (16, 131.0)]:
        pts = rs.uniform(-R * 0.999, R * 0.999, size=(5000, 3)).astype(np.float32)
        q = oracle.quantize(pts, B, R)
        step = 2.0 * R / (1 << B)
        rec = -R + (q + 0.5) * step
        assert np.abs(rec - pts.astype(np.float64)).max() <= step / 2 * (1 + 1e-9)
    assert 2 * 131.0 / (1 << 14) / 2 == pytest.approx(0.008, rel=0.01)     # +-8 mm
    assert 2 * 131.0 / (1 << 12) / 2 == pytest.approx(0.032, rel=0.01)     # +-3.2 cm


def test_quantize_rejects_nonfinite():
    with pytest.raises(ValueError):
        oracle.quantize(np.array([[0, np.nan, 0]], np.float32), 10, 51.2)
    with pytest.raises(ValueError):
        oracle.Pyramid.from_points(np.array([[np.inf, 0, 0]], np.float32), 10, 4, 51.2)


# ---- FOG / FCG worked example -----------------------------------------------------------

def test_fog_tiny_fixture():
    g = _load("fog_tiny.json")
    P = oracle.Pyramid.from_voxels(np.array(g["input_xyz"]), g["B"], g["b0"])
    for b_s, lv in g["levels"].items():
        b = int(b_s)
        assert P.xyz(b).tolist() == lv["xyz"]
        assert P.keys(b).tolist() == lv["keys"]
        assert P.parent(b).tolist() == lv["parent"]
        if "codes" in lv:
            assert P.codes(b).tolist() == lv["codes"]
    # FCG reproduces the finest scale
    assert P.expand(1, np.array(g["levels"]["1"]["codes"], np.uint8)).tolist() == g["levels"]["2"]["xyz"]


# ---- P4: FOG(FCG(c)) = c for every code -----------------------------------------------

def test_fog_fcg_bijection_all_codes():
    for c in range(1, 256):
        for base in ([0, 0, 0], [3, 1, 2]):
            # expand one voxel of scale 2 with code c, then rebuild its code by FOG
            kids = [[2 * base[0] + (d & 1), 2 * base[1] + ((d >> 1) & 1), 2 * base[2] + ((d >> 2) & 1)]
                    for d in range(8) if (c >> d) & 1]
            P = oracle.Pyramid.from_voxels(np.array(kids), 3, 2)
            assert P.xyz(2).tolist() == [base]
            assert P.codes(2).tolist() == [c]
            assert P.expand(2, np.array([c], np.uint8)).tolist() == P.xyz(3).tolist()


# ---- P1-P3: invariants on random clouds and a real scan ---------------------------------

def _check_invariants(P):
    for b in range(P.b0, P.B):
        codes = P.codes(b)
        assert codes.min() >= 1 and codes.max() <= 255                 # Eq. 1 range
        assert int(np.unpackbits(codes).sum()) == P.num(b + 1)          # popcounts sum to N_{b+1}
        assert P.num(b) <= P.num(b + 1) <= 8 * P.num(b)
        # expansion of every scale reproduces the next scale's array exactly (Eq. 2)
        assert np.array_equal(P.expand(b, codes), P.xyz(b + 1))
    for b in range(P.b0, P.B + 1):
        keys = P.keys(b)
        assert np.all(keys[1:] > keys[:-1])                             # strictly ascending
        xyz = P.xyz(b)
        if b > P.b0:
            par = P.parent(b)
            assert np.array_equal(P.xyz(b - 1)[par], xyz >> 1)


def test_invariants_random_clouds():
    rs = np.random.default_rng(7)
    for trial in range(20):
        B = int(rs.integers(2, 9))
        b0 = int(rs.integers(0, B))
        n = int(rs.integers(1, 400))
        xyz = rs.integers(0, 1 << B, size=(n, 3))
        if trial % 3 == 0:                                               # clustered
            xyz = np.clip(xyz // 4 + (1 << (B - 1)), 0, (1 << B) - 1)
        P = oracle.Pyramid.from_voxels(xyz, B, b0)
        _check_invariants(P)
        # brute force: scale b is the set of distinct (xyz >> (B-b))
        for b in range(b0, B + 1):
            expect = {tuple(v) for v in (xyz >> (B - b)).tolist()}
            assert {tuple(v) for v in P.xyz(b).tolist()} == expect


def test_invariants_tiny_scan(scan_cache):
    c = CONFIGS[0]
    P = oracle.Pyramid.from_points(scan_cache(0), c.bit_depth, c.min_bit_depth, c.range_m)
    _check_invariants(P)


def test_recomposition_from_codes(scan_cache):
    # Eq. 2: the initial state plus O_{b0..B-1} reproduce every scale
    c = CONFIGS[0]
    P = oracle.Pyramid.from_points(scan_cache(0), c.bit_depth, c.min_bit_depth, c.range_m)
    codes = [P.codes(b) for b in range(c.min_bit_depth, c.bit_depth)]
    D = oracle.Pyramid.from_codes(P.xyz(c.min_bit_depth), c.min_bit_depth, c.bit_depth, codes)
    for b in range(c.min_bit_depth, c.bit_depth + 1):
        assert np.array_equal(D.xyz(b), P.xyz(b))
        assert np.array_equal(D.parent(b), P.parent(b))


# ---- P13 / P14: metamorphic ---------------------------------------------------------------

def test_shuffle_and_duplicates_invariance(scan_cache):
    c = CONFIGS[0]
    pts = scan_cache(0)
    P = oracle.Pyramid.from_points(pts, c.bit_depth, c.min_bit_depth, c.range_m)
    rs = np.random.default_rng(3)
    pts2 = np.concatenate([pts, pts[rs.integers(0, len(pts), 500)]])[rs.permutation(len(pts) + 500)]
    Q = oracle.Pyramid.from_points(pts2, c.bit_depth, c.min_bit_depth, c.range_m)
    assert Q.raw_points == len(pts) + 500
    for b in range(c.min_bit_depth, c.bit_depth + 1):
        assert np.array_equal(P.xyz(b), Q.xyz(b))
        if b < c.bit_depth:
            assert np.array_equal(P.codes(b), Q.codes(b))


def test_translation_by_coarse_cell():
    rs = np.random.default_rng(11)
    B, b0 = 8, 3
    xyz = rs.integers(40, 200, size=(600, 3))
    shift = 1 << (B - b0)                                                 # one coarse cell
    P = oracle.Pyramid.from_voxels(xyz, B, b0)
    Q = oracle.Pyramid.from_voxels(xyz + shift, B, b0)
    for b in range(b0, B):
        # the voxel -> code map is translated; the Morton order of whole coarse
        # cells may change, so compare as maps
        s = shift >> (B - b)
        mp = {tuple(np.add(v, s).tolist()): c for v, c in zip(P.xyz(b).tolist(), P.codes(b).tolist())}
        mq = {tuple(v): c for v, c in zip(Q.xyz(b).tolist(), Q.codes(b).tolist())}
        assert mp == mq


# ---- neighbour map ----------------------------------------------------------------------

def test_neighbor_map_brute_force():
    rs = np.random.default_rng(2)
    B = 5
    xyz = rs.integers(0, 1 << B, size=(300, 3))
    P = oracle.Pyramid.from_voxels(xyz, B, 2)
    for b in (3, 4, 5):
        v = P.xyz(b)
        nb = P.neighbors(b)
        index = {tuple(p): i for i, p in enumerate(v.tolist())}
        for i, p in enumerate(v.tolist()):
            for dz, dy, dx in itertools.product((-1, 0, 1), repeat=3):
                k = (dx + 1) + 3 * (dy + 1) + 9 * (dz + 1)
                q = (p[0] + dx, p[1] + dy, p[2] + dz)
                expect = index.get(q, -1)
                assert nb[i, k] == expect
        assert np.array_equal(nb[:, 13], np.arange(len(v)))


def test_neighbor_map_brute_force_kernel5():
    """5 x 5 x 5 neighbourhoods: k = (dx+2) + 5(dy+2) + 25(dz+2), centre 62."""
    rs = np.random.default_rng(12)
    B = 5
    xyz = rs.integers(0, 1 << B, size=(250, 3))
    P = oracle.Pyramid.from_voxels(xyz, B, 2)
    for b in (3, 5):
        v = P.xyz(b)
        nb = P.neighbors(b, 5)
        assert nb.shape == (len(v), 125)
        index = {tuple(p): i for i, p in enumerate(v.tolist())}
        lim = 1 << b
        for i, p in enumerate(v.tolist()):
            for dz, dy, dx in itertools.product(range(-2, 3), repeat=3):
                k = (dx + 2) + 5 * (dy + 2) + 25 * (dz + 2)
                q = (p[0] + dx, p[1] + dy, p[2] + dz)
                inside = all(0 <= c < lim for c in q)
                assert nb[i, k] == (index.get(q, -1) if inside else -1)
        assert np.array_equal(nb[:, 62], np.arange(len(v)))
        # the 3 x 3 x 3 map is the centre of the 5 x 5 x 5 one
        sub = [(dx + 2) + 5 * (dy + 2) + 25 * (dz + 2) for dz in (-1, 0, 1) for dy in (-1, 0, 1) for dx in (-1, 0, 1)]
        np.testing.assert_array_equal(nb[:, sub], P.neighbors(b))


# ---- P7 / P8: sparse conv vs dense conv3d ------------------------------------------------

def test_sparse_conv_equals_dense_conv3d():
    import torch
    rs = np.random.default_rng(4)
    b = 4
    G = 1 << b                                                            # the 16^3 grid
    flat = rs.choice(G ** 3, size=400, replace=False)
    xyz = np.stack([flat % G, (flat // G) % G, flat // (G * G)], axis=1)
    for c_in, c_out, relu in [(11, 16, True), (32, 32, True), (5, 7, False)]:
        feats = rs.normal(size=(400, c_in))
        W = rs.normal(size=(27, c_in, c_out)).astype(np.float32)
        bias = rs.normal(size=c_out).astype(np.float32)
        y = oracle.sparse_conv(xyz, b, feats, W, bias, relu)
        # dense: grid [c][z][y][x], weight[co][ci][dz+1][dy+1][dx+1] = W[k][ci][co]
        grid = torch.zeros((1, c_in, G, G, G), dtype=torch.float64)
        grid[0, :, xyz[:, 2], xyz[:, 1], xyz[:, 0]] = torch.from_numpy(feats.T)
        Wt = torch.zeros((c_out, c_in, 3, 3, 3), dtype=torch.float64)
        for k in range(27):
            dx, dy, dz = k % 3, (k // 3) % 3, k // 9
            Wt[:, :, dz, dy, dx] = torch.from_numpy(W[k].astype(np.float64).T)
        out = torch.nn.functional.conv3d(grid, Wt, torch.from_numpy(bias.astype(np.float64)), padding=1)
        if relu:
            out = torch.relu(out)
        dense = out[0, :, xyz[:, 2], xyz[:, 1], xyz[:, 0]].T.numpy()       # mask to the voxels
        np.testing.assert_allclose(y, dense, rtol=1e-12, atol=1e-12)


def test_sparse_conv_kernel5_equals_dense_conv3d():
    import torch
    rs = np.random.default_rng(14)
    b = 4
    G = 1 << b
    flat = rs.choice(G ** 3, size=500, replace=False)
    xyz = np.stack([flat % G, (flat // G) % G, flat // (G * G)], axis=1)
    for c_in, c_out, relu in [(16, 16, True), (6, 9, False)]:
        feats = rs.normal(size=(500, c_in))
        W = rs.normal(size=(125, c_in, c_out)).astype(np.float32)
        bias = rs.normal(size=c_out).astype(np.float32)
        y = oracle.sparse_conv(xyz, b, feats, W, bias, relu)
        grid = torch.zeros((1, c_in, G, G, G), dtype=torch.float64)
        grid[0, :, xyz[:, 2], xyz[:, 1], xyz[:, 0]] = torch.from_numpy(feats.T)
        Wt = torch.zeros((c_out, c_in, 5, 5, 5), dtype=torch.float64)
        for k in range(125):
            dx, dy, dz = k % 5, (k // 5) % 5, k // 25
            Wt[:, :, dz, dy, dx] = torch.from_numpy(W[k].astype(np.float64).T)
        out = torch.nn.functional.conv3d(grid, Wt, torch.from_numpy(bias.astype(np.float64)), padding=2)
        if relu:
            out = torch.relu(out)
        dense = out[0, :, xyz[:, 2], xyz[:, 1], xyz[:, 0]].T.numpy()
        np.testing.assert_allclose(y, dense, rtol=1e-12, atol=1e-12)


def test_isolated_voxel_uses_centre_tap_only():
    rs = np.random.default_rng(9)
    xyz = np.array([[1, 1, 1], [9, 9, 9]])
    feats = rs.normal(size=(2, 6))
    W = rs.normal(size=(27, 6, 4)).astype(np.float32)
    bias = rs.normal(size=4).astype(np.float32)
    y = oracle.sparse_conv(xyz, 4, feats, W, bias, False)
    expect = bias.astype(np.float64) + feats @ W[13].astype(np.float64)
    np.testing.assert_allclose(y, expect, rtol=1e-13, atol=1e-13)


# ---- features (Eqs. 7-8) -----------------------------------------------------------------

def test_features_from_fixture():
    g = _load("fog_tiny.json")
    P = oracle.Pyramid.from_voxels(np.array(g["input_xyz"]), g["B"], g["b0"])
    f = P.features(2)
    # V_2 = (0,0,0) (1,0,0) (0,1,1) (2,3,3) (3,3,3); deltas 0 1 6 6 7; parent codes 67 67 67 192 192
    deltas = [0, 1, 6, 6, 7]
    pcode = [67, 67, 67, 192, 192]
    for i in range(5):
        assert f[i, :3].tolist() == [(deltas[i] >> j) & 1 for j in range(3)]
        assert f[i, 3:].tolist() == [(pcode[i] >> j) & 1 for j in range(8)]


# ---- P9-P11: head, softmax and bits -------------------------------------------------------

def _zero_weights(C, L):
    w = gen_weights(C, L, seed=5)
    w["conv_w"] = [np.zeros_like(x) for x in w["conv_w"]]
    w["conv_b"] = [np.zeros_like(x) for x in w["conv_b"]]
    w["head_w"] = np.zeros_like(w["head_w"])
    w["head_b"] = np.zeros_like(w["head_b"])
    return w


def test_zero_weights_give_8_bits_and_closed_form_total(scan_cache):
    c = CONFIGS[0]
    P = oracle.Pyramid.from_points(scan_cache(0), c.bit_depth, c.min_bit_depth, c.range_m)
    w = _zero_weights(c.channels, c.layers)
    for b in range(c.min_bit_depth + 1, c.bit_depth):
        lg, lse, bits = P.model(b, w)
        np.testing.assert_allclose(bits, 8.0, rtol=0, atol=1e-12)
        np.testing.assert_allclose(lse, math.log(256.0), atol=1e-12)
    T, per = P.totals(w)
    Nb0 = P.num(c.min_bit_depth)
    expect = 32 + Nb0 * (3 * c.min_bit_depth + 8) + 8 * sum(P.num(b) for b in range(c.min_bit_depth + 1, c.bit_depth))
    assert T == pytest.approx(expect, rel=1e-12)


def test_one_hot_bias_closed_form(scan_cache):
    c = CONFIGS[0]
    P = oracle.Pyramid.from_points(scan_cache(0), c.bit_depth, c.min_bit_depth, c.range_m)
    w = _zero_weights(c.channels, c.layers)
    s, cval = 85, 2.5
    w["head_b"][s] = cval
    b = c.min_bit_depth + 3
    _, _, bits = P.model(b, w)
    codes = P.codes(b)
    ec = math.exp(cval)
    expect = np.where(codes == s, -math.log2(ec / (ec + 255)), -math.log2(1 / (ec + 255)))
    np.testing.assert_allclose(bits, expect, rtol=1e-12)


def test_probability_rows_sum_to_one_and_bits_match_logits(scan_cache):
    c = CONFIGS[0]
    P = oracle.Pyramid.from_points(scan_cache(0), c.bit_depth, c.min_bit_depth, c.range_m)
    w = gen_weights(c.channels, c.layers, bias_std=0.1, head_scale=10.0)
    b = c.bit_depth - 1
    lg, lse, bits = P.model(b, w)
    p = np.exp(lg - lse[:, None])
    np.testing.assert_allclose(p.sum(1), 1.0, atol=1e-6)
    codes = P.codes(b)
    np.testing.assert_allclose(bits, -np.log2(p[np.arange(len(codes)), codes]), rtol=1e-9)


def test_model_rows_subset_matches_full(scan_cache):
    # the receptive-field evaluation of a subset equals the full evaluation
    c = CONFIGS[0]
    P = oracle.Pyramid.from_points(scan_cache(0), c.bit_depth, c.min_bit_depth, c.range_m)
    w = gen_weights(c.channels, c.layers, bias_std=0.1)
    b = c.bit_depth - 2
    full, _, _ = P.model(b, w)
    rows = np.array([0, 5, 17, P.num(b) - 1])
    sub, _, _ = P.model(b, w, rows=rows)
    np.testing.assert_array_equal(sub, full[rows])


def test_model_two_layer_by_hand():
    """Logits of a tiny two-voxel scale computed by hand with numpy:
    features -> conv (centre tap + the one neighbour) -> ReLU -> head."""
    rs = np.random.default_rng(12)
    # scale 2 voxels (0,0,0) and (1,0,0): neighbours of each other at dx = +-1
    P = oracle.Pyramid.from_voxels(np.array([[0, 0, 0], [1, 0, 0], [3, 3, 3]]), 2, 0)
    w = gen_weights(4, 1, seed=8, bias_std=0.3)
    x = P.features(2)                                   # [3][11]
    W = w["conv_w"][0].astype(np.float64)
    bias = w["conv_b"][0].astype(np.float64)
    # k for dx = +1: (2) + 3*1 + 9*1 = 14; for dx = -1: 0 + 3 + 9 = 12; centre 13
    h = np.zeros((3, 4))
    h[0] = bias + x[0] @ W[13] + x[1] @ W[14]
    h[1] = bias + x[1] @ W[13] + x[0] @ W[12]
    h[2] = bias + x[2] @ W[13]
    h = np.maximum(h, 0)
    z = w["head_b"].astype(np.float64) + h @ w["head_w"].astype(np.float64)
    lg, _, _ = P.model(2, w)
    np.testing.assert_allclose(lg, z, rtol=1e-12, atol=1e-12)


def _plain_model_by_composition(P, b, w):
    """The plain model of scale b (Sec. 3.2, Eqs. 7-10 in the configured form)
    rebuilt from pinned pieces: input features written out with numpy from the
    coordinates (octant bits of each voxel, bits of its parent's code, parent
    found by halving the coordinates), then every layer l = 1..L through the
    standalone sparse conv pinned against a dense conv3d, with layer l's own
    weights and bias, then the linear head with numpy."""
    xyz = P.xyz(b)
    coarse = {tuple(v): i for i, v in enumerate(P.xyz(b - 1).tolist())}
    par = np.array([coarse[tuple(v)] for v in (xyz >> 1).tolist()], dtype=np.int64)
    pcode = P.codes(b - 1)[par].astype(np.int64)
    x = np.zeros((len(xyz), 11))
    for a in range(3):
        x[:, a] = xyz[:, a] & 1
    for j in range(8):
        x[:, 3 + j] = (pcode >> j) & 1
    h = x
    for l in range(w["layers"]):
        h = oracle.sparse_conv(xyz, b, h, w["conv_w"][l], w["conv_b"][l], True)
    return h @ w["head_w"].astype(np.float64) + w["head_b"].astype(np.float64)


@pytest.mark.parametrize("C,L", [(16, 2), (32, 3), (16, 4)])
def test_model_layer_chain_equals_composition(scan_cache, C, L):
    """Pins the layer loop of the plain model for L >= 2: a wrong layer-to-weight
    index, a bias taken from another layer, or a broken C_in hand-over between
    layers changes the logits far beyond the 1e-9 bound.  Biases are non-zero
    and differ per layer so that each of them is exercised."""
    c = CONFIGS[0]
    P = oracle.Pyramid.from_points(scan_cache(0), c.bit_depth, c.min_bit_depth, c.range_m)
    w = gen_weights(C, L, seed=31 + L, bias_std=0.2, head_scale=3.0)
    for b in (c.min_bit_depth + 2, c.bit_depth - 1):
        lg, lse, bits = P.model(b, w)
        ref = _plain_model_by_composition(P, b, w)
        np.testing.assert_allclose(lg, ref, rtol=0, atol=1e-9)
        code = P.codes(b).astype(np.int64)
        m = ref.max(1)
        ref_lse = m + np.log(np.exp(ref - m[:, None]).sum(1))
        np.testing.assert_allclose(lse, ref_lse, rtol=0, atol=1e-9)
        np.testing.assert_allclose(bits, (ref_lse - ref[np.arange(len(code)), code]) / math.log(2),
                                   rtol=0, atol=1e-9)


# ---- P12: rANS ------------------------------------------------------------------------------

def test_rans_round_trip_and_length():
    rs = np.random.default_rng(21)
    n = 20000
    logits = rs.normal(size=(n, 256)) * 3
    p = np.exp(logits - logits.max(1, keepdims=True))
    p /= p.sum(1, keepdims=True)
    freq = oracle.freqs_from_probs(p)
    assert np.all(freq.sum(1) == 65536) and freq.min() >= 1
    sym = np.array([rs.choice(256, p=pi) for pi in p], dtype=np.uint8)
    words = oracle.rans_encode(sym, freq)
    dec = oracle.rans_decode(words, freq, n)
    assert np.array_equal(dec, sym)
    ideal = -np.log2(freq[np.arange(n), sym] / 65536.0).sum()
    coded = 32 * words.size
    # state in [2^31, 2^63): per-symbol excess below log2(1 + 2^-15); 64 flush bits + <32 padding
    assert coded >= ideal - n * math.log2(1 + 2 ** -15) - 1e-6
    assert coded <= ideal + n * math.log2(1 + 2 ** -15) + 96


def test_rans_rejects_corruption():
    rs = np.random.default_rng(22)
    n = 500
    freq = np.full((n, 256), 256, dtype=np.uint32)
    sym = rs.integers(0, 256, n).astype(np.uint8)
    words = oracle.rans_encode(sym, freq)
    with pytest.raises(ValueError):
        oracle.rans_decode(words[:-1], freq, n)


# ---- bitwise two-stage head (Sec. 3.2, Eqs. 11-13) -------------------------------------

def _two_stage_weights(C, L, seed=9):
    return gen_weights(C, L, seed=seed, bias_std=0.2, two_stage=True)


def _factorised_one_stage(w, shift=None):
    """One-stage head whose logits split as z(O) = u(O & 15) + v(O >> 4): with no
    S1 dependence in stage 2, P(O) = softmax(u)[S1] * softmax(v)[S2] exactly."""
    o = np.arange(256)
    f = dict(w)
    f["head_w"] = (w["head1_w"][:, o & 15].astype(np.float64) + w["head2_w"][:, o >> 4]).astype(np.float32)
    hb = w["head1_b"][o & 15].astype(np.float64) + w["head2_b"][o >> 4]
    if shift is not None:
        hb = hb + shift[o >> 4]
    f["head_b"] = hb.astype(np.float32)
    return f


def _fp32_exact(w):
    """Weights whose fp32 sums used above are exact (values on a 2^-10 grid)."""
    out = dict(w)
    for k in ("head1_w", "head2_w", "head1_b", "head2_b", "emb_s1"):
        out[k] = (np.round(np.asarray(w[k], np.float64) * 1024) / 1024).astype(np.float32)
    return out


def test_two_stage_without_embedding_equals_factorised_one_stage(scan_cache):
    c = CONFIGS[0]
    P = oracle.Pyramid.from_points(scan_cache(0), c.bit_depth, c.min_bit_depth, c.range_m)
    w = _fp32_exact(_two_stage_weights(c.channels, c.layers))
    w["emb_s1"] = np.zeros_like(w["emb_s1"])
    one = _factorised_one_stage(w)
    for b in range(c.min_bit_depth + 1, c.bit_depth):
        _, _, _, _, bits2 = P.model2(b, w)
        _, _, bits1 = P.model(b, one)
        np.testing.assert_allclose(bits2, bits1, rtol=0, atol=1e-9)
    # the same with one embedding vector for every S1: it only moves stage-2 logits by head2_w^T e
    e = (np.arange(c.channels) % 7 - 3).astype(np.float32) / 8
    w["emb_s1"] = np.tile(e, (16, 1))
    one = _factorised_one_stage(w, shift=w["head2_w"].astype(np.float64).T @ e)
    b = c.bit_depth - 1
    np.testing.assert_allclose(P.model2(b, w)[4], P.model(b, one)[2], rtol=0, atol=1e-9)
    T2, _ = P.totals(w)
    T1, _ = P.totals(one)
    assert T2 == pytest.approx(T1, rel=1e-12)


def test_two_stage_embedding_limit_selects_s2():
    """Stage 2 reads the first 16 channels (head2_w = [I; 0]) and Emb(S1) puts a
    large logit on symbol g(S1): S2 costs ~0 bits where S2 = g(S1) and about
    gamma / ln 2 elsewhere, which fixes S1 = low nibble, S2 = high nibble and the
    row of the embedding that is used."""
    rs = np.random.default_rng(4)
    B, b0 = 7, 3
    xyz = rs.integers(0, 1 << B, size=(1500, 3)) // 2 + 20
    P = oracle.Pyramid.from_voxels(xyz, B, b0)
    C, L, gamma = 16, 2, 60.0
    w = _two_stage_weights(C, L, seed=5)
    w["head2_w"] = np.eye(C, 16, dtype=np.float32)
    w["head2_b"] = np.zeros(16, np.float32)
    g = (5 * np.arange(16) + 3) % 16
    emb = np.zeros((16, C), np.float32)
    emb[np.arange(16), g] = gamma
    w["emb_s1"] = emb
    hits = misses = 0
    for b in range(b0 + 1, B):
        l1, l2, lse1, lse2, bits = P.model2(b, w)
        code = P.codes(b).astype(np.int64)
        s1, s2 = code & 15, code >> 4
        stage1 = (lse1 - l1[np.arange(len(code)), s1]) / math.log(2)
        stage2 = bits - stage1
        hit = s2 == g[s1]
        hits += hit.sum()
        misses += (~hit).sum()
        assert np.all(stage2[hit] < 1e-12 + 1e-9)
        assert np.all(stage2[~hit] > 40.0)
        # the winning stage-2 logit is symbol g(S1) for every voxel
        assert np.array_equal(l2.argmax(1), g[s1])
    assert hits > 0 and misses > 0


def test_two_stage_zero_heads_give_8_bits(scan_cache):
    c = CONFIGS[0]
    P = oracle.Pyramid.from_points(scan_cache(0), c.bit_depth, c.min_bit_depth, c.range_m)
    w = _two_stage_weights(c.channels, c.layers)
    for k in ("head1_w", "head1_b", "head2_w", "head2_b"):
        w[k] = np.zeros_like(w[k])
    for b in range(c.min_bit_depth + 1, c.bit_depth):
        _, _, lse1, lse2, bits = P.model2(b, w)
        np.testing.assert_allclose(bits, 8.0, rtol=0, atol=1e-12)
        np.testing.assert_allclose(lse1, math.log(16.0), atol=1e-12)


def test_two_stage_rows_normalised_and_s1_input_path(scan_cache):
    c = CONFIGS[0]
    P = oracle.Pyramid.from_points(scan_cache(0), c.bit_depth, c.min_bit_depth, c.range_m)
    w = _two_stage_weights(c.channels, c.layers, seed=12)
    b = c.bit_depth - 2
    l1, l2, lse1, lse2, bits = P.model2(b, w)
    np.testing.assert_allclose(np.exp(l1 - lse1[:, None]).sum(1), 1.0, atol=1e-12)
    np.testing.assert_allclose(np.exp(l2 - lse2[:, None]).sum(1), 1.0, atol=1e-12)
    code = P.codes(b).astype(np.int64)
    ref = -(l1[np.arange(len(code)), code & 15] - lse1 + l2[np.arange(len(code)), code >> 4] - lse2) / math.log(2)
    np.testing.assert_allclose(bits, ref, atol=1e-12)
    # S1 handed in (as a decoder would after decoding it) gives the same stage 2
    rows = np.arange(0, P.num(b), 3)
    s1 = (code[rows] & 15).astype(np.uint8)
    m1, m2, _, _, none = P.model2(b, w, rows=rows, s1=s1)
    assert none is None
    np.testing.assert_allclose(m2, l2[rows], atol=1e-12)
    np.testing.assert_allclose(m1, l1[rows], atol=1e-12)
    # and a different S1 changes stage 2 only
    m1b, m2b, _, _, _ = P.model2(b, w, rows=rows, s1=(s1 + 1) % 16)
    np.testing.assert_allclose(m1b, m1, atol=0)
    assert np.abs(m2b - m2).max() > 1e-3


def test_freqs_rule_16_symbols_worked_values():
    """f_s = 1 + floor(p_s * (2^16 - 2K)) in fp32, leftover to the lowest-index
    largest: hand-computed for K = 16."""
    p = np.zeros(16)
    p[:3] = [0.5, 0.25, 0.25]
    f = oracle.freqs_from_probs(p, 16)[0]
    # 1 + floor(0.5 * 65504) = 32753, 1 + floor(0.25 * 65504) = 16377, 13 ones: sum 65520
    assert list(f[:3]) == [32753 + 16, 16377, 16377] and list(f[3:]) == [1] * 13
    u = oracle.freqs_from_probs(np.full(16, 1 / 16), 16)[0]
    assert list(u) == [4095 + 16] + [4095] * 15          # 16 * 4095 = 65520
    # ties for the largest go to the lowest index; the total is always 2^16
    t = oracle.freqs_from_probs(np.array([0.1] * 2 + [0.4, 0.4] + [0.0] * 12), 16)[0]
    assert t[2] > t[3] and t.sum() == 65536 and t.min() >= 1


# ---- full target occupancy predictor (Sec. 3.2, Eqs. 6-9) ------------------------------

def _top_weights(C, seed=21, **kw):
    return gen_weights(C, 2, seed=seed, bias_std=0.1, top=True, **kw)


def _top_by_composition(P, b, w):
    """The predictor rebuilt from pinned pieces: residual blocks from the
    sparse conv pinned against a dense conv3d, the target embedding and the
    head written out with numpy."""
    def block(xyz, bits, x, i1, i2):
        t = oracle.sparse_conv(xyz, bits, x, w["top_w"][i1], w["top_b"][i1], True)
        y = oracle.sparse_conv(xyz, bits, t, w["top_w"][i2], w["top_b"][i2], False)
        return np.maximum(x + y, 0.0)
    xp = P.xyz(b - 1)
    fa = block(xp, b - 1, w["emb_o"].astype(np.float64)[P.codes(b - 1)], 0, 1)
    xyz = P.xyz(b)
    par = P.parent(b).astype(np.int64)
    delta = (xyz[:, 0] & 1) + 2 * (xyz[:, 1] & 1) + 4 * (xyz[:, 2] & 1)
    fb = block(xyz, b, fa[par] + w["emb_d"].astype(np.float64)[delta], 2, 3)
    return fb @ w["head_w"].astype(np.float64) + w["head_b"].astype(np.float64)


def test_top_equals_composition_of_pinned_pieces():
    rs = np.random.default_rng(8)
    B, b0 = 7, 3
    xyz = rs.integers(0, 1 << B, size=(900, 3)) // 2 + 16
    P = oracle.Pyramid.from_voxels(xyz, B, b0)
    w = _top_weights(16)
    for b in (b0 + 1, B - 1):
        lg, lse, bits = P.model(b, w)
        ref = _top_by_composition(P, b, w)
        np.testing.assert_allclose(lg, ref, rtol=0, atol=1e-9)
        code = P.codes(b).astype(np.int64)
        np.testing.assert_allclose(bits, (lse - ref[np.arange(len(code)), code]) / math.log(2), atol=1e-9)


@pytest.mark.parametrize("C,ks", [(16, 5), (64, 3), (128, 5)])
def test_top_wide_and_kernel5_equal_composition(C, ks):
    """Other widths and the 5 x 5 x 5 kernel (the large model: c128, k5)."""
    rs = np.random.default_rng(18)
    B, b0 = 6, 2
    xyz = rs.integers(0, 1 << B, size=(300 if C == 128 else 600, 3)) // 2 + 8
    P = oracle.Pyramid.from_voxels(xyz, B, b0)
    w = _top_weights(C, kernel_size=ks)
    assert w["top_w"][0].shape == (ks ** 3, C, C)
    for b in (b0 + 1, B - 1):
        lg, lse, bits = P.model(b, w)
        ref = _top_by_composition(P, b, w)
        np.testing.assert_allclose(lg, ref, rtol=0, atol=1e-9)
        code = P.codes(b).astype(np.int64)
        np.testing.assert_allclose(bits, (lse - ref[np.arange(len(code)), code]) / math.log(2), atol=1e-9)


def test_top_zero_convs_reduce_to_embeddings(scan_cache):
    """With every conv weight and bias zero each residual block is a ReLU, so a
    voxel's logits depend only on its parent's code and its octant."""
    c = CONFIGS[0]
    P = oracle.Pyramid.from_points(scan_cache(0), c.bit_depth, c.min_bit_depth, c.range_m)
    w = _top_weights(c.channels)
    w["top_w"] = [np.zeros_like(x) for x in w["top_w"]]
    w["top_b"] = [np.zeros_like(x) for x in w["top_b"]]
    b = c.bit_depth - 1
    lg, _, _ = P.model(b, w)
    xyz = P.xyz(b)
    delta = (xyz[:, 0] & 1) + 2 * (xyz[:, 1] & 1) + 4 * (xyz[:, 2] & 1)
    pcode = P.codes(b - 1)[P.parent(b)]
    eo, ed = w["emb_o"].astype(np.float64), w["emb_d"].astype(np.float64)
    f = np.maximum(np.maximum(eo[pcode], 0.0) + ed[delta], 0.0)
    np.testing.assert_allclose(lg, f @ w["head_w"].astype(np.float64) + w["head_b"], rtol=0, atol=1e-9)
    # the same (parent code, octant) gives the same row
    key = pcode.astype(np.int64) * 8 + delta
    _, first = np.unique(key, return_index=True)
    np.testing.assert_array_equal(lg, lg[first[np.searchsorted(np.unique(key), key)]])


def test_top_two_stage_head_and_totals(scan_cache):
    c = CONFIGS[0]
    P = oracle.Pyramid.from_points(scan_cache(0), c.bit_depth, c.min_bit_depth, c.range_m)
    w = _top_weights(c.channels, two_stage=True)
    b = c.bit_depth - 2
    l1, l2, lse1, lse2, bits = P.model2(b, w)
    np.testing.assert_allclose(np.exp(l1 - lse1[:, None]).sum(1), 1.0, atol=1e-12)
    T, per = P.totals(w)
    assert per[b] == pytest.approx(bits.sum(), rel=1e-12)
    assert T == pytest.approx(per.sum(), rel=1e-12)
