"""The seeded input generators: determinism, shapes and workload ranges."""
import numpy as np

from synth import CONFIGS, gen_scan, gen_weights
from synth import rng


def test_splitmix_reference_values():
    # splitmix64 from state 0: the first outputs of the published generator
    # (Steele, Lea & Flood 2014) are 0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4
    from synth.rng import _mix, _GOLDEN
    s = np.array([1, 2], dtype=np.uint64) * _GOLDEN
    out = _mix(s)
    assert int(out[0]) == 0xE220A8397B1DCDAF
    assert int(out[1]) == 0x6E789E6AA1B965F4


def test_uniform_and_normal_ranges():
    u = rng.uniform(3, 1, 0, 100000)
    assert u.min() >= 0.0 and u.max() < 1.0 and abs(u.mean() - 0.5) < 0.01
    z = rng.normal(3, 2, 0, 100000)
    assert abs(z.mean()) < 0.02 and abs(z.std() - 1.0) < 0.02
    # counter-based: a window equals the slice of a longer draw
    assert np.array_equal(rng.uniform(3, 1, 50, 10), u[50:60])


def test_scan_deterministic(scan_cache):
    a = scan_cache(0)
    b = gen_scan(CONFIGS[0])
    assert a.dtype == np.float32 and a.shape[1] == 3
    assert np.array_equal(a, b)
    assert 3000 < a.shape[0] < 8192
    r = np.linalg.norm(a.astype(np.float64), axis=1)
    assert r.max() <= CONFIGS[0].max_range_m + 0.2 and r.min() > 1.0


def test_stream_frames_differ_but_share_scene():
    from synth.lidar import _scene
    c = CONFIGS[4]
    b1, c1 = _scene(c)
    assert b1.shape == (c.boxes, 6) and c1.shape == (c.cylinders, 4)


def test_weights_layout():
    w = gen_weights(32, 3, seed=2)
    assert [x.shape for x in w["conv_w"]] == [(27, 11, 32), (27, 32, 32), (27, 32, 32)]
    assert w["head_w"].shape == (32, 256) and w["head_b"].shape == (256,)
    assert all(np.all(b == 0) for b in w["conv_b"])
    std = w["conv_w"][1].std()
    assert abs(std - np.sqrt(2.0 / (27 * 32))) / std < 0.05
    w2 = gen_weights(32, 3, seed=2)
    assert np.array_equal(w["head_w"], w2["head_w"])
