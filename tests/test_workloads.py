"""The seeded input generator: determinism, shapes, distinct indices, Zipf frequencies."""
import numpy as np

from workloads import WORKLOADS, Stream, Workload, ZipfSampler


def test_deterministic_and_shapes():
    w = WORKLOADS["sq_D2k_d32_m16_K3"]
    a, b = Stream(w), Stream(w)
    assert a.V0.dtype == np.float32 and a.V0.shape == (2000, 32)
    assert np.array_equal(a.V0, b.V0)
    for _ in range(3):
        (H1, i1, v1), (H2, i2, v2) = a.batch(), b.batch()
        assert H1.dtype == np.float32 and i1.dtype == np.int32 and v1.dtype == np.float32
        assert H1.shape == (16, 32) and i1.shape == (16, 3)
        assert np.array_equal(H1, H2) and np.array_equal(i1, i2) and np.array_equal(v1, v2)
        assert all(len(set(r)) == 3 for r in i1.tolist())
        assert i1.min() >= 0 and i1.max() < 2000


def test_distributions():
    w = Workload("t", "squared", 10_000, 64, 512, 5)
    s = Stream(w)
    H, idx, val = s.batch()
    assert abs(H.var() * 64 - 1) < 0.05
    assert abs(s.V0.var() * 64 - 1) < 0.01
    assert abs(val.std() - 1) < 0.1


def test_zipf_top_class_frequency():
    z = ZipfSampler(200_000, 1.1)
    rng = np.random.default_rng(0)
    x = z.draw(rng, 200_000)
    p0 = z.p(0)
    assert 0.12 < p0 < 0.14
    assert abs((x == 0).mean() - p0) < 0.005
    assert x.min() >= 0 and x.max() < 200_000
