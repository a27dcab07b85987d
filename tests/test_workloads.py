"""The seeded input generator and the workload definitions."""
import numpy as np

import workloads


def test_splitmix64_published_vectors():
    # SplitMix64 reference outputs for seed 1234567 and for seed 0.
    got = [int(v) for v in workloads.splitmix64(1234567, 3)]
    assert got == [6457827717110365317, 3203168211198807973, 9817491932198370423]
    assert int(workloads.splitmix64(0, 1)[0]) == 0xE220A8397B1DCDAF


def test_uniform_and_normal_ranges():
    u = workloads.uniform(5, (200000,), -1.0, 1.0)
    assert u.dtype == np.float32 and u.min() >= -1.0 and u.max() < 1.0
    assert abs(float(u.mean())) < 0.01
    z = workloads.normal(6, (200001,), 0.0, 2.0)
    assert z.shape == (200001,) and abs(float(z.mean())) < 0.02 and abs(float(z.std()) - 2.0) < 0.02
    i = workloads.small_ints(7, (10000,))
    assert set(np.unique(i).tolist()) == {-2.0, -1.0, 0.0, 1.0, 2.0}


def test_determinism():
    a = workloads.VGG_EARLY.inputs()
    b = workloads.VGG_EARLY.inputs()
    for x, y in zip(a, b):
        np.testing.assert_array_equal(x, y)


def test_case_shapes():
    x, w, b = workloads.TINY.inputs()
    assert x.shape == (1, 3, 32, 32) and w.shape == (16, 3, 3, 3) and b.shape == (16,) and not b.any()
    x, w, b = workloads.RESNET_STRIDED.inputs()
    assert x.shape == (1, 128, 28, 28) and w.shape == (256, 128, 3, 3) and b is None
    assert abs(float(w.std()) - workloads.he_std(128, 3)) < 0.01 * workloads.he_std(128, 3) * 10
    x4a, _, _ = workloads.DEEP_1X1.inputs()
    x4b, w4b, _ = workloads.DEEP_5X5.inputs()
    np.testing.assert_array_equal(x4a, x4b)   # shared input
    assert w4b.shape == (512, 512, 5, 5)


def test_vgg16_stack():
    layers = workloads.vgg16_layers()
    assert len(layers) == 13
    assert [l[4] for l in layers].count(True) == 4
    assert layers[0][1:4] == (3, 64, 224) and layers[-1][1:4] == (512, 512, 14)


def test_fuzz_shapes_valid():
    shapes = workloads.fuzz_shapes(99, 50)
    assert len(shapes) == 50
    for s in shapes:
        assert s["h"] + 2 * s["pad"] >= s["k"] and s["w"] + 2 * s["pad"] >= s["k"]
