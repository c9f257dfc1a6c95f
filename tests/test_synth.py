"""Seeded input generators: determinism, shapes and the stated statistics."""
import numpy as np

import synth


def test_grf_unit_variance_and_determinism():
    wl = synth.WORKLOADS[1]
    a = synth.make_x(wl, np.float32)
    b = synth.make_x(wl, np.float32)
    assert a.shape == (2, 16, 64, 64)
    assert np.array_equal(a, b)
    v = float(np.var(a.astype(np.float64)))
    assert 0.5 < v < 1.6


def test_fp16_is_rne_of_fp32_master():
    wl = synth.WORKLOADS[1]
    x16 = synth.make_x(wl, np.float16)
    x32 = synth.make_x(wl, np.float32)
    d = np.abs(x16.astype(np.float64) - x32.astype(np.float64))
    assert np.all(d <= 2.0 ** -11 * np.abs(x32.astype(np.float64)) + 2.0 ** -24)


def test_weight_statistics():
    wl = synth.WORKLOADS[1]
    w = synth.make_dense_weight(wl, np.float32)
    assert w.shape == (16, 16, 16, 8, 2)
    s = float(np.std(w.astype(np.float64)))
    assert abs(s - 1.0 / 16.0) < 0.01


def test_tucker_shapes():
    wl = synth.WORKLOADS[5]
    t = synth.make_tucker_weight(wl, np.float16)
    assert t["core"].shape == (13, 13, 6, 3, 2)
    assert t["u_in"].shape == (128, 13, 2)
    assert t["u_out"].shape == (128, 13, 2)
    assert [u.shape for u in t["u_mode"]] == [(64, 6, 2), (32, 3, 2)]
    # fp16 normal range for every entry (no subnormals from the scaling)
    for a in [t["core"], t["u_in"]]:
        nz = np.abs(a.astype(np.float64))
        assert np.mean(nz < 6.1e-5) < 0.01


def test_mixing_workload_shape():
    wl = synth.WORKLOADS[2].with_batch(1)
    x = synth.make_x(wl, np.float16)
    assert x.shape == (1, 64, 128, 128)
    v = float(np.var(x.astype(np.float64)))
    assert 0.3 < v < 3.0
