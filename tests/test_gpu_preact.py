"""GPU parity of the pre-activation variants against the float64 oracle:
tanh in fp32 storage (the full-precision + tanh ablation, App. B.8), fp16
storage without pre-activation (the unstabilised baseline), the hard clip
of the pre-FFT comparison (App. B.6), also at the FP8-E5M2 bound 57344 (the
clipping of Sec. 4.6), and the statistics-based 2-sigma clip of App. B.6
(each (batch, channel) plane clipped to its mean +- 2 population standard
deviations, the bounds held constant in the gradient).

Tolerances (relative L2): 1e-5 for fp32 storage, 3e-3 for fp16.  In the clip
modes some inputs sit exactly on +-c, where the derivative counts the point as
inside the bound on both sides.
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

from oracle import fno_oracle as O  # noqa: E402
import synth  # noqa: E402
from tests import gpu_util as U  # noqa: E402
from tests.test_gpu_parity import EDGE, SPECIAL_SHAPES  # noqa: E402

MODES = ["fp32_tanh", "fp16", "fp16_clip:0.75", "fp32_clip:1.0", "fp16_sigma:2",
         "fp32_sigma:2"]


def _check(name, got, ref, prec):
    r = U.rel(got, ref)
    U.say(f"  {name}: rel_l2 = {r:.3e} (tol {U.TOL[prec]:.0e})")
    assert np.isfinite(r) and r <= U.TOL[prec], f"{name}: {r:.3e}"


def _on_bounds(x, prec, step=53):
    """Every step-th input set to +-c (exact in both storage types here)."""
    kind, c = O.preact_kind(prec)
    if kind != "clip":
        return x
    flat = x.reshape(-1)
    idx = np.arange(0, flat.size, step)
    flat[idx] = np.where(idx % 2 == 0, c, -c).astype(x.dtype)
    assert float(np.float16(c)) == c
    return x


def _oracle(x, w, gy, n, modes, oprec):
    wc = U.cplx(w)
    return (O.fwd(x, wc, n, modes, oprec), O.bwd_data(x, wc, gy, n, modes, oprec),
            O.bwd_weight(x, gy, n, modes, oprec))


@pytest.mark.parametrize("prec", MODES)
@pytest.mark.parametrize("case", range(len(EDGE)))
def test_preact_edge_cases(case, prec):
    n, modes, Bt, ci, co = EDGE[case]
    _, npdt, oprec = U.prec_codes(prec)
    U.say(f"pre-activation case {case}: n={n} modes={modes} B={Bt} Cin={ci} Cout={co} {prec}")
    x, w, gy = synth.random_dense_case(700 + case, Bt, ci, co, n, modes, npdt)
    x = _on_bounds(x, prec)
    layer = U.make_layer(n, modes, Bt, ci, co, prec)
    y, gx, gw = U.run_all(layer, x, w, gy)
    ry, rgx, rgw = _oracle(x, w, gy, n, modes, oprec)
    _check("y", y, ry, prec)
    _check("gx", gx, rgx, prec)
    _check("gW", U.cplx(gw), rgw, prec)


@pytest.mark.parametrize("prec", ["fp16_clip:0.7", "fp32_tanh", "fp16_sigma:2"])
def test_preact_workload_128(prec):
    """The 128^2 workload (B32 C64, 32x32 modes) at full size; 0.7 is not an
    fp16 value, so clipped inputs become fp16(0.7) on the GPU."""
    wl = synth.WORKLOADS[2]
    _, npdt, oprec = U.prec_codes(prec)
    U.say(f"workload {wl.name} {prec}")
    x, gy, w = synth.make_x(wl, npdt), synth.make_gy(wl, npdt), synth.make_weight(wl, npdt)
    layer = U.make_layer(wl.n, wl.modes, wl.batch, wl.c_in, wl.c_out, prec)
    y, gx, gw = U.run_all(layer, x, w, gy)
    ry, rgx, rgw = _oracle(x, w, gy, wl.n, wl.modes, oprec)
    _check("y", y, ry, prec)
    _check("gx", gx, rgx, prec)
    _check("gW", U.cplx(gw), rgw, prec)


@pytest.mark.parametrize("shape", range(len(SPECIAL_SHAPES)))
def test_fp8_e5m2_clip(shape):
    """Clipping at the FP8-E5M2 limit 57344 on inputs that reach +-inf in
    fp16: the clipped values and the zero derivative beyond the bound match
    the oracle (the wide-plane kernels' table is then 63 KB)."""
    (n, modes), Bt, ci, co = SPECIAL_SHAPES[shape], 2, 3, 3
    prec = O.clip_mode("fp16", 57344.0)
    U.say(f"fp8-e5m2 clip n={n}")
    with np.errstate(over="ignore"):
        x, w, gy = synth.random_dense_case(81, Bt, ci, co, n, modes, np.float16, x_scale=2e4)
    x[0, 0, 0, :6] = np.array([65504.0, -65504.0, np.inf, -np.inf, 57344.0, -57344.0],
                              dtype=np.float16)
    w = (w.astype(np.float32) * 1e-3).astype(np.float16)
    assert (np.abs(x) > 57344.0).sum() > 10
    layer = U.make_layer(n, modes, Bt, ci, co, prec)
    y, gx, gw = U.run_all(layer, x, w, gy)
    ry, rgx, rgw = _oracle(x, w, gy, n, modes, prec)
    _check("y", y, ry, prec)
    _check("gx", gx, rgx, prec)
    _check("gW", U.cplx(gw), rgw, prec)
    assert np.all(gx[np.abs(x) > 57344.0] == 0)


@pytest.mark.parametrize("prec", ["fp16_clip:0.75", "fp32_clip:1.0", "fp32_tanh"])
@pytest.mark.parametrize("shape", range(len(SPECIAL_SHAPES)))
def test_preact_nan(shape, prec):
    """A NaN input spoils its own sample's output and, through f', exactly its
    own element of the data gradient."""
    (n, modes), Bt, ci, co = SPECIAL_SHAPES[shape], 2, 3, 3
    _, npdt, _ = U.prec_codes(prec)
    U.say(f"nan n={n} {prec}")
    x, w, gy = synth.random_dense_case(82, Bt, ci, co, n, modes, npdt)
    x[0, 1, 5, 7] = np.nan
    layer = U.make_layer(n, modes, Bt, ci, co, prec)
    xd, wd, gyd = U.dev(x), U.dev(w), U.dev(gy)
    y = U.host(layer.fwd(xd, wd))
    gx = U.host(layer.bwd_data(xd, wd, gyd))
    assert np.isnan(y[0]).any() and np.isfinite(y[1]).all()
    assert np.array_equal(np.isnan(gx), np.isnan(x))


SIGMA_SHAPES = [((32, 32), (8, 8)), ((256, 256), (32, 32)), ((6, 10, 12), (2, 3, 4)),
                ((96,), (17,))]


@pytest.mark.parametrize("prec", ["fp16_sigma:2", "fp32_sigma:1.5"])
@pytest.mark.parametrize("shape", range(len(SIGMA_SHAPES)))
def test_sigma_clip_special_planes(shape, prec):
    """Planes whose statistics are extreme: a constant plane (deviation 0:
    every value sits on both bounds and passes with derivative 1), a plane
    with a large offset (mean far from 0 against its spread) and one with a
    few large outliers (clipped, derivative 0), beside ordinary planes; the
    combined backward with and without the input-spectrum cache agrees with
    the separate calls."""
    n, modes = SIGMA_SHAPES[shape]
    Bt, ci, co = 2, 4, 3
    _, npdt, oprec = U.prec_codes(prec)
    U.say(f"sigma clip special planes n={n} {prec}")
    x, w, gy = synth.random_dense_case(83, Bt, ci, co, n, modes, npdt)
    x[0, 1] = npdt(0.625)
    x[1, 2] = (x[1, 2].astype(np.float64) * 2.0 + 300.0).astype(npdt)
    flat = x[1, 3].reshape(-1)
    flat[::37] = npdt(40.0)
    layer = U.make_layer(n, modes, Bt, ci, co, prec)
    y, gx, gw = U.run_all(layer, x, w, gy)
    ry, rgx, rgw = _oracle(x, w, gy, n, modes, oprec)
    _check("y", y, ry, prec)
    _check("gx", gx, rgx, prec)
    _check("gW", U.cplx(gw), rgw, prec)
    fp = O.preactivation_grad(x, oprec)
    assert np.all(fp[0, 1] == 1.0)
    assert np.all(gx[fp == 0.0] == 0)
    assert np.any(fp[1, 3] == 0.0)
    xd, wd, gyd = U.dev(x), U.dev(w), U.dev(gy)
    for cache in (True, False):
        xh = layer.spectrum_buffer(0)
        layer.fwd(xd, wd, x_hat=xh)
        gxc, gwc = layer.bwd(xd, wd, gyd, x_hat=xh if cache else None)
        assert np.array_equal(U.host(gxc), gx), cache
        assert np.array_equal(U.host(gwc), gw), cache


@pytest.mark.parametrize("shape", range(len(SIGMA_SHAPES)))
def test_sigma_clip_nan_plane(shape):
    """A NaN makes its plane's statistics NaN: that whole plane of f(x) and
    f'(x) is NaN (its sample's output and exactly its plane of the data
    gradient), every other plane stays finite."""
    n, modes = SIGMA_SHAPES[shape]
    Bt, ci, co = 2, 3, 3
    prec = "fp16_sigma:2"
    U.say(f"sigma clip nan n={n}")
    x, w, gy = synth.random_dense_case(84, Bt, ci, co, n, modes, np.float16)
    x[0, 1].reshape(-1)[5] = np.nan
    layer = U.make_layer(n, modes, Bt, ci, co, prec)
    xd, wd, gyd = U.dev(x), U.dev(w), U.dev(gy)
    y = U.host(layer.fwd(xd, wd))
    gx = U.host(layer.bwd_data(xd, wd, gyd))
    assert np.isnan(y[0]).any() and np.isfinite(y[1]).all()
    mask = np.zeros(x.shape, dtype=bool)
    mask[0, 1] = True
    assert np.array_equal(np.isnan(gx), mask)
