"""Pins of the CPU oracle against what the paper and the mathematics fix.

None of these re-types the oracle's own formula: each compares it with a
brute-force sum, a library FFT, an identity (Parseval, shift, adjointness,
round trip), a closed form, a theorem's bound, finite differences or
hand-derived integer tables.  The mutation tests at the end plant plausible
mistakes in the oracle and check that at least one pin catches each.
"""
import itertools
import json
import os

import numpy as np
import pytest

from oracle import fno_oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
F32, F16T = O.PREC_FP32, O.PREC_FP16_TANH


def _rng(seed):
    return np.random.default_rng(np.random.SeedSequence([77, seed]))


def _cplx(rng, shape, scale=1.0):
    return (rng.standard_normal(shape) + 1j * rng.standard_normal(shape)) * scale


# ---------------------------------------------------------------------------
# Pin functions (return the error; used by tests and by mutation tests)
# ---------------------------------------------------------------------------

def pin_brute_force_2d():
    """Quadruple-loop double sum on an 8x8 grid vs the separable oracle."""
    rng = _rng(1)
    n, modes = (8, 8), (2, 3)
    u = rng.standard_normal(n)
    k1 = [0, 1, 6, 7]
    k2 = [0, 1, 2]
    ref = np.zeros((4, 3), dtype=np.complex128)
    for a, ka in enumerate(k1):
        for c, kb in enumerate(k2):
            s = 0j
            for x1 in range(8):
                for x2 in range(8):
                    s += u[x1, x2] * np.exp(-2j * np.pi * (ka * x1 / 8 + kb * x2 / 8))
            ref[a, c] = s / 64.0
    got = O.forward_spectrum(u[None, None], n, modes)[0, 0]
    return np.abs(got - ref).max()


def pin_brute_force_3d():
    rng = _rng(2)
    n, modes = (4, 6, 8), (1, 2, 3)
    u = rng.standard_normal(n)
    ks = [[0, 3], [0, 1, 4, 5], [0, 1, 2]]
    ref = np.zeros((2, 4, 3), dtype=np.complex128)
    for ia, ka in enumerate(ks[0]):
        for ib, kb in enumerate(ks[1]):
            for ic, kc in enumerate(ks[2]):
                s = 0j
                for x1, x2, x3 in itertools.product(range(4), range(6), range(8)):
                    s += u[x1, x2, x3] * np.exp(
                        -2j * np.pi * (ka * x1 / 4 + kb * x2 / 6 + kc * x3 / 8))
                ref[ia, ib, ic] = s / (4 * 6 * 8)
    got = O.forward_spectrum(u[None, None], n, modes)[0, 0]
    return np.abs(got - ref).max()


def pin_numpy_rfftn(n=(16, 12), modes=(5, 4)):
    """numpy's real FFT divided by N, read at the retained frequencies."""
    rng = _rng(3)
    u = rng.standard_normal((2, 3) + n)
    lib = np.fft.rfftn(u, axes=tuple(range(2, 2 + len(n)))) / np.prod(n)
    ks = O.retained(n, modes)
    sel = lib[np.ix_(range(2), range(3), *ks)]
    got = O.forward_spectrum(u, n, modes)
    return np.abs(got - sel).max()


def pin_parseval(n=(8, 10)):
    """(1/N) sum u^2 = sum_k c(k) |Xhat_k|^2 over the half spectrum, all modes."""
    rng = _rng(4)
    u = rng.standard_normal(n)
    modes = (n[0] // 2, n[1] // 2 + 1)
    xh = O.forward_spectrum(u[None, None], n, modes)[0, 0]
    c = O.multiplicity(O.retained(n, modes)[-1], n[-1])
    lhs = np.mean(u * u)
    rhs = np.sum(c * np.abs(xh) ** 2)
    return abs(lhs - rhs) / lhs


def pin_ramp(n_last=16, m=9):
    """u[x1, x2] = x2: Xhat[0, k] = -1/2 + (i/2) cot(pi k / N) (k != 0),
    Xhat[0, 0] = (N - 1)/2, other rows zero.  Imaginary part at k = 1 is the
    closed form sum_j j sin(2 pi j / m) = -(m/2) cot(pi / m) used in the proof
    of Thm 3.1."""
    n = (4, n_last)
    u = np.tile(np.arange(n_last, dtype=np.float64), (4, 1))
    xh = O.forward_spectrum(u[None, None], n, (2, m))[0, 0]
    k = np.arange(m)
    ref_row = np.empty(m, dtype=np.complex128)
    ref_row[0] = (n_last - 1) / 2.0
    with np.errstate(divide="ignore"):
        ref_row[1:] = -0.5 + 0.5j / np.tan(np.pi * k[1:] / n_last)
    if 2 * (m - 1) == n_last:
        ref_row[m - 1] = -0.5           # cot(pi/2) = 0 at Nyquist
    ref = np.zeros_like(xh)
    ref[0] = ref_row
    return np.abs(xh - ref).max()


def pin_shift(n=(8, 12), modes=(3, 5), s=(3, 5)):
    """Circular shift by s multiplies Xhat_k by exp(-2 pi i <k, s/N>)."""
    rng = _rng(5)
    u = rng.standard_normal(n)
    us = np.roll(u, shift=s, axis=(0, 1))
    ks = O.retained(n, modes)
    ph = np.exp(-2j * np.pi * (np.outer(ks[0], np.ones_like(ks[1])) * s[0] / n[0]
                               + np.outer(np.ones_like(ks[0]), ks[1]) * s[1] / n[1]))
    a = O.forward_spectrum(u[None, None], n, modes)[0, 0] * ph
    b = O.forward_spectrum(us[None, None], n, modes)[0, 0]
    return np.abs(a - b).max()


def pin_round_trip(n=(8, 6), c=3):
    """Identity weights with every mode retained reproduce u exactly."""
    rng = _rng(6)
    modes = tuple(nj // 2 for nj in n[:-1]) + (n[-1] // 2 + 1,)
    kd = tuple(2 * m for m in modes[:-1]) + (modes[-1],)
    u = rng.standard_normal((2, c) + n)
    w = np.zeros((c, c) + kd, dtype=np.complex128)
    for i in range(c):
        w[i, i] = 1.0
    y = O.fwd(u, w, n, modes, F32)
    return np.abs(y - u).max()


def pin_single_mode(n=(16, 12), modes=(3, 4), a=(14, 2), wv=0.7 - 0.4j):
    """u = cos(theta_a) with a_d >= 1 retained, W = w delta_io at mode a only:
    y = Re(w exp(i theta_a)).  Pins the sign, the phase and c(k)."""
    x1, x2 = np.meshgrid(np.arange(n[0]), np.arange(n[1]), indexing="ij")
    th = 2 * np.pi * (a[0] * x1 / n[0] + a[1] * x2 / n[1])
    u = np.cos(th)
    ks = O.retained(n, modes)
    t0 = int(np.where(ks[0] == a[0])[0][0])
    t1 = int(np.where(ks[1] == a[1])[0][0])
    kd = (len(ks[0]), len(ks[1]))
    w = np.zeros((1, 1) + kd, dtype=np.complex128)
    w[0, 0, t0, t1] = wv
    y = O.fwd(u[None, None], w, n, modes, F32)[0, 0]
    ref = np.real(wv * np.exp(1j * th))
    return np.abs(y - ref).max()


def pin_irfftn(n=(8, 10), modes=(4, 6)):
    """With all modes kept and a Hermitian-consistent half spectrum Z (taken
    from the real FFT of a real field), inverse_spectrum(Z) equals N times
    numpy's irfftn of Z placed on the full half grid."""
    rng = _rng(7)
    v = rng.standard_normal(n)
    half = np.fft.rfftn(v)                       # consistent half spectrum
    ks = O.retained(n, modes)
    z = half[np.ix_(*ks)]
    y = O.inverse_spectrum(z[None, None], n, modes)[0, 0]
    ref = np.fft.irfftn(half, s=n, axes=(0, 1)) * np.prod(n)
    return np.abs(y - ref).max() / np.abs(ref).max()


def pin_fd_dense(precision, seed=11):
    """Central finite differences of L = <gy, y> for x, Re W, Im W."""
    rng = _rng(seed)
    n, modes = (8, 8), (2, 2)
    b, ci, co = 1, 2, 2
    x = rng.standard_normal((b, ci) + n) * 0.8
    w = _cplx(rng, (ci, co, 4, 2), 0.5)
    gy = rng.standard_normal((b, co) + n)

    def loss(xx, ww):
        return float(np.sum(gy * O.fwd(xx, ww, n, modes, precision)))

    h = 1e-6
    gx = O.bwd_data(x, w, gy, n, modes, precision)
    gw = O.bwd_weight(x, gy, n, modes, precision)
    err = 0.0
    for idx in [(0, 0, 0, 0), (0, 1, 3, 5), (0, 0, 7, 2), (0, 1, 4, 4)]:
        e = np.zeros_like(x)
        e[idx] = h
        fd = (loss(x + e, w) - loss(x - e, w)) / (2 * h)
        err = max(err, abs(fd - gx[idx]) / max(1e-3, abs(gx[idx])))
    for idx in [(0, 0, 0, 0), (1, 0, 3, 1), (0, 1, 2, 0), (1, 1, 1, 1)]:
        for comp in (1.0, 1j):
            e = np.zeros_like(w)
            e[idx] = h * comp
            fd = (loss(x, w + e) - loss(x, w - e)) / (2 * h)
            ref = gw[idx].real if comp == 1.0 else gw[idx].imag
            err = max(err, abs(fd - ref) / max(1e-3, abs(ref)))
    return err


def pin_adjoint(seed=12):
    """<gy, fwd(dx)> = <bwd_data(gy), dx> and Re<gW, dW> = <gy, y(dW)> in the
    linear (full-precision) mode."""
    rng = _rng(seed)
    n, modes = (8, 12), (3, 4)
    b, ci, co = 2, 3, 2
    w = _cplx(rng, (ci, co, 6, 4))
    dx = rng.standard_normal((b, ci) + n)
    gy = rng.standard_normal((b, co) + n)
    lhs = np.sum(gy * O.fwd(dx, w, n, modes, F32))
    rhs = np.sum(O.bwd_data(dx, w, gy, n, modes, F32) * dx)
    e1 = abs(lhs - rhs) / abs(lhs)
    x = rng.standard_normal((b, ci) + n)
    dw = _cplx(rng, w.shape)
    lhs2 = np.sum(gy * O.fwd(x, dw, n, modes, F32))
    rhs2 = np.real(np.sum(np.conj(O.bwd_weight(x, gy, n, modes, F32)) * dw))
    e2 = abs(lhs2 - rhs2) / abs(lhs2)
    return max(e1, e2)


def pin_identity_self_adjoint(seed=13):
    """Identity weights: bwd_data(gy) == fwd(gy) in full precision (the
    truncation projector is self-adjoint)."""
    rng = _rng(seed)
    n, modes = (8, 12), (2, 5)
    c = 3
    w = np.zeros((c, c, 4, 5), dtype=np.complex128)
    for i in range(c):
        w[i, i] = 1.0
    gy = rng.standard_normal((2, c) + n)
    a = O.bwd_data(gy, w, gy, n, modes, F32)
    b = O.fwd(gy, w, n, modes, F32)
    return np.abs(a - b).max()


def pin_fd_clip(seed=14, c=0.5):
    """Central finite differences of L = <gy, y> in x through the hard clip,
    at points inside and outside [-c, c] (none within 1e-3 of the bound)."""
    rng = _rng(seed)
    n, modes = (8, 8), (2, 2)
    prec = O.clip_mode("fp16", c)
    x = rng.standard_normal((1, 2) + n) * 0.8
    w = _cplx(rng, (2, 2, 4, 2), 0.5)
    gy = rng.standard_normal((1, 2) + n)
    gx = O.bwd_data(x, w, gy, n, modes, prec)
    far = np.abs(np.abs(x) - c) > 1e-3
    inside = np.argwhere(far & (np.abs(x) < c))[:3]
    outside = np.argwhere(far & (np.abs(x) > c))[:3]
    if len(inside) < 3 or len(outside) < 3:
        return np.inf
    h = 1e-6
    err = 0.0
    for idx in [tuple(i) for i in inside] + [tuple(i) for i in outside]:
        e = np.zeros_like(x)
        e[idx] = h
        fd = (np.sum(gy * O.fwd(x + e, w, n, modes, prec)) -
              np.sum(gy * O.fwd(x - e, w, n, modes, prec))) / (2 * h)
        err = max(err, abs(fd - gx[idx]) / max(1e-3, abs(gx[idx])))
    # outside the bound the input does not reach the output
    err = max(err, float(np.abs(gx[far & (np.abs(x) > c)]).max()))
    return err


def pin_clip_saturated(seed=15, c=0.25):
    """Every |x| > c: the clipped input is c sign(x), so the layer output is
    c times the full-precision output for sign(x)."""
    rng = _rng(seed)
    n, modes = (8, 6), (2, 3)
    x = rng.standard_normal((2, 3) + n)
    x = np.where(np.abs(x) < 2 * c, np.copysign(2 * c, x), x)
    w = _cplx(rng, (3, 2, 4, 3), 0.5)
    got = O.fwd(x, w, n, modes, O.clip_mode("fp32", c))
    ref = c * O.fwd(np.sign(x), w, n, modes, F32)
    return np.abs(got - ref).max() / np.abs(ref).max()


def pin_clip_wide_is_identity(seed=16):
    """A bound above every |x| leaves the layer and its gradients as in
    full precision without pre-activation."""
    rng = _rng(seed)
    n, modes = (8, 6), (2, 3)
    x = rng.standard_normal((2, 3) + n)
    w = _cplx(rng, (3, 2, 4, 3), 0.5)
    gy = rng.standard_normal((2, 2) + n)
    prec = O.clip_mode("fp16", float(np.abs(x).max()) * 1.01)
    err = np.abs(O.fwd(x, w, n, modes, prec) - O.fwd(x, w, n, modes, F32)).max()
    err = max(err, np.abs(O.bwd_data(x, w, gy, n, modes, prec) -
                          O.bwd_data(x, w, gy, n, modes, F32)).max())
    return err


def pin_tanh_constant_field(seed=17):
    """A constant input a_i per channel has only the zero mode: y[o] =
    sum_i Re(W[i, o, 0, 0]) tanh(a_i) at every point, for the tanh modes of
    both storage precisions (scalar math.tanh as the closed form)."""
    import math
    rng = _rng(seed)
    n, modes = (8, 6), (2, 3)
    a = np.array([-3.0, -0.4, 0.7, 5.0])
    x = np.broadcast_to(a[None, :, None, None], (1, 4) + n).copy()
    w = _cplx(rng, (4, 3, 4, 3), 0.5)
    ref = np.array([sum(w[i, o, 0, 0].real * math.tanh(a[i]) for i in range(4))
                    for o in range(3)])
    err = 0.0
    for prec in (O.PREC_FP32_TANH, F16T):
        y = O.fwd(x, w, n, modes, prec)[0]
        err = max(err, np.abs(y - ref[:, None, None]).max())
    return err


def _cp_small(seed, d=2, rank=3):
    rng = _rng(seed)
    n = (8, 8) if d == 2 else (4, 4, 6)
    modes = (2, 3) if d == 2 else (1, 2, 2)
    kd = tuple(2 * m for m in modes[:-1]) + (modes[-1],)
    ci, co = 3, 4
    lam = _cplx(rng, (rank,), 0.5)
    u_in, u_out = _cplx(rng, (ci, rank), 0.5), _cplx(rng, (co, rank), 0.5)
    u_mode = [_cplx(rng, (kd[j], rank), 0.5) for j in range(d)]
    x = rng.standard_normal((2, ci) + n) * 0.7
    gy = rng.standard_normal((2, co) + n)
    return rng, n, modes, kd, lam, u_in, u_out, u_mode, x, gy


def pin_cp_explicit(seed=80):
    """CP reconstruction against the rank-one sum written out (relative)."""
    _, n, modes, kd, lam, u_in, u_out, u_mode, _, _ = _cp_small(seed)
    w = O.cp_dense(lam, u_in, u_out, u_mode)
    err = 0.0
    for (i, o, t1, t2) in [(0, 0, 0, 0), (2, 1, 3, 2), (1, 3, 2, 1)]:
        ref = sum(lam[r] * u_in[i, r] * u_out[o, r] * u_mode[0][t1, r] * u_mode[1][t2, r]
                  for r in range(lam.shape[0]))
        err = max(err, abs(w[i, o, t1, t2] - ref) / abs(ref))
    return err


def pin_cp_tucker(seed=81):
    """The CP layer equals the Tucker layer with lambda on the core's
    superdiagonal: outputs, data gradients, and lambda = the core gradient's
    superdiagonal (relative errors)."""
    _, n, modes, kd, lam, u_in, u_out, u_mode, x, gy = _cp_small(seed)
    r = lam.shape[0]
    core = np.zeros((r,) * 4, dtype=np.complex128)
    for k in range(r):
        core[k, k, k, k] = lam[k]
    rel = lambda a, b: np.abs(a - b).max() / np.abs(b).max()  # noqa: E731
    err = 0.0
    for prec in (F32, F16T):
        err = max(err, rel(O.cp_fwd(x, lam, u_in, u_out, u_mode, n, modes, prec),
                           O.tucker_fwd(x, core, u_in, u_out, u_mode, n, modes, prec)))
        err = max(err, rel(O.cp_bwd_data(x, lam, u_in, u_out, u_mode, gy, n, modes, prec),
                           O.tucker_bwd_data(x, core, u_in, u_out, u_mode, gy, n, modes,
                                             prec)))
        g = O.cp_bwd_weight(x, gy, lam, u_in, u_out, u_mode, n, modes, prec)
        t = O.tucker_bwd_weight(x, gy, core, u_in, u_out, u_mode, n, modes, prec)
        err = max(err, rel(g[0], np.array([t[0][k, k, k, k] for k in range(r)])))
        err = max(err, rel(g[1], t[1]), rel(g[2], t[2]), rel(g[3][0], t[3][0]),
                  rel(g[3][1], t[3][1]))
    return err


def pin_rel_l2_hand():
    """rel_l2 against values worked by hand: a real vector, a 2-D tensor (the
    norm runs over the whole tensor), complex values and the same values as
    (re, im) pairs, fp16 inputs whose squares overflow fp16, the zero
    reference, and scale invariance.  Returns the largest deviation."""
    f16 = np.float16
    cases = [
        (np.array([1.0, 2.0, 2.0]), np.array([1.0, 0.0, 0.0]), np.sqrt(8.0)),
        (np.array([[3.0, 0.0], [0.0, 0.0]]), np.array([[0.0, 0.0], [0.0, 4.0]]), 1.25),
        (np.array([1 + 1j, 0j]), np.array([1 + 0j, 1j]), 1.0),
        (np.array([2 + 0j]), np.array([1j]), np.sqrt(5.0)),
        (np.array([[2.0, 0.0]]), np.array([[0.0, 1.0]]), np.sqrt(5.0)),
        (np.full(4, 60000, f16), np.full(4, 30000, f16), 1.0),
        (np.array([3.0, 4.0]), np.zeros(2), 5.0),
        (np.zeros(3), np.zeros(3), 0.0),
        (np.array([4.0, 8.0, 8.0]), np.array([4.0, 0.0, 0.0]), np.sqrt(8.0)),
    ]
    err = 0.0
    for a, b, want in cases:
        got = O.rel_l2(a, b)
        err = max(err, abs(got - want)) if np.isfinite(got) else np.inf
    return err


def pin_max_plane_hand():
    """max_plane_rel_l2 on a [2, 2, 3] tensor of ones with one element of
    plane (1, 0) off by 3: that plane's error is 3 / sqrt(3) = sqrt(3), while
    the whole-tensor figure is only 3 / sqrt(12).  A NaN in any plane makes
    the worst plane NaN, wherever the plane comes in the scan."""
    b = np.ones((2, 2, 3))
    a = b.copy()
    a[1, 0, 2] += 3.0
    n = a.copy()
    n[0, 0, 1] = np.nan
    nan_ok = np.isnan(O.max_plane_rel_l2(n, b)) and np.isnan(O.max_plane_rel_l2(n[::-1], b))
    return max(abs(O.max_plane_rel_l2(a, b) - np.sqrt(3.0)),
               abs(O.max_plane_rel_l2(b, b) - 0.0),
               abs(O.rel_l2(a, b) - 3.0 / np.sqrt(12.0)),
               0.0 if nan_ok else np.inf)


def pin_sigma_closed_form():
    """The 2-sigma clip on planes whose statistics are known in closed form:
    63 zeros and one value A (mean A/64, population deviation A sqrt(63)/64,
    so A clips to A (1 + 2 sqrt 63) / 64 and the zeros stay), the same with
    -A, values +-1 alternating (mean 0, deviation 1: nothing clips), and the
    first plane scaled by 1000 (each plane's own statistics: the result
    scales with it).  Returns the largest relative deviation."""
    A = 10.0
    x = np.zeros((1, 4, 8, 8))
    x[0, 0, 2, 5] = A
    x[0, 1, 7, 0] = -A
    x[0, 2] = np.where((np.arange(64) % 2).reshape(8, 8) == 0, 1.0, -1.0)
    x[0, 3] = 1000.0 * x[0, 0]
    u = O.preactivation(x, O.sigma_mode("fp32", 2.0))
    want = np.zeros_like(x)
    clipped = A * (1.0 + 2.0 * np.sqrt(63.0)) / 64.0
    want[0, 0, 2, 5] = clipped
    want[0, 1, 7, 0] = -clipped
    want[0, 2] = x[0, 2]
    want[0, 3, 2, 5] = 1000.0 * clipped
    g = O.preactivation_grad(x, O.sigma_mode("fp32", 2.0))
    gwant = np.ones_like(x)
    gwant[0, 0, 2, 5] = gwant[0, 1, 7, 0] = gwant[0, 3, 2, 5] = 0.0
    return max(float(np.abs(u - want).max()) / 1000.0, float(np.abs(g - gwant).max()))


def pin_sigma_fd_frozen():
    """The data gradient through the 2-sigma clip equals central finite
    differences of the layer whose clip bounds are held at the values the
    statistics of x give (the reading: no gradient through the statistics),
    for inside and clipped elements alike."""
    rng = _rng(91)
    n, modes = (8, 8), (2, 3)
    kd = (4, 3)
    x = rng.standard_normal((1, 2) + n)
    x[0, 0, 0, 0] = 6.0
    x[0, 1, 3, 3] = -7.0
    w = _cplx(rng, (2, 2) + kd, 0.5)
    gy = rng.standard_normal((1, 2) + n)
    prec = O.sigma_mode("fp32", 2.0)
    lo, hi = O.sigma_bounds(x, 2.0)

    def loss(xx):
        u = np.where(xx < lo, lo, np.where(xx > hi, hi, xx))
        xh = O.forward_spectrum(u, n, modes)
        y = O.inverse_spectrum(O.contract_dense(xh, w), n, modes)
        return float(np.sum(gy * y))

    gx = O.bwd_data(x, w, gy, n, modes, prec)
    h = 1e-6
    err = 0.0
    for idx in [(0, 0, 0, 0), (0, 1, 3, 3), (0, 0, 4, 2), (0, 1, 6, 7), (0, 0, 7, 1)]:
        xp, xm = x.copy(), x.copy()
        xp[idx] += h
        xm[idx] -= h
        fd = (loss(xp) - loss(xm)) / (2 * h)
        err = max(err, abs(fd - gx[idx]) / max(1.0, abs(gx[idx])))
    return err


def pin_gelu_values():
    """GELU against values fixed by the normal distribution: Phi(1) and
    phi(1) from the standard normal table (so GELU(1) = Phi(1),
    GELU(-1) = -(1 - Phi(1)), GELU'(1) = Phi(1) + phi(1)), GELU(0) = 0,
    GELU'(0) = 1/2, z Phi(z) on a grid against scipy.stats.norm.cdf, and the
    derivative against central differences of the function."""
    from scipy.stats import norm
    phi1, dens1 = 0.8413447460685429, 0.24197072451914337
    errs = [abs(O.gelu(np.array([1.0]))[0] - phi1),
            abs(O.gelu(np.array([-1.0]))[0] + (1.0 - phi1)),
            abs(O.gelu(np.array([0.0]))[0]),
            abs(O.gelu_grad(np.array([0.0]))[0] - 0.5),
            abs(O.gelu_grad(np.array([1.0]))[0] - (phi1 + dens1))]
    z = np.linspace(-7.0, 7.0, 141)
    errs.append(float(np.abs(O.gelu(z) - z * norm.cdf(z)).max()))
    h = 1e-5
    fd = (O.gelu(z + h) - O.gelu(z - h)) / (2 * h)
    errs.append(float(np.abs(fd - O.gelu_grad(z)).max()) * 1e-3)
    return max(errs)


def _torch_epilogue(x, y, w, b, act, residual):
    """The epilogue and its gradients through torch's own 1x1 convolution,
    GELU and autograd (CPU, float64)."""
    import torch
    import torch.nn.functional as F
    d = x.ndim - 2
    conv = {1: F.conv1d, 2: F.conv2d, 3: F.conv3d}[d]
    xt = torch.tensor(x, dtype=torch.float64, requires_grad=True)
    yt = torch.tensor(y, dtype=torch.float64, requires_grad=True)
    wt = torch.tensor(w, dtype=torch.float64, requires_grad=True)
    bt = torch.tensor(b, dtype=torch.float64, requires_grad=True)
    z = conv(xt, wt.reshape(wt.shape + (1,) * d), bt) + yt
    out = F.gelu(z, approximate="none") if act == O.EPI_ACT_GELU else z
    if residual:
        out = out + xt
    g = torch.tensor(_rng(95).standard_normal(out.shape), dtype=torch.float64)
    out.backward(g)
    return (out.detach().numpy(), g.numpy(), yt.grad.numpy(), xt.grad.numpy(),
            wt.grad.numpy(), bt.grad.numpy())


def pin_epilogue_torch():
    """The block epilogue (1x1 skip with bias, activation, residual) and its
    gradients against torch's convolution, GELU and autograd in float64, in
    1-D, 2-D and 3-D, with and without GELU and the residual, C_in != C_out
    where there is no residual."""
    err = 0.0
    cases = [((7,), 3, 5, O.EPI_ACT_GELU, False), ((5, 6), 4, 4, O.EPI_ACT_GELU, True),
             ((3, 4, 5), 2, 3, O.EPI_ACT_NONE, False), ((6, 5), 3, 3, O.EPI_ACT_NONE, True)]
    for k, (sp, ci, co, act, res) in enumerate(cases):
        rng = _rng(96 + k)
        x = rng.standard_normal((2, ci) + sp)
        y = rng.standard_normal((2, co) + sp)
        w = rng.standard_normal((co, ci))
        b = rng.standard_normal(co)
        out_t, g, gy_t, gx_t, gw_t, gb_t = _torch_epilogue(x, y, w, b, act, res)
        out, z = O.block_epilogue_fwd(x, y, w, b, act, res)
        g_z, g_x, g_w, g_b = O.block_epilogue_bwd(x, z, g, w, act, res)
        for a, t in [(out, out_t), (g_z, gy_t), (g_x, gx_t), (g_w, gw_t), (g_b, gb_t)]:
            err = max(err, float(np.abs(a - t).max()) / max(1.0, float(np.abs(t).max())))
    return err


def pin_block_fd():
    """Gradients of the whole block act(W_skip x + b + K x) + x (spectral
    path in tanh mode) against central differences of its loss
    sum(g_out * out), for entries of x, W_skip, b and the real and imaginary
    parts of the spectral weight."""
    rng = _rng(97)
    n, modes = (8, 6), (2, 3)
    kd = (4, 3)
    c = 3
    x = rng.standard_normal((2, c) + n)
    w = _cplx(rng, (c, c) + kd, 0.4)
    ws = rng.standard_normal((c, c)) * 0.5
    b = rng.standard_normal(c) * 0.3
    g = rng.standard_normal((2, c) + n)
    args = (n, modes, F16T, O.EPI_ACT_GELU, True)

    def loss(x_, w_, ws_, b_):
        out, _ = O.block_fwd(x_, w_, ws_, b_, *args)
        return float(np.sum(g * out))

    gx, gw, gws, gb = O.block_bwd(x, w, ws, b, g, *args)
    h = 1e-6
    err = 0.0

    def check(fd, an):
        return abs(fd - an) / max(1.0, abs(an))

    for idx in [(0, 0, 0, 0), (1, 2, 5, 3), (0, 1, 7, 5)]:
        xp, xm = x.copy(), x.copy()
        xp[idx] += h
        xm[idx] -= h
        err = max(err, check((loss(xp, w, ws, b) - loss(xm, w, ws, b)) / (2 * h), gx[idx]))
    for idx in [(0, 1), (2, 0), (1, 1)]:
        wp, wm = ws.copy(), ws.copy()
        wp[idx] += h
        wm[idx] -= h
        err = max(err, check((loss(x, w, wp, b) - loss(x, w, wm, b)) / (2 * h), gws[idx]))
    for o in range(c):
        bp, bm = b.copy(), b.copy()
        bp[o] += h
        bm[o] -= h
        err = max(err, check((loss(x, w, ws, bp) - loss(x, w, ws, bm)) / (2 * h), gb[o]))
    for idx in [(0, 1, 1, 2), (2, 2, 3, 0)]:
        for unit, part in [(1.0, np.real), (1j, np.imag)]:
            wp, wm = w.copy(), w.copy()
            wp[idx] += h * unit
            wm[idx] -= h * unit
            fd = (loss(x, wp, ws, b) - loss(x, wm, ws, b)) / (2 * h)
            err = max(err, check(fd, part(gw[idx])))
    return err


ALL_PINS = {
    "gelu_values": (pin_gelu_values, 1e-12),
    "epilogue_torch": (pin_epilogue_torch, 1e-12),
    "block_fd": (pin_block_fd, 1e-6),
    "sigma_closed_form": (pin_sigma_closed_form, 1e-12),
    "sigma_fd_frozen": (pin_sigma_fd_frozen, 1e-7),
    "rel_l2_hand": (pin_rel_l2_hand, 1e-15),
    "max_plane_hand": (pin_max_plane_hand, 1e-15),
    "cp_explicit": (pin_cp_explicit, 1e-13),
    "cp_tucker": (pin_cp_tucker, 1e-12),
    "brute2d": (pin_brute_force_2d, 1e-13),
    "brute3d": (pin_brute_force_3d, 1e-13),
    "rfftn": (pin_numpy_rfftn, 1e-13),
    "parseval": (pin_parseval, 1e-12),
    "ramp": (pin_ramp, 1e-12),
    "shift": (pin_shift, 1e-13),
    "round_trip": (pin_round_trip, 1e-13),
    "single_mode": (pin_single_mode, 1e-13),
    "irfftn": (pin_irfftn, 1e-13),
    "fd_fp32": (lambda: pin_fd_dense(F32), 1e-7),
    "fd_tanh": (lambda: pin_fd_dense(F16T), 1e-7),
    "fd_fp32_tanh": (lambda: pin_fd_dense(O.PREC_FP32_TANH), 1e-7),
    "fd_clip": (pin_fd_clip, 1e-7),
    "clip_saturated": (pin_clip_saturated, 1e-13),
    "tanh_constant": (pin_tanh_constant_field, 1e-13),
    "clip_wide_identity": (pin_clip_wide_is_identity, 1e-13),
    "adjoint": (pin_adjoint, 1e-12),
    "identity_adjoint": (pin_identity_self_adjoint, 1e-13),
}


@pytest.mark.parametrize("name", sorted(ALL_PINS))
def test_pin(name):
    fn, tol = ALL_PINS[name]
    err = fn()
    assert err <= tol, f"{name}: {err:.3e} > {tol:.1e}"


# ---------------------------------------------------------------------------
# Further pins
# ---------------------------------------------------------------------------

def test_mode_maps_golden():
    with open(os.path.join(GOLDEN, "mode_maps.json")) as f:
        g = json.load(f)
    for ax in g["axes"]:
        k = O.mode_freq(ax["n"], ax["m"], ax["last"])
        if "k" in ax:
            assert k.tolist() == ax["k"]
        else:
            m = ax["m"]
            assert [int(k[0]), int(k[m - 1])] == ax["k_low"]
            if not ax["last"]:
                assert [int(k[m]), int(k[2 * m - 1])] == ax["k_high"]
                assert k.tolist() == sorted(k.tolist())   # ascending FFT order
                assert len(set(k.tolist())) == 2 * m
    for row in g["multiplicity"]:
        assert O.multiplicity(np.array(row["k"]), row["n"]).tolist() == row["c"]


@pytest.mark.parametrize("n,m,last", [(8, 5, False), (8, 0, False), (8, 6, True),
                                      (8, 0, True)])
def test_mode_freq_rejects(n, m, last):
    with pytest.raises(ValueError):
        O.mode_freq(n, m, last)


def test_ramp_closed_form_odd_and_nyquist():
    assert pin_ramp(15, 8) < 1e-12
    assert pin_ramp(16, 9) < 1e-12     # Nyquist bin retained


def test_parseval_3d_and_odd():
    assert pin_parseval((6, 8)) < 1e-12
    rng = _rng(21)
    n = (4, 6, 7)
    u = rng.standard_normal(n)
    modes = (2, 3, 4)
    xh = O.forward_spectrum(u[None, None], n, modes)[0, 0]
    c = O.multiplicity(O.retained(n, modes)[-1], n[-1])
    assert abs(np.mean(u * u) - np.sum(c * np.abs(xh) ** 2)) < 1e-12


def test_rfftn_3d():
    assert pin_numpy_rfftn((6, 8, 10), (2, 3, 4)) < 1e-13
    assert pin_numpy_rfftn((16,), (5,)) < 1e-13


def test_round_trip_3d_odd():
    assert pin_round_trip((4, 6, 8), 2) < 1e-13
    assert pin_round_trip((6, 7), 2) < 1e-13


def test_tanh_bounds_spectrum():
    """|Xhat_k| <= ||tanh(x)||_inf <= 1 for any x, even near the fp16 limit."""
    rng = _rng(22)
    n = (16, 16)
    x = rng.standard_normal((2, 3) + n) * 6e4
    xh = O.forward_spectrum(O.preactivation(x, F16T), n, (8, 9))
    assert np.abs(xh).max() <= 1.0 + 1e-15
    assert np.isfinite(xh).all()


@pytest.mark.parametrize("nn", [64, 256])
def test_thm32_precision_bound(nn):
    """Thm 3.2: quantising v and the basis values to fp16 (unit roundoff
    eps = 2^-11) moves every retained coefficient by at most 4 eps ||v||_inf."""
    rng = _rng(23)
    n, modes = (nn, nn), (8, 8)
    v = np.tanh(rng.standard_normal(n) * 2.0)
    exact = O.forward_spectrum(v[None, None], n, modes)[0, 0]
    qv = v.astype(np.float16).astype(np.float64)
    ks = O.retained(n, modes)
    eps = 2.0 ** -11
    M = np.abs(v).max()
    x1, x2 = np.meshgrid(np.arange(nn), np.arange(nn), indexing="ij")
    worst = 0.0
    for ka in ks[0][[0, 3, 9, 15]]:
        for kb in ks[1][[0, 5, 7]]:
            ph = 2 * np.pi * (((ka * x1) % nn) / nn + ((kb * x2) % nn) / nn)
            qc = np.cos(ph).astype(np.float16).astype(np.float64)
            qs = np.sin(ph).astype(np.float16).astype(np.float64)
            quant = np.sum(qv * (qc - 1j * qs)) / (nn * nn)
            ta = int(np.where(ks[0] == ka)[0][0])
            tb = int(np.where(ks[1] == kb)[0][0])
            err = abs(quant - exact[ta, tb])
            worst = max(worst, err)
            assert err <= 4 * eps * M
    assert worst > 0.0


def test_bandlimited_reproduction():
    """A field supported on the Hermitian-closed part of the retained set is
    reproduced exactly by identity weights; adding the unpaired k1 = -m1
    column on the k_d = 0 plane is not."""
    n, modes = (16, 16), (3, 4)
    rng = _rng(24)
    x1, x2 = np.meshgrid(np.arange(16), np.arange(16), indexing="ij")
    u = np.zeros(n)
    for k1 in range(-2, 3):            # |k1| <= m1 - 1 on the k_d = 0 plane
        a = rng.standard_normal()
        u += a * np.cos(2 * np.pi * k1 * x1 / 16 + 0.3 * k1)
    for k1 in range(-3, 3):            # any retained k1 for k_d >= 1
        for k2 in range(1, 4):
            a = rng.standard_normal()
            u += a * np.cos(2 * np.pi * (k1 * x1 + k2 * x2) / 16 + 0.1 * k2)
    w = np.ones((1, 1, 6, 4), dtype=np.complex128)
    y = O.fwd(u[None, None], w, n, modes, F32)[0, 0]
    assert np.abs(y - u).max() < 1e-12
    u2 = u + np.cos(2 * np.pi * (-3) * x1 / 16 + 0.5)
    y2 = O.fwd(u2[None, None], w, n, modes, F32)[0, 0]
    assert np.abs(y2 - u2).max() > 1e-3


def test_identity_pass_through():
    rng = _rng(25)
    xh = _cplx(rng, (2, 3, 4, 5))
    w = np.zeros((3, 3, 4, 5), dtype=np.complex128)
    for i in range(3):
        w[i, i] = 1.0
    assert np.abs(O.contract_dense(xh, w) - xh).max() == 0.0


def test_adjoint_3d():
    rng = _rng(26)
    n, modes = (4, 6, 8), (1, 2, 3)
    w = _cplx(rng, (2, 3, 2, 4, 3))
    dx = rng.standard_normal((1, 2) + n)
    gy = rng.standard_normal((1, 3) + n)
    lhs = np.sum(gy * O.fwd(dx, w, n, modes, F32))
    rhs = np.sum(O.bwd_data(dx, w, gy, n, modes, F32) * dx)
    assert abs(lhs - rhs) / abs(lhs) < 1e-12


# ---------------------------------------------------------------------------
# Tucker and the greedy path
# ---------------------------------------------------------------------------

def _tucker_case(rng, d=2):
    n = (8, 8) if d == 2 else (4, 4, 6)
    modes = (2, 3) if d == 2 else (1, 2, 2)
    kd = tuple(2 * m for m in modes[:-1]) + (modes[-1],)
    ci, co = 3, 4
    rank = (2, 3) + tuple([2] * d)
    core = _cplx(rng, rank, 0.5)
    u_in = _cplx(rng, (ci, rank[0]), 0.5)
    u_out = _cplx(rng, (co, rank[1]), 0.5)
    u_mode = [_cplx(rng, (kd[j], rank[2 + j]), 0.5) for j in range(d)]
    return n, modes, kd, ci, co, rank, core, u_in, u_out, u_mode


@pytest.mark.parametrize("d", [2, 3])
def test_tucker_all_orders_agree(d):
    """Dense reconstruction, both greedy policies and random pairwise orders
    all give the same spectrum product."""
    rng = _rng(30 + d)
    n, modes, kd, ci, co, rank, core, u_in, u_out, u_mode = _tucker_case(rng, d)
    xh = _cplx(rng, (2, ci) + kd)
    dense = O.contract_dense(xh, O.tucker_dense(core, u_in, u_out, u_mode))
    scale = np.abs(dense).max()
    for pol in (O.POLICY_MIN_RESULT, O.POLICY_MIN_NET):
        got = O.tucker_contract(xh, core, u_in, u_out, u_mode, n, modes, pol)
        assert np.abs(got - dense).max() <= 1e-12 * scale
    ops, out = O.tucker_labels(d)
    for trial in range(6):
        # random order: repeatedly pick a random pair; result keeps needed indices
        cur = list(ops)
        steps = []
        while len(cur) > 2:
            p, q = sorted(rng.choice(len(cur), 2, replace=False).tolist())
            res = O.pair_result(cur, p, q, out)
            steps.append((p, q, res))
            cur = [o for r, o in enumerate(cur) if r not in (p, q)] + [res]
        steps.append((0, 1, out))
        got = O.tucker_contract(xh, core, u_in, u_out, u_mode, n, modes, steps=steps)
        assert np.abs(got - dense).max() <= 1e-12 * scale


def test_tucker_dense_mode_products():
    """The dense reconstruction equals explicit sums over the core."""
    rng = _rng(33)
    n, modes, kd, ci, co, rank, core, u_in, u_out, u_mode = _tucker_case(rng, 2)
    w = O.tucker_dense(core, u_in, u_out, u_mode)
    i, o, t1, t2 = 2, 1, 3, 2
    s = 0j
    for a, e, c, dd in itertools.product(*[range(r) for r in rank]):
        s += core[a, e, c, dd] * u_in[i, a] * u_out[o, e] * u_mode[0][t1, c] * u_mode[1][t2, dd]
    assert abs(w[i, o, t1, t2] - s) < 1e-13


@pytest.mark.parametrize("policy", ["min_result", "min_net"])
def test_greedy_paths_golden(policy):
    with open(os.path.join(GOLDEN, "tucker_paths.json")) as f:
        g = json.load(f)
    steps = O.greedy_path(g["operands"], g["sizes"], g["output"], policy)
    exp = g[policy]["steps"]
    assert len(steps) == len(exp)
    for (p, q, res), (ep, eq, eres, esize) in zip(steps, exp):
        assert (p, q) == (ep, eq)
        assert sorted(res) == sorted(eres)
        assert O._size(res, g["sizes"]) == esize
    assert steps[-1][2] == g["output"]
    assert O.path_macs(g["operands"], g["sizes"], steps) == g[policy]["macs"]
    peak = max(O._size(r, g["sizes"]) for _, _, r in steps)
    assert peak == g[policy]["peak"]


@pytest.mark.parametrize("policy", ["min_result", "min_net"])
def test_greedy_adjoint_golden(policy):
    """The data gradient's contraction (G with the conjugated factors) follows
    its own hand-derived greedy sequence (tests/golden/tucker_paths.json,
    "adjoint"), ties included."""
    with open(os.path.join(GOLDEN, "tucker_paths.json")) as f:
        g = json.load(f)
    ops_a, out_a = O.tucker_labels(2, adjoint=True)
    ga = g["adjoint"]
    assert ops_a == ga["operands"] and out_a == ga["output"]
    sz = O.tucker_sizes(16, 128, 128, (64, 32), (13, 13, 6, 3))
    assert sz == g["sizes"]
    steps = O.greedy_path(ops_a, sz, out_a, policy)
    exp = ga[policy]["steps"]
    assert len(steps) == len(exp)
    for (p, q, res), (ep, eq, eres, esize) in zip(steps, exp):
        assert (p, q) == (ep, eq)
        assert sorted(res) == sorted(eres)
        assert O._size(res, sz) == esize
    assert steps[-1][2] == out_a
    assert O.path_macs(ops_a, sz, steps) == ga[policy]["macs"]
    assert max(O._size(r, sz) for _, _, r in steps) == ga[policy]["peak"]


@pytest.mark.parametrize("precision", [F32, F16T])
def test_tucker_gradients_fd(precision):
    """Central finite differences for the core and every factor."""
    rng = _rng(40)
    n, modes, kd, ci, co, rank, core, u_in, u_out, u_mode = _tucker_case(rng, 2)
    x = rng.standard_normal((1, ci) + n) * 0.7
    gy = rng.standard_normal((1, co) + n)

    def loss(cr, ui, uo, um):
        return float(np.sum(gy * O.tucker_fwd(x, cr, ui, uo, um, n, modes, precision)))

    g_core, g_in, g_out, g_mode = O.tucker_bwd_weight(x, gy, core, u_in, u_out, u_mode,
                                                      n, modes, precision)
    h = 1e-6
    params = [("core", core, g_core), ("in", u_in, g_in), ("out", u_out, g_out),
              ("m0", u_mode[0], g_mode[0]), ("m1", u_mode[1], g_mode[1])]
    for name, arr, grad in params:
        flat_idx = [0, arr.size - 1, arr.size // 2]
        for fi in flat_idx:
            idx = np.unravel_index(fi, arr.shape)
            for comp in (1.0, 1j):
                def bump(sgn):
                    a2 = arr.copy()
                    a2[idx] += sgn * h * comp
                    args = {"core": core, "in": u_in, "out": u_out,
                            "m0": u_mode[0], "m1": u_mode[1]}
                    args[name] = a2
                    return loss(args["core"], args["in"], args["out"],
                                [args["m0"], args["m1"]])
                fd = (bump(1) - bump(-1)) / (2 * h)
                ref = grad[idx].real if comp == 1.0 else grad[idx].imag
                assert abs(fd - ref) <= 1e-7 * max(1.0, abs(ref)), (name, idx, comp)


def test_tucker_bwd_data_matches_dense():
    rng = _rng(41)
    n, modes, kd, ci, co, rank, core, u_in, u_out, u_mode = _tucker_case(rng, 2)
    x = rng.standard_normal((2, ci) + n)
    gy = rng.standard_normal((2, co) + n)
    w = O.tucker_dense(core, u_in, u_out, u_mode)
    for pol in ("min_result", "min_net"):
        a = O.tucker_bwd_data(x, core, u_in, u_out, u_mode, gy, n, modes, F16T, pol)
        b = O.bwd_data(x, w, gy, n, modes, F16T)
        assert np.abs(a - b).max() <= 1e-12 * np.abs(b).max()


# ---------------------------------------------------------------------------
# CP-factorised weights (Sec. 4.6)
# ---------------------------------------------------------------------------

def _cp_case(rng, d=2, rank=3):
    n = (8, 8) if d == 2 else (4, 4, 6)
    modes = (2, 3) if d == 2 else (1, 2, 2)
    kd = tuple(2 * m for m in modes[:-1]) + (modes[-1],)
    ci, co = 3, 4
    lam = _cplx(rng, (rank,), 0.5)
    u_in = _cplx(rng, (ci, rank), 0.5)
    u_out = _cplx(rng, (co, rank), 0.5)
    u_mode = [_cplx(rng, (kd[j], rank), 0.5) for j in range(d)]
    return n, modes, kd, ci, co, rank, lam, u_in, u_out, u_mode


def _superdiagonal_core(lam, d):
    """The Tucker core of a CP tensor: lam[r] on the superdiagonal."""
    r = lam.shape[0]
    core = np.zeros((r,) * (2 + d), dtype=np.complex128)
    for k in range(r):
        core[(k,) * (2 + d)] = lam[k]
    return core


def test_cp_dense_explicit_sum():
    """The dense reconstruction equals the rank-one sum written out."""
    rng = _rng(60)
    n, modes, kd, ci, co, rank, lam, u_in, u_out, u_mode = _cp_case(rng, 2)
    w = O.cp_dense(lam, u_in, u_out, u_mode)
    assert w.shape == (ci, co) + kd
    for (i, o, t1, t2) in [(0, 0, 0, 0), (2, 1, 3, 2), (1, 3, 2, 1)]:
        s = sum(lam[r] * u_in[i, r] * u_out[o, r] * u_mode[0][t1, r] * u_mode[1][t2, r]
                for r in range(rank))
        assert abs(w[i, o, t1, t2] - s) < 1e-13


@pytest.mark.parametrize("d", [2, 3])
def test_cp_is_superdiagonal_tucker(d):
    """A CP tensor is a Tucker tensor whose core holds lambda on its
    superdiagonal (Kolda-Bader): the CP layer equals the Tucker layer with
    that core, and the lambda gradient is the core gradient's superdiagonal
    while the factor gradients coincide."""
    rng = _rng(61 + d)
    n, modes, kd, ci, co, rank, lam, u_in, u_out, u_mode = _cp_case(rng, d)
    core = _superdiagonal_core(lam, d)
    x = rng.standard_normal((2, ci) + n) * 0.7
    gy = rng.standard_normal((2, co) + n)
    wt = O.tucker_dense(core, u_in, u_out, u_mode)
    wc = O.cp_dense(lam, u_in, u_out, u_mode)
    assert np.abs(wt - wc).max() <= 1e-13
    for prec in (F32, F16T):
        a = O.cp_fwd(x, lam, u_in, u_out, u_mode, n, modes, prec)
        b = O.tucker_fwd(x, core, u_in, u_out, u_mode, n, modes, prec)
        assert np.abs(a - b).max() <= 1e-12 * np.abs(b).max()
        a = O.cp_bwd_data(x, lam, u_in, u_out, u_mode, gy, n, modes, prec)
        b = O.tucker_bwd_data(x, core, u_in, u_out, u_mode, gy, n, modes, prec)
        assert np.abs(a - b).max() <= 1e-12 * np.abs(b).max()
        g_lam, g_in, g_out, g_mode = O.cp_bwd_weight(x, gy, lam, u_in, u_out, u_mode, n,
                                                     modes, prec)
        t_core, t_in, t_out, t_mode = O.tucker_bwd_weight(x, gy, core, u_in, u_out, u_mode,
                                                          n, modes, prec)
        diag = np.array([t_core[(k,) * (2 + d)] for k in range(rank)])
        for got, ref in [(g_lam, diag), (g_in, t_in), (g_out, t_out)] + \
                list(zip(g_mode, t_mode)):
            assert np.abs(got - ref).max() <= 1e-12 * max(np.abs(ref).max(), 1e-30)


@pytest.mark.parametrize("d", [2, 3])
def test_cp_all_orders_agree(d):
    """Dense reconstruction, both greedy policies and random pairwise orders
    all give the same spectrum product (forward and adjoint)."""
    rng = _rng(64 + d)
    n, modes, kd, ci, co, rank, lam, u_in, u_out, u_mode = _cp_case(rng, d)
    w = O.cp_dense(lam, u_in, u_out, u_mode)
    for adjoint in (False, True):
        spec = _cplx(rng, (2, co if adjoint else ci) + kd)
        if adjoint:
            ref = np.einsum("bo...,io...->bi...", spec, np.conj(w))
        else:
            ref = O.contract_dense(spec, w)
        scale = np.abs(ref).max()
        for pol in (O.POLICY_MIN_RESULT, O.POLICY_MIN_NET):
            got = O.cp_contract(spec, lam, u_in, u_out, u_mode, pol, adjoint)
            assert np.abs(got - ref).max() <= 1e-12 * scale
        ops, out = O.cp_labels(d, adjoint)
        for trial in range(6):
            cur = list(ops)
            steps = []
            while len(cur) > 2:
                p, q = sorted(rng.choice(len(cur), 2, replace=False).tolist())
                res = O.pair_result(cur, p, q, out)
                steps.append((p, q, res))
                cur = [o for r, o in enumerate(cur) if r not in (p, q)] + [res]
            steps.append((0, 1, out))
            got = O.cp_contract(spec, lam, u_in, u_out, u_mode, adjoint=adjoint, steps=steps)
            assert np.abs(got - ref).max() <= 1e-12 * scale


@pytest.mark.parametrize("policy", ["min_result", "min_net"])
def test_cp_greedy_paths_golden(policy):
    with open(os.path.join(GOLDEN, "cp_paths.json")) as f:
        g = json.load(f)
    ops, out = O.cp_labels(2)
    assert ops == g["operands"] and out == g["output"]
    steps = O.greedy_path(g["operands"], g["sizes"], g["output"], policy)
    exp = g[policy]["steps"]
    assert len(steps) == len(exp)
    for (p, q, res), (ep, eq, eres, esize) in zip(steps, exp):
        assert (p, q) == (ep, eq)
        assert sorted(res) == sorted(eres)
        assert O._size(res, g["sizes"]) == esize
    assert steps[-1][2] == g["output"]
    assert O.path_macs(g["operands"], g["sizes"], steps) == g[policy]["macs"]
    peak = max(O._size(r, g["sizes"]) for _, _, r in steps)
    assert peak == g[policy]["peak"]


@pytest.mark.parametrize("precision", [F32, F16T])
def test_cp_gradients_fd(precision):
    """Central finite differences for lambda and every factor."""
    rng = _rng(70)
    n, modes, kd, ci, co, rank, lam, u_in, u_out, u_mode = _cp_case(rng, 2)
    x = rng.standard_normal((1, ci) + n) * 0.7
    gy = rng.standard_normal((1, co) + n)

    def loss(lm, ui, uo, um):
        return float(np.sum(gy * O.cp_fwd(x, lm, ui, uo, um, n, modes, precision)))

    g_lam, g_in, g_out, g_mode = O.cp_bwd_weight(x, gy, lam, u_in, u_out, u_mode, n, modes,
                                                 precision)
    h = 1e-6
    params = [("lam", lam, g_lam), ("in", u_in, g_in), ("out", u_out, g_out),
              ("m0", u_mode[0], g_mode[0]), ("m1", u_mode[1], g_mode[1])]
    for name, arr, grad in params:
        for fi in [0, arr.size - 1, arr.size // 2]:
            idx = np.unravel_index(fi, arr.shape)
            for comp in (1.0, 1j):
                def bump(sgn):
                    a2 = arr.copy()
                    a2[idx] += sgn * h * comp
                    args = {"lam": lam, "in": u_in, "out": u_out,
                            "m0": u_mode[0], "m1": u_mode[1]}
                    args[name] = a2
                    return loss(args["lam"], args["in"], args["out"],
                                [args["m0"], args["m1"]])
                fd = (bump(1) - bump(-1)) / (2 * h)
                ref = grad[idx].real if comp == 1.0 else grad[idx].imag
                assert abs(fd - ref) <= 1e-7 * max(1.0, abs(ref)), (name, idx, comp)


def test_cp_bwd_data_matches_dense():
    rng = _rng(71)
    n, modes, kd, ci, co, rank, lam, u_in, u_out, u_mode = _cp_case(rng, 2)
    x = rng.standard_normal((2, ci) + n)
    gy = rng.standard_normal((2, co) + n)
    w = O.cp_dense(lam, u_in, u_out, u_mode)
    for pol in ("min_result", "min_net"):
        a = O.cp_bwd_data(x, lam, u_in, u_out, u_mode, gy, n, modes, F16T, pol)
        b = O.bwd_data(x, w, gy, n, modes, F16T)
        assert np.abs(a - b).max() <= 1e-12 * np.abs(b).max()


# ---------------------------------------------------------------------------
# Failure mode the tanh stabiliser addresses (Sec. 4.3), emulated on the CPU
# ---------------------------------------------------------------------------

def test_fp16_overflow_without_tanh():
    """An unnormalised DC coefficient accumulated in fp16 with a pairwise
    (butterfly-like) sum overflows on a 1024^2 grid for a field of mean ~1,
    whereas the 1/N-normalised spectrum of tanh(x) is bounded by 1."""
    rng = _rng(50)
    a = (1.0 + rng.standard_normal(1024 * 1024) * 0.5).astype(np.float16)
    with np.errstate(over="ignore", invalid="ignore"):
        while a.size > 1:
            a = (a[0::2] + a[1::2]).astype(np.float16)
    assert not np.isfinite(a[0])
    n = (32, 32)
    x = (1.0 + rng.standard_normal((1, 1) + n) * 0.5) * 1e4
    xh = O.forward_spectrum(O.preactivation(x, F16T), n, (4, 4))
    assert np.abs(xh).max() <= 1.0


# ---------------------------------------------------------------------------
# Planted mistakes: each must make at least one pin fail
# ---------------------------------------------------------------------------

def _pins_fail():
    failing = []
    for name, (fn, tol) in ALL_PINS.items():
        try:
            err = fn()
        except Exception:
            failing.append(name)
            continue
        if not (err <= tol):
            failing.append(name)
    return failing


def _rel_l2_abs_not_squared(a, b):
    a = np.asarray(a, dtype=np.complex128)
    b = np.asarray(b, dtype=np.complex128)
    den = np.sqrt(np.sum(np.abs(b)))
    num = np.sqrt(np.sum(np.abs(a - b)))
    return float(num / den) if den else float(num)


def _rel_l2_in_input_dtype(a, b):
    a = np.asarray(a)
    b = np.asarray(b)
    with np.errstate(over="ignore", invalid="ignore"):
        num = np.sqrt(np.sum((a - b) * np.conj(a - b)).real)
        den = np.sqrt(np.sum(b * np.conj(b)).real)
    return float(num / den) if den else float(num)


def _sigma_bounds_sample_std(x, k):
    xf = np.asarray(x, dtype=np.float64)
    axes = tuple(range(2, xf.ndim))
    mu = xf.mean(axis=axes, keepdims=True)
    sd = xf.std(axis=axes, ddof=1, keepdims=True)
    return mu - k * sd, mu + k * sd


def _sigma_bounds_whole_tensor(x, k):
    xf = np.asarray(x, dtype=np.float64)
    mu, sd = xf.mean(), xf.std()
    shape = xf.shape[:2] + (1,) * (xf.ndim - 2)
    return np.full(shape, mu - k * sd), np.full(shape, mu + k * sd)


def _gelu_tanh_form(z):
    z = np.asarray(z, dtype=np.float64)
    return 0.5 * z * (1.0 + np.tanh(np.sqrt(2.0 / np.pi) * (z + 0.044715 * z ** 3)))


def _epi_fwd_residual_inside(orig):
    def f(x, y, w, b, act, residual):
        if not residual:
            return orig(x, y, w, b, act, residual)
        yy = np.asarray(y, dtype=np.float64) + np.asarray(x, dtype=np.float64)
        return orig(x, yy, w, b, act, False)
    return f


def _epi_bwd_variant(kind):
    def make(orig):
        def f(x, z, g_out, w, act, residual):
            g_z, g_x, g_w, g_b = orig(x, z, g_out, w, act, residual)
            if kind == "no_act_grad":
                g_z2, g_x2, g_w2, g_b2 = orig(x, np.zeros_like(z), g_out, w, O.EPI_ACT_NONE,
                                              residual)
                return g_z2, g_x2, g_w2, g_b2
            if kind == "no_residual" and residual:
                g_x = g_x - np.asarray(g_out, dtype=np.float64)
            if kind == "gw_transposed":
                g_w = g_w.T
            if kind == "gb_mean":
                g_b = g_b / np.prod(np.shape(g_z)[2:])
            return g_z, g_x, g_w, g_b
        return f
    return make


MUTATIONS = {
    "gelu_tanh_approximation": ("gelu", lambda orig: _gelu_tanh_form),
    "gelu_grad_no_density": ("gelu_grad", lambda orig: (
        lambda z: 0.5 * (1.0 + __import__("scipy.special").special.erf(
            np.asarray(z, dtype=np.float64) / np.sqrt(2.0))))),
    "epi_bias_dropped": ("block_epilogue_fwd", lambda orig: (
        lambda x, y, w, b, act, res: orig(x, y, w, None, act, res))),
    "epi_skip_transposed": ("channel_mix", lambda orig: (
        lambda w, v: orig(np.asarray(w).T, v))),
    "epi_residual_before_activation": ("block_epilogue_fwd", _epi_fwd_residual_inside),
    "epi_gz_without_act_grad": ("block_epilogue_bwd", _epi_bwd_variant("no_act_grad")),
    "epi_gx_without_residual": ("block_epilogue_bwd", _epi_bwd_variant("no_residual")),
    "epi_gw_transposed": ("block_epilogue_bwd", _epi_bwd_variant("gw_transposed")),
    "epi_gb_mean": ("block_epilogue_bwd", _epi_bwd_variant("gb_mean")),
    "sigma_sample_std": ("sigma_bounds", lambda orig: _sigma_bounds_sample_std),
    "sigma_whole_tensor": ("sigma_bounds", lambda orig: _sigma_bounds_whole_tensor),
    "sigma_one_sigma": ("sigma_bounds", lambda orig: (lambda x, k: orig(x, k / 2.0))),
    "sigma_one_sided": ("sigma_bounds", lambda orig: (
        lambda x, k: (np.full_like(orig(x, k)[0], -np.inf), orig(x, k)[1]))),
    "sigma_grad_ones": ("preactivation_grad", lambda orig: (
        lambda x, p: np.ones(np.shape(x)) if O.preact_kind(p)[0] == "sigma" else orig(x, p))),
    "rel_l2_divides_by_a": ("rel_l2", lambda orig: (lambda a, b: orig(b, a))),
    "rel_l2_no_sqrt": ("rel_l2", lambda orig: (lambda a, b: orig(a, b) ** 2)),
    "rel_l2_real_part_only": ("rel_l2", lambda orig: (
        lambda a, b: orig(np.real(a), np.real(b)))),
    "rel_l2_abs_not_squared": ("rel_l2", lambda orig: _rel_l2_abs_not_squared),
    "rel_l2_squares_in_fp16": ("rel_l2", lambda orig: _rel_l2_in_input_dtype),
    "rel_l2_max_norm": ("rel_l2", lambda orig: (
        lambda a, b: float(np.abs(np.asarray(a, dtype=np.complex128) - b).max()
                           / max(np.abs(np.asarray(b, dtype=np.complex128)).max(), 1e-300)))),
    "rel_l2_zero_ref_is_zero": ("rel_l2", lambda orig: (
        lambda a, b: 0.0 if not np.any(np.asarray(b)) else orig(a, b))),
    "max_plane_is_whole_tensor": ("max_plane_rel_l2", lambda orig: (
        lambda a, b, nlead=2: O.rel_l2(a, b))),
    "no_multiplicity": ("multiplicity", lambda orig: (lambda k, n: np.ones(np.shape(k)))),
    "c_everywhere_2": ("multiplicity", lambda orig: (lambda k, n: 2.0 * np.ones(np.shape(k)))),
    "wrong_sign": ("dft_matrix", lambda orig: (lambda n, ks, s: orig(n, ks, -s))),
    "high_block_off_by_one": ("mode_freq", lambda orig: (
        lambda n, m, last: orig(n, m, last) if last else
        np.where(np.arange(2 * m) < m, np.arange(2 * m), n - 2 * m + np.arange(2 * m) - 1))),
    "transposed_weight": ("contract_dense", lambda orig: (
        lambda xh, w: np.einsum("bi...,oi...->bo...", xh, w))),
    "conj_weight": ("contract_dense", lambda orig: (lambda xh, w: orig(xh, np.conj(w)))),
    "no_normalisation": ("forward_spectrum", lambda orig: (
        lambda u, n, m: orig(u, n, m) * float(np.prod(n)))),
    "drop_imag_in_inverse": ("inverse_spectrum", lambda orig: (
        lambda z, n, m, with_c=True: orig(np.real(z) + 0j, n, m, with_c))),
    "tanh_prime_wrong": ("bwd_data", lambda orig: (
        lambda x, w, gy, n, m, p: orig(x, w, gy, n, m, O.PREC_FP32))),
    "clip_one_sided": ("preactivation", lambda orig: (
        lambda x, p: np.minimum(np.asarray(x, dtype=np.float64), O.preact_kind(p)[1])
        if O.preact_kind(p)[0] == "clip" else orig(x, p))),
    "clip_grad_ones": ("preactivation_grad", lambda orig: (
        lambda x, p: np.ones(np.shape(x)) if O.preact_kind(p)[0] == "clip" else orig(x, p))),
    "fp32_tanh_as_identity": ("preact_kind", lambda orig: (
        lambda p: ("none", None) if p == O.PREC_FP32_TANH else orig(p))),
    "grad_no_c": ("grad_spectrum", lambda orig: (
        lambda gy, n, m: O.forward_spectrum(gy, n, m) * float(np.prod(n)))),
    "cp_drop_lambda": ("cp_dense", lambda orig: (
        lambda lam, ui, uo, um: orig(np.ones_like(lam), ui, uo, um))),
    "cp_adjoint_no_conj": ("cp_contract", lambda orig: (
        lambda spec, lam, ui, uo, um, policy=O.POLICY_MIN_RESULT, adjoint=False, steps=None:
        O.contract_path([spec, lam, ui, uo] + list(um), O.cp_labels(len(um), adjoint)[0],
                        O.greedy_path(O.cp_labels(len(um), adjoint)[0],
                                      O.cp_sizes(spec.shape[0], ui.shape[0], uo.shape[0],
                                                 spec.shape[2:], lam.shape[0]),
                                      O.cp_labels(len(um), adjoint)[1], policy)))),
    "cp_wgrad_lambda_no_conj": ("cp_bwd_weight", lambda orig: (
        lambda x, gy, lam, ui, uo, um, n, m, p: (
            np.conj(orig(x, gy, lam, ui, uo, um, n, m, p)[0]),) +
        tuple(orig(x, gy, lam, ui, uo, um, n, m, p)[1:]))),
    "wgrad_no_conj": ("bwd_weight", lambda orig: (
        lambda x, gy, n, m, p: np.einsum(
            "bi...,bo...->io...",
            O.forward_spectrum(O.preactivation(x, p), n, m),
            O.grad_spectrum(gy, n, m)))),
}


@pytest.mark.parametrize("mut", sorted(MUTATIONS))
def test_planted_mistake_is_caught(mut, monkeypatch):
    attr, make = MUTATIONS[mut]
    orig = getattr(O, attr)
    monkeypatch.setattr(O, attr, make(orig))
    failing = _pins_fail()
    assert failing, f"mutation {mut} passed every pin"
