"""GPU parity: the HIP path (through the C ABI) against the float64 oracle on
the same seeded stored inputs.

Tolerances (relative L2): 1e-5 in fp32 mode, 3e-3 in fp16+tanh mode, held
both over the whole output and over every plane of it (each (batch, channel)
plane of y and gx, each (c_in, c_out) plane of gW), so that an error confined
to one plane cannot hide in the norm of the rest.  Full-size workloads that
the oracle cannot finish in seconds are compared on sampled outputs (the
first and the last batch sample for y and gx; all modes of gW with the
spectra computed sample by sample).
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

from oracle import fno_oracle as O  # noqa: E402
import synth  # noqa: E402
from tests import gpu_util as U  # noqa: E402

PRECS = ["fp32", "fp16_tanh"]


def test_native_library_loaded():
    import os
    from paper_2307_15034_amd import binding as B
    here = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    assert os.path.realpath(B.LIB_PATH).startswith(os.path.realpath(here))
    assert B.lib()._name == B.LIB_PATH


def _oracle_dense(x, w, gy, n, modes, oprec):
    wc = U.cplx(w)
    y = O.fwd(x, wc, n, modes, oprec)
    gx = O.bwd_data(x, wc, gy, n, modes, oprec)
    gw = O.bwd_weight(x, gy, n, modes, oprec)
    return y, gx, gw


def _assert_close(name, got, ref, prec, planes=True):
    """Whole-tensor relative L2 and, for tensors with two leading axes and at
    least one more, the largest per-plane relative L2, both within the mode's
    tolerance."""
    r = U.rel(got, ref)
    rp = O.max_plane_rel_l2(got, ref) if planes and np.ndim(ref) >= 3 else None
    extra = f", max per plane {rp:.3e}" if rp is not None else ""
    U.say(f"  {name}: rel_l2 = {r:.3e}{extra} (tol {U.TOL[prec]:.0e})")
    assert np.isfinite(r) and r <= U.TOL[prec], f"{name}: {r:.3e}"
    if rp is not None:
        assert np.isfinite(rp) and rp <= U.TOL[prec], f"{name} (worst plane): {rp:.3e}"


EDGE = [
    # (n, modes, B, Cin, Cout)
    ((20, 24), (3, 5), 3, 5, 7),        # ragged tiles, K = 30 (scalar mode path)
    ((12, 18), (2, 10), 2, 3, 4),       # Nyquist retained, row length not a multiple of 8
    ((8, 6), (4, 4), 2, 3, 3),          # every mode retained
    ((96,), (17,), 2, 3, 5),            # 1-D
    ((6, 10, 12), (2, 3, 4), 2, 3, 2),  # 3-D, ragged
    ((32, 32), (5, 7), 37, 33, 18),     # batch / channels past the 32-wide tiles
    ((1000, 40), (6, 9), 1, 2, 3),      # several row chunks, rows not a multiple of 32
    ((16, 256), (8, 100), 1, 2, 2),     # 100 retained last-axis modes (widest tile)
    ((64, 64), (32, 33), 1, 2, 2),      # 64 leading-axis slots, Nyquist
    ((256, 256), (32, 32), 2, 3, 2),    # wide-plane transforms: one 256-row chunk
    ((512, 128), (16, 64), 1, 2, 3),    # wide-plane transforms: two chunks, 64 last-axis modes
    ((256, 256), (32, 32), 9, 30, 31),  # wide-plane transforms: more planes than work-groups
    # radix-2 wide-plane transforms: odd and even slot classes of unequal
    # padding, several items per plane, leading-axis tiles padded per class
    ((512, 256), (20, 20), 2, 3, 2),    # 10 + 10 last-axis slots, 2 x 20 leading
    ((256, 512), (40, 36), 1, 2, 3),    # 18 + 18 last-axis slots (four column tiles)
    ((1024, 256), (8, 12), 3, 2, 2),    # four items per plane, 6 + 6 slots
    # four column tiles: the plain inverse's 64-column blocks (Nb / 2 not a
    # multiple of 256) beside the 128-column ones of (256, 512) above
    ((256, 256), (40, 36), 1, 2, 3),    # two 64-column blocks
    ((768, 768), (40, 40), 1, 2, 2),    # six 64-column blocks, three chunks
]


@pytest.mark.parametrize("prec", PRECS)
@pytest.mark.parametrize("case", range(len(EDGE)))
def test_dense_edge_cases(case, prec):
    n, modes, Bt, ci, co = EDGE[case]
    _, npdt, oprec = U.prec_codes(prec)
    U.say(f"edge case {case}: n={n} modes={modes} B={Bt} Cin={ci} Cout={co} {prec}")
    x, w, gy = synth.random_dense_case(case, Bt, ci, co, n, modes, npdt)
    layer = U.make_layer(n, modes, Bt, ci, co, prec)
    y, gx, gw = U.run_all(layer, x, w, gy)
    ry, rgx, rgw = _oracle_dense(x, w, gy, n, modes, oprec)
    _assert_close("y", y, ry, prec)
    _assert_close("gx", gx, rgx, prec)
    _assert_close("gW", U.cplx(gw), rgw, prec)


_CACHE = {}


def _workload_inputs(wid, prec, batch=None):
    key = (wid, prec, batch)
    if key not in _CACHE:
        wl = synth.WORKLOADS[wid]
        _, npdt, _ = U.prec_codes(prec)
        x = synth.make_x(wl, npdt, batch)
        gy = synth.make_gy(wl, npdt, batch)
        w = synth.make_weight(wl, npdt)
        _CACHE.clear()
        _CACHE[key] = (x, w, gy)
    return _CACHE[key]


@pytest.mark.parametrize("prec", PRECS)
@pytest.mark.parametrize("wid", [1, 2, 4])
def test_workload_dense_full(wid, prec):
    wl = synth.WORKLOADS[wid]
    _, _, oprec = U.prec_codes(prec)
    U.say(f"workload {wid} {wl.name} {prec}")
    x, w, gy = _workload_inputs(wid, prec)
    layer = U.make_layer(wl.n, wl.modes, wl.batch, wl.c_in, wl.c_out, prec)
    y, gx, gw = U.run_all(layer, x, w, gy)
    ry, rgx, rgw = _oracle_dense(x, w, gy, wl.n, wl.modes, oprec)
    _assert_close("y", y, ry, prec)
    _assert_close("gx", gx, rgx, prec)
    _assert_close("gW", U.cplx(gw), rgw, prec)


def _spectra_by_sample(x, gy, n, modes, oprec):
    xs = np.concatenate([O.forward_spectrum(O.preactivation(x[b:b + 1], oprec), n, modes)
                         for b in range(x.shape[0])])
    gs = np.concatenate([O.grad_spectrum(gy[b:b + 1], n, modes) for b in range(gy.shape[0])])
    return xs, gs


@pytest.mark.parametrize("prec", PRECS)
def test_workload_hires_sampled(prec):
    """1024^2 workload at full size: y and gx of the first and the last batch
    sample compared with the oracle (whole and per plane); gW compared over
    every mode."""
    wid = 3
    wl = synth.WORKLOADS[wid]
    _, _, oprec = U.prec_codes(prec)
    U.say(f"workload {wid} {wl.name} {prec}")
    x, w, gy = _workload_inputs(wid, prec)
    layer = U.make_layer(wl.n, wl.modes, wl.batch, wl.c_in, wl.c_out, prec)
    y, gx, gw = U.run_all(layer, x, w, gy)
    wc = U.cplx(w)
    for b in (0, wl.batch - 1):
        ry = O.fwd(x[b:b + 1], wc, wl.n, wl.modes, oprec)
        _assert_close(f"y[b={b}]", y[b:b + 1], ry, prec)
        rgx = O.bwd_data(x[b:b + 1], wc, gy[b:b + 1], wl.n, wl.modes, oprec)
        _assert_close(f"gx[b={b}]", gx[b:b + 1], rgx, prec)
    xs, gs = _spectra_by_sample(x, gy, wl.n, wl.modes, oprec)
    rgw = np.einsum("bi...,bo...->io...", np.conj(xs), gs)
    _assert_close("gW", U.cplx(gw), rgw, prec)


def test_wide_narrow_multi_item():
    """1024^2 planes through the narrow radix-2 wide-plane transforms (24 x 24
    modes: two column tiles per class, ragged leading-axis tiles) with four
    work items per plane and more planes (3 x 96 = 288) than work-groups, so
    that the early step-B tables, the next item's rows and the inverse's
    next-item epilogue inputs all cross item and plane boundaries.  y and gx
    of the last batch sample (planes 192..287, the second plane of the first
    work-groups among them) against the oracle; gW over every mode."""
    n, modes, Bt, ci, co, prec = (1024, 1024), (24, 24), 3, 96, 96, "fp16_tanh"
    _, _, oprec = U.prec_codes(prec)
    U.say(f"narrow wide-plane transforms n={n} modes={modes} B={Bt} C={ci}->{co}")
    x, w, gy = synth.random_dense_case(81, Bt, ci, co, n, modes, np.float16)
    layer = U.make_layer(n, modes, Bt, ci, co, prec)
    y, gx, gw = U.run_all(layer, x, w, gy)
    wc = U.cplx(w)
    b = Bt - 1
    _assert_close(f"y[b={b}]", y[b:b + 1], O.fwd(x[b:b + 1], wc, n, modes, oprec), prec)
    _assert_close(f"gx[b={b}]", gx[b:b + 1],
                  O.bwd_data(x[b:b + 1], wc, gy[b:b + 1], n, modes, oprec), prec)
    xs, gs = _spectra_by_sample(x, gy, n, modes, oprec)
    _assert_close("gW", U.cplx(gw), np.einsum("bi...,bo...->io...", np.conj(xs), gs), prec)


@pytest.mark.parametrize("policy", ["min_result", "min_net"])
@pytest.mark.parametrize("prec", PRECS)
def test_workload_tucker(prec, policy):
    """Tucker workload at full size: y and gx of the first and the last batch
    sample; the core and factor gradients from all samples."""
    wid = 5
    wl = synth.WORKLOADS[wid]
    _, _, oprec = U.prec_codes(prec)
    U.say(f"workload {wid} {wl.name} {prec} {policy}")
    x, w, gy = _workload_inputs(wid, prec)
    pol = 0 if policy == "min_result" else 1
    layer = U.make_layer(wl.n, wl.modes, wl.batch, wl.c_in, wl.c_out, prec, wl.rank, pol)
    y, gx, gw = U.run_all(layer, x, w, gy)
    core, u_in, u_out = U.cplx(w["core"]), U.cplx(w["u_in"]), U.cplx(w["u_out"])
    u_mode = [U.cplx(u) for u in w["u_mode"]]
    for b in (0, wl.batch - 1):
        ry = O.tucker_fwd(x[b:b + 1], core, u_in, u_out, u_mode, wl.n, wl.modes, oprec,
                          policy)
        _assert_close(f"y[b={b}]", y[b:b + 1], ry, prec)
        rgx = O.tucker_bwd_data(x[b:b + 1], core, u_in, u_out, u_mode, gy[b:b + 1], wl.n,
                                wl.modes, oprec, policy)
        _assert_close(f"gx[b={b}]", gx[b:b + 1], rgx, prec)
    g_core, g_in, g_out, g_mode = O.tucker_bwd_weight(x, gy, core, u_in, u_out, u_mode,
                                                      wl.n, wl.modes, oprec)
    gwc = U.gw_complex(gw)
    _assert_close("g_core", gwc["core"], g_core, prec)
    _assert_close("g_u_in", gwc["u_in"], g_in, prec)
    _assert_close("g_u_out", gwc["u_out"], g_out, prec)
    for j in range(wl.ndim):
        _assert_close(f"g_u_mode{j}", gwc["u_mode"][j], g_mode[j], prec)


TUCKER_EDGE = [
    ((8, 8), (2, 3), 2, 3, 4, (2, 3, 2, 2)),
    ((6, 10, 12), (2, 3, 4), 2, 3, 2, (2, 2, 2, 3, 2)),
    ((40,), (7,), 3, 2, 5, (3, 2, 4)),
    # ranks and C_in multiples of 4 but not of 16: GEMM steps whose operands
    # are staged as 16-byte quads of contiguous contracted elements, with
    # contractions that end in a partial stage
    ((16, 24), (4, 5), 3, 12, 20, (4, 8, 2, 4)),
    # B r_in + B r_out + r_in r_out > 1024: the weight gradient's R, Z1 and
    # Z2 as three launches instead of the fused one
    ((8, 8), (2, 3), 40, 16, 16, (14, 14, 2, 2)),
]


@pytest.mark.parametrize("policy", ["min_result", "min_net"])
@pytest.mark.parametrize("prec", PRECS)
@pytest.mark.parametrize("case", range(len(TUCKER_EDGE)))
def test_tucker_edge_cases(case, prec, policy):
    n, modes, Bt, ci, co, rank = TUCKER_EDGE[case]
    _, npdt, oprec = U.prec_codes(prec)
    U.say(f"tucker edge {case}: n={n} modes={modes} rank={rank} {prec} {policy}")
    rng = np.random.default_rng(np.random.SeedSequence([2000 + case]))
    d = len(n)
    kd = tuple(2 * m if j < d - 1 else m for j, m in enumerate(modes))

    def cp(shape, std):
        return (rng.standard_normal(tuple(shape) + (2,)) * std).astype(npdt)

    w = {"core": cp(rank, 0.5), "u_in": cp((ci, rank[0]), 0.5),
         "u_out": cp((co, rank[1]), 0.5),
         "u_mode": [cp((kd[j], rank[2 + j]), 0.5) for j in range(d)]}
    x = rng.standard_normal((Bt, ci) + n).astype(npdt)
    gy = rng.standard_normal((Bt, co) + n).astype(npdt)
    pol = 0 if policy == "min_result" else 1
    layer = U.make_layer(n, modes, Bt, ci, co, prec, rank, pol)
    y, gx, gw = U.run_all(layer, x, w, gy)
    core, u_in, u_out = U.cplx(w["core"]), U.cplx(w["u_in"]), U.cplx(w["u_out"])
    u_mode = [U.cplx(u) for u in w["u_mode"]]
    _assert_close("y", y, O.tucker_fwd(x, core, u_in, u_out, u_mode, n, modes, oprec, policy),
                  prec)
    _assert_close("gx", gx, O.tucker_bwd_data(x, core, u_in, u_out, u_mode, gy, n, modes,
                                               oprec, policy), prec)
    g_core, g_in, g_out, g_mode = O.tucker_bwd_weight(x, gy, core, u_in, u_out, u_mode, n,
                                                      modes, oprec)
    gwc = U.gw_complex(gw)
    _assert_close("g_core", gwc["core"], g_core, prec)
    _assert_close("g_u_in", gwc["u_in"], g_in, prec)
    _assert_close("g_u_out", gwc["u_out"], g_out, prec)
    for j in range(d):
        _assert_close(f"g_u_mode{j}", gwc["u_mode"][j], g_mode[j], prec)


# ---------------------------------------------------------------------------
# Invariants
# ---------------------------------------------------------------------------

def test_identity_round_trip_fp32():
    """Identity weights with every mode retained reproduce x (fp32 mode)."""
    n, modes = (16, 12), (8, 7)
    c = 4
    U.say("identity round trip")
    rng = np.random.default_rng(3)
    x = rng.standard_normal((2, c) + n).astype(np.float32)
    w = np.zeros((c, c, 16, 7, 2), dtype=np.float32)
    for i in range(c):
        w[i, i, :, :, 0] = 1.0
    layer = U.make_layer(n, modes, 2, c, c, "fp32")
    y = U.host(layer.fwd(U.dev(x), U.dev(w)))
    assert np.abs(y - x).max() < 1e-5


@pytest.mark.parametrize("prec", PRECS)
def test_deterministic_repeat(prec):
    """Two runs give bitwise-identical outputs (fixed reduction order)."""
    n, modes, Bt, ci, co = (32, 32), (5, 7), 37, 33, 18
    _, npdt, _ = U.prec_codes(prec)
    U.say(f"determinism {prec}")
    x, w, gy = synth.random_dense_case(77, Bt, ci, co, n, modes, npdt)
    layer = U.make_layer(n, modes, Bt, ci, co, prec)
    a = U.run_all(layer, x, w, gy)
    b = U.run_all(layer, x, w, gy)
    for u, v in zip(a, b):
        assert np.array_equal(u, v)


@pytest.mark.timeout(300)
@pytest.mark.parametrize("wid,reps", [(3, 24), (5, 6), (2, 12), (4, 12), (6, 8)])
def test_deterministic_repeat_workloads(wid, reps):
    """Repeated calls on a benchmark workload in its launch configuration are
    bit-identical to the first call: the forward and data gradient of the
    dense layers (chained, leading-axis and radix-2 transforms), and the
    Tucker and CP layers' combined backward (their weight gradients on the
    side streams).  A race in a kernel, such as a store handed another
    segment's values in a few lanes now and then, shows as a difference
    between repetitions."""
    wl = synth.WORKLOADS[wid]
    prec = "fp16_tanh"
    _, npdt, _ = U.prec_codes(prec)
    U.say(f"repeat {wl.name} x{reps}")
    x, w, gy = _workload_inputs(wid, prec)
    tucker = isinstance(w, dict)
    if wl.weight == "cp":
        layer = U.make_layer(wl.n, wl.modes, wl.batch, wl.c_in, wl.c_out, prec, policy=1,
                             cp_rank=wl.rank[0])
    elif tucker:
        layer = U.make_layer(wl.n, wl.modes, wl.batch, wl.c_in, wl.c_out, prec, wl.rank, 1)
    else:
        layer = U.make_layer(wl.n, wl.modes, wl.batch, wl.c_in, wl.c_out, prec)
    xd, gyd = U.dev(x), U.dev(gy)
    wd = ({"core": U.dev(w["core"]), "u_in": U.dev(w["u_in"]), "u_out": U.dev(w["u_out"]),
           "u_mode": [U.dev(u) for u in w["u_mode"]]} if tucker else U.dev(w))
    y, gx = torch.empty_like(xd), torch.empty_like(xd)
    xh = layer.spectrum_buffer(0)
    gw = layer.alloc_grads()

    def outputs():
        layer.fwd(xd, wd, y=y, x_hat=xh)
        if tucker:
            layer.bwd(xd, wd, gyd, x_hat=xh, gx=gx, gw=gw)
            return [y, gx, gw["core"], gw["u_in"], gw["u_out"]] + list(gw["u_mode"])
        layer.bwd_data(xd, wd, gyd, gx=gx)
        return [y, gx]

    first = [t.clone() for t in outputs()]
    for r in range(1, reps):
        cur = outputs()
        for k, (a, b) in enumerate(zip(cur, first)):
            assert torch.equal(a, b), f"repetition {r}: output {k} differs"
    torch.cuda.synchronize()


@pytest.mark.parametrize("prec", PRECS)
def test_caches_match_recompute(prec):
    n, modes, Bt, ci, co = (20, 24), (3, 5), 3, 5, 7
    _, npdt, _ = U.prec_codes(prec)
    U.say(f"caches vs recompute {prec}")
    x, w, gy = synth.random_dense_case(78, Bt, ci, co, n, modes, npdt)
    layer = U.make_layer(n, modes, Bt, ci, co, prec)
    a = U.run_all(layer, x, w, gy, caches=True)
    b = U.run_all(layer, x, w, gy, caches=False)
    for u, v in zip(a, b):
        assert np.array_equal(u, v)


# small planes, and planes that take the wide-plane transforms
SPECIAL_SHAPES = [((32, 32), (4, 5)), ((256, 256), (32, 32))]


@pytest.mark.parametrize("shape", range(len(SPECIAL_SHAPES)))
def test_fp16_extremes_stay_finite(shape):
    """tanh bounds the transform input: +-65504 and +-inf give finite outputs
    that still match the oracle."""
    (n, modes), Bt, ci, co = SPECIAL_SHAPES[shape], 2, 3, 3
    U.say(f"fp16 extremes n={n}")
    x, w, gy = synth.random_dense_case(79, Bt, ci, co, n, modes, np.float16, x_scale=3.0)
    x[0, 0, 0, :4] = np.array([65504.0, -65504.0, np.inf, -np.inf], dtype=np.float16)
    layer = U.make_layer(n, modes, Bt, ci, co, "fp16_tanh")
    y, gx, gw = U.run_all(layer, x, w, gy)
    assert np.isfinite(y).all() and np.isfinite(gx).all() and np.isfinite(gw).all()
    ry, rgx, rgw = _oracle_dense(x, w, gy, n, modes, O.PREC_FP16_TANH)
    _assert_close("y", y, ry, "fp16_tanh")
    _assert_close("gW", U.cplx(gw), rgw, "fp16_tanh")


@pytest.mark.parametrize("shape", range(len(SPECIAL_SHAPES)))
def test_nan_propagates(shape):
    (n, modes), Bt, ci, co = SPECIAL_SHAPES[shape], 2, 3, 3
    U.say(f"nan propagation n={n}")
    x, w, gy = synth.random_dense_case(80, Bt, ci, co, n, modes, np.float16)
    x[0, 1, 5, 7] = np.nan
    layer = U.make_layer(n, modes, Bt, ci, co, "fp16_tanh")
    y = U.host(layer.fwd(U.dev(x), U.dev(w)))
    assert np.isnan(y[0]).any()
    assert np.isfinite(y[1]).all()


# ---------------------------------------------------------------------------
# The combined backward call (data + weight gradient in one call)
# ---------------------------------------------------------------------------
BWD_CASES = [
    # (n, modes, B, Cin, Cout, prec): K % 16 == 0 fp16 takes the shared launch
    ((64, 64), (8, 8), 2, 16, 16, "fp16_tanh"),
    ((32, 32), (5, 7), 37, 33, 18, "fp16_tanh"),   # K = 70: separate kernels
    ((32, 32), (8, 8), 17, 20, 36, "fp16_tanh"),   # ragged rows / columns / batch
    ((6, 10, 12), (2, 3, 4), 2, 3, 2, "fp16_tanh"),
    ((32, 32), (8, 8), 3, 5, 7, "fp32"),
    ((64, 64), (8, 8), 2, 16, 16, "fp16_clip:0.75"),   # shared launch, clip derivative
    ((32, 32), (8, 8), 3, 5, 7, "fp32_tanh"),
]


@pytest.mark.parametrize("case", range(len(BWD_CASES)))
@pytest.mark.parametrize("cache", [True, False])
def test_combined_bwd(case, cache):
    """fno_spectral_conv_bwd gives the oracle's gx and gW, and exactly what the
    separate bwd_data / bwd_weight calls give."""
    n, modes, Bt, ci, co, prec = BWD_CASES[case]
    U.say(f"combined bwd case {case}: n={n} modes={modes} B={Bt} {ci}->{co} {prec} "
          f"cache={cache}")
    _, npdt, oprec = U.prec_codes(prec)
    x, w, gy = synth.random_dense_case(500 + case, Bt, ci, co, n, modes, npdt)
    layer = U.make_layer(n, modes, Bt, ci, co, prec)
    xd, wd, gyd = U.dev(x), U.dev(w), U.dev(gy)
    xh = layer.spectrum_buffer(0)
    gh = layer.spectrum_buffer(1)
    layer.fwd(xd, wd, x_hat=xh)
    gx, gw = layer.bwd(xd, wd, gyd, x_hat=xh if cache else None, gy_hat=gh)
    gx_sep = layer.bwd_data(xd, wd, gyd)
    gw_sep = layer.bwd_weight(xd, gyd, wd)
    torch.cuda.synchronize()
    U.say("  done")
    ref_gx = O.bwd_data(x, U.cplx(w), gy, n, modes, oprec)
    ref_gw = O.bwd_weight(x, gy, n, modes, oprec)
    _assert_close("gx", U.host(gx), ref_gx, prec)
    _assert_close("gW", U.cplx(U.host(gw)), ref_gw, prec)
    assert np.array_equal(U.host(gx), U.host(gx_sep))
    assert np.array_equal(U.host(gw), U.host(gw_sep))


@pytest.mark.parametrize("prec", PRECS)
def test_combined_bwd_tucker(prec):
    n, modes, Bt, ci, co, rank = (32, 32), (4, 5), 2, 6, 5, (3, 4, 2, 3)
    U.say(f"combined bwd tucker {prec}")
    _, npdt, oprec = U.prec_codes(prec)
    rng = np.random.default_rng(77)
    x = (rng.standard_normal((Bt, ci) + n)).astype(npdt)
    gy = (rng.standard_normal((Bt, co) + n)).astype(npdt)
    kd = (2 * modes[0], modes[1])
    core = (rng.standard_normal(rank + (2,)) * 0.3).astype(npdt)
    u_in = (rng.standard_normal((ci, rank[0], 2)) * 0.4).astype(npdt)
    u_out = (rng.standard_normal((co, rank[1], 2)) * 0.4).astype(npdt)
    u_mode = [(rng.standard_normal((kd[j], rank[2 + j], 2)) * 0.4).astype(npdt)
              for j in range(2)]
    layer = U.make_layer(n, modes, Bt, ci, co, prec, tucker_rank=rank)
    wd = {"core": U.dev(core), "u_in": U.dev(u_in), "u_out": U.dev(u_out),
          "u_mode": [U.dev(u) for u in u_mode]}
    xd, gyd = U.dev(x), U.dev(gy)
    gx, gw = layer.bwd(xd, wd, gyd)
    gx_sep = layer.bwd_data(xd, wd, gyd)
    gw_sep = layer.bwd_weight(xd, gyd, wd)
    torch.cuda.synchronize()
    assert np.array_equal(U.host(gx), U.host(gx_sep))
    for k in ("core", "u_in", "u_out"):
        assert np.array_equal(U.host(gw[k]), U.host(gw_sep[k]))
    for a, b in zip(gw["u_mode"], gw_sep["u_mode"]):
        assert np.array_equal(U.host(a), U.host(b))


# ---------------------------------------------------------------------------
# CP-factorised weights (Sec. 4.6)
# ---------------------------------------------------------------------------

def _cp_check(w, x, gy, n, modes, y, gx, gw, prec, oprec, policy):
    lam, u_in, u_out = U.cplx(w["core"]), U.cplx(w["u_in"]), U.cplx(w["u_out"])
    u_mode = [U.cplx(u) for u in w["u_mode"]]
    _assert_close("y", y, O.cp_fwd(x, lam, u_in, u_out, u_mode, n, modes, oprec, policy), prec)
    _assert_close("gx", gx, O.cp_bwd_data(x, lam, u_in, u_out, u_mode, gy, n, modes, oprec,
                                          policy), prec)
    g_lam, g_in, g_out, g_mode = O.cp_bwd_weight(x, gy, lam, u_in, u_out, u_mode, n, modes,
                                                 oprec)
    gwc = U.gw_complex(gw)
    _assert_close("g_lambda", gwc["core"], g_lam, prec)
    _assert_close("g_u_in", gwc["u_in"], g_in, prec)
    _assert_close("g_u_out", gwc["u_out"], g_out, prec)
    for j in range(len(n)):
        _assert_close(f"g_u_mode{j}", gwc["u_mode"][j], g_mode[j], prec)


CP_EDGE = [
    # (n, modes, B, Cin, Cout, R)
    ((8, 8), (2, 3), 2, 3, 4, 3),
    ((6, 10, 12), (2, 3, 4), 2, 3, 2, 5),
    ((40,), (7,), 3, 2, 5, 4),
    ((32, 48), (5, 9), 3, 7, 6, 1),      # rank one
    ((64, 64), (16, 16), 4, 32, 32, 24),  # chained-transform shapes, K % 32 == 0
]


@pytest.mark.parametrize("policy", ["min_result", "min_net"])
@pytest.mark.parametrize("prec", PRECS)
@pytest.mark.parametrize("case", range(len(CP_EDGE)))
def test_cp_edge_cases(case, prec, policy):
    n, modes, Bt, ci, co, r = CP_EDGE[case]
    _, npdt, oprec = U.prec_codes(prec)
    U.say(f"cp edge {case}: n={n} modes={modes} B={Bt} C={ci}->{co} R={r} {prec} {policy}")
    rng = np.random.default_rng(np.random.SeedSequence([3000 + case]))
    d = len(n)
    kd = tuple(2 * m if j < d - 1 else m for j, m in enumerate(modes))

    def cpx(shape, std):
        return (rng.standard_normal(tuple(shape) + (2,)) * std).astype(npdt)

    w = {"core": cpx((r,), 0.5), "u_in": cpx((ci, r), 0.5), "u_out": cpx((co, r), 0.5),
         "u_mode": [cpx((kd[j], r), 0.5) for j in range(d)]}
    x = rng.standard_normal((Bt, ci) + n).astype(npdt)
    gy = rng.standard_normal((Bt, co) + n).astype(npdt)
    pol = 0 if policy == "min_result" else 1
    layer = U.make_layer(n, modes, Bt, ci, co, prec, policy=pol, cp_rank=r)
    y, gx, gw = U.run_all(layer, x, w, gy)
    _cp_check(w, x, gy, n, modes, y, gx, gw, prec, oprec, policy)
    if case == 0:
        # bwd_weight recomputing both spectra (no caches) gives the same grads
        _, _, gw2 = U.run_all(layer, x, w, gy, caches=False)
        for k in ("core", "u_in", "u_out"):
            assert np.array_equal(gw[k], gw2[k]), k


@pytest.mark.parametrize("policy", ["min_result", "min_net"])
@pytest.mark.parametrize("prec", PRECS)
def test_workload_cp(prec, policy):
    """CP workload at full size: y and gx of the first and the last batch
    sample; lambda and factor gradients from all samples."""
    wid = 6
    wl = synth.WORKLOADS[wid]
    _, _, oprec = U.prec_codes(prec)
    U.say(f"workload {wid} {wl.name} {prec} {policy}")
    x, w, gy = _workload_inputs(wid, prec)
    pol = 0 if policy == "min_result" else 1
    layer = U.make_layer(wl.n, wl.modes, wl.batch, wl.c_in, wl.c_out, prec, policy=pol,
                         cp_rank=wl.rank[0])
    y, gx, gw = U.run_all(layer, x, w, gy)
    lam, u_in, u_out = U.cplx(w["core"]), U.cplx(w["u_in"]), U.cplx(w["u_out"])
    u_mode = [U.cplx(u) for u in w["u_mode"]]
    for b in (0, wl.batch - 1):
        ry = O.cp_fwd(x[b:b + 1], lam, u_in, u_out, u_mode, wl.n, wl.modes, oprec, policy)
        _assert_close(f"y[b={b}]", y[b:b + 1], ry, prec)
        rgx = O.cp_bwd_data(x[b:b + 1], lam, u_in, u_out, u_mode, gy[b:b + 1], wl.n,
                            wl.modes, oprec, policy)
        _assert_close(f"gx[b={b}]", gx[b:b + 1], rgx, prec)
    g_lam, g_in, g_out, g_mode = O.cp_bwd_weight(x, gy, lam, u_in, u_out, u_mode, wl.n,
                                                 wl.modes, oprec)
    gwc = U.gw_complex(gw)
    _assert_close("g_lambda", gwc["core"], g_lam, prec)
    _assert_close("g_u_in", gwc["u_in"], g_in, prec)
    _assert_close("g_u_out", gwc["u_out"], g_out, prec)
    for j in range(wl.ndim):
        _assert_close(f"g_u_mode{j}", gwc["u_mode"][j], g_mode[j], prec)


@pytest.mark.parametrize("prec", PRECS)
def test_combined_bwd_cp(prec):
    """fno_spectral_conv_bwd with CP weights equals the two separate calls."""
    n, modes, Bt, ci, co, r = (32, 32), (4, 5), 2, 6, 5, 7
    U.say(f"combined bwd cp {prec}")
    _, npdt, oprec = U.prec_codes(prec)
    rng = np.random.default_rng(78)
    x = (rng.standard_normal((Bt, ci) + n)).astype(npdt)
    gy = (rng.standard_normal((Bt, co) + n)).astype(npdt)
    kd = (2 * modes[0], modes[1])
    w = {"core": (rng.standard_normal((r, 2)) * 0.3).astype(npdt),
         "u_in": (rng.standard_normal((ci, r, 2)) * 0.4).astype(npdt),
         "u_out": (rng.standard_normal((co, r, 2)) * 0.4).astype(npdt),
         "u_mode": [(rng.standard_normal((kd[j], r, 2)) * 0.4).astype(npdt) for j in range(2)]}
    layer = U.make_layer(n, modes, Bt, ci, co, prec, cp_rank=r)
    wd = {"core": U.dev(w["core"]), "u_in": U.dev(w["u_in"]), "u_out": U.dev(w["u_out"]),
          "u_mode": [U.dev(u) for u in w["u_mode"]]}
    xd, gyd = U.dev(x), U.dev(gy)
    gx, gw = layer.bwd(xd, wd, gyd)
    gx_sep = layer.bwd_data(xd, wd, gyd)
    gw_sep = layer.bwd_weight(xd, gyd, wd)
    torch.cuda.synchronize()
    assert np.array_equal(U.host(gx), U.host(gx_sep))
    for k in ("core", "u_in", "u_out"):
        assert np.array_equal(U.host(gw[k]), U.host(gw_sep[k]))
    for a, b in zip(gw["u_mode"], gw_sep["u_mode"]):
        assert np.array_equal(U.host(a), U.host(b))
