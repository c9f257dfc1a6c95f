"""GPU parity of the FNO block epilogue (the rest of the block after the
spectral convolution, Sec. 2: 1x1 skip with bias, GELU, residual) and of the
whole block (spectral convolution + epilogue) against the float64 oracle,
through the C ABI.

Tolerances (relative L2, whole tensor and worst (batch, channel) plane): 1e-5
in fp32 mode, 3e-3 in fp16 mode.  The parameter gradients are compared whole.
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

from oracle import fno_oracle as O  # noqa: E402
import synth  # noqa: E402
from tests import gpu_util as U  # noqa: E402
from paper_2307_15034_amd import binding as B  # noqa: E402
from paper_2307_15034_amd.layer import BlockEpilogue  # noqa: E402

ACTS = {"gelu": (B.FNO_EPI_ACT_GELU, O.EPI_ACT_GELU), "none": (B.FNO_EPI_ACT_NONE, O.EPI_ACT_NONE)}


def _close(name, got, ref, prec, planes=True):
    r = U.rel(got, ref)
    rp = O.max_plane_rel_l2(got, ref) if planes and np.ndim(ref) >= 3 else None
    extra = f", max per plane {rp:.3e}" if rp is not None else ""
    U.say(f"  {name}: rel_l2 = {r:.3e}{extra} (tol {U.TOL[prec]:.0e})")
    if not np.isfinite(r):
        U.say("  " + U.nonfinite_report(got, ref))
    assert np.isfinite(r) and r <= U.TOL[prec], f"{name}: {r:.3e}"
    if rp is not None:
        assert np.isfinite(rp) and rp <= U.TOL[prec], f"{name} (worst plane): {rp:.3e}"


def _epi(grid, bt, ci, co, prec, act, residual):
    pc, npdt, _ = U.prec_codes(prec)
    return BlockEpilogue(grid, bt, ci, co, pc, ACTS[act][0], residual), npdt


EPI_CASES = [
    # (grid, B, Cin, Cout, act, residual, bias)
    ((20, 24), 3, 5, 7, "gelu", False, True),      # ragged channels, matrix-core path
    ((15, 17), 2, 6, 6, "gelu", True, True),       # 255 points: generic kernels
    ((96,), 4, 16, 16, "none", True, False),        # 1-D, no activation, no bias
    ((6, 10, 12), 2, 3, 2, "gelu", False, True),   # 3-D
    ((32, 32), 3, 33, 18, "gelu", False, True),    # channel tiles past 32 / 16
    ((16, 16), 2, 130, 20, "gelu", False, True),   # 130 input channels: generic mix and sums
    ((16, 16), 2, 20, 200, "gelu", False, True),   # 200 output channels (13 tiles)
    ((8, 16), 2, 64, 300, "none", False, True),    # 300 output channels: generic sums
    ((64, 64), 2, 64, 64, "gelu", True, True),     # the workloads' channel count
    ((40, 40), 3, 128, 128, "gelu", True, True),   # 128 channels, ragged last tile
    ((1000,), 1, 24, 40, "gelu", False, True),     # several tiles, partial sums past one wave
]


@pytest.mark.parametrize("prec", ["fp32", "fp16_tanh"])
@pytest.mark.parametrize("case", range(len(EPI_CASES)))
def test_epilogue_edge_cases(case, prec):
    grid, bt, ci, co, act, res, bias = EPI_CASES[case]
    U.say(f"epilogue case {case}: grid={grid} B={bt} {ci}->{co} {act} residual={res} "
          f"bias={bias} {prec}")
    epi, npdt = _epi(grid, bt, ci, co, prec, act, res)
    x, y, w, b, g = synth.random_block_case(case, bt, ci, co, grid, npdt)
    if not bias:
        b = None
    # the spectral input gradient, standing in for the spectral backward
    gxs = synth.random_block_case(100 + case, bt, ci, ci, grid, npdt)[0]
    xd, yd, wd, gd, gxsd = U.dev(x), U.dev(y), U.dev(w), U.dev(g), U.dev(gxs)
    bd = U.dev(b) if b is not None else None
    out, z = epi.fwd(xd, yd, wd, bd)
    gz, gw, gb = epi.bwd_weight(xd, z, gd, bias=bias)
    gx = epi.bwd_data(gz, wd, gxsd, gd if res else None)
    torch.cuda.synchronize()
    oact = ACTS[act][1]
    r_out, r_z = O.block_epilogue_fwd(x, y, w, b, oact, res)
    r_gz, r_gx, r_gw, r_gb = O.block_epilogue_bwd(x, r_z, g, w, oact, res)
    _close("out", U.host(out), r_out, prec)
    if z is not None:
        _close("z", U.host(z), r_z, prec)
    _close("g_z", U.host(gz), r_gz, prec)
    _close("gx", U.host(gx), r_gx + gxs.astype(np.float64), prec)
    _close("g_w_skip", U.host(gw), r_gw, prec, planes=False)
    if bias:
        _close("g_b", U.host(gb), r_gb, prec, planes=False)


def test_epilogue_deterministic_and_in_place():
    """Bit-identical reruns (the parameter gradients are summed in a fixed
    order), and bwd_data in place on gx_spec gives the out-of-place result."""
    grid, bt, ci, co = (64, 64), 4, 64, 64
    epi, npdt = _epi(grid, bt, ci, co, "fp16_tanh", "gelu", True)
    x, y, w, b, g = synth.random_block_case(40, bt, ci, co, grid, npdt)
    xd, yd, wd, bd, gd = U.dev(x), U.dev(y), U.dev(w), U.dev(b), U.dev(g)
    res = []
    for _ in range(2):
        out, z = epi.fwd(xd, yd, wd, bd)
        gz, gw, gb = epi.bwd_weight(xd, z, gd)
        res.append([U.host(t) for t in (out, z, gz, gw, gb)])
    for a, c in zip(*res):
        assert np.array_equal(a, c)
    gxs = U.dev(synth.random_block_case(41, bt, ci, ci, grid, npdt)[0])
    gx = U.host(epi.bwd_data(gz, wd, gxs, gd))
    epi.bwd_data(gz, wd, gxs, gd, gx=gxs)
    assert np.array_equal(U.host(gxs), gx)


def test_epilogue_rejections_enqueue_nothing():
    """Malformed calls are refused on the host: aliasing outputs, a missing
    z or g_z with GELU, a short workspace."""
    epi, npdt = _epi((16, 16), 2, 8, 8, "fp16_tanh", "gelu", True)
    x, y, w, b, g = (U.dev(a) for a in synth.random_block_case(7, 2, 8, 8, (16, 16), npdt))
    d = epi.desc
    st = B.fno_block_epilogue_fwd(d, x.data_ptr(), y.data_ptr(), w.data_ptr(), 0, x.data_ptr(),
                                  0, 0, check=False)
    assert st == B.FNO_ERR_INVALID_ARGUMENT
    ws = torch.empty(epi.ws_bytes, dtype=torch.uint8, device="cuda")
    gw = torch.empty((8, 8), dtype=torch.float32, device="cuda")
    st = B.fno_block_epilogue_bwd_weight(d, x.data_ptr(), 0, g.data_ptr(), y.data_ptr(),
                                         gw.data_ptr(), 0, ws.data_ptr(), epi.ws_bytes, 0,
                                         check=False)
    assert st == B.FNO_ERR_INVALID_ARGUMENT
    st = B.fno_block_epilogue_bwd_weight(d, x.data_ptr(), y.data_ptr(), g.data_ptr(),
                                         b.data_ptr(), gw.data_ptr(), 0, ws.data_ptr(),
                                         epi.ws_bytes - 256, 0, check=False)
    assert st == B.FNO_ERR_WORKSPACE_TOO_SMALL
    with pytest.raises(ValueError):
        epi.fwd(x.float(), y, w)
    torch.cuda.synchronize()


def _block_run(wl, prec, act, residual, g_samples=None):
    """The whole block on the GPU: spectral forward into y, epilogue forward,
    epilogue parameter gradients, spectral backward at g_z, epilogue data
    gradient.  g_samples: batch samples whose output gradient is kept (the
    others get zero)."""
    pc, npdt, oprec = U.prec_codes(prec)
    x = synth.make_x(wl, npdt)
    g = synth.make_gy(wl, npdt)
    if g_samples is not None:
        keep = np.zeros(g.shape[0], dtype=bool)
        keep[list(g_samples)] = True
        g[~keep] = 0
    w = synth.make_weight(wl, npdt)
    ws, bs = synth.make_block_params(wl, npdt)
    bt = x.shape[0]
    layer = U.make_layer(wl.n, wl.modes, bt, wl.c_in, wl.c_out, prec)
    epi = BlockEpilogue(wl.n, bt, wl.c_in, wl.c_out, pc, ACTS[act][0], residual)
    xd, wd, gd, wsd, bsd = U.dev(x), U.dev(w), U.dev(g), U.dev(ws), U.dev(bs)
    xh = layer.spectrum_buffer(0)
    U.say(f"  block forward {wl.name} B={bt} {prec} {act} residual={residual}")
    y = layer.fwd(xd, wd, x_hat=xh)
    out, z = epi.fwd(xd, y, wsd, bsd)
    U.say("  block backward")
    gz, gws, gbs = epi.bwd_weight(xd, z, gd)
    gxs, gw = layer.bwd(xd, wd, gz, x_hat=xh)
    gx = epi.bwd_data(gz, wsd, gxs, gd if residual else None, gx=gxs)
    torch.cuda.synchronize()
    U.say("  done")
    return (x, w, ws, bs, g, oprec), (U.host(out), U.host(gx), U.host(gw), U.host(gws),
                                      U.host(gbs))


def _oracle_block(x, wc, ws, bs, g, wl, oprec, oact, residual, weight_grad=True):
    """The oracle's block, its pieces in order (one forward)."""
    r_out, r_z = O.block_fwd(x, wc, ws, bs, wl.n, wl.modes, oprec, oact, residual)
    r_gz, r_gxs, r_gws, r_gbs = O.block_epilogue_bwd(x, r_z, g, ws, oact, residual)
    r_gx = O.bwd_data(x, wc, r_gz, wl.n, wl.modes, oprec) + r_gxs
    r_gw = O.bwd_weight(x, r_gz, wl.n, wl.modes, oprec) if weight_grad else None
    return r_out, r_gx, r_gw, r_gws, r_gbs


@pytest.mark.parametrize("act,residual", [("gelu", True), ("none", False)])
def test_block_workload_128(act, residual):
    """The whole block on the 128^2 workload (B32, C64, 32x32 modes), fp16,
    every output against the oracle's block."""
    wl = synth.WORKLOADS[2]
    U.say(f"block workload {wl.name}")
    (x, w, ws, bs, g, oprec), (out, gx, gw, gws, gbs) = _block_run(wl, "fp16_tanh", act,
                                                                   residual)
    r_out, r_gx, r_gw, r_gws, r_gbs = _oracle_block(x, U.cplx(w), ws, bs, g, wl, oprec,
                                                    ACTS[act][1], residual)
    _close("out", out, r_out, "fp16_tanh")
    _close("gx", gx, r_gx, "fp16_tanh")
    _close("gW", U.cplx(gw), r_gw, "fp16_tanh")
    _close("g_w_skip", gws, r_gws, "fp16_tanh", planes=False)
    _close("g_b", gbs, r_gbs, "fp16_tanh", planes=False)


@pytest.mark.timeout(600)
def test_block_workload_1024_sampled():
    """The whole block on the 1024^2 workload (B8, C64, 64x64 modes), fp16,
    GELU and residual, in the benchmark's launch configuration.  Only the
    first and the last batch sample carry an output gradient: out and gx of
    those two against the oracle's block on each, the skip parameters'
    gradients against the oracle's sum over the two, and gx of every other
    sample exactly zero (its g_z is zero)."""
    wl = synth.WORKLOADS[3]
    last = wl.batch - 1
    U.say(f"block workload {wl.name}")
    (x, w, ws, bs, g, oprec), (out, gx, gw, gws, gbs) = _block_run(
        wl, "fp16_tanh", "gelu", True, g_samples=(0, last))
    wc = U.cplx(w)
    r_gws = np.zeros(gws.shape)
    r_gbs = np.zeros(gbs.shape)
    for s in (0, last):
        U.say(f"  oracle sample {s}")
        r_out, r_gx, _, gw_s, gb_s = _oracle_block(x[s:s + 1], wc, ws, bs, g[s:s + 1], wl,
                                                   oprec, O.EPI_ACT_GELU, True,
                                                   weight_grad=False)
        _close(f"out[{s}]", out[s:s + 1], r_out, "fp16_tanh")
        _close(f"gx[{s}]", gx[s:s + 1], r_gx, "fp16_tanh")
        r_gws += gw_s
        r_gbs += gb_s
    assert not np.any(gx[1:last])
    _close("g_w_skip", gws, r_gws, "fp16_tanh", planes=False)
    _close("g_b", gbs, r_gbs, "fp16_tanh", planes=False)
