"""The layer's calls captured in a HIP graph (through torch.cuda.graph) and
replayed: every replay must reproduce the eager calls bit for bit on the same
inputs, with eager work of the same layer and device synchronisations between
the replays, and the inputs changed before each replay (the graph reads the
live buffers).  The last replay is also checked against the float64 oracle.  Dense weights
in both precisions; Tucker and CP weights (the pairwise steps) in fp16 with
both greedy policies.
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

from oracle import fno_oracle as O  # noqa: E402
import synth  # noqa: E402
from tests import gpu_util as U  # noqa: E402

# (n, modes, B, Cin, Cout): the fp16 case runs the chained transforms and the
# slab contractions, the fp32 case the generic kernels
CASES = {"fp16_tanh": ((64, 64), (16, 16), 4, 32, 32),
         "fp32": ((40, 48), (6, 9), 3, 5, 7)}


@pytest.mark.parametrize("prec", ["fp16_tanh", "fp32"])
def test_graph_replay_matches_eager(prec):
    n, modes, Bt, ci, co = CASES[prec]
    _, npdt, oprec = U.prec_codes(prec)
    U.say(f"graph replay {prec}: n={n} modes={modes} B={Bt} C={ci}->{co}")
    layer = U.make_layer(n, modes, Bt, ci, co, prec)
    x0, w0, gy0 = synth.random_dense_case(40, Bt, ci, co, n, modes, npdt)
    xs, ws, gys = U.dev(x0), U.dev(w0), U.dev(gy0)           # the graph's inputs
    xh, gh = layer.spectrum_buffer(0), layer.spectrum_buffer(1)
    y = torch.empty((Bt, co) + n, dtype=layer.dtype, device="cuda")
    gx = torch.empty((Bt, ci) + n, dtype=layer.dtype, device="cuda")
    gw = layer.alloc_grads()

    def step(stream=None):
        layer.fwd(xs, ws, y=y, x_hat=xh, stream=stream)
        layer.bwd(xs, ws, gys, x_hat=xh, gx=gx, gw=gw, stream=stream)

    step()  # plans, tables and workspaces exist before the capture
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    torch.cuda.synchronize()

    for r in range(3):
        x, w, gyv = synth.random_dense_case(41 + r, Bt, ci, co, n, modes, npdt)
        xs.copy_(U.dev(x))
        ws.copy_(U.dev(w))
        gys.copy_(U.dev(gyv))
        torch.cuda.synchronize()
        U.say(f"  replay {r}")
        g.replay()
        torch.cuda.synchronize()
        got = [U.host(t).copy() for t in (y, gx, gw)]
        # eager calls of the same layer on the same inputs (separate outputs)
        xd, wd, gd = U.dev(x), U.dev(w), U.dev(gyv)
        xh_e, gh_e = layer.spectrum_buffer(0), layer.spectrum_buffer(1)
        ye = layer.fwd(xd, wd, x_hat=xh_e)
        gxe, gwe = layer.bwd(xd, wd, gd, x_hat=xh_e)
        torch.cuda.synchronize()
        ref = [U.host(t) for t in (ye, gxe, gwe)]
        for name, a, b in zip(("y", "gx", "gw"), got, ref):
            assert a.shape == b.shape
            assert np.array_equal(a.view(np.uint8), b.view(np.uint8)), f"replay {r}: {name}"
    # the last replay against the oracle
    wc = U.cplx(w)
    oy = O.fwd(x, wc, n, modes, oprec)
    ogx = O.bwd_data(x, wc, gyv, n, modes, oprec)
    ogw = O.bwd_weight(x, gyv, n, modes, oprec)
    for name, a, b in zip(("y", "gx", "gw"), got, (oy, ogx, ogw)):
        if name == "gw":
            a = U.cplx(a)
        r_ = U.rel(a, b)
        U.say(f"  {name}: rel_l2 = {r_:.3e}")
        assert r_ <= U.TOL[prec], name


# Factorised weights: the pairwise steps (GEMM tiles with split-K partial
# sums, the generic kernels) replayed from a graph.  (n, modes, B, Cin, Cout,
# ranks): Tucker ranks (r_in, r_out, r_1, r_2), CP rank (R,).
FACTOR_CASES = {"tucker": ((32, 32), (8, 8), 4, 32, 24, (8, 6, 4, 4)),
                "cp": ((32, 32), (8, 8), 4, 32, 24, (12,))}


def _factor_weights(rng, kind, ci, co, kd, rank, npdt):
    def cp(shape, std):
        return (rng.standard_normal(tuple(shape) + (2,)) * std).astype(npdt)
    if kind == "tucker":
        return {"core": cp(rank, 0.5), "u_in": cp((ci, rank[0]), 0.5),
                "u_out": cp((co, rank[1]), 0.5),
                "u_mode": [cp((kd[j], rank[2 + j]), 0.5) for j in range(len(kd))]}
    r = rank[0]
    return {"core": cp((r,), 0.5), "u_in": cp((ci, r), 0.5), "u_out": cp((co, r), 0.5),
            "u_mode": [cp((kd[j], r), 0.5) for j in range(len(kd))]}


def _flat(t):
    if isinstance(t, dict):
        return [t["core"], t["u_in"], t["u_out"]] + list(t["u_mode"])
    return [t]


@pytest.mark.parametrize("separate", [False, True])
@pytest.mark.parametrize("policy", [0, 1])
@pytest.mark.parametrize("kind", ["tucker", "cp"])
def test_graph_replay_factorized(kind, policy, separate):
    """separate: the backward as bwd_data (keeping the gradient spectrum) and
    bwd_weight from the two spectra, instead of the combined call."""
    n, modes, Bt, ci, co, rank = FACTOR_CASES[kind]
    prec = "fp16_tanh"
    _, npdt, oprec = U.prec_codes(prec)
    U.say(f"graph replay {kind} policy {policy}: n={n} modes={modes} B={Bt} C={ci}->{co} "
          f"rank={rank} separate={separate}")
    kd = tuple(2 * m if j < len(n) - 1 else m for j, m in enumerate(modes))
    if kind == "tucker":
        layer = U.make_layer(n, modes, Bt, ci, co, prec, rank, policy)
    else:
        layer = U.make_layer(n, modes, Bt, ci, co, prec, policy=policy, cp_rank=rank[0])
    rng = np.random.default_rng(np.random.SeedSequence([3100, policy]))
    x0 = rng.standard_normal((Bt, ci) + n).astype(npdt)
    gy0 = rng.standard_normal((Bt, co) + n).astype(npdt)
    w0 = _factor_weights(rng, kind, ci, co, kd, rank, npdt)
    xs, gys = U.dev(x0), U.dev(gy0)
    ws = {"core": U.dev(w0["core"]), "u_in": U.dev(w0["u_in"]), "u_out": U.dev(w0["u_out"]),
          "u_mode": [U.dev(u) for u in w0["u_mode"]]}
    xh = layer.spectrum_buffer(0)
    y = torch.empty((Bt, co) + n, dtype=layer.dtype, device="cuda")
    gx = torch.empty((Bt, ci) + n, dtype=layer.dtype, device="cuda")
    gw = layer.alloc_grads()

    gh = layer.spectrum_buffer(1)

    def backward(x_, w_, gy_, xh_, gx_=None, gw_=None, gh_=None, stream=None):
        if not separate:
            return layer.bwd(x_, w_, gy_, x_hat=xh_, gx=gx_, gw=gw_, stream=stream)
        gh_ = layer.spectrum_buffer(1) if gh_ is None else gh_
        gx_ = layer.bwd_data(x_, w_, gy_, gx=gx_, gy_hat=gh_, stream=stream)
        gw_ = layer.bwd_weight(None, None, w_, x_hat=xh_, gy_hat=gh_, gw=gw_, stream=stream)
        return gx_, gw_

    def step(stream=None):
        layer.fwd(xs, ws, y=y, x_hat=xh, stream=stream)
        backward(xs, ws, gys, xh, gx_=gx, gw_=gw, gh_=gh, stream=stream)

    step()  # plans, tables and workspaces exist before the capture
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    torch.cuda.synchronize()

    for r in range(3):
        x = rng.standard_normal((Bt, ci) + n).astype(npdt)
        gyv = rng.standard_normal((Bt, co) + n).astype(npdt)
        w = _factor_weights(rng, kind, ci, co, kd, rank, npdt)
        xs.copy_(U.dev(x))
        gys.copy_(U.dev(gyv))
        for dst, src in zip(_flat(ws), _flat(w)):
            dst.copy_(U.dev(src))
        torch.cuda.synchronize()
        U.say(f"  replay {r}")
        g.replay()
        torch.cuda.synchronize()
        got = [U.host(t).copy() for t in [y, gx] + _flat(gw)]
        # eager calls of the same layer on the same inputs (separate outputs)
        xd, gd = U.dev(x), U.dev(gyv)
        wd = {"core": U.dev(w["core"]), "u_in": U.dev(w["u_in"]), "u_out": U.dev(w["u_out"]),
              "u_mode": [U.dev(u) for u in w["u_mode"]]}
        xh_e = layer.spectrum_buffer(0)
        ye = layer.fwd(xd, wd, x_hat=xh_e)
        gxe, gwe = backward(xd, wd, gd, xh_e)
        torch.cuda.synchronize()
        ref = [U.host(t) for t in [ye, gxe] + _flat(gwe)]
        assert len(got) == len(ref)
        for k, (a, b) in enumerate(zip(got, ref)):
            assert a.shape == b.shape
            assert np.array_equal(a.view(np.uint8), b.view(np.uint8)), f"replay {r}: output {k}"
    # the last replay's y and gx against the oracle
    core, u_in, u_out = U.cplx(w["core"]), U.cplx(w["u_in"]), U.cplx(w["u_out"])
    u_mode = [U.cplx(u) for u in w["u_mode"]]
    pol = "min_result" if policy == 0 else "min_net"
    if kind == "tucker":
        oy = O.tucker_fwd(x, core, u_in, u_out, u_mode, n, modes, oprec, pol)
        ogx = O.tucker_bwd_data(x, core, u_in, u_out, u_mode, gyv, n, modes, oprec, pol)
    else:
        oy = O.cp_fwd(x, core, u_in, u_out, u_mode, n, modes, oprec, pol)
        ogx = O.cp_bwd_data(x, core, u_in, u_out, u_mode, gyv, n, modes, oprec, pol)
    for name, a, b in zip(("y", "gx"), got[:2], (oy, ogx)):
        r_ = U.rel(a, b)
        U.say(f"  {name}: rel_l2 = {r_:.3e}")
        assert r_ <= U.TOL[prec], name
