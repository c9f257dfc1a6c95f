"""The layer's calls captured in a HIP graph (through torch.cuda.graph) and
replayed: every replay must reproduce the eager calls bit for bit on the same
inputs, with eager work of the same layer and device synchronisations between
the replays, and the inputs changed before each replay (the graph reads the
live buffers).  The last replay is also checked against the float64 oracle.
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
