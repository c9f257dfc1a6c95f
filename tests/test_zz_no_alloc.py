"""The allocation-free forward call (fno_spectral_conv_fwd_noalloc) through
the C ABI against the ordinary forward call on the same inputs: bit-identical
outputs and spectral caches, on two allocation-free calls in a row (the
second on a smaller layer, so it runs on what the first left in the shared
scratch), and host-side rejections that enqueue nothing."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

import synth  # noqa: E402
from tests import gpu_util as U  # noqa: E402


def _setup(wid, batch=None):
    """Inputs on the GPU, the layer, and the ordinary forward call's results
    (which also builds the descriptor's plan)."""
    from paper_2307_15034_amd.layer import SpectralConv
    from paper_2307_15034_amd import binding as B
    wl = synth.WORKLOADS[wid]
    Bt = wl.batch if batch is None else batch
    x = synth.make_x(wl, np.float16, Bt)
    w = synth.make_dense_weight(wl, np.float16)
    layer = SpectralConv(wl.n, wl.modes, Bt, wl.c_in, wl.c_out, B.FNO_PREC_FP16_TANH)
    xd, wd = U.dev(x), U.dev(w)
    xh = layer.spectrum_buffer(0)
    U.say(f"  ordinary fwd: {wl.name} B={Bt}")
    y = layer.fwd(xd, wd, x_hat=xh)
    torch.cuda.synchronize()
    return layer, xd, wd, U.host(y), U.host(xh)


def _noalloc(layer, xd, wd):
    from paper_2307_15034_amd import binding as B
    y = torch.full((layer.batch, layer.c_out) + layer.n, 7.0, dtype=layer.dtype, device="cuda")
    xh = layer.spectrum_buffer(0)
    xh.fill_(0xAB)
    s = torch.cuda.current_stream().cuda_stream
    U.say(f"  fwd_noalloc: n={layer.n} B={layer.batch} C={layer.c_in}->{layer.c_out}")
    B.fno_spectral_conv_fwd_noalloc(layer.desc, xd.data_ptr(), layer.weights_struct(wd),
                                    y.data_ptr(), xh.data_ptr(), s)
    return y, xh


def test_noalloc_matches_fwd_two_calls():
    big = _setup(2)          # 128 x 128, B = 32, C = 64: 33.6 MB of scratch
    small = _setup(1)        # 64 x 64, B = 2, C = 16
    yb, xhb = _noalloc(*big[:3])
    ys, xhs = _noalloc(*small[:3])
    torch.cuda.synchronize()
    for name, (got_y, got_xh), ref in [("128^2", (yb, xhb), big), ("64^2", (ys, xhs), small)]:
        y_ref, xh_ref = ref[3], ref[4]
        U.say(f"  {name}: comparing y and the spectrum cache bit for bit")
        assert np.array_equal(U.host(got_y).view(np.uint16), y_ref.view(np.uint16)), name
        assert np.array_equal(U.host(got_xh), xh_ref), name


def test_noalloc_rejections_enqueue_nothing():
    from paper_2307_15034_amd import binding as B
    from paper_2307_15034_amd.layer import SpectralConv
    # a descriptor with no plan on this device yet
    layer = SpectralConv((32, 48), (5, 7), 3, 4, 6, B.FNO_PREC_FP16_TANH)
    x = torch.zeros((3, 4, 32, 48), dtype=torch.float16, device="cuda")
    w = torch.zeros((4, 6, 10, 7, 2), dtype=torch.float16, device="cuda")
    y = torch.full((3, 6, 32, 48), 5.0, dtype=torch.float16, device="cuda")
    s = torch.cuda.current_stream().cuda_stream
    st = B.fno_spectral_conv_fwd_noalloc(layer.desc, x.data_ptr(), layer.weights_struct(w),
                                         y.data_ptr(), 0, s, check=False)
    assert st == B.FNO_ERR_INVALID_ARGUMENT
    # a forward workspace beyond the scratch: two 33.6 MB spectra
    big = SpectralConv((16, 16), (8, 8), 1024, 64, 64, B.FNO_PREC_FP16_TANH)
    need = B.fno_spectral_conv_workspace_size(big.desc, B.FNO_OP_FWD)
    assert need > B.FNO_NOALLOC_SCRATCH_BYTES
    xb = torch.zeros((1024, 64, 16, 16), dtype=torch.float16, device="cuda")
    wb = torch.zeros((64, 64, 16, 8, 2), dtype=torch.float16, device="cuda")
    yb = big.fwd(xb, wb)                     # the plan exists from here on
    yb.fill_(3.0)
    st = B.fno_spectral_conv_fwd_noalloc(big.desc, xb.data_ptr(), big.weights_struct(wb),
                                         yb.data_ptr(), 0, s, check=False)
    assert st == B.FNO_ERR_WORKSPACE_TOO_SMALL
    torch.cuda.synchronize()
    assert bool((y == 5.0).all()) and bool((yb == 3.0).all())
