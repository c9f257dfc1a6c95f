"""Shared helpers of the GPU parity tests: seeded inputs, the HIP path through
the C ABI, and the float64 oracle on the same stored values."""
from __future__ import annotations

import sys

import numpy as np
import torch

from oracle import fno_oracle as O
import synth

class _Tol(dict):
    """Relative L2 tolerance of a mode: 1e-5 for fp32 storage, 3e-3 for fp16."""

    def __missing__(self, prec):
        return 1e-5 if prec.startswith("fp32") else 3e-3


TOL = _Tol({"fp32": 1e-5, "fp16_tanh": 3e-3})


def say(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def prec_codes(prec: str):
    """(library precision code, numpy storage dtype, oracle mode) of a mode
    name: "fp32", "fp16_tanh", "fp32_tanh", "fp16", "fp16_clip:<c>" /
    "fp32_clip:<c>" or "fp16_sigma:<k>" / "fp32_sigma:<k>" (the oracle's mode
    strings)."""
    from paper_2307_15034_amd import binding as B
    O.preact_kind(prec)  # rejects unknown names
    if prec.startswith("fp32"):
        return B.FNO_PREC_FP32, np.float32, prec
    return B.FNO_PREC_FP16_TANH, np.float16, prec


def preact_codes(prec: str):
    """(library pre-activation code, clip bound) of a mode name."""
    from paper_2307_15034_amd import binding as B
    kind, c = O.preact_kind(prec)
    if prec in ("fp32", "fp16_tanh"):
        return B.FNO_PREACT_DEFAULT, 0.0
    if kind == "clip":
        return B.FNO_PREACT_HARD_CLIP, float(c)
    if kind == "sigma":
        return B.FNO_PREACT_SIGMA_CLIP, float(c)
    return (B.FNO_PREACT_TANH if kind == "tanh" else B.FNO_PREACT_NONE), 0.0


def dev(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a)).to("cuda")


def host(t: torch.Tensor) -> np.ndarray:
    return t.detach().to("cpu").numpy()


def cplx(pairs: np.ndarray) -> np.ndarray:
    return synth.pairs_to_complex(pairs)


def make_layer(n, modes, batch, c_in, c_out, prec, tucker_rank=None, policy=0, cp_rank=None):
    from paper_2307_15034_amd import binding as B
    from paper_2307_15034_amd.layer import SpectralConv
    pc, _, _ = prec_codes(prec)
    pa, clip = preact_codes(prec)
    if cp_rank is not None:
        return SpectralConv(n, modes, batch, c_in, c_out, pc, B.FNO_WEIGHT_CP, (cp_rank,),
                            policy, preact=pa, clip=clip)
    kind = B.FNO_WEIGHT_TUCKER if tucker_rank is not None else B.FNO_WEIGHT_DENSE
    return SpectralConv(n, modes, batch, c_in, c_out, pc, kind, tucker_rank, policy,
                        preact=pa, clip=clip)


def run_all(layer, x, w, gy, caches=True):
    """fwd, bwd_data and bwd_weight on the GPU; returns host arrays."""
    xd, gyd = dev(x), dev(gy)
    if isinstance(w, dict):
        wd = {"core": dev(w["core"]), "u_in": dev(w["u_in"]), "u_out": dev(w["u_out"]),
              "u_mode": [dev(u) for u in w["u_mode"]]}
    else:
        wd = dev(w)
    xh = layer.spectrum_buffer(0) if caches else None
    gh = layer.spectrum_buffer(1) if caches else None
    say(f"  launch fwd n={layer.n} modes={layer.modes} B={layer.batch} "
        f"C={layer.c_in}->{layer.c_out} caches={caches}")
    y = layer.fwd(xd, wd, x_hat=xh)
    say("  launch bwd_data")
    gx = layer.bwd_data(xd, wd, gyd, gy_hat=gh)
    say("  launch bwd_weight")
    if caches:
        gw = layer.bwd_weight(None, None, wd, x_hat=xh, gy_hat=gh)
    else:
        gw = layer.bwd_weight(xd, gyd, wd)
    torch.cuda.synchronize()
    say("  done")
    if isinstance(gw, dict):
        gwh = {"core": host(gw["core"]), "u_in": host(gw["u_in"]),
               "u_out": host(gw["u_out"]), "u_mode": [host(u) for u in gw["u_mode"]]}
    else:
        gwh = host(gw)
    return host(y), host(gx), gwh


def rel(a, b) -> float:
    return O.rel_l2(a, b)


def nonfinite_report(got, ref, nlead: int = 2, show: int = 8) -> str:
    """Where the non-finite values of got and of ref are: their counts and
    the first few (leading-index plane, position) of each."""
    out = []
    for name, arr in (("got", np.asarray(got)), ("ref", np.asarray(ref))):
        bad = ~np.isfinite(arr)
        idx = np.argwhere(bad)[:show]
        planes = sorted({tuple(int(v) for v in i[:nlead]) for i in np.argwhere(bad)})
        out.append(f"{name}: {int(bad.sum())} non-finite in planes {planes[:show]}"
                   f"{' ...' if len(planes) > show else ''} first {idx.tolist()}")
    return "; ".join(out)


def gw_complex(gw):
    if isinstance(gw, dict):
        return {"core": cplx(gw["core"]), "u_in": cplx(gw["u_in"]),
                "u_out": cplx(gw["u_out"]), "u_mode": [cplx(u) for u in gw["u_mode"]]}
    return cplx(gw)
