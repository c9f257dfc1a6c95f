"""Torch-facing wrapper of the C ABI: allocates device buffers with PyTorch and
forwards raw device addresses and the current HIP stream to the library.

PyTorch supplies memory and streams only; every step of the layer runs in the
HIP kernels behind the three entry points.
"""
from __future__ import annotations

from typing import Dict, List, Optional, Sequence

import torch

from . import binding as B


def _addr(t: Optional[torch.Tensor]) -> int:
    if t is None:
        return 0
    if not t.is_cuda:
        raise ValueError("tensor must live on the GPU")
    if not t.is_contiguous():
        raise ValueError("tensor must be contiguous")
    return t.data_ptr()


class SpectralConv:
    """One FNO spectral-convolution layer bound to a descriptor.

    Weights are device tensors of interleaved (re, im) pairs:
      dense: [c_in, c_out, K_1..K_d, 2]
      tucker: core [r_in, r_out, r_1..r_d, 2], u_in [c_in, r_in, 2],
              u_out [c_out, r_out, 2], u_mode[j] [K_j, r_j, 2]
      cp (rank R): core = lambda [R, 2], u_in [c_in, R, 2], u_out [c_out, R, 2],
              u_mode[j] [K_j, R, 2]
    The storage dtype is float16 in fp16+tanh mode and float32 in fp32 mode;
    `preact` / `clip` choose the pre-activation (the precision's own by default).
    """

    def __init__(self, n: Sequence[int], modes: Sequence[int], batch: int, c_in: int,
                 c_out: int, precision: int = B.FNO_PREC_FP16_TANH,
                 weight_kind: int = B.FNO_WEIGHT_DENSE, rank: Optional[Sequence[int]] = None,
                 path_policy: int = B.FNO_PATH_MIN_RESULT, device: str = "cuda",
                 preact: int = B.FNO_PREACT_DEFAULT, clip: float = 0.0):
        self.n = tuple(int(v) for v in n)
        self.modes = tuple(int(v) for v in modes)
        self.batch, self.c_in, self.c_out = int(batch), int(c_in), int(c_out)
        self.precision = precision
        self.weight_kind = weight_kind
        self.rank = tuple(rank) if rank is not None else None
        self.desc = B.make_desc(self.n, self.modes, batch, c_in, c_out, precision,
                                weight_kind, rank, path_policy, preact, clip)
        self.dtype = torch.float16 if precision == B.FNO_PREC_FP16_TANH else torch.float32
        self.device = torch.device(device)
        d = len(self.n)
        self.kdims = tuple(2 * m if j < d - 1 else m for j, m in enumerate(self.modes))
        self._ws: Dict[str, torch.Tensor] = {}

    # -- buffers ---------------------------------------------------------------
    def workspace(self, op: int, caches: bool = True) -> torch.Tensor:
        key = f"{op}:{int(caches)}"
        if key not in self._ws:
            nbytes = B.fno_spectral_conv_workspace_size(self.desc, op, caches)
            self._ws[key] = torch.empty(nbytes, dtype=torch.uint8, device=self.device)
        return self._ws[key]

    def spectrum_buffer(self, which: int) -> torch.Tensor:
        nbytes = B.fno_spectrum_bytes(self.desc, which)
        return torch.empty(max(nbytes, 16), dtype=torch.uint8, device=self.device)

    def weights_struct(self, w) -> B.FnoWeights:
        if self.weight_kind == B.FNO_WEIGHT_DENSE:
            return B.weights_struct(dense=_addr(w))
        return B.weights_struct(core=_addr(w["core"]), u_in=_addr(w["u_in"]),
                                u_out=_addr(w["u_out"]),
                                u_mode=[_addr(u) for u in w["u_mode"]])

    def alloc_grads(self):
        f = dict(dtype=torch.float32, device=self.device)
        if self.weight_kind == B.FNO_WEIGHT_DENSE:
            return torch.empty((self.c_in, self.c_out) + self.kdims + (2,), **f)
        r = self.rank
        d = len(self.n)
        if self.weight_kind == B.FNO_WEIGHT_CP:
            # the lambda gradient travels in the "core" slot
            return {"core": torch.empty((r[0], 2), **f),
                    "u_in": torch.empty((self.c_in, r[0], 2), **f),
                    "u_out": torch.empty((self.c_out, r[0], 2), **f),
                    "u_mode": [torch.empty((k, r[0], 2), **f) for k in self.kdims]}
        return {"core": torch.empty(tuple(r[:2]) + tuple(r[2:2 + d]) + (2,), **f),
                "u_in": torch.empty((self.c_in, r[0], 2), **f),
                "u_out": torch.empty((self.c_out, r[1], 2), **f),
                "u_mode": [torch.empty((self.kdims[j], r[2 + j], 2), **f) for j in range(d)]}

    def grads_struct(self, g) -> B.FnoWeightGrads:
        if self.weight_kind == B.FNO_WEIGHT_DENSE:
            return B.grads_struct(dense=_addr(g))
        return B.grads_struct(core=_addr(g["core"]), u_in=_addr(g["u_in"]),
                              u_out=_addr(g["u_out"]), u_mode=[_addr(u) for u in g["u_mode"]])

    # -- the calls ---------------------------------------------------------------
    def fwd(self, x: torch.Tensor, w, y: Optional[torch.Tensor] = None,
            x_hat: Optional[torch.Tensor] = None, stream: Optional[int] = None):
        if y is None:
            y = torch.empty((self.batch, self.c_out) + self.n, dtype=self.dtype,
                            device=self.device)
        ws = self.workspace(B.FNO_OP_FWD)
        s = torch.cuda.current_stream().cuda_stream if stream is None else stream
        B.fno_spectral_conv_fwd(self.desc, _addr(x), self.weights_struct(w), _addr(y),
                                _addr(x_hat), _addr(ws), ws.numel(), s)
        return y

    def bwd_data(self, x: torch.Tensor, w, gy: torch.Tensor, gx: Optional[torch.Tensor] = None,
                 gy_hat: Optional[torch.Tensor] = None, stream: Optional[int] = None):
        if gx is None:
            gx = torch.empty((self.batch, self.c_in) + self.n, dtype=self.dtype,
                             device=self.device)
        ws = self.workspace(B.FNO_OP_BWD_DATA)
        s = torch.cuda.current_stream().cuda_stream if stream is None else stream
        B.fno_spectral_conv_bwd_data(self.desc, _addr(x), self.weights_struct(w), _addr(gy),
                                     _addr(gx), _addr(gy_hat), _addr(ws), ws.numel(), s)
        return gx

    def bwd_weight(self, x: Optional[torch.Tensor], gy: Optional[torch.Tensor], w=None,
                   x_hat: Optional[torch.Tensor] = None, gy_hat: Optional[torch.Tensor] = None,
                   gw=None, stream: Optional[int] = None):
        if gw is None:
            gw = self.alloc_grads()
        caches = x_hat is not None and gy_hat is not None
        ws = self.workspace(B.FNO_OP_BWD_WEIGHT, caches)
        s = torch.cuda.current_stream().cuda_stream if stream is None else stream
        wstruct = self.weights_struct(w) if w is not None else B.weights_struct()
        B.fno_spectral_conv_bwd_weight(self.desc, _addr(x), _addr(gy), wstruct, _addr(x_hat),
                                       _addr(gy_hat), self.grads_struct(gw), _addr(ws),
                                       ws.numel(), s)
        return gw

    def bwd(self, x: Optional[torch.Tensor], w, gy: torch.Tensor,
            x_hat: Optional[torch.Tensor] = None, gx: Optional[torch.Tensor] = None, gw=None,
            gy_hat: Optional[torch.Tensor] = None, stream: Optional[int] = None):
        """Data and weight gradients in one call (returns gx, gw)."""
        if gx is None:
            gx = torch.empty((self.batch, self.c_in) + self.n, dtype=self.dtype,
                             device=self.device)
        if gw is None:
            gw = self.alloc_grads()
        ws = self.workspace(B.FNO_OP_BWD, x_hat is not None)
        s = torch.cuda.current_stream().cuda_stream if stream is None else stream
        B.fno_spectral_conv_bwd(self.desc, _addr(x), self.weights_struct(w), _addr(gy),
                                _addr(x_hat), _addr(gx), self.grads_struct(gw), _addr(gy_hat),
                                _addr(ws), ws.numel(), s)
        return gx, gw
