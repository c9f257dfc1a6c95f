"""Torch-facing wrapper of the C ABI: allocates device buffers with PyTorch and
forwards raw device addresses and the current HIP stream to the library.

PyTorch supplies memory and streams only; every step of the layer runs in the
HIP kernels behind the three entry points.
"""
from __future__ import annotations

from typing import Dict, List, Optional, Sequence

import torch

from . import binding as B


def _addr(t: Optional[torch.Tensor], shape=None, dtype=None, name: str = "tensor",
          device: Optional[torch.device] = None, min_bytes: Optional[int] = None) -> int:
    """Device address of t after checking what the kernels assume of it: its
    dtype and exact shape (or, for raw byte buffers, a minimum size), that it
    is contiguous, and that it lives on the layer's GPU.  None gives 0."""
    if t is None:
        return 0
    if not isinstance(t, torch.Tensor):
        raise ValueError(f"{name}: expected a torch.Tensor, got {type(t).__name__}")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name}: dtype {t.dtype}, expected {dtype}")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name}: shape {tuple(t.shape)}, expected {tuple(shape)}")
    if min_bytes is not None and t.numel() * t.element_size() < min_bytes:
        raise ValueError(f"{name}: {t.numel() * t.element_size()} bytes, "
                         f"at least {min_bytes} needed")
    if not t.is_contiguous():
        raise ValueError(f"{name}: tensor must be contiguous")
    if device is False:      # layout checks only (the caller checks devices later)
        return 0
    if not t.is_cuda:
        raise ValueError(f"{name}: tensor must live on the GPU")
    if device is not None and device.index is not None and t.device.index != device.index:
        raise ValueError(f"{name}: on {t.device}, the layer runs on {device}")
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

    def _param_shapes(self):
        """Shapes (without the trailing (re, im) axis) of the weight tensors:
        {"dense": ...} or {"core", "u_in", "u_out", "u_mode": [...]}."""
        if self.weight_kind == B.FNO_WEIGHT_DENSE:
            return {"dense": (self.c_in, self.c_out) + self.kdims}
        r = self.rank
        d = len(self.n)
        if self.weight_kind == B.FNO_WEIGHT_CP:
            return {"core": (r[0],), "u_in": (self.c_in, r[0]), "u_out": (self.c_out, r[0]),
                    "u_mode": [(k, r[0]) for k in self.kdims]}
        return {"core": tuple(r[:2]) + tuple(r[2:2 + d]), "u_in": (self.c_in, r[0]),
                "u_out": (self.c_out, r[1]),
                "u_mode": [(self.kdims[j], r[2 + j]) for j in range(d)]}

    def _params(self, w, dtype, what, device=None):
        """Checked addresses of a weight (or gradient) set of this layer
        (device=False: the layout checks only)."""
        sh = self._param_shapes()
        dev = self.device if device is None else device
        chk = lambda t, shp, nm: _addr(t, shp + (2,), dtype, f"{what}.{nm}", dev)  # noqa: E731
        if self.weight_kind == B.FNO_WEIGHT_DENSE:
            if isinstance(w, dict):
                raise ValueError(f"{what}: a dense layer takes one tensor")
            return {"dense": chk(w, sh["dense"], "dense")}
        if not isinstance(w, dict) or len(w.get("u_mode", [])) != len(self.n):
            raise ValueError(f"{what}: expected core, u_in, u_out and {len(self.n)} u_mode")
        return {"core": chk(w["core"], sh["core"], "core"),
                "u_in": chk(w["u_in"], sh["u_in"], "u_in"),
                "u_out": chk(w["u_out"], sh["u_out"], "u_out"),
                "u_mode": [chk(u, shp, f"u_mode[{j}]")
                           for j, (u, shp) in enumerate(zip(w["u_mode"], sh["u_mode"]))]}

    def weights_struct(self, w) -> B.FnoWeights:
        return B.weights_struct(**self._params(w, self.dtype, "w"))

    def _x(self, t, name, c, device=None):
        return _addr(t, (self.batch, c) + self.n, self.dtype, name,
                     self.device if device is None else device)

    def _spec(self, t, name, which, device=None):
        return _addr(t, None, None, name, self.device if device is None else device,
                     min_bytes=B.fno_spectrum_bytes(self.desc, which))

    def _validate(self, x=None, w=None, gy=None, y=None, gx=None, x_hat=None, gy_hat=None,
                  gw=None):
        """Layout checks (dtype, shape, size, contiguity) of every argument of a
        call, then device checks of every argument: a mistake in any argument
        is reported before anything is allocated or enqueued."""
        for dev in (False, None):
            self._x(x, "x", self.c_in, dev)
            self._x(gy, "gy", self.c_out, dev)
            self._x(y, "y", self.c_out, dev)
            self._x(gx, "gx", self.c_in, dev)
            if w is not None:
                self._params(w, self.dtype, "w", dev)
            if gw is not None:
                self._params(gw, torch.float32, "gw", dev)
            self._spec(x_hat, "x_hat", 0, dev)
            self._spec(gy_hat, "gy_hat", 1, dev)

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
        return B.grads_struct(**self._params(g, torch.float32, "gw"))

    # -- the calls ---------------------------------------------------------------
    # Every tensor argument is checked (dtype, shape, device) before anything
    # is allocated or enqueued; outputs left as None are allocated afterwards.
    def _out(self, t, c):
        if t is None:
            t = torch.empty((self.batch, c) + self.n, dtype=self.dtype, device=self.device)
        return t

    def fwd(self, x: torch.Tensor, w, y: Optional[torch.Tensor] = None,
            x_hat: Optional[torch.Tensor] = None, stream: Optional[int] = None):
        self._validate(x=x, w=w, y=y, x_hat=x_hat)
        y = self._out(y, self.c_out)
        ws = self.workspace(B.FNO_OP_FWD)
        s = torch.cuda.current_stream().cuda_stream if stream is None else stream
        B.fno_spectral_conv_fwd(self.desc, self._x(x, "x", self.c_in), self.weights_struct(w),
                                self._x(y, "y", self.c_out), self._spec(x_hat, "x_hat", 0),
                                _addr(ws), ws.numel(), s)
        return y

    def bwd_data(self, x: torch.Tensor, w, gy: torch.Tensor, gx: Optional[torch.Tensor] = None,
                 gy_hat: Optional[torch.Tensor] = None, stream: Optional[int] = None):
        self._validate(x=x, w=w, gy=gy, gx=gx, gy_hat=gy_hat)
        gx = self._out(gx, self.c_in)
        ws = self.workspace(B.FNO_OP_BWD_DATA)
        s = torch.cuda.current_stream().cuda_stream if stream is None else stream
        B.fno_spectral_conv_bwd_data(self.desc, self._x(x, "x", self.c_in),
                                     self.weights_struct(w), self._x(gy, "gy", self.c_out),
                                     self._x(gx, "gx", self.c_in),
                                     self._spec(gy_hat, "gy_hat", 1), _addr(ws), ws.numel(), s)
        return gx

    def bwd_weight(self, x: Optional[torch.Tensor], gy: Optional[torch.Tensor], w=None,
                   x_hat: Optional[torch.Tensor] = None, gy_hat: Optional[torch.Tensor] = None,
                   gw=None, stream: Optional[int] = None):
        self._validate(x=x, w=w, gy=gy, x_hat=x_hat, gy_hat=gy_hat, gw=gw)
        gw = self.alloc_grads() if gw is None else gw
        caches = x_hat is not None and gy_hat is not None
        ws = self.workspace(B.FNO_OP_BWD_WEIGHT, caches)
        s = torch.cuda.current_stream().cuda_stream if stream is None else stream
        wst = self.weights_struct(w) if w is not None else B.weights_struct()
        B.fno_spectral_conv_bwd_weight(self.desc, self._x(x, "x", self.c_in),
                                       self._x(gy, "gy", self.c_out), wst,
                                       self._spec(x_hat, "x_hat", 0),
                                       self._spec(gy_hat, "gy_hat", 1), self.grads_struct(gw),
                                       _addr(ws), ws.numel(), s)
        return gw

    def bwd(self, x: Optional[torch.Tensor], w, gy: torch.Tensor,
            x_hat: Optional[torch.Tensor] = None, gx: Optional[torch.Tensor] = None, gw=None,
            gy_hat: Optional[torch.Tensor] = None, stream: Optional[int] = None):
        """Data and weight gradients in one call (returns gx, gw)."""
        self._validate(x=x, w=w, gy=gy, gx=gx, x_hat=x_hat, gy_hat=gy_hat, gw=gw)
        gx = self._out(gx, self.c_in)
        gw = self.alloc_grads() if gw is None else gw
        ws = self.workspace(B.FNO_OP_BWD, x_hat is not None)
        s = torch.cuda.current_stream().cuda_stream if stream is None else stream
        B.fno_spectral_conv_bwd(self.desc, self._x(x, "x", self.c_in), self.weights_struct(w),
                                self._x(gy, "gy", self.c_out), self._spec(x_hat, "x_hat", 0),
                                self._x(gx, "gx", self.c_in), self.grads_struct(gw),
                                self._spec(gy_hat, "gy_hat", 1), _addr(ws), ws.numel(), s)
        return gx, gw


class BlockEpilogue:
    """The rest of one FNO block after the spectral convolution K (the
    fno_block_epilogue_* calls): out = act(W_skip x + b + y) (+ x).

    x [batch, c_in, *grid], y and out [batch, c_out, *grid] in the
    precision's dtype (float16 in fp16 mode, float32 in fp32 mode); w_skip
    [c_out, c_in] and b [c_out] in the same dtype; the parameter gradients are
    float32.  `grid` is the spatial shape (its product is the descriptor's
    points).
    """

    def __init__(self, grid: Sequence[int], batch: int, c_in: int, c_out: int,
                 precision: int = B.FNO_PREC_FP16_TANH, activation: int = B.FNO_EPI_ACT_GELU,
                 residual: bool = False, device: str = "cuda"):
        self.grid = tuple(int(v) for v in grid)
        points = 1
        for v in self.grid:
            points *= v
        self.batch, self.c_in, self.c_out = batch, c_in, c_out
        self.activation, self.residual = activation, residual
        self.desc = B.make_block_desc(batch, c_in, c_out, points, precision, activation,
                                      residual)
        self.dtype = torch.float16 if precision == B.FNO_PREC_FP16_TANH else torch.float32
        self.device = torch.device(device)
        # descriptor checks run in the library
        self.ws_bytes = B.fno_block_epilogue_workspace_size(self.desc, B.FNO_OP_BWD_WEIGHT)

    def _t(self, t, c, name, optional=False):
        if t is None and optional:
            return 0
        if t is None:
            raise ValueError(f"{name} is required")
        return _addr(t, (self.batch, c) + self.grid, self.dtype, name, self.device)

    def _new(self, c):
        return torch.empty((self.batch, c) + self.grid, dtype=self.dtype, device=self.device)

    def fwd(self, x, y, w_skip, b=None, out=None, z_out=None, keep_z: bool = True,
            stream: Optional[int] = None):
        """Returns (out, z); z is None unless kept (needed by the backward
        with GELU)."""
        ax, ay = self._t(x, self.c_in, "x"), self._t(y, self.c_out, "y")
        aw = _addr(w_skip, (self.c_out, self.c_in), self.dtype, "w_skip", self.device)
        ab = _addr(b, (self.c_out,), self.dtype, "b", self.device)
        out = self._new(self.c_out) if out is None else out
        if z_out is None and keep_z and self.activation != B.FNO_EPI_ACT_NONE:
            z_out = self._new(self.c_out)
        ao = self._t(out, self.c_out, "out")
        az = self._t(z_out, self.c_out, "z_out", optional=True)
        s = torch.cuda.current_stream().cuda_stream if stream is None else stream
        B.fno_block_epilogue_fwd(self.desc, ax, ay, aw, ab, ao, az, s)
        return out, z_out

    def bwd_weight(self, x, z, g_out, g_z=None, bias: bool = True,
                   stream: Optional[int] = None):
        """Returns (g_z, g_w_skip, g_b); with activation NONE g_z is g_out
        itself."""
        gelu = self.activation != B.FNO_EPI_ACT_NONE
        ax, ago = self._t(x, self.c_in, "x"), self._t(g_out, self.c_out, "g_out")
        az = self._t(z, self.c_out, "z", optional=not gelu)
        if gelu and g_z is None:
            g_z = self._new(self.c_out)
        agz = self._t(g_z, self.c_out, "g_z", optional=not gelu) if gelu else 0
        gw = torch.empty((self.c_out, self.c_in), dtype=torch.float32, device=self.device)
        gb = torch.empty((self.c_out,), dtype=torch.float32, device=self.device) if bias else None
        ws = torch.empty(max(self.ws_bytes, 1), dtype=torch.uint8, device=self.device)
        s = torch.cuda.current_stream().cuda_stream if stream is None else stream
        B.fno_block_epilogue_bwd_weight(self.desc, ax, az if gelu else 0, ago, agz,
                                        gw.data_ptr(), gb.data_ptr() if bias else 0,
                                        ws.data_ptr(), self.ws_bytes, s)
        return (g_z if gelu else g_out), gw, gb

    def bwd_data(self, g_z, w_skip, gx_spec, g_out=None, gx=None,
                 stream: Optional[int] = None):
        """gx = gx_spec + W_skip^T g_z (+ g_out); gx may be gx_spec (in place)."""
        agz = self._t(g_z, self.c_out, "g_z")
        aw = _addr(w_skip, (self.c_out, self.c_in), self.dtype, "w_skip", self.device)
        ags = self._t(gx_spec, self.c_in, "gx_spec")
        ago = self._t(g_out, self.c_out, "g_out", optional=not self.residual)
        gx = self._new(self.c_in) if gx is None else gx
        agx = self._t(gx, self.c_in, "gx")
        s = torch.cuda.current_stream().cuda_stream if stream is None else stream
        B.fno_block_epilogue_bwd_data(self.desc, agz, aw, ags, ago, agx, s)
        return gx
