"""ctypes binding of libfno_spectral_conv.so (argument marshalling only).

Every function here has the name of the C entry point it calls and passes
plain integers (device addresses, sizes, the HIP stream handle) straight
through; all computation happens in the HIP library.  If the library has not
been built the import fails loudly: there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libfno_spectral_conv.so")

FNO_OK = 0
FNO_ERR_INVALID_ARGUMENT = 1
FNO_ERR_UNSUPPORTED = 2
FNO_ERR_WORKSPACE_TOO_SMALL = 3
FNO_ERR_HIP = 4
FNO_ERR_INTERNAL = 5

FNO_PREC_FP32 = 0
FNO_PREC_FP16_TANH = 1
FNO_PREACT_DEFAULT = 0
FNO_PREACT_NONE = 1
FNO_PREACT_TANH = 2
FNO_PREACT_HARD_CLIP = 3
FNO_PREACT_SIGMA_CLIP = 4
FNO_WEIGHT_DENSE = 0
FNO_WEIGHT_TUCKER = 1
FNO_WEIGHT_CP = 2
FNO_PATH_MIN_RESULT = 0
FNO_PATH_MIN_NET = 1
FNO_OP_FWD = 0
FNO_OP_BWD_DATA = 1
FNO_OP_BWD_WEIGHT = 2
FNO_OP_BWD = 3

LABEL_BITS = {"b": 0, "i": 1, "o": 2, "a": 3, "e": 4, "x": 5, "y": 6, "z": 7,
              "c": 8, "d": 9, "f": 10, "r": 11}


class FnoError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        msg = f"{where}: {status_string(status)} ({status})"
        if status == FNO_ERR_HIP:
            msg += f": {_lib.fno_last_error().decode()}"
        super().__init__(msg)


class FnoConvDesc(ctypes.Structure):
    _fields_ = [
        ("ndim", ctypes.c_int32),
        ("precision", ctypes.c_int32),
        ("weight_kind", ctypes.c_int32),
        ("path_policy", ctypes.c_int32),
        ("batch", ctypes.c_int64),
        ("c_in", ctypes.c_int64),
        ("c_out", ctypes.c_int64),
        ("n", ctypes.c_int64 * 3),
        ("modes", ctypes.c_int64 * 3),
        ("rank", ctypes.c_int64 * 5),
        ("preact", ctypes.c_int32),
        ("clip", ctypes.c_float),
    ]


FNO_EPI_ACT_NONE = 0
FNO_EPI_ACT_GELU = 1


class FnoBlockDesc(ctypes.Structure):
    _fields_ = [
        ("precision", ctypes.c_int32),
        ("batch", ctypes.c_int64),
        ("c_in", ctypes.c_int64),
        ("c_out", ctypes.c_int64),
        ("points", ctypes.c_int64),
        ("activation", ctypes.c_int32),
        ("residual", ctypes.c_int32),
    ]


class FnoWeights(ctypes.Structure):
    _fields_ = [
        ("dense", ctypes.c_void_p),
        ("core", ctypes.c_void_p),
        ("u_in", ctypes.c_void_p),
        ("u_out", ctypes.c_void_p),
        ("u_mode", ctypes.c_void_p * 3),
    ]


class FnoWeightGrads(ctypes.Structure):
    _fields_ = list(FnoWeights._fields_)


def _load() -> ctypes.CDLL:
    if not os.path.exists(LIB_PATH):
        raise ImportError(
            f"{LIB_PATH} is missing: build it with `python -m paper_2307_15034_amd.build` "
            "(no CPU fallback exists)")
    # One HIP runtime per process: PyTorch ships its own libamdhip64 with the
    # same soname as the system one.  Loading torch first makes this library
    # bind to that copy instead of starting a second runtime (and a second
    # HSA runtime) beside it.
    try:
        import torch  # noqa: F401
    except ImportError:  # pragma: no cover - the library also works without torch
        pass
    lib = ctypes.CDLL(LIB_PATH)
    P = ctypes.POINTER
    D = P(FnoConvDesc)
    vp, sz, i32, i64 = ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int32, ctypes.c_int64
    BD = P(FnoBlockDesc)
    sig = {
        "fno_status_string": (ctypes.c_char_p, [ctypes.c_int]),
        "fno_last_error": (ctypes.c_char_p, []),
        "fno_mode_frequency": (ctypes.c_int, [D, i32, i64, P(i64)]),
        "fno_contraction_path": (ctypes.c_int, [D, ctypes.c_int, P(i32), i32, P(i32)]),
        "fno_contraction_path_cost": (ctypes.c_int, [D, ctypes.c_int, P(i64), P(i64)]),
        "fno_spectrum_bytes": (ctypes.c_int, [D, ctypes.c_int, P(sz)]),
        "fno_spectral_conv_workspace_size": (ctypes.c_int, [D, ctypes.c_int, P(sz)]),
        "fno_spectral_conv_workspace_size_nocache": (ctypes.c_int, [D, ctypes.c_int, P(sz)]),
        "fno_spectral_conv_fwd": (ctypes.c_int, [D, vp, P(FnoWeights), vp, vp, vp, sz, vp]),
        "fno_spectral_conv_fwd_noalloc": (ctypes.c_int, [D, vp, P(FnoWeights), vp, vp, vp]),
        "fno_spectral_conv_bwd_data": (ctypes.c_int,
                                       [D, vp, P(FnoWeights), vp, vp, vp, vp, sz, vp]),
        "fno_spectral_conv_bwd_weight": (ctypes.c_int,
                                         [D, vp, vp, P(FnoWeights), vp, vp,
                                          P(FnoWeightGrads), vp, sz, vp]),
        "fno_spectral_conv_bwd": (ctypes.c_int,
                                  [D, vp, P(FnoWeights), vp, vp, vp, P(FnoWeightGrads), vp, vp,
                                   sz, vp]),
        "fno_block_epilogue_workspace_size": (ctypes.c_int, [BD, ctypes.c_int, P(sz)]),
        "fno_block_epilogue_fwd": (ctypes.c_int, [BD, vp, vp, vp, vp, vp, vp, vp]),
        "fno_block_epilogue_bwd_weight": (ctypes.c_int,
                                          [BD, vp, vp, vp, vp, vp, vp, vp, sz, vp]),
        "fno_block_epilogue_bwd_data": (ctypes.c_int, [BD, vp, vp, vp, vp, vp, vp]),
        "fno_release_caches": (ctypes.c_int, []),
        "fno_profile_enable": (ctypes.c_int, [i32]),
        "fno_profile_reset": (ctypes.c_int, []),
        "fno_profile_read": (ctypes.c_int, [i32, ctypes.c_char_p, i32, P(i64),
                                            P(ctypes.c_double)]),
    }
    for name, (res, args) in sig.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    return lib


_lib = _load()

EXPORTED = [
    "fno_status_string", "fno_last_error", "fno_mode_frequency", "fno_contraction_path",
    "fno_contraction_path_cost", "fno_spectrum_bytes", "fno_spectral_conv_workspace_size",
    "fno_spectral_conv_workspace_size_nocache", "fno_spectral_conv_fwd",
    "fno_spectral_conv_fwd_noalloc",
    "fno_spectral_conv_bwd_data", "fno_spectral_conv_bwd_weight", "fno_spectral_conv_bwd",
    "fno_release_caches",
    "fno_profile_enable", "fno_profile_reset", "fno_profile_read",
    "fno_block_epilogue_workspace_size", "fno_block_epilogue_fwd",
    "fno_block_epilogue_bwd_weight", "fno_block_epilogue_bwd_data",
]


def lib() -> ctypes.CDLL:
    return _lib


def status_string(status: int) -> str:
    return _lib.fno_status_string(int(status)).decode()


def _check(status: int, where: str) -> None:
    if status != FNO_OK:
        raise FnoError(status, where)


def make_desc(n: Sequence[int], modes: Sequence[int], batch: int, c_in: int, c_out: int,
              precision: int = FNO_PREC_FP16_TANH, weight_kind: int = FNO_WEIGHT_DENSE,
              rank: Optional[Sequence[int]] = None,
              path_policy: int = FNO_PATH_MIN_RESULT, preact: int = FNO_PREACT_DEFAULT,
              clip: float = 0.0) -> FnoConvDesc:
    d = FnoConvDesc()
    d.ndim = len(n)
    d.precision = precision
    d.weight_kind = weight_kind
    d.path_policy = path_policy
    d.preact = preact
    d.clip = clip
    d.batch, d.c_in, d.c_out = batch, c_in, c_out
    for j, v in enumerate(n):
        d.n[j] = int(v)
    for j, v in enumerate(modes):
        d.modes[j] = int(v)
    if rank is not None:
        for j, v in enumerate(rank):
            d.rank[j] = int(v)
    return d


def fno_mode_frequency(desc: FnoConvDesc, axis: int, t: int) -> int:
    k = ctypes.c_int64()
    _check(_lib.fno_mode_frequency(ctypes.byref(desc), axis, t, ctypes.byref(k)),
           "fno_mode_frequency")
    return k.value


def fno_contraction_path(desc: FnoConvDesc, op: int):
    """[(p, q, result_mask)] of the greedy Tucker order."""
    n = ctypes.c_int32()
    buf = (ctypes.c_int32 * 96)()
    _check(_lib.fno_contraction_path(ctypes.byref(desc), op, buf, 32, ctypes.byref(n)),
           "fno_contraction_path")
    return [(buf[3 * i], buf[3 * i + 1], buf[3 * i + 2]) for i in range(n.value)]


def fno_contraction_path_cost(desc: FnoConvDesc, op: int):
    macs, peak = ctypes.c_int64(), ctypes.c_int64()
    _check(_lib.fno_contraction_path_cost(ctypes.byref(desc), op, ctypes.byref(macs),
                                          ctypes.byref(peak)), "fno_contraction_path_cost")
    return macs.value, peak.value


def fno_spectrum_bytes(desc: FnoConvDesc, which: int) -> int:
    b = ctypes.c_size_t()
    _check(_lib.fno_spectrum_bytes(ctypes.byref(desc), which, ctypes.byref(b)),
           "fno_spectrum_bytes")
    return b.value


def fno_spectral_conv_workspace_size(desc: FnoConvDesc, op: int, caches: bool = True) -> int:
    b = ctypes.c_size_t()
    f = (_lib.fno_spectral_conv_workspace_size if caches
         else _lib.fno_spectral_conv_workspace_size_nocache)
    _check(f(ctypes.byref(desc), op, ctypes.byref(b)), "fno_spectral_conv_workspace_size")
    return b.value


def _weights(dense=0, core=0, u_in=0, u_out=0, u_mode=(0, 0, 0), cls=FnoWeights):
    w = cls()
    w.dense = dense or None
    w.core = core or None
    w.u_in = u_in or None
    w.u_out = u_out or None
    for j in range(3):
        w.u_mode[j] = (u_mode[j] if j < len(u_mode) else 0) or None
    return w


def weights_struct(**kw) -> FnoWeights:
    return _weights(cls=FnoWeights, **kw)


def grads_struct(**kw) -> FnoWeightGrads:
    return _weights(cls=FnoWeightGrads, **kw)


def fno_spectral_conv_fwd(desc, x: int, w: FnoWeights, y: int, x_hat: int, ws: int,
                          ws_bytes: int, stream: int, check: bool = True) -> int:
    st = _lib.fno_spectral_conv_fwd(ctypes.byref(desc), x or None, ctypes.byref(w), y or None,
                                     x_hat or None, ws or None, ws_bytes, stream or None)
    if check:
        _check(st, "fno_spectral_conv_fwd")
    return st


# the fixed per-GPU scratch of the allocation-free forward call
FNO_NOALLOC_SCRATCH_BYTES = 64 << 20


def fno_spectral_conv_fwd_noalloc(desc, x: int, w: FnoWeights, y: int, x_hat: int, stream: int,
                                  check: bool = True) -> int:
    st = _lib.fno_spectral_conv_fwd_noalloc(ctypes.byref(desc), x or None, ctypes.byref(w),
                                            y or None, x_hat or None, stream or None)
    if check:
        _check(st, "fno_spectral_conv_fwd_noalloc")
    return st


def fno_spectral_conv_bwd_data(desc, x: int, w: FnoWeights, gy: int, gx: int, gy_hat: int,
                               ws: int, ws_bytes: int, stream: int, check: bool = True) -> int:
    st = _lib.fno_spectral_conv_bwd_data(ctypes.byref(desc), x or None, ctypes.byref(w),
                                         gy or None, gx or None, gy_hat or None, ws or None,
                                         ws_bytes, stream or None)
    if check:
        _check(st, "fno_spectral_conv_bwd_data")
    return st


def fno_spectral_conv_bwd_weight(desc, x: int, gy: int, w: FnoWeights, x_hat: int,
                                 gy_hat: int, gw: FnoWeightGrads, ws: int, ws_bytes: int,
                                 stream: int, check: bool = True) -> int:
    st = _lib.fno_spectral_conv_bwd_weight(ctypes.byref(desc), x or None, gy or None,
                                           ctypes.byref(w), x_hat or None, gy_hat or None,
                                           ctypes.byref(gw), ws or None, ws_bytes,
                                           stream or None)
    if check:
        _check(st, "fno_spectral_conv_bwd_weight")
    return st


def fno_spectral_conv_bwd(desc, x: int, w: FnoWeights, gy: int, x_hat: int, gx: int,
                          gw: FnoWeightGrads, gy_hat_out: int, ws: int, ws_bytes: int,
                          stream: int, check: bool = True) -> int:
    st = _lib.fno_spectral_conv_bwd(ctypes.byref(desc), x or None, ctypes.byref(w), gy or None,
                                    x_hat or None, gx or None, ctypes.byref(gw),
                                    gy_hat_out or None, ws or None, ws_bytes, stream or None)
    if check:
        _check(st, "fno_spectral_conv_bwd")
    return st


def make_block_desc(batch: int, c_in: int, c_out: int, points: int,
                    precision: int = FNO_PREC_FP16_TANH, activation: int = FNO_EPI_ACT_GELU,
                    residual: bool = False) -> FnoBlockDesc:
    d = FnoBlockDesc()
    d.precision = precision
    d.batch, d.c_in, d.c_out, d.points = batch, c_in, c_out, points
    d.activation = activation
    d.residual = 1 if residual else 0
    return d


def fno_block_epilogue_workspace_size(desc: FnoBlockDesc, op: int) -> int:
    b = ctypes.c_size_t()
    _check(_lib.fno_block_epilogue_workspace_size(ctypes.byref(desc), op, ctypes.byref(b)),
           "fno_block_epilogue_workspace_size")
    return b.value


def fno_block_epilogue_fwd(desc, x: int, y: int, w_skip: int, b: int, out: int, z_out: int,
                           stream: int, check: bool = True) -> int:
    st = _lib.fno_block_epilogue_fwd(ctypes.byref(desc), x or None, y or None, w_skip or None,
                                     b or None, out or None, z_out or None, stream or None)
    if check:
        _check(st, "fno_block_epilogue_fwd")
    return st


def fno_block_epilogue_bwd_weight(desc, x: int, z: int, g_out: int, g_z: int, g_w_skip: int,
                                  g_b: int, ws: int, ws_bytes: int, stream: int,
                                  check: bool = True) -> int:
    st = _lib.fno_block_epilogue_bwd_weight(ctypes.byref(desc), x or None, z or None,
                                            g_out or None, g_z or None, g_w_skip or None,
                                            g_b or None, ws or None, ws_bytes, stream or None)
    if check:
        _check(st, "fno_block_epilogue_bwd_weight")
    return st


def fno_block_epilogue_bwd_data(desc, g_z: int, w_skip: int, gx_spec: int, g_out: int, gx: int,
                                stream: int, check: bool = True) -> int:
    st = _lib.fno_block_epilogue_bwd_data(ctypes.byref(desc), g_z or None, w_skip or None,
                                          gx_spec or None, g_out or None, gx or None,
                                          stream or None)
    if check:
        _check(st, "fno_block_epilogue_bwd_data")
    return st


def fno_release_caches() -> None:
    _check(_lib.fno_release_caches(), "fno_release_caches")


def fno_profile_enable(enable: bool) -> None:
    _check(_lib.fno_profile_enable(1 if enable else 0), "fno_profile_enable")


def fno_profile_reset() -> None:
    _check(_lib.fno_profile_reset(), "fno_profile_reset")


def fno_profile_read():
    """{kernel name: (launches, total_ms)} of the launches timed so far."""
    out = {}
    i = 0
    name = ctypes.create_string_buffer(64)
    n = ctypes.c_int64()
    ms = ctypes.c_double()
    while _lib.fno_profile_read(i, name, 64, ctypes.byref(n), ctypes.byref(ms)) == FNO_OK:
        out[name.value.decode()] = (n.value, ms.value)
        i += 1
    return out
