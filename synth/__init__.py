"""Seeded synthetic inputs for the FNO spectral-convolution layer.

This module only draws random numbers and shapes them into inputs; it holds
none of the layer's arithmetic (no truncated transform, no contraction).  Both
the CPU oracle's tests and the GPU path's tests and benchmark take their inputs
from here, so the two sides always see the same stored values.

Workloads (the five layer shapes the paper's PDE settings suggest):

  1  2-D 64x64,    B=2,  Cin=Cout=16,  modes (8, 8),    dense weights
  2  2-D 128x128,  B=32, Cin=Cout=64,  modes (32, 32),  dense, GRF + channel mixing
     (shaped like the Navier-Stokes TFNO setting of Sec. 4.1)
  3  2-D 1024x1024,B=8,  Cin=Cout=64,  modes (64, 64),  dense
     (the 1024^2 zero-shot super-resolution resolution of Sec. 4.4)
  4  3-D 64^3,     B=4,  Cin=Cout=32,  modes (16,16,16), dense
     (the 64^3 latent grid of the GINO setting, Sec. 4.1)
  5  2-D 256x256,  B=16, Cin=Cout=128, modes (32, 32),  Tucker core (13,13,6,3)
     (a tensorised FNO, Sec. 2 "FNO and extensions")
  6  2-D 128x128,  B=32, Cin=Cout=64,  modes (32, 32),  CP rank 16, GRF + mixing
     (the CP-factorised Navier-Stokes setting of Sec. 4.6; the paper does not
     give the rank: 16 keeps the parameter count near the Tucker workload's)

Synthetic Gaussian random fields stand in for the paper's datasets (none are
available here).  Recipe (one independent field per (sample, channel)):

  * per-mode variance  lam_k = (|k|^2 + 49)^(-5/2), k the folded integer
    wavenumber (k_j - N_j when k_j > N_j / 2);
  * u = irfftn(sqrt(lam) * rfftn(w)) with w iid N(0, 1), divided by
    sqrt(mean_k lam_k) so each field has unit expected variance;
  * workload 2 additionally mixes channels, x[b] = M @ g[b] with
    M_ij ~ N(0, 1/Cin);
  * dense weights: real and imaginary parts iid N(0, 1/(Cin*Cout));
  * Tucker: factor entries re, im ~ N(0, 1/(2 r)), core entries re, im ~
    N(0, 1/(Cin*Cout));
  * CP (rank R): factor entries re, im ~ N(0, 1/2), lambda re, im ~
    N(0, 1/(Cin*Cout*R)), so that W has the dense weights' variance;
  * upstream gradient gy: iid N(0, 1).

Seeds: numpy SeedSequence([workload_id, stream]) with streams x=0, W=1, gy=2,
M=3.  Values are drawn in float64 and rounded to the storage dtype with
round-to-nearest-even (numpy's float16/float32 casts).
"""
from __future__ import annotations

import dataclasses
import os
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np
import scipy.fft

STREAM_X, STREAM_W, STREAM_GY, STREAM_M = 0, 1, 2, 3
STREAM_SKIP = 4  # the block's skip weight and bias

GRF_SHIFT = 49.0
GRF_POWER = 2.5


@dataclasses.dataclass(frozen=True)
class Workload:
    wid: int
    name: str
    batch: int
    c_in: int
    c_out: int
    n: Tuple[int, ...]
    modes: Tuple[int, ...]
    weight: str = "dense"            # "dense" | "tucker" | "cp"
    rank: Optional[Tuple[int, ...]] = None   # (r_in, r_out, r_1..r_d) tucker; (R,) cp
    mixing: bool = False

    @property
    def ndim(self) -> int:
        return len(self.n)

    @property
    def kdims(self) -> Tuple[int, ...]:
        """Retained-mode extents: 2 m_j on leading axes, m_d on the last."""
        d = self.ndim
        return tuple(2 * m if j < d - 1 else m for j, m in enumerate(self.modes))

    def with_batch(self, batch: int) -> "Workload":
        return dataclasses.replace(self, batch=batch)


WORKLOADS: Dict[int, Workload] = {
    1: Workload(1, "grf2d-64x64-b2-c16-m8x8", 2, 16, 16, (64, 64), (8, 8)),
    2: Workload(2, "ns2d-128x128-b32-c64-m32x32", 32, 64, 64, (128, 128), (32, 32),
                mixing=True),
    3: Workload(3, "grf2d-1024x1024-b8-c64-m64x64", 8, 64, 64, (1024, 1024), (64, 64)),
    4: Workload(4, "grf3d-64x64x64-b4-c32-m16x16x16", 4, 32, 32, (64, 64, 64),
                (16, 16, 16)),
    5: Workload(5, "tfno2d-256x256-b16-c128-m32x32-tucker13x13x6x3", 16, 128, 128,
                (256, 256), (32, 32), weight="tucker", rank=(13, 13, 6, 3)),
    6: Workload(6, "cpfno2d-128x128-b32-c64-m32x32-cp16", 32, 64, 64, (128, 128), (32, 32),
                weight="cp", rank=(16,), mixing=True),
}


def rng_for(wid: int, stream: int) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([int(wid), int(stream)]))


def grf_variance(n: Sequence[int]) -> np.ndarray:
    """Per-mode variance (|k|^2 + 49)^(-2.5) on the full FFT grid (folded k)."""
    grids = []
    for nj in n:
        k = np.arange(nj)
        k = np.where(k > nj // 2, k - nj, k).astype(np.float64)
        grids.append(k)
    mesh = np.meshgrid(*grids, indexing="ij")
    k2 = sum(g * g for g in mesh)
    return (k2 + GRF_SHIFT) ** (-GRF_POWER)


def grf_fields(rng: np.random.Generator, count: int, n: Sequence[int],
               chunk: int = 64) -> np.ndarray:
    """`count` independent unit-variance GRFs of shape n, float64 [count, *n].

    The amplitude sqrt(lam) is even in k, so shaping the half spectrum of the
    real noise and transforming back gives the real field directly."""
    n = tuple(int(v) for v in n)
    lam = grf_variance(n)
    amp = np.sqrt(lam / lam.mean())
    amp_half = amp[..., : n[-1] // 2 + 1]
    axes = tuple(range(1, len(n) + 1))
    workers = os.cpu_count() or 1
    out = np.empty((count,) + n, dtype=np.float64)
    for s in range(0, count, chunk):
        e = min(count, s + chunk)
        w = rng.standard_normal((e - s,) + n)
        spec = scipy.fft.rfftn(w, axes=axes, workers=workers) * amp_half
        out[s:e] = scipy.fft.irfftn(spec, s=n, axes=axes, workers=workers)
    return out


def _round(a: np.ndarray, dtype) -> np.ndarray:
    return np.ascontiguousarray(a.astype(dtype))


def make_x(wl: Workload, dtype=np.float16, batch: Optional[int] = None) -> np.ndarray:
    """Input activations x[B, Cin, *n] in the storage dtype."""
    B = wl.batch if batch is None else batch
    rng = rng_for(wl.wid, STREAM_X)
    planes = B * wl.c_in
    out = np.empty((B, wl.c_in) + wl.n, dtype=dtype)
    flat = out.reshape((planes,) + wl.n)
    if wl.mixing:
        mrng = rng_for(wl.wid, STREAM_M)
        M = mrng.standard_normal((wl.c_in, wl.c_in)) / np.sqrt(wl.c_in)
        for b in range(B):
            g = grf_fields(rng, wl.c_in, wl.n)
            mixed = np.tensordot(M, g, axes=([1], [0]))
            out[b] = mixed.astype(dtype)
    else:
        chunk = max(1, min(64, (1 << 22) // int(np.prod(wl.n))))
        for s in range(0, planes, chunk):
            e = min(planes, s + chunk)
            flat[s:e] = grf_fields(rng, e - s, wl.n).astype(dtype)
    return out


def make_gy(wl: Workload, dtype=np.float16, batch: Optional[int] = None) -> np.ndarray:
    """Upstream gradient gy[B, Cout, *n] ~ N(0, 1) in the storage dtype."""
    B = wl.batch if batch is None else batch
    rng = rng_for(wl.wid, STREAM_GY)
    shape = (B, wl.c_out) + wl.n
    out = np.empty(shape, dtype=dtype)
    flat = out.reshape(B * wl.c_out, -1)
    step = max(1, (1 << 22) // flat.shape[1])
    for s in range(0, flat.shape[0], step):
        e = min(flat.shape[0], s + step)
        flat[s:e] = rng.standard_normal((e - s, flat.shape[1])).astype(dtype)
    return out


def _complex_pairs(rng: np.random.Generator, shape, std: float, dtype) -> np.ndarray:
    """Complex values as interleaved (re, im) pairs: array [*shape, 2]."""
    v = rng.standard_normal(tuple(shape) + (2,)) * std
    return _round(v, dtype)


def make_dense_weight(wl: Workload, dtype=np.float16) -> np.ndarray:
    """Dense spectral weight W[Cin, Cout, K_1..K_d, 2] (re, im pairs)."""
    rng = rng_for(wl.wid, STREAM_W)
    std = 1.0 / np.sqrt(wl.c_in * wl.c_out)
    return _complex_pairs(rng, (wl.c_in, wl.c_out) + wl.kdims, std, dtype)


def make_tucker_weight(wl: Workload, dtype=np.float16) -> Dict[str, object]:
    """Tucker weights: core[r_in, r_out, r_1..r_d], u_in[Cin, r_in],
    u_out[Cout, r_out], u_mode[j][K_j, r_j], all as (re, im) pairs."""
    assert wl.rank is not None
    rng = rng_for(wl.wid, STREAM_W)
    r_in, r_out = wl.rank[0], wl.rank[1]
    rm = wl.rank[2:]
    core = _complex_pairs(rng, (r_in, r_out) + tuple(rm),
                          1.0 / np.sqrt(wl.c_in * wl.c_out), dtype)
    u_in = _complex_pairs(rng, (wl.c_in, r_in), 1.0 / np.sqrt(2 * r_in), dtype)
    u_out = _complex_pairs(rng, (wl.c_out, r_out), 1.0 / np.sqrt(2 * r_out), dtype)
    u_mode = [_complex_pairs(rng, (k, r), 1.0 / np.sqrt(2 * r), dtype)
              for k, r in zip(wl.kdims, rm)]
    return {"core": core, "u_in": u_in, "u_out": u_out, "u_mode": u_mode}


def make_cp_weight(wl: Workload, dtype=np.float16) -> Dict[str, object]:
    """CP weights of rank R: lambda ("core" slot) [R], u_in[Cin, R],
    u_out[Cout, R], u_mode[j][K_j, R], all as (re, im) pairs."""
    assert wl.rank is not None
    rng = rng_for(wl.wid, STREAM_W)
    r = wl.rank[0]
    lam = _complex_pairs(rng, (r,), 1.0 / np.sqrt(wl.c_in * wl.c_out * r), dtype)
    u_in = _complex_pairs(rng, (wl.c_in, r), np.sqrt(0.5), dtype)
    u_out = _complex_pairs(rng, (wl.c_out, r), np.sqrt(0.5), dtype)
    u_mode = [_complex_pairs(rng, (k, r), np.sqrt(0.5), dtype) for k in wl.kdims]
    return {"core": lam, "u_in": u_in, "u_out": u_out, "u_mode": u_mode}


def make_weight(wl: Workload, dtype=np.float16):
    """The workload's weights: dense array, or dict of Tucker / CP factors."""
    if wl.weight == "tucker":
        return make_tucker_weight(wl, dtype)
    if wl.weight == "cp":
        return make_cp_weight(wl, dtype)
    return make_dense_weight(wl, dtype)


def make_block_params(wl: Workload, dtype=np.float16):
    """Skip weight w_skip[Cout, Cin] ~ N(0, 1/Cin) and bias b[Cout] ~ N(0, 0.1^2)
    of one FNO block, in the storage dtype."""
    rng = rng_for(wl.wid, STREAM_SKIP)
    w = _round(rng.standard_normal((wl.c_out, wl.c_in)) / np.sqrt(wl.c_in), dtype)
    b = _round(rng.standard_normal(wl.c_out) * 0.1, dtype)
    return w, b


def random_block_case(seed: int, batch: int, c_in: int, c_out: int, grid: Sequence[int],
                      dtype=np.float16):
    """Small iid-normal case for the block epilogue: x[B, Cin, *grid],
    y[B, Cout, *grid] (standing in for the spectral output), w_skip[Cout, Cin]
    ~ N(0, 1/Cin), b[Cout] ~ N(0, 0.1^2) and g_out[B, Cout, *grid]."""
    rng = np.random.default_rng(np.random.SeedSequence([2000 + int(seed)]))
    grid = tuple(grid)
    x = _round(rng.standard_normal((batch, c_in) + grid), dtype)
    y = _round(rng.standard_normal((batch, c_out) + grid), dtype)
    w = _round(rng.standard_normal((c_out, c_in)) / np.sqrt(c_in), dtype)
    b = _round(rng.standard_normal(c_out) * 0.1, dtype)
    g = _round(rng.standard_normal((batch, c_out) + grid), dtype)
    return x, y, w, b, g


def pairs_to_complex(a: np.ndarray) -> np.ndarray:
    """Exact upcast of stored (re, im) pairs to complex128."""
    a = np.asarray(a)
    return a[..., 0].astype(np.float64) + 1j * a[..., 1].astype(np.float64)


def random_dense_case(seed: int, batch: int, c_in: int, c_out: int,
                      n: Sequence[int], modes: Sequence[int], dtype=np.float16,
                      x_scale: float = 1.0):
    """Small iid-normal case for parity tests of odd shapes: x, W pairs, gy."""
    rng = np.random.default_rng(np.random.SeedSequence([1000 + int(seed)]))
    n = tuple(n)
    d = len(n)
    kd = tuple(2 * m if j < d - 1 else m for j, m in enumerate(modes))
    x = _round(rng.standard_normal((batch, c_in) + n) * x_scale, dtype)
    w = _complex_pairs(rng, (c_in, c_out) + kd, 1.0 / np.sqrt(c_in * c_out), dtype)
    gy = _round(rng.standard_normal((batch, c_out) + n), dtype)
    return x, w, gy


def decaying_sinusoids(seed: int, count: int, length: int, kmax: int = 10,
                       decay: float = 1.0) -> np.ndarray:
    """`count` 1-D signals of `length` samples, float64 [count, length]: sums of
    a cosine and a sine at each integer frequency k = 1..kmax (cycles per
    signal), with amplitudes r 2^(-decay (k-1)), r ~ U(0.5, 1) drawn per wave
    (the synthetic signal of the frequency-mode ablation, App. B.10)."""
    rng = np.random.default_rng(np.random.SeedSequence([3000 + int(seed)]))
    x = np.arange(length, dtype=np.float64) / length
    out = np.zeros((count, length))
    for k in range(1, kmax + 1):
        a = rng.uniform(0.5, 1.0, (count, 2)) * 2.0 ** (-decay * (k - 1))
        out += a[:, :1] * np.cos(2 * np.pi * k * x) + a[:, 1:] * np.sin(2 * np.pi * k * x)
    return out
