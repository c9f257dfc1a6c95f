"""CPU float64 oracle of the FNO spectral-convolution layer.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
execute this module: only the test suite, the package's smoke check and the
benchmark's CPU-baseline leg use it.  It shares no code with the HIP library.

What it computes (Tu et al., "Guaranteed Approximation Bounds for
Mixed-Precision Neural Operators", ICLR 2024):

* The Fourier convolution operator (K v)(x) = F^-1(R . T_K(F v))(x) of Sec. 2
  ("FNO and extensions"), evaluated with discrete transforms on a regular grid.
* The forward transform is the Riemann sum of the discretisation error's
  definition in Sec. 3 (the sum of v(xi_j) phi(xi_j) |Q_j| with |Q_j| = 1/N),
  i.e. the DFT normalised by 1/N ("forward" normalisation), sign e^{-i theta}
  (the paper's basis uses e^{+}; for real data this is only conjugation, we
  take the usual forward-FFT sign).
* T_K keeps, on every axis but the last, the m_j lowest non-negative and the
  m_j highest (negative) frequencies in ascending FFT order; on the last,
  real-FFT axis it keeps k = 0..m_d-1.
* R is a complex weight per retained mode mixing channels (Sec. 2), dense,
  Tucker-factorised (the tensorised FNO of Sec. 2; Kolda-Bader mode products)
  or CP-factorised (the factorisation of the Navier-Stokes and Darcy runs,
  Sec. 4.6).
* A pre-activation u = f(x) before the forward transform: tanh in
  half-precision mode (Sec. 4.3), none in full precision; as variants, tanh in
  full precision (the ablation of App. B.8), none in half precision (the
  unstabilised baseline) and the hard clip to [-c, c] of the pre-FFT
  comparison (App. B.6; with c = 57344 the FP8-E5M2 clipping of Sec. 4.6),
  and the 2-sigma clip of the same comparison: each (batch, channel) plane
  clipped to its mean plus or minus two (population) standard deviations,
  the bounds held constant in the gradient.
* The inverse takes y = sum_t c(k_d) Re(Yhat_t e^{+i theta}) with c = 1 on the
  k_d = 0 and Nyquist planes and 2 elsewhere, and no 1/N.
* The Tucker and CP contractions are split into two-operand steps in the
  order a greedy rule picks (Sec. 4.2: the next step is the one whose intermediate is
  smallest).
* Gradients use the real-gradient convention g = dL/dRe + i dL/dIm.
* The rest of the FNO block (Sec. 2): the pointwise channel-mixing skip with
  bias, the activation (GELU) and an optional residual connection, applied
  to the block input and the spectral output, with their gradients.

Everything runs in float64/complex128 on the exact stored input values.

Parity status: every function here is pinned by the oracle tests (brute-force
sums, a library FFT, Parseval, closed forms, adjoint identities, finite
differences, hand-derived greedy sequences of the forward and the adjoint
contraction, and hand-computed values of the comparison functions rel_l2 and
max_plane_rel_l2), each with planted mistakes that a pin must catch.
"""
from __future__ import annotations

import itertools
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

# A mode names the storage precision and the pre-activation f.  The storage
# precision does not change this module's arithmetic (it works on the stored
# values in float64); it only names which library mode a result stands for.
PREC_FP32 = "fp32"            # f(x) = x
PREC_FP16_TANH = "fp16_tanh"  # f(x) = tanh(x)
PREC_FP32_TANH = "fp32_tanh"  # f(x) = tanh(x)
PREC_FP16 = "fp16"            # f(x) = x
# "fp16_clip:<c>" / "fp32_clip:<c>": f(x) = min(max(x, -c), c), built by clip_mode
# "fp16_sigma:<k>" / "fp32_sigma:<k>": the statistics-based clip to
# [mu - k sigma, mu + k sigma] per (batch, channel) plane (k = 2: the 2-sigma
# clip), built by sigma_mode


def clip_mode(storage: str, c: float) -> str:
    """Mode string of the hard clip to [-c, c] with the given storage."""
    if storage not in ("fp16", "fp32"):
        raise ValueError(storage)
    return f"{storage}_clip:{float(c)!r}"


def sigma_mode(storage: str, k: float = 2.0) -> str:
    """Mode string of the k-sigma clip with the given storage."""
    if storage not in ("fp16", "fp32"):
        raise ValueError(storage)
    return f"{storage}_sigma:{float(k)!r}"


def preact_kind(precision: str) -> Tuple[str, Optional[float]]:
    """("none" | "tanh" | "clip" | "sigma", the clip bound / the number of
    standard deviations, or None) of a mode."""
    if precision in (PREC_FP32, PREC_FP16):
        return "none", None
    if precision in (PREC_FP16_TANH, PREC_FP32_TANH):
        return "tanh", None
    if isinstance(precision, str) and precision.split(":")[0] in ("fp16_clip", "fp32_clip"):
        c = float(precision.split(":", 1)[1])
        if not (c > 0.0 and np.isfinite(c)):
            raise ValueError(precision)
        return "clip", c
    if isinstance(precision, str) and precision.split(":")[0] in ("fp16_sigma", "fp32_sigma"):
        k = float(precision.split(":", 1)[1])
        if not (k > 0.0 and np.isfinite(k)):
            raise ValueError(precision)
        return "sigma", k
    raise ValueError(precision)

POLICY_MIN_RESULT = "min_result"
POLICY_MIN_NET = "min_net"


# ---------------------------------------------------------------------------
# Retained modes (T_K)
# ---------------------------------------------------------------------------

def mode_freq(n: int, m: int, last: bool) -> np.ndarray:
    """FFT index k(t) of retained slot t on an axis of length n with m modes.

    Leading axes keep 2m slots: t < m -> k = t, else k = n - 2m + t (the
    negative frequencies -m..-1).  The last (real-FFT) axis keeps m slots,
    k = t.  Sec. 2 names the truncation T_K without fixing the set; this is
    the low-pass set the workloads use.
    """
    n, m = int(n), int(m)
    if last:
        if not (1 <= m <= n // 2 + 1):
            raise ValueError("last-axis modes must satisfy 1 <= m <= n/2+1")
        return np.arange(m, dtype=np.int64)
    if not (1 <= m and 2 * m <= n):
        raise ValueError("leading-axis modes must satisfy 1 <= m and 2m <= n")
    t = np.arange(2 * m, dtype=np.int64)
    return np.where(t < m, t, n - 2 * m + t)


def retained(n: Sequence[int], modes: Sequence[int]) -> List[np.ndarray]:
    d = len(n)
    if len(modes) != d:
        raise ValueError("modes must have one entry per spatial axis")
    return [mode_freq(n[j], modes[j], j == d - 1) for j in range(d)]


def multiplicity(k_last: np.ndarray, n_last: int) -> np.ndarray:
    """c(k): 1 on the k_d = 0 and Nyquist (2 k_d = N_d) planes, 2 elsewhere."""
    k = np.asarray(k_last)
    return np.where((k == 0) | (2 * k == n_last), 1.0, 2.0)


def dft_matrix(n: int, ks: np.ndarray, sign: int) -> np.ndarray:
    """Naive DFT matrix E[t, x] = exp(sign * 2 pi i k_t x / n), phase reduced
    exactly in integers before the float64 evaluation."""
    r = np.outer(np.asarray(ks, dtype=np.int64), np.arange(n, dtype=np.int64)) % n
    return np.exp(sign * 2j * np.pi * r.astype(np.float64) / n)


# ---------------------------------------------------------------------------
# Transforms
# ---------------------------------------------------------------------------

def _apply_axis(a: np.ndarray, mat: np.ndarray, axis: int) -> np.ndarray:
    """Contract axis `axis` of a with mat[new, old]; the new axis stays put."""
    out = np.tensordot(a, mat, axes=([axis], [1]))
    return np.moveaxis(out, -1, axis)


def sigma_bounds(x: np.ndarray, k: float) -> Tuple[np.ndarray, np.ndarray]:
    """Bounds of the statistics-based clip (App. B.6: clipping from the data's
    mean and standard deviation): for every (batch, channel) plane of x
    [B, C, N...], mu - k sigma and mu + k sigma with mu the plane's mean and
    sigma its population standard deviation (divide by the number of points).
    A plane holding a non-finite value has NaN bounds.  Returned with the
    spatial axes kept (size 1) for broadcasting."""
    xf = np.asarray(x, dtype=np.float64)
    if xf.ndim < 3:
        raise ValueError("the sigma clip needs [batch, channel, spatial...] input")
    axes = tuple(range(2, xf.ndim))
    with np.errstate(invalid="ignore", over="ignore"):
        mu = xf.mean(axis=axes, keepdims=True)
        sd = np.sqrt(((xf - mu) ** 2).mean(axis=axes, keepdims=True))
        lo, hi = mu - k * sd, mu + k * sd
    bad = ~(np.isfinite(lo) & np.isfinite(hi))
    lo = np.where(bad, np.nan, lo)
    hi = np.where(bad, np.nan, hi)
    return lo, hi


def preactivation(x: np.ndarray, precision: str) -> np.ndarray:
    """u = f(x): tanh (Sec. 4.3), the identity, the hard clip that moves
    every value outside [-c, c] to the nearer bound, or the statistics-based
    clip to each plane's [mu - k sigma, mu + k sigma] (App. B.6).  NaN stays
    NaN; a plane whose statistics are not finite is NaN throughout."""
    xf = np.asarray(x, dtype=np.float64)
    kind, c = preact_kind(precision)
    if kind == "tanh":
        return np.tanh(xf)
    if kind == "clip":
        return np.where(np.abs(xf) > c, np.copysign(c, xf), xf)
    if kind == "sigma":
        lo, hi = sigma_bounds(xf, c)
        u = np.where(xf < lo, lo, np.where(xf > hi, hi, xf))
        return np.where(np.isnan(lo), np.nan, u)
    return xf


def preactivation_grad(x: np.ndarray, precision: str) -> Optional[np.ndarray]:
    """f'(x), or None for the identity.  tanh: 1 - tanh(x)^2.  Hard clip: 1
    where |x| <= c (a value on the bound counts as inside, as for a clamp whose
    gradient passes at its limits), 0 beyond, NaN where x is NaN."""
    xf = np.asarray(x, dtype=np.float64)
    kind, c = preact_kind(precision)
    if kind == "tanh":
        t = np.tanh(xf)
        return 1.0 - t * t
    if kind == "clip":
        return np.where(np.isnan(xf), np.nan, np.where(np.abs(xf) <= c, 1.0, 0.0))
    if kind == "sigma":
        # the bounds depend on x too; this reading holds them constant (no
        # gradient through the mean and the standard deviation), as for a
        # clip with given bounds
        lo, hi = sigma_bounds(xf, c)
        inside = (xf >= lo) & (xf <= hi)
        return np.where(np.isnan(xf) | np.isnan(lo), np.nan, np.where(inside, 1.0, 0.0))
    return None


def forward_spectrum(u: np.ndarray, n: Sequence[int], modes: Sequence[int]) -> np.ndarray:
    """Xhat[..., t] = (1/N) sum_x u[..., x] exp(-i theta(k(t), x)).

    u has leading (batch, channel) axes followed by the d spatial axes.  The
    sum is the Riemann sum of Sec. 3 with |Q_j| = 1/N, applied axis by axis
    with naive DFT matrices (the d-dimensional exponential factorises).
    """
    d = len(n)
    ks = retained(n, modes)
    a = np.asarray(u, dtype=np.float64)
    lead = a.ndim - d
    for j in range(d - 1, -1, -1):
        a = _apply_axis(a, dft_matrix(n[j], ks[j], -1), lead + j)
    return a / float(np.prod(n))


def inverse_spectrum(z: np.ndarray, n: Sequence[int], modes: Sequence[int],
                     with_c: bool = True) -> np.ndarray:
    """y[..., x] = sum_t c(k_d(t)) Re(z[..., t] exp(+i theta(k(t), x))), no 1/N.

    with_c=False drops the multiplicity (used by the data gradient)."""
    d = len(n)
    ks = retained(n, modes)
    a = np.asarray(z, dtype=np.complex128)
    if with_c:
        a = a * multiplicity(ks[-1], n[-1])
    lead = a.ndim - d
    for j in range(d):
        a = _apply_axis(a, dft_matrix(n[j], ks[j], +1).T, lead + j)
    return a.real


# ---------------------------------------------------------------------------
# Dense layer: forward and gradients
# ---------------------------------------------------------------------------

def contract_dense(xh: np.ndarray, w: np.ndarray) -> np.ndarray:
    """Yhat[b, o, t] = sum_i Xhat[b, i, t] W[i, o, t] (R acting per mode)."""
    return np.einsum("bi...,io...->bo...", xh, w)


def fwd(x, w, n, modes, precision):
    """y = F^-1(R . T_K(F tanh(x))) for dense complex w[Cin, Cout, K...]."""
    u = preactivation(x, precision)
    xh = forward_spectrum(u, n, modes)
    return inverse_spectrum(contract_dense(xh, w), n, modes, with_c=True)


def grad_spectrum(gy, n, modes) -> np.ndarray:
    """G[b, o, t] = c(k_d) sum_x gy[b, o, x] exp(-i theta): the gradient of the
    loss with respect to Yhat (unnormalised)."""
    ks = retained(n, modes)
    g = forward_spectrum(gy, n, modes) * float(np.prod(n))
    return g * multiplicity(ks[-1], n[-1])


def bwd_data(x, w, gy, n, modes, precision):
    """gx: G -> gXhat = sum_o G conj(W) -> gu = (1/N) sum_t Re(gXhat e^{+i theta})
    -> gx = gu f'(x) (the chain rule through the pre-activation)."""
    g = grad_spectrum(gy, n, modes)
    gxh = np.einsum("bo...,io...->bi...", g, np.conj(w))
    gu = inverse_spectrum(gxh, n, modes, with_c=False) / float(np.prod(n))
    fp = preactivation_grad(x, precision)
    return gu if fp is None else gu * fp


def bwd_weight(x, gy, n, modes, precision):
    """gW[i, o, t] = sum_b conj(Xhat[b, i, t]) G[b, o, t]."""
    xh = forward_spectrum(preactivation(x, precision), n, modes)
    g = grad_spectrum(gy, n, modes)
    return np.einsum("bi...,bo...->io...", np.conj(xh), g)


# ---------------------------------------------------------------------------
# Greedy two-operand contraction order (Sec. 4.2)
# ---------------------------------------------------------------------------

def _size(idx: str, sizes: Dict[str, int]) -> int:
    s = 1
    for ch in idx:
        s *= int(sizes[ch])
    return s


def pair_result(operands: Sequence[str], p: int, q: int, output: str) -> str:
    """Indices kept by contracting operands p and q: those still needed by the
    output or by another remaining operand; p's order first, then q's new
    indices."""
    others = set(output)
    for r, op in enumerate(operands):
        if r != p and r != q:
            others.update(op)
    res = [c for c in operands[p] if c in others]
    res += [c for c in operands[q] if c in others and c not in res]
    return "".join(res)


def greedy_path(operands: Sequence[str], sizes: Dict[str, int], output: str,
                policy: str = POLICY_MIN_RESULT) -> List[Tuple[int, int, str]]:
    """Pairwise contraction order chosen greedily (Sec. 4.2).

    At every step, among pairs that share an index (all pairs if none do),
    take the one whose result is smallest (policy min_result: element count
    of the intermediate) or that shrinks memory most (policy min_net: result
    minus both inputs); ties go to the lexicographically smallest (p, q) of
    the current list.  The two inputs leave the list and the result is
    appended.  The final step produces the output index order.

    Returns [(p, q, result_indices)] with p < q positions in the list at the
    time of the step.
    """
    ops = list(operands)
    steps: List[Tuple[int, int, str]] = []
    while len(ops) > 1:
        if len(ops) == 2:
            steps.append((0, 1, output))
            break
        pairs = [(p, q) for p in range(len(ops)) for q in range(p + 1, len(ops))]
        sharing = [(p, q) for (p, q) in pairs if set(ops[p]) & set(ops[q])]
        cand = sharing if sharing else pairs
        best = None
        for (p, q) in cand:
            res = pair_result(ops, p, q, output)
            cost = _size(res, sizes)
            if policy == POLICY_MIN_NET:
                cost -= _size(ops[p], sizes) + _size(ops[q], sizes)
            elif policy != POLICY_MIN_RESULT:
                raise ValueError(policy)
            if best is None or cost < best[0]:
                best = (cost, p, q, res)
        _, p, q, res = best
        steps.append((p, q, res))
        ops = [op for r, op in enumerate(ops) if r not in (p, q)] + [res]
    return steps


def path_macs(operands: Sequence[str], sizes: Dict[str, int],
              steps: Sequence[Tuple[int, int, str]]) -> int:
    """Complex multiply-adds of a path: result size x contracted extent."""
    ops = list(operands)
    total = 0
    for p, q, res in steps:
        shared = (set(ops[p]) | set(ops[q])) - set(res)
        k = 1
        for ch in shared:
            k *= int(sizes[ch])
        total += _size(res, sizes) * k
        ops = [op for r, op in enumerate(ops) if r not in (p, q)] + [res]
    return total


def contract_path(arrays: Sequence[np.ndarray], operands: Sequence[str],
                  steps: Sequence[Tuple[int, int, str]]) -> np.ndarray:
    """Evaluate a pairwise path with two-operand einsums."""
    arrs = list(arrays)
    ops = list(operands)
    for p, q, res in steps:
        r = np.einsum(f"{ops[p]},{ops[q]}->{res}", arrs[p], arrs[q])
        arrs = [a for i, a in enumerate(arrs) if i not in (p, q)] + [r]
        ops = [o for i, o in enumerate(ops) if i not in (p, q)] + [res]
    assert len(arrs) == 1
    return arrs[0]


# ---------------------------------------------------------------------------
# Tucker-factorised weights
# ---------------------------------------------------------------------------

SPATIAL = "xyz"
RANKS = "cdf"


def tucker_labels(d: int, adjoint: bool = False) -> Tuple[List[str], str]:
    """Index strings of [spectrum, core, u_in, u_out, u_1..u_d] and the output.

    Forward: Xhat(b i x..) core(a e c..) u_in(i a) u_out(o e) u_j(x_j c_j)
    -> (b o x..).  Adjoint (data gradient): G(b o x..) with the same factor
    labels -> (b i x..)."""
    sp = SPATIAL[:d]
    rk = RANKS[:d]
    first = ("bo" if adjoint else "bi") + sp
    out = ("bi" if adjoint else "bo") + sp
    ops = [first, "ae" + rk, "ia", "oe"] + [sp[j] + rk[j] for j in range(d)]
    return ops, out


def tucker_sizes(batch, c_in, c_out, kdims, rank) -> Dict[str, int]:
    d = len(kdims)
    s = {"b": batch, "i": c_in, "o": c_out, "a": rank[0], "e": rank[1]}
    for j in range(d):
        s[SPATIAL[j]] = kdims[j]
        s[RANKS[j]] = rank[2 + j]
    return s


def tucker_dense(core, u_in, u_out, u_mode) -> np.ndarray:
    """W[i, o, t_1..t_d] = core x_1 u_in x_2 u_out x_3 u_1 ... (mode products)."""
    d = len(u_mode)
    w = np.asarray(core, dtype=np.complex128)
    # mode product along core axis 0 with u_in[i, a]
    w = np.tensordot(u_in, w, axes=([1], [0]))               # i, e, r..
    w = np.moveaxis(np.tensordot(u_out, w, axes=([1], [1])), 0, 1)  # i, o, r..
    for j in range(d):
        w = np.tensordot(w, u_mode[j], axes=([2], [1]))      # rank axis -> K_j last
    return w


def tucker_contract(spec, core, u_in, u_out, u_mode, n, modes,
                    policy: str = POLICY_MIN_RESULT, adjoint: bool = False,
                    steps=None):
    """Contract a spectrum with Tucker weights along a greedy path.

    forward:  Yhat[b, o, t] = sum_i spec[b, i, t] W[i, o, t]
    adjoint:  gXhat[b, i, t] = sum_o spec[b, o, t] conj(W[i, o, t])
    """
    d = len(n)
    ops, out = tucker_labels(d, adjoint)
    if adjoint:
        facs = [np.conj(core), np.conj(u_in), np.conj(u_out)] + [np.conj(u) for u in u_mode]
    else:
        facs = [core, u_in, u_out] + list(u_mode)
    b = spec.shape[0]
    c_first = spec.shape[1]
    kd = spec.shape[2:]
    c_in = u_in.shape[0]
    c_out = u_out.shape[0]
    rank = (core.shape[0], core.shape[1]) + tuple(core.shape[2:])
    sizes = tucker_sizes(b, c_in, c_out, kd, rank)
    if steps is None:
        steps = greedy_path(ops, sizes, out, policy)
    return contract_path([spec] + facs, ops, steps)


def tucker_fwd(x, core, u_in, u_out, u_mode, n, modes, precision,
               policy: str = POLICY_MIN_RESULT):
    xh = forward_spectrum(preactivation(x, precision), n, modes)
    yh = tucker_contract(xh, core, u_in, u_out, u_mode, n, modes, policy)
    return inverse_spectrum(yh, n, modes, with_c=True)


def tucker_bwd_data(x, core, u_in, u_out, u_mode, gy, n, modes, precision,
                    policy: str = POLICY_MIN_RESULT):
    g = grad_spectrum(gy, n, modes)
    gxh = tucker_contract(g, core, u_in, u_out, u_mode, n, modes, policy, adjoint=True)
    gu = inverse_spectrum(gxh, n, modes, with_c=False) / float(np.prod(n))
    fp = preactivation_grad(x, precision)
    return gu if fp is None else gu * fp


def tucker_bwd_weight(x, gy, core, u_in, u_out, u_mode, n, modes, precision):
    """Chain rule through the multilinear map W(core, factors):
    g_F = sum gW * conj(dW/dF) for each factor F, with gW the dense gradient."""
    d = len(n)
    gw = bwd_weight(x, gy, n, modes, precision)             # i, o, t..
    sp = SPATIAL[:d]
    rk = RANKS[:d]
    core = np.asarray(core)
    cu_in, cu_out = np.conj(u_in), np.conj(u_out)
    cmode = [np.conj(u) for u in u_mode]
    ccore = np.conj(core)
    gw_l = "io" + sp
    mode_terms = ",".join(sp[j] + rk[j] for j in range(d))
    opt = dict(optimize=True)   # evaluation order only; the sum is the same
    g_core = np.einsum(f"{gw_l},ia,oe,{mode_terms}->ae{rk}", gw, cu_in, cu_out, *cmode, **opt)
    g_in = np.einsum(f"{gw_l},ae{rk},oe,{mode_terms}->ia", gw, ccore, cu_out, *cmode, **opt)
    g_out = np.einsum(f"{gw_l},ae{rk},ia,{mode_terms}->oe", gw, ccore, cu_in, *cmode, **opt)
    g_mode = []
    for j in range(d):
        others = [sp[q] + rk[q] for q in range(d) if q != j]
        arrs = [cmode[q] for q in range(d) if q != j]
        spec = ",".join([gw_l, "ae" + rk, "ia", "oe"] + others)
        g_mode.append(np.einsum(f"{spec}->{sp[j]}{rk[j]}", gw, ccore, cu_in, cu_out, *arrs,
                                **opt))
    return g_core, g_in, g_out, g_mode


# ---------------------------------------------------------------------------
# CP-factorised weights
# ---------------------------------------------------------------------------

CP_RANK = "r"


def cp_labels(d: int, adjoint: bool = False) -> Tuple[List[str], str]:
    """Index strings of [spectrum, lambda, u_in, u_out, u_1..u_d] and the output.

    CP (canonical polyadic) form of the weight tensor, the factorisation the
    paper uses on Navier-Stokes and Darcy flow (Sec. 4.6; Kolda-Bader, cited in
    Sec. 2): W[i, o, t_1..t_d] = sum_r lambda[r] u_in[i, r] u_out[o, r]
    prod_j u_j[t_j, r], one rank index r shared by every factor.
    Forward: Xhat(b i x..) lambda(r) u_in(i r) u_out(o r) u_j(x_j r) -> (b o x..);
    adjoint: G(b o x..) with the same factor labels -> (b i x..)."""
    sp = SPATIAL[:d]
    first = ("bo" if adjoint else "bi") + sp
    out = ("bi" if adjoint else "bo") + sp
    ops = [first, CP_RANK, "i" + CP_RANK, "o" + CP_RANK] + [sp[j] + CP_RANK for j in range(d)]
    return ops, out


def cp_sizes(batch, c_in, c_out, kdims, rank: int) -> Dict[str, int]:
    s = {"b": batch, "i": c_in, "o": c_out, CP_RANK: int(rank)}
    for j in range(len(kdims)):
        s[SPATIAL[j]] = kdims[j]
    return s


def cp_dense(lam, u_in, u_out, u_mode) -> np.ndarray:
    """W[i, o, t_1..t_d] = sum_r lam[r] u_in[i, r] u_out[o, r] prod_j u_j[t_j, r]."""
    w = np.asarray(lam, dtype=np.complex128)[None, None, :] * \
        np.asarray(u_in, dtype=np.complex128)[:, None, :] * \
        np.asarray(u_out, dtype=np.complex128)[None, :, :]          # i, o, r
    for u in u_mode:
        u = np.asarray(u, dtype=np.complex128)
        w = w[..., None, :] * u.reshape((1,) * (w.ndim - 1) + u.shape)  # ..., t_j, r
    return w.sum(axis=-1)


def cp_contract(spec, lam, u_in, u_out, u_mode, policy: str = POLICY_MIN_RESULT,
                adjoint: bool = False, steps=None):
    """Contract a spectrum with CP weights along a greedy two-operand path
    (Sec. 4.2), the same rule as for Tucker weights.

    forward:  Yhat[b, o, t] = sum_i spec[b, i, t] W[i, o, t]
    adjoint:  gXhat[b, i, t] = sum_o spec[b, o, t] conj(W[i, o, t])
    """
    d = len(u_mode)
    ops, out = cp_labels(d, adjoint)
    facs = [lam, u_in, u_out] + list(u_mode)
    if adjoint:
        facs = [np.conj(f) for f in facs]
    sizes = cp_sizes(spec.shape[0], u_in.shape[0], u_out.shape[0], spec.shape[2:],
                     np.asarray(lam).shape[0])
    if steps is None:
        steps = greedy_path(ops, sizes, out, policy)
    return contract_path([spec] + facs, ops, steps)


def cp_fwd(x, lam, u_in, u_out, u_mode, n, modes, precision,
           policy: str = POLICY_MIN_RESULT):
    xh = forward_spectrum(preactivation(x, precision), n, modes)
    yh = cp_contract(xh, lam, u_in, u_out, u_mode, policy)
    return inverse_spectrum(yh, n, modes, with_c=True)


def cp_bwd_data(x, lam, u_in, u_out, u_mode, gy, n, modes, precision,
                policy: str = POLICY_MIN_RESULT):
    g = grad_spectrum(gy, n, modes)
    gxh = cp_contract(g, lam, u_in, u_out, u_mode, policy, adjoint=True)
    gu = inverse_spectrum(gxh, n, modes, with_c=False) / float(np.prod(n))
    fp = preactivation_grad(x, precision)
    return gu if fp is None else gu * fp


def cp_bwd_weight(x, gy, lam, u_in, u_out, u_mode, n, modes, precision):
    """Chain rule through W(lambda, factors): g_F = sum gW * conj(dW/dF) for
    each parameter F, with gW the dense weight gradient."""
    d = len(n)
    gw = bwd_weight(x, gy, n, modes, precision)             # i, o, t..
    sp = SPATIAL[:d]
    r = CP_RANK
    clam, cu_in, cu_out = np.conj(lam), np.conj(u_in), np.conj(u_out)
    cmode = [np.conj(u) for u in u_mode]
    gw_l = "io" + sp
    mode_terms = [sp[j] + r for j in range(d)]
    opt = dict(optimize=True)   # evaluation order only; the sum is the same
    g_lam = np.einsum(",".join([gw_l, "i" + r, "o" + r] + mode_terms) + "->" + r,
                      gw, cu_in, cu_out, *cmode, **opt)
    g_in = np.einsum(",".join([gw_l, r, "o" + r] + mode_terms) + "->i" + r,
                     gw, clam, cu_out, *cmode, **opt)
    g_out = np.einsum(",".join([gw_l, r, "i" + r] + mode_terms) + "->o" + r,
                      gw, clam, cu_in, *cmode, **opt)
    g_mode = []
    for j in range(d):
        others = [mode_terms[q] for q in range(d) if q != j]
        arrs = [cmode[q] for q in range(d) if q != j]
        spec = ",".join([gw_l, r, "i" + r, "o" + r] + others)
        g_mode.append(np.einsum(f"{spec}->{sp[j]}{r}", gw, clam, cu_in, cu_out, *arrs, **opt))
    return g_lam, g_in, g_out, g_mode


# ---------------------------------------------------------------------------
# The rest of the FNO block (Sec. 2; Sec. 4.2 leaves these real-valued
# operations to automatic mixed precision)
# ---------------------------------------------------------------------------
#
# One FNO block maps v to act(W v + b + K v) (+ v with a residual connection):
# K is the spectral convolution above, W v + b a pointwise linear map over the
# channels (a 1x1 convolution with bias, the "skip" path), act a pointwise
# nonlinearity.  The epilogue below is everything after K: it takes the
# block input x and the spectral output y = K x.

EPI_ACT_NONE = "none"
EPI_ACT_GELU = "gelu"


def gelu(z: np.ndarray) -> np.ndarray:
    """GELU, the Gaussian error linear unit z Phi(z) with the exact normal
    distribution function Phi(z) = (1 + erf(z / sqrt 2)) / 2."""
    from scipy.special import erf
    z = np.asarray(z, dtype=np.float64)
    return 0.5 * z * (1.0 + erf(z / np.sqrt(2.0)))


def gelu_grad(z: np.ndarray) -> np.ndarray:
    """d/dz z Phi(z) = Phi(z) + z phi(z), phi the standard normal density."""
    from scipy.special import erf
    z = np.asarray(z, dtype=np.float64)
    return 0.5 * (1.0 + erf(z / np.sqrt(2.0))) + z * np.exp(-0.5 * z * z) / np.sqrt(2.0 * np.pi)


def _epi_act(z, act):
    if act == EPI_ACT_GELU:
        return gelu(z)
    if act == EPI_ACT_NONE:
        return np.asarray(z, dtype=np.float64)
    raise ValueError(act)


def _epi_act_grad(z, act):
    if act == EPI_ACT_GELU:
        return gelu_grad(z)
    if act == EPI_ACT_NONE:
        return np.ones(np.shape(z))
    raise ValueError(act)


def channel_mix(w: np.ndarray, v: np.ndarray) -> np.ndarray:
    """(W v)[b, o, x] = sum_i W[o, i] v[b, i, x]: the 1x1 convolution (one
    matrix product per batch item over the flattened grid)."""
    w = np.asarray(w, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    out = np.matmul(w, v.reshape(v.shape[:2] + (-1,)))
    return out.reshape((v.shape[0], w.shape[0]) + v.shape[2:])


def block_epilogue_fwd(x, y, w_skip, bias, act: str, residual: bool):
    """z = W_skip x + b + y (b broadcast over batch and space, absent when
    None), out = act(z) (+ x when residual, which needs C_in = C_out).
    Returns (out, z)."""
    z = channel_mix(w_skip, x) + np.asarray(y, dtype=np.float64)
    if bias is not None:
        z = z + np.asarray(bias, dtype=np.float64).reshape((1, -1) + (1,) * (z.ndim - 2))
    out = _epi_act(z, act)
    if residual:
        if np.shape(x) != np.shape(out):
            raise ValueError("the residual connection needs C_in = C_out")
        out = out + np.asarray(x, dtype=np.float64)
    return out, z


def block_epilogue_bwd(x, z, g_out, w_skip, act: str, residual: bool):
    """Gradients of the epilogue given dL/d out (chain rule):
    g_z = g_out act'(z) (also the gradient of y, so the spectral convolution's
    backward takes it as its output gradient), the skip path's share of the
    input gradient W_skip^T g_z (+ g_out when residual), and the parameter
    gradients g_W[o, i] = sum_{b, x} g_z[b, o, x] x[b, i, x] and
    g_b[o] = sum_{b, x} g_z[b, o, x].  Returns (g_z, g_x_skip, g_w, g_b)."""
    g_out = np.asarray(g_out, dtype=np.float64)
    g_z = g_out * _epi_act_grad(z, act)
    g_x = channel_mix(np.asarray(w_skip, dtype=np.float64).T, g_z)
    if residual:
        g_x = g_x + g_out
    xf = np.asarray(x, dtype=np.float64)
    gz2 = g_z.reshape(g_z.shape[:2] + (-1,))
    g_w = np.matmul(gz2, xf.reshape(xf.shape[:2] + (-1,)).transpose(0, 2, 1)).sum(axis=0)
    g_b = g_z.sum(axis=(0,) + tuple(range(2, g_z.ndim)))
    return g_z, g_x, g_w, g_b


def block_fwd(x, w, w_skip, bias, n, modes, precision, act, residual):
    """The whole block with a dense spectral weight w: act(W_skip x + b + K x)
    (+ x).  Returns (out, z)."""
    return block_epilogue_fwd(x, fwd(x, w, n, modes, precision), w_skip, bias, act, residual)


def block_bwd(x, w, w_skip, bias, g_out, n, modes, precision, act, residual):
    """Gradients of block_fwd: (g_x, g_w_spectral, g_w_skip, g_b).  The input
    gradient adds the spectral path's data gradient (taken at g_z) to the
    skip path's."""
    _, z = block_fwd(x, w, w_skip, bias, n, modes, precision, act, residual)
    g_z, g_x_skip, g_ws, g_b = block_epilogue_bwd(x, z, g_out, w_skip, act, residual)
    g_x = bwd_data(x, w, g_z, n, modes, precision) + g_x_skip
    g_w = bwd_weight(x, g_z, n, modes, precision)
    return g_x, g_w, g_ws, g_b


# ---------------------------------------------------------------------------
# Comparison
# ---------------------------------------------------------------------------

def rel_l2(a, b) -> float:
    """||a - b||_2 / ||b||_2 over the whole tensor in float64 (complex values
    count as real pairs: |z|^2 = Re^2 + Im^2).  b is the reference.  When b is
    zero everywhere the relative error is undefined and the absolute error
    ||a - b||_2 is returned instead (0 when a is zero too)."""
    a = np.asarray(a)
    b = np.asarray(b)
    if np.iscomplexobj(a) or np.iscomplexobj(b):
        a = np.asarray(a, dtype=np.complex128)
        b = np.asarray(b, dtype=np.complex128)
        num = np.sqrt(np.sum(np.abs(a - b) ** 2))
        den = np.sqrt(np.sum(np.abs(b) ** 2))
    else:
        a = a.astype(np.float64)
        b = b.astype(np.float64)
        num = np.sqrt(np.sum((a - b) ** 2))
        den = np.sqrt(np.sum(b ** 2))
    if den == 0.0:
        return float(num)
    return float(num / den)


def max_plane_rel_l2(a, b, nlead: int = 2) -> float:
    """The largest rel_l2 over the planes of the first `nlead` axes: for a
    [B, C, N...] tensor with nlead = 2, rel_l2(a[b, c], b[b, c]) for every
    (b, c), maximised.  A whole-tensor norm can hide an error confined to one
    plane; this cannot."""
    a = np.asarray(a)
    b = np.asarray(b)
    if a.shape != b.shape:
        raise ValueError("shapes differ")
    lead = a.shape[:nlead]
    worst = 0.0
    for idx in itertools.product(*[range(s) for s in lead]):
        r = rel_l2(a[idx], b[idx])
        if np.isnan(r):
            return r  # a non-finite plane is the worst plane
        worst = max(worst, r)
    return worst
