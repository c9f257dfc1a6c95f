"""Host-side checks of the C ABI (no GPU needed).

The library loads and exports every symbol the header declares; the integer
logic (mode map, greedy contraction order, path cost, spectrum and workspace
sizes) matches the oracle bit for bit; invalid requests are rejected with the
documented status codes before any device call.
"""
import os
import re

import numpy as np
import pytest

from oracle import fno_oracle as O
import synth

B = pytest.importorskip("paper_2307_15034_amd.binding")

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_symbols():
    names = set()
    inc = os.path.join(ROOT, "include")
    for fn in os.listdir(inc):
        if fn.endswith(".h"):
            txt = open(os.path.join(inc, fn)).read()
            names.update(re.findall(r"^\s*(?:fno_status|const char\s*\*)\s*(fno_\w+)\s*\(",
                                    txt, flags=re.M))
    return sorted(names)


def test_exports_every_declared_symbol():
    names = _declared_symbols()
    assert len(names) >= 10
    lib = B.lib()
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) <= set(B.EXPORTED)


def test_status_strings():
    for code, name in [(0, "FNO_OK"), (1, "FNO_ERR_INVALID_ARGUMENT"), (2, "FNO_ERR_UNSUPPORTED"),
                       (3, "FNO_ERR_WORKSPACE_TOO_SMALL"), (4, "FNO_ERR_HIP")]:
        assert B.status_string(code) == name


def _desc_for(wl, precision=B.FNO_PREC_FP16_TANH, policy=B.FNO_PATH_MIN_RESULT, batch=None):
    kind = {"tucker": B.FNO_WEIGHT_TUCKER, "cp": B.FNO_WEIGHT_CP}.get(wl.weight,
                                                                    B.FNO_WEIGHT_DENSE)
    return B.make_desc(wl.n, wl.modes, batch or wl.batch, wl.c_in, wl.c_out, precision, kind,
                       wl.rank, policy)


@pytest.mark.parametrize("wid", sorted(synth.WORKLOADS))
def test_mode_frequency_matches_oracle(wid):
    wl = synth.WORKLOADS[wid]
    d = _desc_for(wl)
    for j, (n, m) in enumerate(zip(wl.n, wl.modes)):
        last = j == wl.ndim - 1
        ref = O.mode_freq(n, m, last)
        got = [B.fno_mode_frequency(d, j, t) for t in range(len(ref))]
        assert got == ref.tolist()


def test_mode_frequency_random_shapes():
    rng = np.random.default_rng(5)
    for _ in range(200):
        nd = int(rng.integers(1, 4))
        n = [int(rng.integers(2, 300)) for _ in range(nd)]
        modes = [int(rng.integers(1, v // 2 + 1)) for v in n[:-1]]
        modes.append(int(rng.integers(1, min(128, n[-1] // 2 + 1) + 1)))
        d = B.make_desc(n, modes, 1, 1, 1)
        for j in range(nd):
            ref = O.mode_freq(n[j], modes[j], j == nd - 1)
            ts = [0, len(ref) - 1, len(ref) // 2]
            for t in ts:
                assert B.fno_mode_frequency(d, j, t) == int(ref[t])
        with pytest.raises(B.FnoError):
            B.fno_mode_frequency(d, 0, 10 ** 6)


def _mask_to_set(mask):
    inv = {v: k for k, v in B.LABEL_BITS.items()}
    return {inv[b] for b in range(12) if mask >> b & 1}


def _check_path(d, wl_like, op, policy, cp=False):
    nd = len(wl_like["n"])
    kd = tuple(2 * m if j < nd - 1 else m for j, m in enumerate(wl_like["modes"]))
    if cp:
        ops, out = O.cp_labels(nd, adjoint=(op == B.FNO_OP_BWD_DATA))
        sizes = O.cp_sizes(wl_like["batch"], wl_like["c_in"], wl_like["c_out"], kd,
                           wl_like["rank"][0])
    else:
        ops, out = O.tucker_labels(nd, adjoint=(op == B.FNO_OP_BWD_DATA))
        sizes = O.tucker_sizes(wl_like["batch"], wl_like["c_in"], wl_like["c_out"], kd,
                               wl_like["rank"])
    ref = O.greedy_path(ops, sizes, out, policy)
    got = B.fno_contraction_path(d, op)
    assert len(got) == len(ref)
    for (p, q, mask), (rp, rq, rres) in zip(got, ref):
        assert (p, q) == (rp, rq)
        assert _mask_to_set(mask) == set(rres)
    macs, peak = B.fno_contraction_path_cost(d, op)
    assert macs == O.path_macs(ops, sizes, ref)
    assert peak == max(O._size(r, sizes) for _, _, r in ref)


@pytest.mark.parametrize("policy", [B.FNO_PATH_MIN_RESULT, B.FNO_PATH_MIN_NET])
@pytest.mark.parametrize("op", [B.FNO_OP_FWD, B.FNO_OP_BWD_DATA])
def test_tucker_path_matches_oracle_workload(policy, op):
    wl = synth.WORKLOADS[5]
    d = _desc_for(wl, policy=policy)
    pol = "min_result" if policy == B.FNO_PATH_MIN_RESULT else "min_net"
    _check_path(d, dict(n=wl.n, modes=wl.modes, batch=wl.batch, c_in=wl.c_in,
                        c_out=wl.c_out, rank=wl.rank), op, pol)


def test_tucker_path_matches_oracle_random():
    rng = np.random.default_rng(9)
    for trial in range(150):
        nd = int(rng.integers(1, 4))
        n = [int(rng.choice([8, 16, 32, 64])) for _ in range(nd)]
        modes = [int(rng.integers(1, v // 2 + 1)) for v in n]
        modes[-1] = int(rng.integers(1, n[-1] // 2 + 2))
        rank = [int(rng.integers(1, 20)) for _ in range(2 + nd)]
        b, ci, co = (int(rng.integers(1, 40)) for _ in range(3))
        for policy, pol in [(B.FNO_PATH_MIN_RESULT, "min_result"),
                            (B.FNO_PATH_MIN_NET, "min_net")]:
            d = B.make_desc(n, modes, b, ci, co, B.FNO_PREC_FP16_TANH, B.FNO_WEIGHT_TUCKER,
                            rank, policy)
            for op in (B.FNO_OP_FWD, B.FNO_OP_BWD_DATA):
                _check_path(d, dict(n=n, modes=modes, batch=b, c_in=ci, c_out=co, rank=rank),
                            op, pol)


@pytest.mark.parametrize("policy", [B.FNO_PATH_MIN_RESULT, B.FNO_PATH_MIN_NET])
@pytest.mark.parametrize("op", [B.FNO_OP_FWD, B.FNO_OP_BWD_DATA])
def test_cp_path_matches_oracle_workload(policy, op):
    wl = synth.WORKLOADS[6]
    d = _desc_for(wl, policy=policy)
    pol = "min_result" if policy == B.FNO_PATH_MIN_RESULT else "min_net"
    _check_path(d, dict(n=wl.n, modes=wl.modes, batch=wl.batch, c_in=wl.c_in,
                        c_out=wl.c_out, rank=wl.rank), op, pol, cp=True)


def test_cp_path_golden():
    """The library's CP path for the workload the golden sequences were worked
    out for (hand-derived, tests/golden/cp_paths.json)."""
    import json
    with open(os.path.join(ROOT, "tests", "golden", "cp_paths.json")) as f:
        g = json.load(f)
    sz = g["sizes"]
    for policy, pol in [(B.FNO_PATH_MIN_RESULT, "min_result"), (B.FNO_PATH_MIN_NET, "min_net")]:
        d = B.make_desc((128, 128), (32, 32), sz["b"], sz["i"], sz["o"], B.FNO_PREC_FP16_TANH,
                        B.FNO_WEIGHT_CP, (sz["r"],), policy)
        got = B.fno_contraction_path(d, B.FNO_OP_FWD)
        exp = g[pol]["steps"]
        assert len(got) == len(exp)
        for (p, q, mask), (ep, eq, eres, _) in zip(got, exp):
            assert (p, q) == (ep, eq)
            assert _mask_to_set(mask) == set(eres)
        macs, peak = B.fno_contraction_path_cost(d, B.FNO_OP_FWD)
        assert (macs, peak) == (g[pol]["macs"], g[pol]["peak"])


def test_tucker_path_golden_both_ops():
    """The library's Tucker paths for the workload the golden sequences were
    worked out for (hand-derived, tests/golden/tucker_paths.json): the
    forward contraction and the data gradient's adjoint contraction."""
    import json
    with open(os.path.join(ROOT, "tests", "golden", "tucker_paths.json")) as f:
        g = json.load(f)
    sz = g["sizes"]
    for policy, pol in [(B.FNO_PATH_MIN_RESULT, "min_result"), (B.FNO_PATH_MIN_NET, "min_net")]:
        d = B.make_desc((256, 256), (32, 32), sz["b"], sz["i"], sz["o"], B.FNO_PREC_FP16_TANH,
                        B.FNO_WEIGHT_TUCKER, (sz["a"], sz["e"], sz["c"], sz["d"]), policy)
        for op, gg in [(B.FNO_OP_FWD, g), (B.FNO_OP_BWD_DATA, g["adjoint"])]:
            got = B.fno_contraction_path(d, op)
            exp = gg[pol]["steps"]
            assert len(got) == len(exp)
            for (p, q, mask), (ep, eq, eres, _) in zip(got, exp):
                assert (p, q) == (ep, eq)
                assert _mask_to_set(mask) == set(eres)
            macs, peak = B.fno_contraction_path_cost(d, op)
            assert (macs, peak) == (gg[pol]["macs"], gg[pol]["peak"])


def test_cp_path_matches_oracle_random():
    rng = np.random.default_rng(19)
    for trial in range(150):
        nd = int(rng.integers(1, 4))
        n = [int(rng.choice([8, 16, 32, 64])) for _ in range(nd)]
        modes = [int(rng.integers(1, v // 2 + 1)) for v in n]
        modes[-1] = int(rng.integers(1, n[-1] // 2 + 2))
        rank = [int(rng.integers(1, 40))]
        b, ci, co = (int(rng.integers(1, 40)) for _ in range(3))
        for policy, pol in [(B.FNO_PATH_MIN_RESULT, "min_result"),
                            (B.FNO_PATH_MIN_NET, "min_net")]:
            d = B.make_desc(n, modes, b, ci, co, B.FNO_PREC_FP16_TANH, B.FNO_WEIGHT_CP,
                            rank, policy)
            for op in (B.FNO_OP_FWD, B.FNO_OP_BWD_DATA):
                _check_path(d, dict(n=n, modes=modes, batch=b, c_in=ci, c_out=co, rank=rank),
                            op, pol, cp=True)


def test_cp_rank_checked():
    d = B.make_desc((16, 16), (4, 4), 2, 3, 3, B.FNO_PREC_FP16_TANH, B.FNO_WEIGHT_CP, (0,))
    with pytest.raises(B.FnoError):
        B.fno_spectral_conv_workspace_size(d, B.FNO_OP_FWD)
    d = B.make_desc((16, 16), (4, 4), 2, 3, 3, B.FNO_PREC_FP16_TANH, B.FNO_WEIGHT_DENSE)
    with pytest.raises(B.FnoError):
        B.fno_contraction_path(d, B.FNO_OP_FWD)


def test_spectrum_bytes():
    wl = synth.WORKLOADS[2]
    d = _desc_for(wl)
    assert B.fno_spectrum_bytes(d, 0) == 32 * 64 * 64 * 32 * 4
    d32 = _desc_for(wl, precision=B.FNO_PREC_FP32)
    assert B.fno_spectrum_bytes(d32, 1) == 32 * 64 * 64 * 32 * 8


@pytest.mark.parametrize("wid", sorted(synth.WORKLOADS))
def test_workspace_sizes(wid):
    wl = synth.WORKLOADS[wid]
    for prec in (B.FNO_PREC_FP32, B.FNO_PREC_FP16_TANH):
        d = _desc_for(wl, prec)
        for op in (B.FNO_OP_FWD, B.FNO_OP_BWD_DATA, B.FNO_OP_BWD_WEIGHT):
            a = B.fno_spectral_conv_workspace_size(d, op)
            b = B.fno_spectral_conv_workspace_size(d, op, caches=False)
            assert a >= 256 and a % 256 == 0
            assert b >= a
        spec = B.fno_spectrum_bytes(d, 0) + B.fno_spectrum_bytes(d, 1)
        assert B.fno_spectral_conv_workspace_size(d, B.FNO_OP_BWD_WEIGHT, False) >= spec


BAD_DESCS = [
    dict(n=(64, 64), modes=(33, 8)),     # 2m > N on a leading axis
    dict(n=(64, 64), modes=(8, 34)),     # m_d > N/2 + 1
    dict(n=(64, 64), modes=(0, 8)),
    dict(n=(0, 64), modes=(1, 8)),
]


@pytest.mark.parametrize("kw", BAD_DESCS)
def test_invalid_descriptor(kw):
    d = B.make_desc(kw["n"], kw["modes"], 2, 4, 4)
    with pytest.raises(B.FnoError) as e:
        B.fno_spectral_conv_workspace_size(d, B.FNO_OP_FWD)
    assert e.value.status == B.FNO_ERR_INVALID_ARGUMENT


def test_invalid_enums_and_counts():
    for field, val in [("ndim", 0), ("ndim", 4), ("precision", 7), ("weight_kind", 3),
                       ("path_policy", 9), ("batch", 0), ("c_in", -1)]:
        d = B.make_desc((16, 16), (4, 4), 2, 4, 4)
        setattr(d, field, val)
        with pytest.raises(B.FnoError) as e:
            B.fno_spectral_conv_workspace_size(d, B.FNO_OP_FWD)
        assert e.value.status == B.FNO_ERR_INVALID_ARGUMENT, field


def test_preactivation_descriptor_checks():
    P16, P32 = B.FNO_PREC_FP16_TANH, B.FNO_PREC_FP32
    SIG = B.FNO_PREACT_SIGMA_CLIP
    bad = [(P16, 5, 1.0), (P16, -1, 1.0), (P16, B.FNO_PREACT_HARD_CLIP, 0.0),
           (P16, SIG, 0.0), (P32, SIG, -2.0), (P16, SIG, float("nan")),
           (P32, SIG, float("inf")),
           (P16, B.FNO_PREACT_HARD_CLIP, -1.0), (P16, B.FNO_PREACT_HARD_CLIP, float("nan")),
           (P32, B.FNO_PREACT_HARD_CLIP, float("inf")),
           (P16, B.FNO_PREACT_HARD_CLIP, 70000.0)]       # beyond fp16's largest value
    for prec, pa, clip in bad:
        d = B.make_desc((16, 16), (4, 4), 2, 4, 4, prec, preact=pa, clip=clip)
        with pytest.raises(B.FnoError) as e:
            B.fno_spectral_conv_workspace_size(d, B.FNO_OP_FWD)
        assert e.value.status == B.FNO_ERR_INVALID_ARGUMENT, (prec, pa, clip)
    good = [(P32, B.FNO_PREACT_HARD_CLIP, 70000.0), (P16, B.FNO_PREACT_HARD_CLIP, 65504.0),
            (P16, B.FNO_PREACT_TANH, float("nan")), (P32, B.FNO_PREACT_NONE, -3.0),
            (P32, B.FNO_PREACT_TANH, 0.0),             # the bound is ignored unless clipping
            (P16, SIG, 2.0), (P32, SIG, 1e30)]
    for prec, pa, clip in good:
        d = B.make_desc((16, 16), (4, 4), 2, 4, 4, prec, preact=pa, clip=clip)
        assert B.fno_spectral_conv_workspace_size(d, B.FNO_OP_FWD) > 0


def test_sigma_clip_workspace_holds_the_bounds():
    """The statistics-based clip adds 16 bytes (lo, hi in double) per (batch,
    input channel) plane, rounded up to 256, to the workspaces of the calls
    that apply it to x: the forward, the data gradient and the weight
    gradient without caches (the combined backward through its data part)."""
    for n, modes, bt, ci in [((32, 32), (4, 4), 3, 5), ((6, 10, 12), (2, 3, 4), 2, 37),
                             ((96,), (17,), 40, 9)]:
        for prec in (B.FNO_PREC_FP16_TANH, B.FNO_PREC_FP32):
            t = B.make_desc(n, modes, bt, ci, 4, prec, preact=B.FNO_PREACT_TANH)
            s = B.make_desc(n, modes, bt, ci, 4, prec, preact=B.FNO_PREACT_SIGMA_CLIP, clip=2.0)
            extra = (bt * ci * 16 + 255) // 256 * 256
            for op in (B.FNO_OP_FWD, B.FNO_OP_BWD_DATA, B.FNO_OP_BWD):
                assert (B.fno_spectral_conv_workspace_size(s, op)
                        == B.fno_spectral_conv_workspace_size(t, op) + extra), (n, prec, op)
            assert (B.fno_spectral_conv_workspace_size(s, B.FNO_OP_BWD_WEIGHT)
                    == B.fno_spectral_conv_workspace_size(t, B.FNO_OP_BWD_WEIGHT))
            assert (B.fno_spectral_conv_workspace_size(s, B.FNO_OP_BWD_WEIGHT, caches=False)
                    == B.fno_spectral_conv_workspace_size(t, B.FNO_OP_BWD_WEIGHT, caches=False)
                    + extra)


def test_preactivation_decides_whether_bwd_data_reads_x():
    """x may be null exactly when there is no pre-activation (no f'(x))."""
    w = B.weights_struct(dense=FAKE)
    for prec, pa, needs_x in [(B.FNO_PREC_FP32, B.FNO_PREACT_TANH, True),
                              (B.FNO_PREC_FP32, B.FNO_PREACT_HARD_CLIP, True),
                              (B.FNO_PREC_FP16_TANH, B.FNO_PREACT_SIGMA_CLIP, True),
                              (B.FNO_PREC_FP16_TANH, B.FNO_PREACT_NONE, False),
                              (B.FNO_PREC_FP32, B.FNO_PREACT_DEFAULT, False)]:
        d = B.make_desc((32, 32), (4, 4), 2, 4, 4, prec, preact=pa, clip=1.0)
        st = B.fno_spectral_conv_bwd_data(d, 0, w, FAKE, FAKE, 0, FAKE, 16, 0, check=False)
        assert st == (B.FNO_ERR_INVALID_ARGUMENT if needs_x else B.FNO_ERR_WORKSPACE_TOO_SMALL)


def test_unsupported_sizes():
    d = B.make_desc((512, 512), (8, 200), 1, 1, 1)
    with pytest.raises(B.FnoError) as e:
        B.fno_spectral_conv_workspace_size(d, B.FNO_OP_FWD)
    assert e.value.status == B.FNO_ERR_UNSUPPORTED


@pytest.mark.parametrize("batch,c_in,c_out,ok", [
    (1, 65535, 3, True), (1, 3, 65535, True), (1, 65536, 3, False), (1, 3, 65536, False),
    (2, 32768, 1, False), (256, 255, 255, True), (256, 256, 2, False)])
def test_3d_channel_batch_limit(batch, c_in, c_out, ok):
    """The 3-D leading-axis kernels hold batch x channels on a grid axis of at
    most 65535 entries (for the larger of the two channel counts); a
    descriptor beyond that is rejected by the descriptor check, before any
    call enqueues work."""
    d = B.make_desc((8, 8, 8), (2, 2, 2), batch, c_in, c_out)
    if ok:
        B.fno_spectral_conv_workspace_size(d, B.FNO_OP_FWD)
    else:
        with pytest.raises(B.FnoError) as e:
            B.fno_spectral_conv_workspace_size(d, B.FNO_OP_FWD)
        assert e.value.status == B.FNO_ERR_UNSUPPORTED


# Fake device addresses are only ever paired with a request that the host
# rejects first (null / misaligned pointer or too small a workspace), so no
# call below can reach a device.
FAKE = 1 << 20


def test_entry_points_reject_before_device_calls():
    d = B.make_desc((32, 32), (4, 4), 2, 4, 4)
    w = B.weights_struct(dense=FAKE)
    st = B.fno_spectral_conv_fwd(d, 0, w, FAKE, 0, FAKE, 1 << 30, 0, check=False)
    assert st == B.FNO_ERR_INVALID_ARGUMENT                      # null x
    st = B.fno_spectral_conv_fwd(d, FAKE + 2, w, FAKE, 0, FAKE, 1 << 30, 0, check=False)
    assert st == B.FNO_ERR_INVALID_ARGUMENT                      # misaligned x
    st = B.fno_spectral_conv_fwd(d, FAKE, B.weights_struct(), FAKE, 0, FAKE, 1 << 30, 0,
                                 check=False)
    assert st == B.FNO_ERR_INVALID_ARGUMENT                      # missing weights
    st = B.fno_spectral_conv_fwd(d, FAKE, w, FAKE, 0, FAKE, 16, 0, check=False)
    assert st == B.FNO_ERR_WORKSPACE_TOO_SMALL
    st = B.fno_spectral_conv_bwd_data(d, FAKE, w, FAKE, FAKE, 0, FAKE, 16, 0, check=False)
    assert st == B.FNO_ERR_WORKSPACE_TOO_SMALL
    st = B.fno_spectral_conv_bwd_data(d, 0, w, FAKE, FAKE, 0, FAKE, 1 << 30, 0, check=False)
    assert st == B.FNO_ERR_INVALID_ARGUMENT                      # tanh mode needs x
    gw = B.grads_struct(dense=FAKE)
    st = B.fno_spectral_conv_bwd_weight(d, 0, FAKE, w, 0, FAKE, gw, FAKE, 1 << 30, 0,
                                        check=False)
    assert st == B.FNO_ERR_INVALID_ARGUMENT                      # no x and no x_hat
    st = B.fno_spectral_conv_bwd_weight(d, FAKE, FAKE, w, 0, 0, gw, FAKE, 16, 0, check=False)
    assert st == B.FNO_ERR_WORKSPACE_TOO_SMALL
    st = B.fno_spectral_conv_bwd_weight(d, FAKE, FAKE, w, 0, 0, B.grads_struct(), FAKE,
                                        1 << 30, 0, check=False)
    assert st == B.FNO_ERR_INVALID_ARGUMENT                      # no gradient output
    dt = B.make_desc((32, 32), (4, 4), 2, 4, 4, weight_kind=B.FNO_WEIGHT_TUCKER,
                     rank=(2, 2, 2, 2))
    st = B.fno_spectral_conv_fwd(dt, FAKE, B.weights_struct(core=FAKE, u_in=FAKE), FAKE, 0,
                                 FAKE, 1 << 30, 0, check=False)
    assert st == B.FNO_ERR_INVALID_ARGUMENT                      # missing factors


def test_path_rejects_dense_and_bad_op():
    d = B.make_desc((32, 32), (4, 4), 2, 4, 4)
    with pytest.raises(B.FnoError):
        B.fno_contraction_path(d, B.FNO_OP_FWD)
    dt = B.make_desc((32, 32), (4, 4), 2, 4, 4, weight_kind=B.FNO_WEIGHT_TUCKER,
                     rank=(2, 2, 2, 2))
    with pytest.raises(B.FnoError):
        B.fno_contraction_path(dt, B.FNO_OP_BWD_WEIGHT)


def test_binding_has_no_cpu_fallback():
    """The package's product path imports nothing from the oracle."""
    pkg = os.path.join(ROOT, "paper_2307_15034_amd")
    pat = re.compile(r"^\s*(from|import)\s+oracle\b|fno_oracle", re.M)
    for dirpath, _, files in os.walk(pkg):
        for fn in files:
            if fn.endswith((".py", ".hip", ".cpp", ".h")):
                txt = open(os.path.join(dirpath, fn)).read()
                assert not pat.search(txt), fn


# ---------------------------------------------------------------------------
# The torch wrapper checks every tensor before anything reaches the library
# (CPU tensors here: the dtype and shape checks come before the device check,
# and every rejection happens before any allocation or call)
# ---------------------------------------------------------------------------

def _layer(**kw):
    from paper_2307_15034_amd.layer import SpectralConv
    args = dict(n=(16, 16), modes=(4, 4), batch=2, c_in=3, c_out=5)
    args.update(kw)
    return SpectralConv(**args)


def _good(layer):
    import torch
    x = torch.zeros((2, 3, 16, 16), dtype=torch.float16)
    w = torch.zeros((3, 5, 8, 4, 2), dtype=torch.float16)
    gy = torch.zeros((2, 5, 16, 16), dtype=torch.float16)
    return x, w, gy


def test_layer_rejects_wrong_dtype():
    import torch
    layer = _layer()
    x, w, gy = _good(layer)
    with pytest.raises(ValueError, match="dtype"):
        layer.fwd(x.float(), w)
    with pytest.raises(ValueError, match="dtype"):
        layer.fwd(x, w.float())
    with pytest.raises(ValueError, match="dtype"):
        layer.bwd_data(x, w, gy.to(torch.float64))
    with pytest.raises(ValueError, match="dtype"):
        layer.bwd(x, w, gy, gw=torch.zeros((3, 5, 8, 4, 2), dtype=torch.float16))


def test_layer_rejects_wrong_shape():
    layer = _layer()
    x, w, gy = _good(layer)
    with pytest.raises(ValueError, match="shape"):
        layer.fwd(x[:1], w)                               # batch smaller than the layer's
    with pytest.raises(ValueError, match="shape"):
        layer.fwd(x, w[:, :, :4])                         # fewer modes
    with pytest.raises(ValueError, match="shape"):
        layer.fwd(x, w[..., 0].contiguous())              # no (re, im) axis
    with pytest.raises(ValueError, match="shape"):
        layer.bwd_data(x, w, gy[:, :3].contiguous())      # gradient with C_in channels
    with pytest.raises(ValueError, match="shape"):
        layer.fwd(x, w, y=gy[:, :4].contiguous())


def test_layer_rejects_factor_shapes_and_kinds():
    import torch
    from paper_2307_15034_amd import binding as B
    layer = _layer(weight_kind=B.FNO_WEIGHT_TUCKER, rank=(2, 3, 2, 2))
    x, _, _ = _good(layer)
    h = dict(dtype=torch.float16)
    w = {"core": torch.zeros((2, 3, 2, 2, 2), **h), "u_in": torch.zeros((3, 2, 2), **h),
         "u_out": torch.zeros((5, 3, 2), **h),
         "u_mode": [torch.zeros((8, 2, 2), **h), torch.zeros((4, 2, 2), **h)]}
    bad = dict(w, u_out=torch.zeros((5, 2, 2), **h))
    with pytest.raises(ValueError, match="u_out.*shape"):
        layer.fwd(x, bad)
    with pytest.raises(ValueError, match="u_mode"):
        layer.fwd(x, dict(w, u_mode=w["u_mode"][:1]))
    with pytest.raises(ValueError, match="one tensor|expected core"):
        layer.fwd(x, torch.zeros((3, 5, 8, 4, 2), **h))
    with pytest.raises(ValueError, match="GPU"):
        layer.fwd(x, w)                                   # right shapes, but on the host


def test_layer_rejects_host_tensors_and_short_spectra():
    import torch
    layer = _layer()
    x, w, gy = _good(layer)
    with pytest.raises(ValueError, match="GPU"):
        layer.fwd(x, w)
    with pytest.raises(ValueError, match="contiguous"):
        layer.fwd(x.transpose(2, 3), w)
    with pytest.raises(ValueError, match="bytes"):
        layer.fwd(x, w, x_hat=torch.zeros(16, dtype=torch.uint8))


def test_block_epilogue_descriptor_checks():
    """The block epilogue's descriptor: sizes, enums, the residual's channel
    condition and the parameter-gradient limit are checked on the host."""
    ok = B.make_block_desc(2, 4, 4, 64, B.FNO_PREC_FP16_TANH, B.FNO_EPI_ACT_GELU, True)
    assert B.fno_block_epilogue_workspace_size(ok, B.FNO_OP_FWD) == 0
    assert B.fno_block_epilogue_workspace_size(ok, B.FNO_OP_BWD_DATA) == 0
    assert B.fno_block_epilogue_workspace_size(ok, B.FNO_OP_BWD_WEIGHT) > 0
    bad = [dict(residual=True, c_out=5), dict(activation=2), dict(precision=3), dict(batch=0),
           dict(points=0), dict(c_in=0), dict(c_out=70000), dict(c_in=65536, c_out=300)]
    for kw in bad:
        args = dict(batch=2, c_in=4, c_out=4, points=64, precision=B.FNO_PREC_FP16_TANH,
                    activation=B.FNO_EPI_ACT_GELU, residual=False)
        args.update(kw)
        d = B.make_block_desc(**args)
        with pytest.raises(B.FnoError) as e:
            B.fno_block_epilogue_workspace_size(d, B.FNO_OP_BWD_WEIGHT)
        assert e.value.status == B.FNO_ERR_INVALID_ARGUMENT, kw
    with pytest.raises(B.FnoError):
        B.fno_block_epilogue_workspace_size(ok, B.FNO_OP_BWD)


def test_block_epilogue_workspace_is_the_partial_sums():
    """One fp32 partial sum of (c_out x c_in + c_out) values per work-group of
    the parameter-gradient kernel, at most 1024 of them, rounded to 256
    bytes."""
    # fp16: 64-point tiles; fp32: 512-point tiles per work-group round (four
    # waves of 128 points); the generic kernels (points not a multiple of 8)
    # take 4096-point slices
    P16, P32 = B.FNO_PREC_FP16_TANH, B.FNO_PREC_FP32
    for bt, ci, co, pts, prec, expect_g in [(8, 64, 64, 1 << 20, P16, 1024),
                                            (1, 16, 16, 256, P16, 4), (2, 5, 7, 480, P16, 16),
                                            (3, 16, 16, 1536, P32, 9), (2, 5, 7, 480, P32, 2),
                                            (40, 6, 6, 255, P16, 3)]:
        d = B.make_block_desc(bt, ci, co, pts, prec)
        e = co * ci + co
        got = B.fno_block_epilogue_workspace_size(d, B.FNO_OP_BWD_WEIGHT)
        assert got == (expect_g * e * 4 + 255) // 256 * 256, (bt, ci, co, pts, prec)


def test_block_epilogue_rejects_bad_pointers_on_the_host():
    """Misaligned or missing pointers are refused before anything is
    enqueued (no GPU needed)."""
    d = B.make_block_desc(2, 4, 4, 64, B.FNO_PREC_FP16_TANH, B.FNO_EPI_ACT_GELU, False)
    st = B.fno_block_epilogue_fwd(d, FAKE, FAKE + 2, FAKE, 0, FAKE + 256, 0, 0, check=False)
    assert st == B.FNO_ERR_INVALID_ARGUMENT
    st = B.fno_block_epilogue_fwd(d, FAKE, FAKE + 512, FAKE, 0, FAKE, 0, 0, check=False)
    assert st == B.FNO_ERR_INVALID_ARGUMENT          # out aliases x
    st = B.fno_block_epilogue_bwd_weight(d, FAKE, 0, FAKE, FAKE + 256, FAKE + 512, 0, FAKE,
                                         1 << 20, 0, check=False)
    assert st == B.FNO_ERR_INVALID_ARGUMENT          # GELU needs z
    st = B.fno_block_epilogue_bwd_weight(d, FAKE, FAKE + 768, FAKE + 256, FAKE + 1024,
                                         FAKE + 512, 0, FAKE + 4096, 16, 0, check=False)
    assert st == B.FNO_ERR_WORKSPACE_TOO_SMALL
    r = B.make_block_desc(2, 4, 4, 64, B.FNO_PREC_FP32, B.FNO_EPI_ACT_NONE, True)
    st = B.fno_block_epilogue_bwd_data(r, FAKE, FAKE + 256, FAKE + 512, 0, FAKE + 768, 0,
                                       check=False)
    assert st == B.FNO_ERR_INVALID_ARGUMENT          # the residual needs g_out
