"""Benchmark of the FNO spectral-convolution layer (fwd + bwd_data + bwd_weight).

One step = one pass of the whole layer over one batch: forward (writing the
input-spectrum cache), data gradient (writing the gradient-spectrum cache)
and weight gradient (reading both caches).  Inputs are seeded synthetic
Gaussian random fields resident in HBM before the timed region.

Prints one JSON line with the throughput (samples/s), the roofline figure of
the dominant kernel (HIP events on the launch stream through the library's
event profiler) and the CPU oracle timed on a bounded sample.

The timed steps replay the step's launches captured once as a HIP graph
(--no-graph launches every kernel from the host instead); the per-kernel
figures come from separate, eagerly launched steps.

    python bench.py [--steps K] [--warmup W] [--workload 3] [--no-cpu-baseline]

The default workload is the largest single-GPU one, the 2-D 1024 x 1024 layer
(B = 8, C_in = C_out = 64, 64 x 64 retained modes): 5.97 GB of algorithmic
HBM traffic per step.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "spectral-conv fwd+bwd samples/s (fp16+tanh) + achieved HBM GB/s fraction"
HBM_PEAK_GBS = 8000.0


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=200)
    p.add_argument("--warmup", type=int, default=20)
    p.add_argument("--workload", type=int, default=3)
    p.add_argument("--precision", choices=["fp16_tanh", "fp32"], default="fp16_tanh")
    p.add_argument("--preact", choices=["default", "none", "tanh", "clip"], default="default",
                   help="pre-activation (default: tanh in fp16_tanh, none in fp32)")
    p.add_argument("--clip", type=float, default=1.0, help="bound of --preact clip")
    p.add_argument("--policy", choices=["min_result", "min_net"], default="min_result")
    p.add_argument("--no-caches", action="store_true",
                   help="bwd_weight recomputes both spectra from x and gy")
    p.add_argument("--no-graph", action="store_true",
                   help="launch every kernel from the host instead of replaying the step "
                        "as a HIP graph")
    p.add_argument("--separate-bwd", action="store_true",
                   help="bwd_data and bwd_weight as two calls instead of the combined one")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--block", action="store_true",
                   help="time the whole FNO block (spectral layer + skip/GELU/residual "
                        "epilogue, forward and backward) instead of the layer alone")
    p.add_argument("--cpu-seconds", type=float, default=12.0)
    p.add_argument("--profile-steps", type=int, default=20)
    p.add_argument("--summarize", metavar="DIR",
                   help="write profiles/ summaries of the workload from rocprofv3 output "
                        "under DIR (trace/, FETCH_SIZE/, WRITE_SIZE/, copy_FETCH_SIZE/, "
                        "copy_WRITE_SIZE/, each holding run_*.csv); no GPU")
    p.add_argument("--summarize-sq", metavar="DIR",
                   help="write profiles/sq_counters_<workload>.md from the two SQ counter "
                        "runs under DIR (sq1/, sq2/) and the kernel trace (trace/); no GPU")
    p.add_argument("--copy-probe", action="store_true",
                   help="only run a plain elementwise kernel that reads 1 GiB and writes "
                        "1 GiB, three times (the calibration of the FETCH_SIZE / WRITE_SIZE "
                        "counters)")
    return p.parse_args()


def kernel_bytes(wl, es, preact="tanh"):
    """Algorithmic HBM bytes of each kernel per step (reads + writes of the
    tensors it must touch once).  Without a pre-activation the input and
    gradient transforms are both "r2c_plane" and both inverses "c2r_plane"
    (the data gradient's inverse then reads no x)."""
    B, Ci, Co = wl.batch, wl.c_in, wl.c_out
    N = int(np.prod(wl.n))
    K = int(np.prod(wl.kdims))
    spec_in = B * Ci * K * 2 * es
    spec_out = B * Co * K * 2 * es
    W = Ci * Co * K * 2 * es
    out = {
        "contract": spec_in + W + spec_out,
        "contract_adjoint": spec_out + W + spec_in,
        "c2r_plane": spec_out + B * Co * N * es,
        "c2r_plane_tanh_grad": spec_in + 2 * B * Ci * N * es,
        "wgrad": spec_in + spec_out + Ci * Co * K * 2 * 4,
    }
    # one launch: G read once (shared by both products), W read, gXhat
    # written, Xhat read, gW written
    out["contract_adjoint_wgrad"] = spec_out + W + spec_in + spec_in + Ci * Co * K * 2 * 4
    out["r2c_plane_tanh"] = B * Ci * N * es + spec_in     # input transform (tanh)
    out["r2c_plane"] = B * Co * N * es + spec_out         # gradient transform
    out["r2c_plane_clip"] = out["r2c_plane_tanh"]
    out["c2r_plane_clip_grad"] = out["c2r_plane_tanh_grad"]
    if preact == "none":
        out["r2c_plane"] += out["r2c_plane_tanh"]
        out["c2r_plane"] += spec_in + B * Ci * N * es
    return out


def block_kernel_bytes(wl, es, residual=True):
    """Algorithmic bytes of the block epilogue's launches: the forward reads x
    and y and writes out and z; the parameter-gradient pass reads x, z and
    g_out and writes g_z (plus W_skip / b and the fp32 parameter gradients);
    the data-gradient pass reads g_z and gx_spec (and g_out with the
    residual) and writes gx."""
    B, Ci, Co = wl.batch, wl.c_in, wl.c_out
    N = int(np.prod(wl.n))
    S_in, S_out = B * Ci * N * es, B * Co * N * es
    P = Co * Ci * es + Co * es
    return {"block_epilogue_fwd": S_in + 3 * S_out + P,
            "block_epilogue_bwd_weight": S_in + 3 * S_out + (Co * Ci + Co) * 4,
            "block_epilogue_bwd_data": 2 * S_in + S_out + (S_out if residual else 0) + P}


def step_bytes(wl, es, caches=True, preact="tanh"):
    """Whole-step algorithmic bytes: 5 spatial passes (4 without a
    pre-activation, whose data gradient reads no x), W twice, gW (fp32), and
    the two spectral caches written once and read once."""
    B, Ci, Co = wl.batch, wl.c_in, wl.c_out
    N = int(np.prod(wl.n))
    K = int(np.prod(wl.kdims))
    S_in, S_out = B * Ci * N * es, B * Co * N * es
    spec = (B * Ci * K + B * Co * K) * 2 * es
    if wl.weight == "tucker":
        r = wl.rank
        nparam = (np.prod(r) + Ci * r[0] + Co * r[1]
                  + sum(k * rr for k, rr in zip(wl.kdims, r[2:])))
        W, gW = 2 * nparam * es, 2 * nparam * 4
    elif wl.weight == "cp":
        r = wl.rank[0]
        nparam = r * (1 + Ci + Co + sum(wl.kdims))
        W, gW = 2 * nparam * es, 2 * nparam * 4
    else:
        W, gW = Ci * Co * K * 2 * es, Ci * Co * K * 2 * 4
    total = S_in + S_out + (S_out + S_in + S_in) + 2 * W + gW
    if preact == "none":
        total -= S_in
    total += 2 * spec if caches else (S_in + S_out)
    return int(total)


def kernel_sources_hash():
    """Hash of the HIP/C++ sources; counter-derived traffic is reported only
    while the kernels are the ones the counters were taken on."""
    import hashlib
    h = hashlib.sha256()
    c = os.path.join(ROOT, "paper_2307_15034_amd", "csrc")
    for f in sorted(os.listdir(c)):
        h.update(f.encode())
        with open(os.path.join(c, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic(wl_name, kernel):
    """HBM bytes per launch of `kernel` from the committed rocprofv3
    FETCH_SIZE / WRITE_SIZE summary (copy-kernel calibrated), or None."""
    path = os.path.join(ROOT, "profiles", f"traffic_{wl_name}.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        t = json.load(f)
    if t.get("src_hash") != kernel_sources_hash():
        return None
    k = t.get("kernels", {}).get(kernel)
    return int(k["bytes"]) if k else None


def cpu_baseline(wl, x, w, gy, prec, seconds):
    """The float64 oracle, as it stands, on a bounded sample of the workload:
    whole batch samples (fwd + bwd_data + bwd_weight), repeated until about
    `seconds` of CPU time."""
    from oracle import fno_oracle as O
    import synth
    host_cores = len(os.sched_getaffinity(0))
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:  # pragma: no cover
        threads = host_cores
    oprec = prec
    done = 0
    t0 = time.perf_counter()
    while True:
        b = done % wl.batch
        xb, gb = x[b:b + 1], gy[b:b + 1]
        if wl.weight in ("tucker", "cp"):
            core = synth.pairs_to_complex(w["core"])
            u_in = synth.pairs_to_complex(w["u_in"])
            u_out = synth.pairs_to_complex(w["u_out"])
            um = [synth.pairs_to_complex(u) for u in w["u_mode"]]
            fw, bd, bw = ((O.tucker_fwd, O.tucker_bwd_data, O.tucker_bwd_weight)
                          if wl.weight == "tucker" else
                          (O.cp_fwd, O.cp_bwd_data, O.cp_bwd_weight))
            fw(xb, core, u_in, u_out, um, wl.n, wl.modes, oprec)
            bd(xb, core, u_in, u_out, um, gb, wl.n, wl.modes, oprec)
            bw(xb, gb, core, u_in, u_out, um, wl.n, wl.modes, oprec)
        else:
            wc = synth.pairs_to_complex(w)
            O.fwd(xb, wc, wl.n, wl.modes, oprec)
            O.bwd_data(xb, wc, gb, wl.n, wl.modes, oprec)
            O.bwd_weight(xb, gb, wl.n, wl.modes, oprec)
        done += 1
        el = time.perf_counter() - t0
        if el >= seconds:
            break
    return {"value": done / el, "unit": "samples/s", "cores": int(threads),
            "host_cores": int(host_cores), "kind": "oracle",
            "sample": f"{done} batch samples of the workload (B=1 slices), float64 oracle "
                      f"fwd+bwd_data+bwd_weight, {el:.1f} s"}


def copy_probe(torch):
    """A plain elementwise kernel that reads 1 GiB and writes 1 GiB (int32
    negation, torch's own kernel), three times: what FETCH_SIZE and
    WRITE_SIZE read for it calibrates them in bytes."""
    assert torch.cuda.is_available(), "the copy probe needs a GPU"
    n = (1 << 30) // 4
    a = torch.ones(n, dtype=torch.int32, device="cuda")
    b = torch.empty_like(a)
    for _ in range(3):
        torch.neg(a, out=b)
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe_bytes_read": n * 4, "copy_probe_bytes_written": n * 4,
                      "dispatches": 3}))


def copy_bandwidth(torch, nbytes=1 << 30, reps=10):
    """A plain device-to-device copy of `nbytes` (torch's copy kernel), timed
    with HIP events: (read + written bytes) / time, in GB/s.  The practical
    streaming rate of this GPU, reported beside the 8 TB/s peak."""
    a = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    a.fill_(1)
    b = torch.empty_like(a)
    for _ in range(2):
        b.copy_(a)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        b.copy_(a)
    e1.record()
    torch.cuda.synchronize()
    gbs = 2.0 * nbytes * reps / (e0.elapsed_time(e1) / 1e3) / 1e9
    del a, b
    torch.cuda.empty_cache()
    return gbs


# rocprofv3 kernel symbols -> the names the library times its launches under
# (first match wins; the template flag "true" marks the pre-activation
# variant of a transform: the last flag; the second argument of the radix-2
# wide-plane forward, the third of its inverse)
KERNEL_NAMES = [
    (r"epi_mix\w*<[^>]*true>", "block_epilogue_fwd"),
    (r"epi_mix\w*<", "block_epilogue_bwd_data"),
    (r"epi_wgrad\w*<", "block_epilogue_bwd_weight"),
    (r"r2c_wide2_kernel<\d+, true", "r2c_plane_tanh"),
    (r"r2c_wide2_kernel<", "r2c_plane"),
    (r"r2c_\w+<[^>]*true>", "r2c_plane_tanh"),
    (r"r2c_\w+<", "r2c_plane"),
    (r"slab_adj_wgrad_kernel", "contract_adjoint_wgrad"),
    (r"slab_kernel<", "contract"),
    (r"c2r_wide2_kernel<\d+, \d+, true", "c2r_plane_tanh_grad"),
    (r"c2r_wide2_kernel<", "c2r_plane"),
    (r"c2r_\w+<[^>]*true>", "c2r_plane_tanh_grad"),
    (r"c2r_\w+<", "c2r_plane"),
]


def _logical(kname):
    import re
    for pat, name in KERNEL_NAMES:
        if re.search(pat, kname):
            return name
    return kname


def _csv(path):
    import csv
    with open(path, newline="") as f:
        return list(csv.DictReader(f))


def summarize(args):
    """profiles/traffic_<workload>.json and profiles/layer_step_<workload>.md
    from the rocprofv3 runs listed in the summary: durations from the kernel
    trace, HBM bytes from FETCH_SIZE / WRITE_SIZE (KiB per dispatch, median
    over the dispatches of a kernel) scaled by what the same counters read for
    the copy probe (1 GiB read, 1 GiB written)."""
    import statistics
    wl = __import__("synth").WORKLOADS[args.workload]
    d = args.summarize
    trace = _csv(os.path.join(d, "trace", "run_kernel_trace.csv"))
    stats = _csv(os.path.join(d, "trace", "run_kernel_stats.csv"))

    def counter(sub, name):
        per = {}
        for r in _csv(os.path.join(d, sub, "run_counter_collection.csv")):
            if r["Counter_Name"] == name:
                per.setdefault(r["Kernel_Name"], []).append(float(r["Counter_Value"]) * 1024)
        return per

    gib = float(1 << 30)
    # counter runs are optional: without them only the trace is summarised
    have_pmc = os.path.isdir(os.path.join(d, "FETCH_SIZE"))
    f_cal = w_cal = 1.0
    fetch, write = {}, {}
    if have_pmc:
        cf = counter("copy_FETCH_SIZE", "FETCH_SIZE")
        cw = counter("copy_WRITE_SIZE", "WRITE_SIZE")
        # the probe's kernel is the one that moves the most bytes
        f_cal = gib / statistics.median(max(cf.values(), key=statistics.median))
        w_cal = gib / statistics.median(max(cw.values(), key=statistics.median))
        fetch = counter("FETCH_SIZE", "FETCH_SIZE")
        write = counter("WRITE_SIZE", "WRITE_SIZE")
    # the HIP-event figures bench.py printed in the same (traced) run
    ev = {}
    tlog = os.path.join(d, "trace.log")
    if os.path.exists(tlog):
        for line in open(tlog):
            line = line.strip()
            if line.startswith("{") and '"kernels"' in line:
                ev = {k: v["avg_ms"] * 1e3 for k, v in json.loads(line)["kernels"].items()}
    dur = {}
    for r in trace:
        dur.setdefault(r["Kernel_Name"], []).append(
            (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)
    es = 2 if args.precision == "fp16_tanh" else 4
    kb = kernel_bytes(wl, es)
    if args.block:
        kb.update(block_kernel_bytes(wl, es, wl.c_in == wl.c_out))
    tr = {"workload": wl.name, "src_hash": kernel_sources_hash(),
          "calibration": {"fetch": f_cal, "write": w_cal}, "kernels": {}}
    rows = []
    for kname, ds in sorted(dur.items(), key=lambda kv: -sum(kv[1])):
        name = _logical(kname)
        evs = f"{ev[name]:.1f}" if name in ev else "-"
        if name not in kb or kname not in fetch or kname not in write:
            if name in kb:
                avg = sum(ds) / len(ds)
                rows.append(f"| {name} | {len(ds)} | {avg:.1f} | {evs} | {min(ds):.1f} | "
                            f"{max(ds):.1f} | {kb[name] / 1e6:.1f} | {kb[name] / avg / 1e3:.0f} | "
                            f"{kb[name] / avg / 1e3 / HBM_PEAK_GBS:.3f} | - | - | - |")
            continue
        fb = statistics.median(fetch[kname]) * f_cal
        wb = statistics.median(write[kname]) * w_cal
        tr["kernels"][name] = {"fetch_bytes": int(fb), "write_bytes": int(wb),
                               "bytes": int(fb + wb)}
        avg = sum(ds) / len(ds)
        rows.append(f"| {name} | {len(ds)} | {avg:.1f} | {evs} | {min(ds):.1f} | {max(ds):.1f} | "
                    f"{kb[name] / 1e6:.1f} | {kb[name] / avg / 1e3:.0f} | "
                    f"{kb[name] / avg / 1e3 / HBM_PEAK_GBS:.3f} | {fb / 1e6:.1f} | "
                    f"{wb / 1e6:.1f} | {(fb + wb) / kb[name]:.2f} |")
    os.makedirs(os.path.join(ROOT, "profiles"), exist_ok=True)
    tag = "block_" if args.block else ""
    if have_pmc:
        with open(os.path.join(ROOT, "profiles", f"traffic_{tag}{wl.name}.json"), "w") as f:
            json.dump(tr, f, indent=1)
    cmd = ("cd /tmp && export TMPDIR=/tmp && rocprofv3 {what} --output-format csv "
           "-d <out>/{sub} -o run -- python3 /root/repo/bench.py {extra}")
    wk = f"--workload {args.workload} " if args.workload != 3 else ""
    if args.block:
        wk += "--block "
    if wl.weight != "dense":
        wk += f"--policy {args.policy} "
    cmds = [
        cmd.format(what="--kernel-trace --stats", sub="trace",
                   extra=f"{wk}--steps 20 --warmup 5 --no-cpu-baseline") + " > <out>/trace.log",
        cmd.format(what="--pmc FETCH_SIZE", sub="FETCH_SIZE",
                   extra=f"{wk}--steps 2 --warmup 1 --profile-steps 1 --no-cpu-baseline"),
        cmd.format(what="--pmc WRITE_SIZE", sub="WRITE_SIZE",
                   extra=f"{wk}--steps 2 --warmup 1 --profile-steps 1 --no-cpu-baseline"),
        cmd.format(what="--pmc FETCH_SIZE", sub="copy_FETCH_SIZE", extra="--copy-probe"),
        cmd.format(what="--pmc WRITE_SIZE", sub="copy_WRITE_SIZE", extra="--copy-probe"),
        f"python3 bench.py {wk}--summarize <out>",
    ]
    if not have_pmc:
        cmds = [cmds[0], cmds[-1]]
    total_avg = sum(sum(ds) / len(ds) for k, ds in dur.items() if _logical(k) in kb)
    pol = f", {args.policy} path" if wl.weight != "dense" else ""
    title = ("FNO block step kernels (spectral layer + skip/GELU/residual epilogue)"
             if args.block else "Layer step kernels")
    lines = [
        f"# {title}, workload {wl.name} (fp16+tanh, {wl.weight}{pol}, spectral "
        "caches, combined backward)", "",
        "MI355X, one GPU. Durations from the rocprofv3 kernel trace of the timed benchmark",
        "(kernel begin/end timestamps, all dispatches of the run)" + (
            "; HBM traffic from the" if have_pmc else "."),
    ]
    if have_pmc:
        lines += [
            "FETCH_SIZE and WRITE_SIZE counters (KiB per dispatch, median over dispatches) "
            "scaled",
            "by the factors that an elementwise probe kernel reading 1 GiB and writing 1 GiB",
            f"(bench.py --copy-probe) gives for the same counters (FETCH x{f_cal:.3f}, "
            f"WRITE x{w_cal:.3f})."]
    lines += [f"Kernel sources hash {tr['src_hash']}.", "", "Commands:", ""]
    lines += ["    " + c for c in cmds]
    lines += ["", "\"avg us\" is the trace's average over all dispatches; \"events us\" the "
                  "average that", "bench.py's own HIP events measured in the same run (the "
                  "figure its JSON line uses);", "\"frac\" = alg MB / trace avg / 8 TB/s.", "",
              "| kernel | dispatches | avg us | events us | min us | max us | alg MB | "
              "alg GB/s (avg) | frac | HBM fetch MB | HBM write MB | traffic / alg |",
              "|---|---|---|---|---|---|---|---|---|---|---|---|"] + rows
    whole = wl.weight == "dense" and wl.ndim < 3 and not args.block
    lines += ["", f"Sum of the averages of the kernels in the table: {total_avg:.1f} us"
                  + (" (the whole step)." if whole else
                     " (the other kernels of the step are in the summary below)."), "",
              "rocprofv3 --stats summary (all dispatches):", "",
              "| name | calls | avg ns | min ns | max ns | % |", "|---|---|---|---|---|---|"]
    for r in stats:
        lines.append(f"| {r['Name'][:70]} | {r['Calls']} | {float(r['AverageNs']):.0f} | "
                     f"{float(r['MinNs']):.0f} | {float(r['MaxNs']):.0f} | "
                     f"{float(r['Percentage']):.2f} |")
    suffix = f"_{args.policy}" if wl.weight != "dense" else ""
    stem = "block_step" if args.block else "layer_step"
    with open(os.path.join(ROOT, "profiles", f"{stem}_{wl.name}{suffix}.md"), "w") as f:
        f.write("\n".join(lines) + "\n")
    print(json.dumps(tr))


SQ_PASSES = {
    "sq1": "SQ_WAVES SQ_INSTS_VALU SQ_INSTS_LDS SQ_INSTS_MFMA SQ_VALU_MFMA_BUSY_CYCLES "
           "SQ_INSTS_VALU_MFMA_MOPS_F16 SQ_WAVE_CYCLES SQ_BUSY_CYCLES GRBM_GUI_ACTIVE",
    "sq2": "SQ_WAIT_ANY SQ_WAIT_INST_ANY SQ_ACTIVE_INST_VALU SQ_ACTIVE_INST_LDS "
           "SQ_ACTIVE_INST_VMEM SQ_LDS_BANK_CONFLICT SQ_INSTS_SALU SQ_INSTS_VMEM_RD",
}
SIMDS = 256 * 4          # MI355X: 256 compute units of four SIMDs
XCDS = 8                 # GRBM_GUI_ACTIVE is summed over the eight XCDs
MFMA_F16_PEAK_TFS = 2500.0


def summarize_sq(args):
    """profiles/sq_counters_<workload>.md: instruction, stall and matrix-core
    counters of one profiled step per kernel (chip-wide sums per dispatch,
    median over a kernel's dispatches).  Matrix-core utilisation is
    SQ_VALU_MFMA_BUSY_CYCLES / (GRBM_GUI_ACTIVE / XCDs x SIMDs), the busy
    cycles of all SIMDs over the cycles of one XCD's kernel; the fp16 matrix rate
    is 512 x SQ_INSTS_VALU_MFMA_MOPS_F16 flops over the kernel's trace
    duration, against the 2.5 PFLOP/s dense fp16 peak."""
    import statistics
    wl = __import__("synth").WORKLOADS[args.workload]
    d = args.summarize_sq
    vals = {}
    for sub in SQ_PASSES:
        for r in _csv(os.path.join(d, sub, "run_counter_collection.csv")):
            key = (r["Kernel_Name"], r.get("Grid_Size", ""))
            vals.setdefault(key, {}).setdefault(r["Counter_Name"], {}).setdefault(
                r.get("Dispatch_Id", "0"), 0.0)
            vals[key][r["Counter_Name"]][r.get("Dispatch_Id", "0")] += float(r["Counter_Value"])
    dur = {}
    tpath = os.path.join(d, "trace", "run_kernel_trace.csv")
    if os.path.exists(tpath):
        for r in _csv(tpath):
            dur.setdefault(r["Kernel_Name"], []).append(
                (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)
    med = lambda m, c: statistics.median(m[c].values()) if c in m else float("nan")  # noqa
    rows = []
    for (kname, grid), m in sorted(vals.items(), key=lambda kv: -med(kv[1], "SQ_WAVE_CYCLES")):
        if _logical(kname) == kname and "fno::" not in kname:
            continue
        wc = med(m, "SQ_WAVE_CYCLES")
        util = 100.0 * med(m, "SQ_VALU_MFMA_BUSY_CYCLES") / (
            med(m, "GRBM_GUI_ACTIVE") / XCDS * SIMDS)
        flops = 512.0 * med(m, "SQ_INSTS_VALU_MFMA_MOPS_F16")
        avg = (sum(dur[kname]) / len(dur[kname])) if kname in dur else float("nan")
        tfs = flops / (avg * 1e-6) / 1e12
        short = kname.replace("void ", "").replace("fno::", "").split("(")[0][:48]
        rows.append(
            f"| {short} | {grid} | {avg:.1f} | {util:.1f} | {flops / 1e9:.2f} | {tfs:.0f} | "
            f"{100 * tfs / MFMA_F16_PEAK_TFS:.1f} | {med(m, 'SQ_INSTS_VALU'):.3g} | "
            f"{med(m, 'SQ_INSTS_MFMA'):.3g} | {med(m, 'SQ_INSTS_LDS'):.3g} | "
            f"{med(m, 'SQ_LDS_BANK_CONFLICT'):.3g} | "
            f"{100 * med(m, 'SQ_WAIT_ANY') / wc:.0f} | "
            f"{100 * med(m, 'SQ_ACTIVE_INST_VALU') / wc:.0f} | "
            f"{100 * med(m, 'SQ_ACTIVE_INST_LDS') / wc:.0f} |")
    wk = f"--workload {args.workload} " if args.workload != 3 else ""
    cmd = ("cd /tmp && export TMPDIR=/tmp && rocprofv3 --pmc {c} --output-format csv "
           "-d <out>/{sub} -o run -- python3 /root/repo/bench.py {wk}--steps 2 --warmup 1 "
           "--profile-steps 1 --no-cpu-baseline")
    lines = [f"# SQ and matrix-core counters, workload {wl.name} (fp16+tanh, one step)", "",
             "MI355X, one GPU. Chip-wide counter sums per dispatch, median over the "
             "dispatches of a", "kernel with the same grid. Durations from the kernel "
             "trace of the same sources.", f"Kernel sources hash {kernel_sources_hash()}.", "",
             "Commands:", ""]
    lines += ["    " + cmd.format(c=c, sub=sub, wk=wk) for sub, c in SQ_PASSES.items()]
    lines += ["    (trace: the kernel-trace command of the layer-step summary, same sources)",
              f"    python3 bench.py {wk}--summarize-sq <out>", "",
              "Columns: trace average (us); MFMA busy = SQ_VALU_MFMA_BUSY_CYCLES / "
              "(GRBM_GUI_ACTIVE / 8 XCDs x 1024 SIMDs);", "fp16 MFMA GFLOP per dispatch = 512 x "
              "SQ_INSTS_VALU_MFMA_MOPS_F16, its rate over the trace average and the",
              "fraction of the 2.5 PFLOP/s dense fp16 peak; instruction counts; LDS bank-"
              "conflict cycles;", "wait / VALU-active / LDS-active as % of SQ_WAVE_CYCLES.", "",
              "| kernel | grid | avg us | MFMA busy % | fp16 MFMA GFLOP | TFLOP/s | % of fp16 "
              "peak | VALU insts | MFMA insts | LDS insts | LDS bank confl. | wait % | "
              "VALU % | LDS % |",
              "|---|---|---|---|---|---|---|---|---|---|---|---|---|---|"] + rows
    with open(os.path.join(ROOT, "profiles", f"sq_counters_{wl.name}.md"), "w") as f:
        f.write("\n".join(lines) + "\n")


def main():
    args = parse()
    if args.summarize:
        summarize(args)
        return
    if args.summarize_sq:
        summarize_sq(args)
        return
    if args.gpus != 1:
        print(json.dumps({"error": "this layer runs on one GPU; multi-GPU runs are not "
                                   "supported (the sharding is a documented design only)",
                          "n_gpus": args.gpus}))
        sys.exit(2)
    import torch
    if args.copy_probe:
        copy_probe(torch)
        return
    import synth
    from paper_2307_15034_amd import binding as B
    from paper_2307_15034_amd.layer import SpectralConv

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    wl = synth.WORKLOADS[args.workload]
    npdt = np.float16 if args.precision == "fp16_tanh" else np.float32
    es = 2 if args.precision == "fp16_tanh" else 4
    pc = B.FNO_PREC_FP16_TANH if args.precision == "fp16_tanh" else B.FNO_PREC_FP32
    preact = args.preact if args.preact != "default" else (
        "tanh" if args.precision == "fp16_tanh" else "none")
    pa = {"default": B.FNO_PREACT_DEFAULT, "none": B.FNO_PREACT_NONE,
          "tanh": B.FNO_PREACT_TANH, "clip": B.FNO_PREACT_HARD_CLIP}[args.preact]
    storage = "fp16" if args.precision == "fp16_tanh" else "fp32"
    # the oracle's name of this mode (cpu_baseline leg)
    omode = {"none": storage, "tanh": storage + "_tanh",
             "clip": f"{storage}_clip:{float(np.float32(args.clip))!r}"}[preact]
    kind = {"tucker": B.FNO_WEIGHT_TUCKER, "cp": B.FNO_WEIGHT_CP}.get(wl.weight,
                                                                    B.FNO_WEIGHT_DENSE)
    pol = B.FNO_PATH_MIN_RESULT if args.policy == "min_result" else B.FNO_PATH_MIN_NET
    x = synth.make_x(wl, npdt)
    gy = synth.make_gy(wl, npdt)
    w = synth.make_weight(wl, npdt)
    layer = SpectralConv(wl.n, wl.modes, wl.batch, wl.c_in, wl.c_out, pc, kind, wl.rank, pol,
                         preact=pa, clip=args.clip)
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()  # noqa: E731
    xd, gyd = dev(x), dev(gy)
    wd = ({"core": dev(w["core"]), "u_in": dev(w["u_in"]), "u_out": dev(w["u_out"]),
           "u_mode": [dev(u) for u in w["u_mode"]]} if isinstance(w, dict) else dev(w))
    caches = not args.no_caches
    if args.block:
        from paper_2307_15034_amd.layer import BlockEpilogue
        if caches is False or args.separate_bwd:
            raise SystemExit("--block times the combined backward with the spectral cache")
        epi = BlockEpilogue(wl.n, wl.batch, wl.c_in, wl.c_out, pc, B.FNO_EPI_ACT_GELU,
                            residual=wl.c_in == wl.c_out)
        wsk, bsk = synth.make_block_params(wl, npdt)
        wskd, bskd = dev(wsk), dev(bsk)
        bout = torch.empty((wl.batch, wl.c_out) + wl.n, dtype=layer.dtype, device="cuda")
        bz = torch.empty_like(bout)
        bgz = torch.empty_like(bout)
    xh = layer.spectrum_buffer(0) if caches else None
    gh = layer.spectrum_buffer(1) if caches else None
    y = torch.empty((wl.batch, wl.c_out) + wl.n, dtype=layer.dtype, device="cuda")
    gx = torch.empty((wl.batch, wl.c_in) + wl.n, dtype=layer.dtype, device="cuda")
    gw = layer.alloc_grads()
    stream = torch.cuda.current_stream()
    sh = stream.cuda_stream
    for op in (B.FNO_OP_FWD, B.FNO_OP_BWD_DATA):
        layer.workspace(op)
    layer.workspace(B.FNO_OP_BWD_WEIGHT, caches)
    layer.workspace(B.FNO_OP_BWD, caches)

    def block_step(s):
        # y = K x; out = GELU(W_skip x + b + y) + x; then the backward with
        # g_out = gy: g_z and the skip gradients, K's backward at g_z, and
        # gx = gx_spec + W_skip^T g_z + g_out (in place)
        layer.fwd(xd, wd, y=y, x_hat=xh, stream=s)
        epi.fwd(xd, y, wskd, bskd, out=bout, z_out=bz, stream=s)
        gzz, _, _ = epi.bwd_weight(xd, bz, gyd, g_z=bgz, stream=s)
        layer.bwd(xd, wd, gzz, x_hat=xh, gx=gx, gw=gw, stream=s)
        epi.bwd_data(gzz, wskd, gx, gyd if epi.residual else None, gx=gx, stream=s)

    def step(s=None):
        s = sh if s is None else s
        if args.block:
            block_step(s)
            return
        layer.fwd(xd, wd, y=y, x_hat=xh, stream=s)
        if not args.separate_bwd:
            # data and weight gradient in one call (the layer's backward)
            layer.bwd(xd, wd, gyd, x_hat=xh, gx=gx, gw=gw, stream=s)
            return
        layer.bwd_data(xd, wd, gyd, gx=gx, gy_hat=gh, stream=s)
        if caches:
            layer.bwd_weight(None, None, wd, x_hat=xh, gy_hat=gh, gw=gw, stream=s)
        else:
            layer.bwd_weight(xd, gyd, wd, gw=gw, stream=s)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    graph, per_graph = None, 1
    if not args.no_graph:
        # The step's launches (every kernel of fwd and bwd) captured once in a
        # HIP graph; a timed step is a replay (per_graph steps per replay).
        per_graph = 10 if args.steps % 10 == 0 else 1
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            cs = torch.cuda.current_stream().cuda_stream
            for _ in range(per_graph):
                step(cs)
        torch.cuda.synchronize()
        for _ in range(2):
            graph.replay()
        torch.cuda.synchronize()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    ev0.record(stream)
    if graph is not None:
        for _ in range(args.steps // per_graph):
            graph.replay()
    else:
        for _ in range(args.steps):
            step()
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_step = ev0.elapsed_time(ev1) / args.steps
    value = wl.batch / (ms_step / 1e3)
    sbytes = step_bytes(wl, es, caches, preact)
    if args.block:
        sbytes += sum(block_kernel_bytes(wl, es, epi.residual).values())

    # per-kernel durations: the library brackets each launch with HIP events
    B.fno_profile_reset()
    B.fno_profile_enable(True)
    for _ in range(args.profile_steps):
        step()
    torch.cuda.synchronize()
    prof = B.fno_profile_read()
    B.fno_profile_enable(False)
    B.fno_profile_reset()
    kb = kernel_bytes(wl, es, preact)
    if args.block:
        kb.update(block_kernel_bytes(wl, es, epi.residual))
    kernels = {}
    for name, (n, tot) in prof.items():
        avg = tot / max(n, 1)
        per_step = tot / args.profile_steps
        e = {"launches_per_step": n / args.profile_steps, "avg_ms": avg,
             "ms_per_step": per_step}
        if kb.get(name):
            # kernel_bytes() is per whole batch; a call may split the batch
            # into several launches (halves on two streams)
            per_launch = kb[name] / max(n / args.profile_steps, 1.0)
            e["alg_bytes"] = int(per_launch)
            e["gbs"] = per_launch / (avg / 1e3) / 1e9
        kernels[name] = e
    dom = max(kernels, key=lambda k: kernels[k]["ms_per_step"])
    dk = kernels[dom]
    copy_gbs = copy_bandwidth(torch)
    roof = {"bound": "hbm", "kernel": dom, "achieved": round(dk.get("gbs", 0.0), 1),
            "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(dk.get("gbs", 0.0) / HBM_PEAK_GBS, 4),
            "traffic": measured_traffic(wl.name, dom),
            "avg_ms": round(dk["avg_ms"], 5), "alg_bytes": dk.get("alg_bytes"),
            "copy_gbs": round(copy_gbs, 1),
            "frac_of_copy": round(dk.get("gbs", 0.0) / copy_gbs, 4)}

    out = {
        "metric": METRIC, "value": round(value, 1), "unit": "samples/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_step, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f16" if args.precision == "fp16_tanh" else "f32",
        "data": "synthetic (seeded Gaussian random fields standing in for the paper's PDE "
                "datasets; random-init weights)",
        "config": {"workload": wl.name, "batch": wl.batch, "c_in": wl.c_in, "c_out": wl.c_out,
                   "grid": list(wl.n), "modes": list(wl.modes), "weights": wl.weight,
                   "precision": args.precision, "preactivation": preact,
                   **({"clip": args.clip} if preact == "clip" else {}),
                   "spectral_caches": caches,
                   "backward": "separate" if args.separate_bwd else "combined",
                   "launch": "stream" if args.no_graph else "hip_graph",
                   "path_policy": args.policy if wl.weight != "dense" else None},
        **({"block": {"activation": "gelu", "residual": bool(epi.residual), "bias": True,
                      "note": "whole FNO block: spectral layer + fused skip/GELU/residual "
                              "epilogue, forward and backward"}} if args.block else {}),
        "step_alg_bytes": sbytes,
        "step_hbm_gbs": round(sbytes / (ms_step / 1e3) / 1e9, 1),
        "step_hbm_frac": round(sbytes / (ms_step / 1e3) / 1e9 / HBM_PEAK_GBS, 4),
        "step_copy_frac": round(sbytes / (ms_step / 1e3) / 1e9 / copy_gbs, 4),
        "roofline": roof,
        "kernels": {k: {kk: (round(vv, 5) if isinstance(vv, float) else vv)
                        for kk, vv in v.items()} for k, v in kernels.items()},
        "wall_s_timed": round(wall, 3),
    }
    if args.block:
        out["metric"] = "FNO block fwd+bwd samples/s (fp16+tanh spectral layer, GELU, residual)"
    if not args.no_cpu_baseline and not args.block:
        out["cpu_baseline"] = cpu_baseline(wl, x, w, gy, omode, args.cpu_seconds)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
