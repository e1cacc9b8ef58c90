#!/usr/bin/env python3
"""Benchmark: chunked CARVE layer forward + backward on one MI355X.

One step = carve_chunk_fwd + carve_chunk_bwd over one batch of the 1.3B-scale
layer (B=4, H=16, T=4096, d_k=d_v=128, r=32, L=64, bf16 token tensors, f32
state and accumulation), inputs already resident in HBM.  Prints ONE JSON
line with tokens/s, the roofline of the dominant kernel and the CPU oracle
timed on a bounded sample of the same workload.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--L 64]
(defaults: 50 timed steps after 10 warm-up steps; the reported step time is
the median of the steps' HIP-event times)
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "layer fwd+bwd tokens/s, H=16 d=128 T=4096 L=64 bf16; % MFMA peak"
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
BF16_PEAK_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
KERNEL_SOURCES = tuple("paper_2606_27229_amd/csrc/" + f for f in (
    "carve_fwd_chain.h", "carve_fwd_chain.hip", "carve_rec.h", "carve_bwd.h", "carve_bwd.hip", "carve_dev.h",
    "carve_kernels.h", "carve_param.h", "carve_variant.hip"))
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_layer_1p3b_T4096_L64.json")


def algorithmic_counts(B, T, H, d, R, L, gated=False, sw=False):
    """Algorithmic bytes and flops per call (every input and output once).

    Bytes per token-head (bf16 token tensors, f32 g and states):
      forward kernel   reads q, k, v (3*2d) + g (4d) + bx, wx (2*2d) + beta (2);
                       writes o (2d) + chunk-start states (4 d^2 / L)
      adjoint          reads the forward inputs + dO (2d); writes dq, dk, dv
                       (3*2d) + dg (4d) + dbx, dwx (2*2d) + dbeta (2)
      backward         the adjoint's bytes + the chunk-start states it needs
                       (4 d^2 / L, read by the recompute); the fused
                       recompute + adjoint kernel is priced at this figure
    With the gate-in-kernel decay the f32 g (4d) is replaced by the bf16 logit
    f (2d) and dg by df (2d); A, tau_f and dA, dtau are per head (negligible).
    With the scalar write gate wx and dwx are one bf16 value per token-head (2
    each instead of 2d) and the fold and the content projection lose their
    write half.
    Flops per token-head (multiply-add = 2): forward
      2 * (2 r d^2 / L + 3 d^2 + 4 r d + 5/2 L d + L^2 / 6)
      (r d^2 / L and 2 r d with the scalar write gate), backward 2x forward.
    """
    th = B * T * H
    decay = 2 * d if gated else 4 * d
    wxb = 2 if sw else 2 * d
    inputs = 3 * 2 * d + decay + 2 * d + wxb + 2
    grads = 3 * 2 * d + decay + 2 * d + wxb + 2
    states = 4 * d * d / L
    rf = 1 if sw else 2       # fold rows per rank unit
    fwd_mac = rf * R * d * d / L + 3 * d * d + 2 * rf * R * d + 2.5 * L * d + L * L / 6.0
    return {
        "fwd_bytes": (inputs + 2 * d + states) * th,
        "adjoint_bytes": (inputs + 2 * d + grads) * th,
        "bwd_bytes": (inputs + 2 * d + grads + states) * th,
        "fwd_flops": 2 * fwd_mac * th, "bwd_flops": 4 * fwd_mac * th,
    }


def kernel_source_hash():
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def load_traffic(kernel):
    """HBM bytes per launch measured with rocprofv3 counters, if they were taken
    on the current kernel sources; None otherwise."""
    try:
        with open(TRAFFIC_FILE) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    if rec.get("source_hash") != kernel_source_hash():
        return None
    k = rec.get("kernels", {}).get(kernel)
    return None if k is None else k.get("hbm_bytes_per_launch")


TRAFFIC_KERNELS = {"carve_chain_fwd_kernel": "carve_chain_fwd_kernel", "carve_bwd_fused_kernel": "carve_bwd_fused_kernel"}


def _pmc_per_dispatch(run_dir, counter):
    """{kernel name: [counter value per dispatch]} from a rocprofv3 --pmc csv run."""
    import csv
    import glob
    vals = {}
    for path in glob.glob(os.path.join(run_dir, "**", "*counter_collection.csv"), recursive=True):
        with open(path) as f:
            for row in csv.DictReader(f):
                if row["Counter_Name"] != counter:
                    continue
                key = (row["Kernel_Name"], row["Dispatch_Id"])
                vals[key] = vals.get(key, 0.0) + float(row["Counter_Value"])
    out = {}
    for (name, _), v in vals.items():
        out.setdefault(name, []).append(v)
    return out


def traffic_summary(fetch_dir, write_dir, copy_fetch_dir, copy_write_dir):
    """Scale the FETCH_SIZE / WRITE_SIZE counters (KiB per dispatch) by what they
    read for a plain copy of known size and write the per-launch HBM traffic of
    the headline kernels to TRAFFIC_FILE, tagged with the kernel-source hash."""
    n_copy = 1 << 30

    def copy_factor(d, counter):
        per = _pmc_per_dispatch(d, counter)
        big = max((sum(v) / len(v), name) for name, v in per.items())
        return n_copy / (big[0] * 1024.0), big[1]

    ff, copy_name = copy_factor(copy_fetch_dir, "FETCH_SIZE")
    wf, _ = copy_factor(copy_write_dir, "WRITE_SIZE")
    fetch = _pmc_per_dispatch(fetch_dir, "FETCH_SIZE")
    write = _pmc_per_dispatch(write_dir, "WRITE_SIZE")
    rec = {"source_hash": kernel_source_hash(), "copy_kernel": copy_name,
           "fetch_factor": ff, "write_factor": wf, "kernels": {}}
    for key, pat in TRAFFIC_KERNELS.items():
        fv = [v for name, vs in fetch.items() if pat in name for v in vs]
        wv = [v for name, vs in write.items() if pat in name for v in vs]
        if not fv or not wv:
            continue
        fb = sum(fv) / len(fv) * 1024.0 * ff
        wb = sum(wv) / len(wv) * 1024.0 * wf
        rec["kernels"][key] = {"fetch_bytes_per_launch": fb, "write_bytes_per_launch": wb,
                               "hbm_bytes_per_launch": fb + wb, "dispatches": len(fv)}
    with open(TRAFFIC_FILE, "w") as f:
        json.dump(rec, f, indent=1)
    print(json.dumps(rec), flush=True)


def counter_summary(run_dirs):
    """Per-kernel averages of every counter in rocprofv3 --pmc csv runs (one line
    of JSON per kernel): the value per dispatch, the number of dispatches and,
    where the csv carries timestamps, the average dispatch duration in us."""
    import csv
    import glob
    acc = {}
    for run_dir in run_dirs:
        for path in glob.glob(os.path.join(run_dir, "**", "*counter_collection.csv"), recursive=True):
            with open(path) as f:
                for row in csv.DictReader(f):
                    k = acc.setdefault(row["Kernel_Name"], {"dispatch": {}, "grid": row.get("Grid_Size")})
                    d = k["dispatch"].setdefault((run_dir, row["Dispatch_Id"]), {})
                    d[row["Counter_Name"]] = d.get(row["Counter_Name"], 0.0) + float(row["Counter_Value"])
                    if row.get("Start_Timestamp") and row.get("End_Timestamp"):
                        d["_us"] = (int(row["End_Timestamp"]) - int(row["Start_Timestamp"])) * 1e-3
    for name, k in sorted(acc.items()):
        per = {}
        for d in k["dispatch"].values():
            for c, v in d.items():
                per.setdefault(c, []).append(v)
        out = {c: sum(v) / len(v) for c, v in per.items()}
        rec = {"kernel": name, "grid": k["grid"], "dispatches": len(k["dispatch"]),
               "duration_us": out.pop("_us", None), "counters": out}
        print(json.dumps(rec), flush=True)


def host_cpu():
    """(cores of the host, cores this process may run on, CPU share of its
    cgroup or None, CPU model) for the CPU baseline's record."""
    host = os.cpu_count() or 1
    try:
        usable = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        usable = host
    share = None
    try:
        with open("/sys/fs/cgroup/cpu.max") as f:
            quota, period = f.read().split()[:2]
        if quota != "max":
            share = max(1, int(int(quota) // int(period)))
    except (OSError, ValueError):
        pass
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return host, usable, share, model


def cpu_baseline(w, L, seed, target_s=12.0, gated=False, sw=False, act=False):
    """Time the CPU oracle (token-serial forward + exact backward, double) on the
    whole workload batch, repeated until about target_s seconds of CPU work.
    One host thread per (batch, head) chain, up to the cores this process may
    use (its affinity set, and its cgroup's CPU share where one is set)."""
    from oracle import oracle as orc
    from paper_2606_27229_amd.inputs import make_inputs

    inp = make_inputs(w, seed=seed, gated=gated, scalar_write=sw, act=act)
    host, usable, share, model = host_cpu()
    avail = min(usable, share) if share else usable
    threads = max(1, min(avail, w.B * w.H))
    if act:
        fwd, bwd = orc.fwd_act, orc.bwd_act
    elif sw:
        fwd, bwd = orc.fwd_sw, orc.bwd_sw
    else:
        fwd = orc.fwd_gated if gated else orc.fwd_serial
        bwd = orc.bwd_gated if gated else orc.bwd
    reps, t_f, t_b = 0, 0.0, 0.0
    while reps == 0 or t_f + t_b < target_s:
        t0 = time.perf_counter()
        fwd(inp, L, nthreads=threads)
        t1 = time.perf_counter()
        bwd(inp, L, inp["dO"], None, nthreads=threads)
        t2 = time.perf_counter()
        t_f += t1 - t0
        t_b += t2 - t1
        reps += 1
    tokens = reps * w.B * w.T   # layer tokens (all heads) processed
    return {"value": tokens / (t_f + t_b), "unit": "tokens/s", "cores": host, "threads": threads,
            "usable_cores": usable, "cgroup_cpu_share": share, "cpu_model": model, "kind": "oracle",
            "sample": f"{reps} x the whole batch (B={w.B}, H={w.H}, T={w.T}, L={L}): token-serial forward + "
                      f"exact reverse-mode backward in double, one thread per (batch, head) chain on "
                      f"{threads} threads (host {host} cores, {usable} usable"
                      + (f", cgroup share {share}" if share else "") + f"; {model}), "
                      f"fwd {t_f:.1f} s, bwd {t_b:.1f} s"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--L", type=int, default=64)
    ap.add_argument("--workload", default=None,
                    help="another bf16 workload of the layer to time (e.g. layer_1p3b_T2048, long_seq_T16384); "
                         "the default is the headline layer_1p3b_T4096")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--gated", action="store_true",
                    help="the gate-in-kernel variant: the decay is formed in the kernels from its raw "
                         "logit f (bf16) and per-head A, tau_f (carve_chunk_fwd_gated / _bwd_gated)")
    ap.add_argument("--act", action="store_true",
                    help="the input activations inside the kernels: q, k, v are the raw projections "
                         "(SiLU, then L2 norm for q, k; carve_chunk_fwd_act / _bwd_act)")
    ap.add_argument("--scalar-write", action="store_true",
                    help="the scalar write gate: one write logit per token and head, no write-side "
                         "content (carve_chunk_fwd_sw / _bwd_sw; with --gated, the decay from f)")
    ap.add_argument("--rmsnorm", action="store_true",
                    help="also run the output RMS normalisation of the layer (carve_rmsnorm_fwd after the "
                         "forward, carve_rmsnorm_bwd before the backward, whose d_o is the layer's dO) inside "
                         "every timed step, and report its kernels next to the layer's")
    ap.add_argument("--traffic-summary", nargs=4, metavar=("FETCH_DIR", "WRITE_DIR", "COPY_FETCH_DIR", "COPY_WRITE_DIR"),
                    help="turn rocprofv3 --pmc FETCH_SIZE / WRITE_SIZE runs of this benchmark and of "
                         "--copy-calibration into the traffic record read by the roofline (no GPU needed)")
    ap.add_argument("--counter-summary", nargs="+", metavar="PMC_DIR",
                    help="print per-kernel averages of the counters in rocprofv3 --pmc csv runs (no GPU needed)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain elementwise copy of 1 GiB (reads 1 GiB, writes 1 GiB) "
                         "five times: the reference kernel for scaling the HBM byte counters")
    args = ap.parse_args()
    if args.traffic_summary:
        traffic_summary(*args.traffic_summary)
        return
    if args.counter_summary:
        counter_summary(args.counter_summary)
        return
    if args.gpus != 1:
        print("bench.py measures one GPU: the layer shards over (batch, head) with no exchange "
              "except a 64 KB parameter-gradient all-reduce, which this benchmark does not run; "
              "use --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2606_27229_amd import carve
    from paper_2606_27229_amd.inputs import HEADLINE, WORKLOADS, make_inputs

    if args.copy_calibration:
        n = 1 << 30
        src = torch.ones(n // 4, dtype=torch.float32, device="cuda:0")
        dst = torch.empty_like(src)
        for _ in range(5):
            torch.mul(src, 1.0, out=dst)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration": {"read_bytes": n, "write_bytes": n, "launches": 5}}), flush=True)
        return

    name = args.workload or HEADLINE
    if name not in WORKLOADS or WORKLOADS[name].dtype != "bf16" or not WORKLOADS[name].backward:
        print(f"--workload must be one of the bf16 training workloads, got {name}", file=sys.stderr)
        sys.exit(2)
    w = WORKLOADS[name].with_(L=args.L)
    L = w.L
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    gated, sw, act = args.gated, args.scalar_write, args.act
    if act and (gated or sw):
        print("--act runs with the default decay and write gate only", file=sys.stderr)
        sys.exit(2)
    inp = make_inputs(w, seed=4, gated=gated, scalar_write=sw, act=act)
    x = {}
    for key, val in inp.items():
        if val is None:
            x[key] = None
            continue
        t = torch.from_numpy(np.ascontiguousarray(val))
        if key not in ("g", "A", "tau_f", "Ub", "Uw", "Vb", "Vw", "S0", "dS_T"):
            t = t.to(torch.bfloat16)
        x[key] = t.to(dev)
    B, T, H, d, R = w.B, w.T, w.H, w.Dk, w.R
    f32, bf = torch.float32, torch.bfloat16
    fwd_out = {"o": torch.empty((B, T, H, d), dtype=bf, device=dev),
               "S_T": torch.empty((B, H, d, d), dtype=f32, device=dev),
               "S_chunks": torch.empty((B, H, T // L, d, d), dtype=f32, device=dev)}
    bwd_out = {"dq": torch.empty((B, T, H, d), dtype=bf, device=dev),
               "dk": torch.empty((B, T, H, d), dtype=bf, device=dev),
               "dv": torch.empty((B, T, H, d), dtype=bf, device=dev),
               "dbeta": torch.empty((B, T, H), dtype=bf, device=dev),
               "dg": torch.empty((B, T, H, d), dtype=f32, device=dev),
               "dbx": torch.empty((B, T, H, d), dtype=bf, device=dev),
               "dwx": torch.empty((B, T, H, d), dtype=bf, device=dev),
               "dUb": torch.empty((R, d), dtype=f32, device=dev), "dUw": torch.empty((R, d), dtype=f32, device=dev),
               "dVb": torch.empty((d, R), dtype=f32, device=dev), "dVw": torch.empty((d, R), dtype=f32, device=dev),
               "dS0": torch.empty((B, H, d, d), dtype=f32, device=dev)}
    if gated:
        del bwd_out["dg"]
        bwd_out.update({"df": torch.empty((B, T, H, d), dtype=bf, device=dev),
                        "dA": torch.empty((H, d), dtype=f32, device=dev),
                        "dtau": torch.empty((H, d), dtype=f32, device=dev)})
    if sw:
        del bwd_out["dUw"], bwd_out["dVw"]
        bwd_out["dwx"] = torch.empty((B, T, H), dtype=bf, device=dev)
    decay = dict(f=x["f"], A=x["A"], tau_f=x["tau_f"]) if gated else dict(g=x["g"])
    dims = carve.make_dims(B, T, H, d, d, R, L, bf)
    ws = torch.empty(max(carve.workspace_size(dims, True), 16), dtype=torch.uint8, device=dev)

    norm = args.rmsnorm
    if norm:
        nw = torch.from_numpy((1.0 + 0.1 * np.random.default_rng(5).standard_normal(H * d)).astype(np.float32)).to(dev)
        norm_y = torch.empty((B, T, H, d), dtype=bf, device=dev)
        norm_out = {"d_o": torch.empty((B, T, H, d), dtype=bf, device=dev),
                    "dweight": torch.empty((H * d,), dtype=f32, device=dev)}
        norm_ws = torch.empty(max(int(carve.load_library().carve_rmsnorm_workspace_size(
            carve.ctypes.byref(carve.make_dims(B, T, H, d, d, R, L, bf)))), 16), dtype=torch.uint8, device=dev)
        norm_dy = x["dO"]       # upstream gradient of y; the norm's d_o feeds the layer backward
        layer_dO = norm_out["d_o"]
    else:
        layer_dO = x["dO"]
    ev_nf = ev_nb = None
    cur = {"s": 0}

    def fwd():
        _fwd_layer()
        if norm:
            if ev_nf is not None:
                carve.profile_events(ev_nf[cur["s"]])
            carve.rmsnorm_fwd(fwd_out["o"], nw, out=norm_y)

    def bwd():
        if norm:
            if ev_nb is not None:
                carve.profile_events(ev_nb[cur["s"]])
            carve.rmsnorm_bwd(fwd_out["o"], nw, norm_dy, out=norm_out, workspace=norm_ws)
            if ev_b_armed[0] is not None:
                carve.profile_events(ev_b_armed[0])
        _bwd_layer()

    ev_b_armed = [None]

    def _fwd_layer():
        if sw:
            carve.chunk_fwd_sw(x["q"], x["k"], x["v"], x["beta"], x["bx"], x["wx"], x["Ub"], x["Vb"], x["S0"],
                               L=L, out=fwd_out, **decay)
        elif gated:
            carve.chunk_fwd_gated(x["q"], x["k"], x["v"], x["beta"], x["f"], x["A"], x["tau_f"], x["bx"], x["wx"],
                                  x["Ub"], x["Uw"], x["Vb"], x["Vw"], x["S0"], L=L, out=fwd_out)
        else:
            carve.chunk_fwd(x["q"], x["k"], x["v"], x["beta"], x["g"], x["bx"], x["wx"], x["Ub"], x["Uw"],
                            x["Vb"], x["Vw"], x["S0"], L=L, out=fwd_out, act=act)

    def _bwd_layer():
        if sw:
            carve.chunk_bwd_sw(x["q"], x["k"], x["v"], x["beta"], x["bx"], x["wx"], x["Ub"], x["Vb"],
                               fwd_out["S_chunks"], layer_dO, None, L=L, out=bwd_out, workspace=ws, **decay)
        elif gated:
            carve.chunk_bwd_gated(x["q"], x["k"], x["v"], x["beta"], x["f"], x["A"], x["tau_f"], x["bx"], x["wx"],
                                  x["Ub"], x["Uw"], x["Vb"], x["Vw"], fwd_out["S_chunks"], layer_dO, None, L=L,
                                  out=bwd_out, workspace=ws)
        else:
            carve.chunk_bwd(x["q"], x["k"], x["v"], x["beta"], x["g"], x["bx"], x["wx"], x["Ub"], x["Uw"],
                            x["Vb"], x["Vw"], fwd_out["S_chunks"], layer_dO, None, L=L, out=bwd_out,
                            workspace=ws, act=act)

    for _ in range(args.warmup):
        fwd()
        bwd()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    # launch-boundary events recorded by the library: forward 1 kernel, backward 4
    # (5 with the gate-in-kernel decay: the reduction of dA, dtau; or with the
    # input activations: their backward)
    NF, NB = 2, (6 if (gated or act) else 5)
    ev_f = [[torch.cuda.Event(enable_timing=True) for _ in range(NF)] for _ in range(args.steps)]
    ev_b = [[torch.cuda.Event(enable_timing=True) for _ in range(NB)] for _ in range(args.steps)]
    if norm:
        ev_nf = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(args.steps)]
        ev_nb = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    for e in [x for row in ev_f + ev_b + (ev_nf or []) + (ev_nb or []) for x in row]:
        e.record(stream)            # create the device events up front
    torch.cuda.synchronize()
    # a step: [forward layer, norm forward] then [norm backward, backward layer];
    # the step's time runs from ev_f[s][0] to ev_b[s][-1] (with the norm, the
    # layer backward's events are armed inside bwd(), after the norm backward)
    t0 = time.perf_counter()
    for s_ in range(args.steps):
        cur["s"] = s_
        carve.profile_events(ev_f[s_])
        fwd()
        if norm:
            ev_b_armed[0] = ev_b[s_]
        else:
            carve.profile_events(ev_b[s_])
        bwd()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    wall_ms_per_step = wall * 1e3 / args.steps
    # a step's time: from the event before its forward's first launch to the
    # event after its backward's last launch (the steps run back to back on
    # one stream); the headline is the median over the timed steps
    step_ms = sorted(ev_f[s_][0].elapsed_time(ev_b[s_][NB - 1]) for s_ in range(args.steps))
    ms_per_step = (step_ms[(args.steps - 1) // 2] + step_ms[args.steps // 2]) / 2

    def avg(rows, i):
        return sum(r[i].elapsed_time(r[i + 1]) for r in rows) / len(rows)

    bwd_names = ["carve_sync_clear_kernel", "carve_bwd_fused_kernel", "carve_bwd_param_kernel",
                 "carve_param_reduce_kernel"]
    if gated:
        bwd_names.append("carve_gate_reduce_kernel")
    if act:
        bwd_names.append("carve_act_bwd_kernel")
    kernels_ms = {"carve_chain_fwd_kernel": avg(ev_f, 0)}
    for i, kname in enumerate(bwd_names):
        kernels_ms[kname] = avg(ev_b, i)
    if norm:
        kernels_ms["carve_rmsnorm_fwd_kernel"] = avg(ev_nf, 0)
        kernels_ms["carve_rmsnorm_bwd_kernel"] = avg(ev_nb, 0)
        kernels_ms["carve_rmsnorm_reduce_kernel"] = avg(ev_nb, 1)
    fwd_ms = kernels_ms["carve_chain_fwd_kernel"]
    bwd_ms = sum(r[0].elapsed_time(r[NB - 1]) for r in ev_b) / args.steps
    tokens = B * T
    cnt = algorithmic_counts(B, T, H, d, R, L, gated, sw)

    alg = {"carve_chain_fwd_kernel": cnt["fwd_bytes"], "carve_bwd_fused_kernel": cnt["bwd_bytes"]}
    dominant = max(alg, key=lambda k_: kernels_ms[k_])
    dom_ms = kernels_ms[dominant]
    dom_bytes = alg[dominant]
    achieved = dom_bytes / (dom_ms * 1e-3) / 1e9
    dom_flops = cnt["fwd_flops"] if dominant == "carve_chain_fwd_kernel" else cnt["bwd_flops"]
    dom_mfma_frac = dom_flops / (dom_ms * 1e-3) / 1e12 / BF16_PEAK_TFLOPS
    # the roofline that binds the kernel's algorithmic counts (bytes / HBM peak
    # against flops / MFMA peak); "limiter" says what the measured fractions
    # show when both are far below 1
    bound = "hbm" if dom_bytes / (HBM_PEAK_GBS * 1e9) >= dom_flops / (BF16_PEAK_TFLOPS * 1e12) else "mfma"
    limiter = bound if max(achieved / HBM_PEAK_GBS, dom_mfma_frac) >= 0.5 else \
        "latency: a dependent chain per (batch, head), far below both rooflines"
    # the counters were taken on the default variant
    traffic = None if (gated or sw or act or name != HEADLINE or L != 64) else load_traffic(dominant)
    layer_tflops = (cnt["fwd_flops"] + cnt["bwd_flops"]) / (ms_per_step * 1e-3) / 1e12
    # achievable HBM bandwidth on this device, for context: a plain 1 GiB
    # device copy (reads 1 GiB, writes 1 GiB), timed after the measured steps
    csrc_ = torch.ones(1 << 28, dtype=torch.float32, device=dev)
    cdst_ = torch.empty_like(csrc_)
    cdst_.copy_(csrc_)
    c0_, c1_ = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    c0_.record(stream)
    for _ in range(5):
        cdst_.copy_(csrc_)
    c1_.record(stream)
    torch.cuda.synchronize()
    copy_gbs = 5 * 2 * (1 << 30) / (c0_.elapsed_time(c1_) * 1e-3) / 1e9
    del csrc_, cdst_
    res = {
        "metric": METRIC if (name == HEADLINE and L == 64) else
                  f"layer fwd+bwd tokens/s, H={H} d={d} T={T} L={L} bf16; % MFMA peak",
        "value": tokens / (ms_per_step * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "ms_per_step_wall": wall_ms_per_step,
        "step_ms_min_max": [step_ms[0], step_ms[-1]],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": w.name, "B": B, "H": H, "T": T, "Dk": d, "Dv": d, "R": R, "L": L,
                   "token_dtype": "bf16", "state_dtype": "f32",
                   "decay": "formed in the kernels from f, A, tau_f" if gated else "g input (f32)",
                   "write_gate": "scalar per token and head" if sw else "per value channel, content-aware",
                   "qkv": "raw projections, activations in the kernels" if act else "activated inputs",
                   "output_norm": "RMSNorm over the H*Dv values of a token (fwd and bwd in every step)"
                                  if norm else "none (the layer's o)"},
        "roofline": {"bound": bound, "kernel": dominant,
                     "achieved": achieved if bound == "hbm" else dom_mfma_frac * BF16_PEAK_TFLOPS,
                     "peak": HBM_PEAK_GBS if bound == "hbm" else BF16_PEAK_TFLOPS,
                     "unit": "GB/s" if bound == "hbm" else "TFLOP/s",
                     "frac": achieved / HBM_PEAK_GBS if bound == "hbm" else dom_mfma_frac,
                     "traffic": None if traffic is None else traffic / (dom_ms * 1e-3) / 1e9,
                     "traffic_bytes_per_launch": traffic,
                     "algorithmic_bytes_per_launch": dom_bytes, "avg_launch_ms": dom_ms,
                     "mfma_frac": dom_mfma_frac, "limiter": limiter},
        "kernels_ms": kernels_ms,
        "fwd_call_ms": fwd_ms,
        "bwd_call_ms": bwd_ms,
        "layer_hbm_frac": (cnt["fwd_bytes"] + cnt["bwd_bytes"]) / (ms_per_step * 1e-3) / 1e9 / HBM_PEAK_GBS,
        "mfma_peak_frac": layer_tflops / BF16_PEAK_TFLOPS,
        "layer_tflops": layer_tflops,
        "hbm_copy_gbs": copy_gbs,
    }
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(w, L, seed=4, gated=gated, sw=sw, act=act)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
