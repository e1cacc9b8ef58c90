"""Parity at the full workload sizes, in the launch configuration the benchmark
times (the whole batch and all heads in one call), on sampled (batch, head)
slices.

Every output of a slice (o, S_T, S_chunks and the token gradients, dS0 too)
depends only on that slice's inputs and the shared parameters, so the oracle
runs on the sampled slices alone.  The parameter gradients are sums over all
slices: the upstream gradients dO and dS_T are zeroed outside the sampled
slices, which makes every other slice's contribution exactly zero, so the
full-size parameter gradients of the GPU must equal the oracle's sum over the
sampled slices.

Bar: bf16 inputs with f32 state and accumulation, max-rel <= 2e-2 per tensor.
"""
import numpy as np
import pytest
import torch

from oracle import oracle as orc
from paper_2606_27229_amd import carve
from paper_2606_27229_amd.inputs import CHUNK_SWEEP, WORKLOADS, make_inputs
from tests.gpu_util import host, max_rel, to_gpu

pytestmark = pytest.mark.gpu

TOL = 2e-2
TOKEN_KEYS = ("q", "k", "v", "beta", "g", "bx", "wx", "dO")
TOKEN_GRADS = ("dq", "dk", "dv", "dbeta", "dg", "dbx", "dwx")
PARAM_GRADS = ("dUb", "dUw", "dVb", "dVw")

CASES = [("layer_1p3b_T2048", 64), ("long_seq_T16384", 64)] + [("layer_1p3b_T4096", L) for L in CHUNK_SWEEP]


def _slice(inp, b, h):
    out = {}
    for key, val in inp.items():
        if val is None:
            out[key] = None
        elif key in TOKEN_KEYS:
            out[key] = np.ascontiguousarray(val[b:b + 1, :, h:h + 1])
        elif key in ("S0", "dS_T"):
            out[key] = np.ascontiguousarray(val[b:b + 1, h:h + 1])
        else:
            out[key] = val
    return out


@pytest.mark.parametrize("name,L,u_std", [c + (None,) for c in CASES] + [("layer_1p3b_T4096", 64, 0.3)])
def test_full_size_sampled(name, L, u_std):
    """u_std = 0.3: the content projections at 15x the paper's initialisation
    scale, so that a broken fold or glue shows at the 2e-2 bar."""
    w = WORKLOADS[name].with_(L=L)
    if u_std is not None:
        w = w.with_(u_std=u_std)
    print(f"case {name} L={L}: B={w.B} H={w.H} T={w.T} u_std={w.u_std}", flush=True)
    inp = make_inputs(w, seed=100 + L, dS_T=True)
    samples = [(0, 0), (w.B - 1, w.H - 1)]
    keep = np.zeros((w.B, w.H), dtype=bool)
    for b, h in samples:
        keep[b, h] = True
    inp["dO"] = inp["dO"] * keep[:, None, :, None]
    inp["dS_T"] = inp["dS_T"] * keep[:, :, None, None]

    x = to_gpu(inp, torch.bfloat16)
    o, S_T, S_chunks = carve.chunk_fwd(x["q"], x["k"], x["v"], x["beta"], x["g"], x["bx"], x["wx"], x["Ub"],
                                       x["Uw"], x["Vb"], x["Vw"], x["S0"], L=L)
    gr = carve.chunk_bwd(x["q"], x["k"], x["v"], x["beta"], x["g"], x["bx"], x["wx"], x["Ub"], x["Uw"],
                         x["Vb"], x["Vw"], S_chunks, x["dO"], x["dS_T"], L=L)
    torch.cuda.synchronize()
    del x

    ref_params = {key: 0.0 for key in PARAM_GRADS}
    errs = {}
    for b, h in samples:
        s = _slice(inp, b, h)
        rf = orc.fwd_serial(s, L, want_chunks=True)
        rb = orc.bwd(s, L, s["dO"], s["dS_T"])
        got = {"o": host(o[b:b + 1, :, h:h + 1]), "S_T": host(S_T[b:b + 1, h:h + 1]),
               "S_chunks": host(S_chunks[b:b + 1, h:h + 1])}
        for key in ("o", "S_T", "S_chunks"):
            errs[f"{key}[{b},{h}]"] = max_rel(got[key], rf[key])
        for key in TOKEN_GRADS:
            g_ = host(gr[key][b:b + 1, :, h:h + 1])
            errs[f"{key}[{b},{h}]"] = max_rel(g_, rb[key])
        errs[f"dS0[{b},{h}]"] = max_rel(host(gr["dS0"][b:b + 1, h:h + 1]), rb["dS0"])
        for key in PARAM_GRADS:
            ref_params[key] = ref_params[key] + rb[key]
    for key in PARAM_GRADS:
        errs[key] = max_rel(host(gr[key]), ref_params[key])
    print("max-rel errors:", {k: float("%.3g" % e) for k, e in errs.items()}, flush=True)
    bad = {k: e for k, e in errs.items() if not e <= TOL}
    assert not bad, bad


def test_full_size_gated_sampled():
    """The gate-in-kernel variant at the headline size (B=4 H=16 T=4096 L=64):
    sampled slices as above; dA and dtau of a head are sums over that head's
    slices, so with the upstream gradients zeroed outside the samples the
    sampled heads' rows must equal the slices' oracle rows and every other
    head's rows must be zero."""
    w = WORKLOADS["layer_1p3b_T4096"].with_(L=64)
    L = 64
    print(f"case gated {w.name} L={L}", flush=True)
    inp = make_inputs(w, seed=7, dS_T=True, gated=True)
    samples = [(0, 0), (w.B - 1, w.H - 1)]
    keep = np.zeros((w.B, w.H), dtype=bool)
    for b, h in samples:
        keep[b, h] = True
    inp["dO"] = inp["dO"] * keep[:, None, :, None]
    inp["dS_T"] = inp["dS_T"] * keep[:, :, None, None]
    x = to_gpu(inp, torch.bfloat16)
    args = (x["q"], x["k"], x["v"], x["beta"], x["f"], x["A"], x["tau_f"], x["bx"], x["wx"],
            x["Ub"], x["Uw"], x["Vb"], x["Vw"])
    o, S_T, S_chunks = carve.chunk_fwd_gated(*args, x["S0"], L=L)
    gr = carve.chunk_bwd_gated(*args, S_chunks, x["dO"], x["dS_T"], L=L)
    torch.cuda.synchronize()
    del x
    errs = {}
    dA, dtau = host(gr["dA"]), host(gr["dtau"])
    for b, h in samples:
        s = {}
        for key, val in inp.items():
            if val is None:
                s[key] = None
            elif key in TOKEN_KEYS + ("f",):
                s[key] = np.ascontiguousarray(val[b:b + 1, :, h:h + 1])
            elif key in ("S0", "dS_T"):
                s[key] = np.ascontiguousarray(val[b:b + 1, h:h + 1])
            elif key in ("A", "tau_f"):
                s[key] = np.ascontiguousarray(val[h:h + 1])
            else:
                s[key] = val
        rf = orc.fwd_gated(s, L, want_chunks=True)
        rb = orc.bwd_gated(s, L, s["dO"], s["dS_T"])
        errs[f"o[{b},{h}]"] = max_rel(host(o[b:b + 1, :, h:h + 1]), rf["o"])
        errs[f"S_chunks[{b},{h}]"] = max_rel(host(S_chunks[b:b + 1, h:h + 1]), rf["S_chunks"])
        for key in ("dq", "dk", "dv", "dbeta", "df", "dbx", "dwx"):
            errs[f"{key}[{b},{h}]"] = max_rel(host(gr[key][b:b + 1, :, h:h + 1]), rb[key])
        errs[f"dA[{h}]"] = max_rel(dA[h:h + 1], rb["dA"])
        errs[f"dtau[{h}]"] = max_rel(dtau[h:h + 1], rb["dtau"])
    others = [h for h in range(w.H) if h not in (0, w.H - 1)]
    assert np.all(dA[others] == 0) and np.all(dtau[others] == 0)
    print("max-rel errors:", {k: float("%.3g" % e) for k, e in errs.items()}, flush=True)
    bad = {k: e for k, e in errs.items() if not e <= TOL}
    assert not bad, bad


def test_full_size_scalar_write_sampled():
    """The scalar-write-gate variant at the headline size (B=4 H=16 T=4096
    L=64), sampled slices as above (dwx is one value per token and head)."""
    w = WORKLOADS["layer_1p3b_T4096"].with_(L=64)
    L = 64
    print(f"case scalar write {w.name} L={L}", flush=True)
    inp = make_inputs(w, seed=8, dS_T=True, scalar_write=True)
    samples = [(0, 0), (w.B - 1, w.H - 1)]
    keep = np.zeros((w.B, w.H), dtype=bool)
    for b, h in samples:
        keep[b, h] = True
    inp["dO"] = inp["dO"] * keep[:, None, :, None]
    inp["dS_T"] = inp["dS_T"] * keep[:, :, None, None]
    x = to_gpu(inp, torch.bfloat16)
    args = (x["q"], x["k"], x["v"], x["beta"], x["bx"], x["wx"], x["Ub"], x["Vb"])
    o, S_T, S_chunks = carve.chunk_fwd_sw(*args, x["S0"], L=L, g=x["g"])
    gr = carve.chunk_bwd_sw(*args, S_chunks, x["dO"], x["dS_T"], L=L, g=x["g"])
    torch.cuda.synchronize()
    del x
    ref_params = {"dUb": 0.0, "dVb": 0.0}
    errs = {}
    for b, h in samples:
        s = _slice(inp, b, h)
        rf = orc.fwd_sw(s, L, want_chunks=True)
        rb = orc.bwd_sw(s, L, s["dO"], s["dS_T"])
        errs[f"o[{b},{h}]"] = max_rel(host(o[b:b + 1, :, h:h + 1]), rf["o"])
        errs[f"S_T[{b},{h}]"] = max_rel(host(S_T[b:b + 1, h:h + 1]), rf["S_T"])
        errs[f"S_chunks[{b},{h}]"] = max_rel(host(S_chunks[b:b + 1, h:h + 1]), rf["S_chunks"])
        for key in TOKEN_GRADS:
            errs[f"{key}[{b},{h}]"] = max_rel(host(gr[key][b:b + 1, :, h:h + 1]), rb[key])
        errs[f"dS0[{b},{h}]"] = max_rel(host(gr["dS0"][b:b + 1, h:h + 1]), rb["dS0"])
        for key in ref_params:
            ref_params[key] = ref_params[key] + rb[key]
    for key in ref_params:
        errs[key] = max_rel(host(gr[key]), ref_params[key])
    print("max-rel errors:", {k: float("%.3g" % e) for k, e in errs.items()}, flush=True)
    bad = {k: e for k, e in errs.items() if not e <= TOL}
    assert not bad, bad
