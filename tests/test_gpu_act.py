"""Parity of the variant with the input activations inside the kernels (Sec.
input projections, Fig. carve_block: q, k = L2-norm(SiLU(raw)), v = SiLU(raw),
fused into the chunk loads of the forward, the recompute and the adjoint)
through the C ABI, against the CPU oracle (the pinned layer composed with the
pinned activations and their reverse mode).

Bars: f32 inputs max-rel <= 1e-4; bf16 inputs max-rel <= 2e-2, on every output
and gradient tensor (dq, dk, dv are the gradients of the raw projections).
"""
import numpy as np
import pytest
import torch

from oracle import oracle as orc
from paper_2606_27229_amd import carve
from paper_2606_27229_amd.inputs import WORKLOADS, Workload, make_inputs
from tests.gpu_util import host, max_rel, to_gpu

pytestmark = pytest.mark.gpu

TOL = {"f32": 1e-4, "bf16": 2e-2}
GRADS = ("dq", "dk", "dv", "dbeta", "dg", "dbx", "dwx", "dUb", "dUw", "dVb", "dVw", "dS0")


def _w(**kw):
    base = dict(name="act", B=2, H=2, T=64, Dk=32, Dv=32, L=16, R=4, dtype="f32", mu=2.0, s0=0.3, u_std=0.3)
    base.update(kw)
    return Workload(**base)


def _args(x):
    return (x["q"], x["k"], x["v"], x["beta"], x["g"], x["bx"], x["wx"], x["Ub"], x["Uw"], x["Vb"], x["Vw"])


def run_gpu(w, inp, L):
    dt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    x = to_gpu(inp, dt)
    o, S_T, S_chunks = carve.chunk_fwd(*_args(x), x["S0"], L=L, act=True)
    gr = carve.chunk_bwd(*_args(x), S_chunks, x["dO"], x["dS_T"], L=L, act=True)
    torch.cuda.synchronize()
    out = {key: host(val) for key, val in gr.items()}
    out.update({"o": host(o), "S_T": host(S_T), "S_chunks": host(S_chunks)})
    return out


def check(w, inp, L=None):
    L = L or w.L
    tol = TOL[w.dtype]
    ref = dict(orc.fwd_act(inp, L, want_chunks=True))
    ref.update(orc.bwd_act(inp, L, inp["dO"], inp["dS_T"]))
    got = run_gpu(w, inp, L)
    keys = ("o", "S_T", "S_chunks") + GRADS
    for key in keys:
        assert np.all(np.isfinite(got[key])), key
    errs = {key: max_rel(got[key], ref[key]) for key in keys}
    print("max-rel errors:", {key: float("%.3g" % e) for key, e in errs.items()}, flush=True)
    bad = {key: e for key, e in errs.items() if e > tol}
    assert not bad, (bad, errs)


@pytest.mark.parametrize("L", [16, 32])
def test_act_fp32_small(L):
    w = _w(L=L, T=128)
    print(f"case act fp32 D=32 L={L}", flush=True)
    check(w, make_inputs(w, seed=L, dS_T=True, act=True))


def test_act_fp32_d64():
    w = _w(Dk=64, Dv=64, L=32, T=96, R=16, B=3, H=2)
    print("case act fp32 D=64", flush=True)
    check(w, make_inputs(w, seed=5, dS_T=True, act=True))


@pytest.mark.parametrize("L", [16, 64, 128])
def test_act_bf16_d128(L):
    w = _w(Dk=128, Dv=128, L=L, T=256, R=32, dtype="bf16", mu=3.0, s0=0.0, u_std=0.02)
    print(f"case act bf16 D=128 L={L}", flush=True)
    check(w, make_inputs(w, seed=L, act=True))


def test_act_bf16_d128_content_amplified():
    w = _w(Dk=128, Dv=128, L=64, T=192, R=32, dtype="bf16", mu=3.0, s0=0.1, u_std=0.3)
    print("case act bf16 D=128 content-amplified", flush=True)
    check(w, make_inputs(w, seed=9, dS_T=True, act=True))


def test_act_forward_matches_plain_layer_on_activated_inputs():
    """The fused forward equals the plain forward fed the activations formed by
    the oracle in double (rounded to f32)."""
    w = _w(T=64, L=16)
    inp = make_inputs(w, seed=3, act=True)
    x = to_gpu(inp, torch.float32)
    o1, s1, _ = carve.chunk_fwd(*_args(x), x["S0"], L=16, act=True)
    a = orc.act_inputs(inp)
    y = dict(x)
    for key in ("q", "k", "v"):
        y[key] = torch.from_numpy(a[key].astype(np.float32)).cuda()
    o2, s2, _ = carve.chunk_fwd(*_args(y), y["S0"], L=16)
    torch.cuda.synchronize()
    assert max_rel(host(o1), host(o2)) < 1e-5 and max_rel(host(s1), host(s2)) < 1e-5


def test_act_full_size_sampled():
    """At the headline size (B=4 H=16 T=4096 d=128 r=32 L=64, bf16), on sampled
    (batch, head) slices, with the upstream gradients zeroed outside them (the
    sampling of the other full-size parity tests)."""
    w = WORKLOADS["layer_1p3b_T4096"].with_(L=64)
    L = 64
    print(f"case act {w.name} L={L}", flush=True)
    inp = make_inputs(w, seed=11, dS_T=True, act=True)
    samples = [(0, 0), (w.B - 1, w.H - 1)]
    keep = np.zeros((w.B, w.H), dtype=bool)
    for b, h in samples:
        keep[b, h] = True
    inp["dO"] = inp["dO"] * keep[:, None, :, None]
    inp["dS_T"] = inp["dS_T"] * keep[:, :, None, None]
    x = to_gpu(inp, torch.bfloat16)
    o, S_T, S_chunks = carve.chunk_fwd(*_args(x), x["S0"], L=L, act=True)
    gr = carve.chunk_bwd(*_args(x), S_chunks, x["dO"], x["dS_T"], L=L, act=True)
    torch.cuda.synchronize()
    del x
    tok = ("q", "k", "v", "beta", "g", "bx", "wx", "dO")
    ref_params = {key: 0.0 for key in ("dUb", "dUw", "dVb", "dVw")}
    errs = {}
    for b, h in samples:
        s = {}
        for key, val in inp.items():
            if val is None:
                s[key] = None
            elif key in tok:
                s[key] = np.ascontiguousarray(val[b:b + 1, :, h:h + 1])
            elif key in ("S0", "dS_T"):
                s[key] = np.ascontiguousarray(val[b:b + 1, h:h + 1])
            else:
                s[key] = val
        rf = orc.fwd_act(s, L, want_chunks=True)
        rb = orc.bwd_act(s, L, s["dO"], s["dS_T"])
        errs[f"o[{b},{h}]"] = max_rel(host(o[b:b + 1, :, h:h + 1]), rf["o"])
        errs[f"S_chunks[{b},{h}]"] = max_rel(host(S_chunks[b:b + 1, h:h + 1]), rf["S_chunks"])
        for key in ("dq", "dk", "dv", "dbeta", "dg", "dbx", "dwx"):
            errs[f"{key}[{b},{h}]"] = max_rel(host(gr[key][b:b + 1, :, h:h + 1]), rb[key])
        errs[f"dS0[{b},{h}]"] = max_rel(host(gr["dS0"][b:b + 1, h:h + 1]), rb["dS0"])
        for key in ref_params:
            ref_params[key] = ref_params[key] + rb[key]
    for key in ref_params:
        errs[key] = max_rel(host(gr[key]), ref_params[key])
    print("max-rel errors:", {k: float("%.3g" % e) for k, e in errs.items()}, flush=True)
    bad = {k: e for k, e in errs.items() if not e <= 2e-2}
    assert not bad, bad


def test_act_backward_deterministic():
    w = _w(Dk=64, Dv=64, L=32, T=128, R=8, B=3)
    inp = make_inputs(w, seed=2, act=True)
    a = run_gpu(w, inp, 32)
    b = run_gpu(w, inp, 32)
    for key in GRADS:
        assert np.array_equal(a[key], b[key]), key
