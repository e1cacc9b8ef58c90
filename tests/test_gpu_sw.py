"""Parity of the scalar-write-gate variant (Sec. scalar write gate: one write
logit per token and head, w = sigmoid(wx) on every value channel, no write-side
content; fold over Ub only) through the C ABI, against the CPU oracle (the
pinned layer composed with the broadcast write logit, its reverse mode summing
dwx over the value channels).  The decay is given as g or, with the
gate-in-kernel option, formed from f, A, tau_f.

Bars: f32 inputs max-rel <= 1e-4; bf16 inputs max-rel <= 2e-2, on every output
and gradient tensor.
"""
import numpy as np
import pytest
import torch

from oracle import oracle as orc
from paper_2606_27229_amd import carve
from paper_2606_27229_amd.inputs import Workload, make_inputs
from tests.gpu_util import host, max_rel, to_gpu

pytestmark = pytest.mark.gpu

TOL = {"f32": 1e-4, "bf16": 2e-2}


def _w(**kw):
    base = dict(name="sw", B=2, H=2, T=64, Dk=32, Dv=32, L=16, R=4, dtype="f32", mu=2.0, s0=0.3, u_std=0.3)
    base.update(kw)
    return Workload(**base)


def _grads(gated):
    dec = ("df", "dA", "dtau") if gated else ("dg",)
    return ("dq", "dk", "dv", "dbeta") + dec + ("dbx", "dwx", "dUb", "dVb", "dS0")


def _decay(x):
    if x.get("f") is not None:
        return dict(f=x["f"], A=x["A"], tau_f=x["tau_f"])
    return dict(g=x["g"])


def run_gpu(w, inp, L):
    dt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    x = to_gpu(inp, dt)
    args = (x["q"], x["k"], x["v"], x["beta"], x["bx"], x["wx"], x["Ub"], x["Vb"])
    o, S_T, S_chunks = carve.chunk_fwd_sw(*args, x["S0"], L=L, **_decay(x))
    gr = carve.chunk_bwd_sw(*args, S_chunks, x["dO"], x["dS_T"], L=L, **_decay(x))
    torch.cuda.synchronize()
    out = {key: host(val) for key, val in gr.items()}
    out.update({"o": host(o), "S_T": host(S_T), "S_chunks": host(S_chunks)})
    return out


def check(w, inp, L=None):
    L = L or w.L
    tol = TOL[w.dtype]
    ref = dict(orc.fwd_sw(inp, L, want_chunks=True))
    ref.update(orc.bwd_sw(inp, L, inp["dO"], inp["dS_T"]))
    got = run_gpu(w, inp, L)
    keys = ("o", "S_T", "S_chunks") + _grads(inp.get("f") is not None)
    for key in keys:
        assert got[key].shape == ref[key].shape, key
        assert np.all(np.isfinite(got[key])), key
    errs = {key: max_rel(got[key], ref[key]) for key in keys}
    print("max-rel errors:", {key: float("%.3g" % e) for key, e in errs.items()}, flush=True)
    bad = {key: e for key, e in errs.items() if e > tol}
    assert not bad, (bad, errs)


@pytest.mark.parametrize("L", [16, 32])
def test_sw_fp32_small(L):
    w = _w(L=L, T=128)
    print(f"case sw fp32 D=32 L={L}", flush=True)
    check(w, make_inputs(w, seed=L, dS_T=True, scalar_write=True))


def test_sw_gated_fp32_d64():
    w = _w(Dk=64, Dv=64, L=32, T=96, R=16, B=3, H=2)
    print("case sw+gated fp32 D=64", flush=True)
    check(w, make_inputs(w, seed=5, dS_T=True, gated=True, scalar_write=True))


def test_sw_fp32_rank_over_32():
    """R = 40: the fold operand and tau span 64 padded rows."""
    w = _w(L=32, T=96, R=40, B=1, H=3)
    print("case sw fp32 D=32 R=40", flush=True)
    check(w, make_inputs(w, seed=40, dS_T=True, scalar_write=True))


@pytest.mark.parametrize("L,gated", [(32, False), (64, False), (128, True)])
def test_sw_bf16_d128(L, gated):
    w = _w(Dk=128, Dv=128, L=L, T=256, R=32, dtype="bf16", mu=3.0, s0=0.0, u_std=0.02)
    print(f"case sw bf16 D=128 L={L} gated={gated}", flush=True)
    check(w, make_inputs(w, seed=L, gated=gated, scalar_write=True))


def test_sw_bf16_d128_content_amplified():
    w = _w(Dk=128, Dv=128, L=64, T=192, R=32, dtype="bf16", mu=3.0, s0=0.1, u_std=0.3)
    print("case sw bf16 D=128 content-amplified", flush=True)
    check(w, make_inputs(w, seed=9, dS_T=True, scalar_write=True))


def test_sw_matches_full_layer_on_broadcast_logit():
    """The scalar-write kernels equal the full kernels fed the write logit on
    every value channel and Uw = Vw = 0; the full layer's dwx summed over the
    value channels is the scalar-write dwx."""
    w = _w(T=64, L=16)
    inp = make_inputs(w, seed=3, dS_T=True, scalar_write=True)
    dt = torch.float32
    x = to_gpu(inp, dt)
    args = (x["q"], x["k"], x["v"], x["beta"], x["bx"], x["wx"], x["Ub"], x["Vb"])
    o1, s1, c1 = carve.chunk_fwd_sw(*args, x["S0"], L=16, g=x["g"])
    g1 = carve.chunk_bwd_sw(*args, c1, x["dO"], x["dS_T"], L=16, g=x["g"])
    wxf = x["wx"][..., None].expand(-1, -1, -1, w.Dv).contiguous()
    zU = torch.zeros((w.R, w.Dv), device="cuda")
    zV = torch.zeros((w.Dv, w.R), device="cuda")
    full = (x["q"], x["k"], x["v"], x["beta"], x["g"], x["bx"], wxf, x["Ub"], zU, x["Vb"], zV)
    o2, s2, c2 = carve.chunk_fwd(*full, x["S0"], L=16)
    g2 = carve.chunk_bwd(*full, c2, x["dO"], x["dS_T"], L=16)
    torch.cuda.synchronize()
    assert max_rel(host(o1), host(o2)) < 1e-5 and max_rel(host(s1), host(s2)) < 1e-5
    assert max_rel(host(g1["dwx"]), host(g2["dwx"]).sum(axis=-1)) < 1e-5
    for key in ("dq", "dk", "dv", "dbeta", "dg", "dbx", "dUb", "dVb", "dS0"):
        assert max_rel(host(g1[key]), host(g2[key])) < 1e-5, key


def test_sw_backward_deterministic():
    w = _w(Dk=64, Dv=64, L=32, T=128, R=8, B=3)
    inp = make_inputs(w, seed=2, scalar_write=True)
    a = run_gpu(w, inp, 32)
    b = run_gpu(w, inp, 32)
    for key in _grads(False):
        assert np.array_equal(a[key], b[key]), key
