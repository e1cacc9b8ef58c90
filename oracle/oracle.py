"""Python access to the CPU oracle (``carve_oracle.c``) for the chunked CARVE layer.

TEST INFRASTRUCTURE ONLY.  This module (and the C library it wraps) may be
imported only by ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline
leg of ``bench.py``.  It shares no code with the HIP path and never imports
the product package.

All arrays are converted to contiguous float64 before the call; layouts are
those documented in ``carve_oracle.h`` ([B,T,H,D] token tensors,
[B,H,Dv,Dk] states, shared [R,Dv] / [Dk,R] / [Dv,R] parameters).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "carve_oracle.c")
_LIB = os.path.join(_HERE, "libcarve_oracle.so")

_lib = None


class _Dims(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int) for n in ("B", "T", "H", "Dk", "Dv", "R", "L")]


def build() -> str:
    """Compile the oracle with gcc (IEEE double, no FMA contraction)."""
    tmp = _LIB + ".tmp"
    cmd = ["gcc", "-O2", "-std=c99", "-fPIC", "-shared", "-ffp-contract=off",
           "-fno-fast-math", "-Wall", "-o", tmp, _SRC, "-lm", "-lpthread"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB):
        build()
    lib = ctypes.CDLL(_LIB)
    P = ctypes.POINTER(ctypes.c_double)
    D = ctypes.POINTER(_Dims)
    lib.cref_fwd_serial.argtypes = [D] + [P] * 17 + [ctypes.c_int]
    lib.cref_fwd_chunked.argtypes = [D] + [P] * 17 + [ctypes.c_int]
    lib.cref_baseline_fwd.argtypes = [D] + [P] * 10 + [ctypes.c_int]
    lib.cref_bwd.argtypes = [D] + [P] * 26 + [ctypes.c_int]
    lib.cref_decay_gate.argtypes = [D] + [P] * 4
    lib.cref_decay_gate_bwd.argtypes = [D] + [P] * 7
    for f in (lib.cref_fwd_serial, lib.cref_fwd_chunked, lib.cref_baseline_fwd, lib.cref_bwd,
              lib.cref_decay_gate, lib.cref_decay_gate_bwd):
        f.restype = ctypes.c_int
    _lib = lib
    return lib


def _f64(x):
    if x is None:
        return None
    return np.ascontiguousarray(np.asarray(x, dtype=np.float64))


def _ptr(x):
    if x is None:
        return ctypes.POINTER(ctypes.c_double)()
    return x.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def dims_of(inp, L):
    B, T, H, Dk = inp["q"].shape
    Dv = inp["v"].shape[-1]
    R = inp["Ub"].shape[0]
    return _Dims(B, T, H, Dk, Dv, R, L)


def default_threads():
    return max(1, os.cpu_count() or 1)


def _check(st, name):
    if st != 0:
        raise ValueError(f"oracle {name} returned {st}")


def _fwd(fn_name, inp, L, want_chunks, want_gates, nthreads):
    lib = _load()
    d = dims_of(inp, L)
    a = {k: _f64(inp.get(k)) for k in ("q", "k", "v", "beta", "g", "bx", "wx", "Ub", "Uw", "Vb", "Vw", "S0")}
    B, T, H, Dk, Dv = d.B, d.T, d.H, d.Dk, d.Dv
    o = np.zeros((B, T, H, Dv))
    S_T = np.zeros((B, H, Dv, Dk))
    S_chunks = np.zeros((B, H, T // L, Dv, Dk)) if want_chunks else None
    gb = np.zeros((B, T, H, Dk)) if want_gates else None
    gw = np.zeros((B, T, H, Dv)) if want_gates else None
    fn = getattr(lib, fn_name)
    st = fn(ctypes.byref(d), *[_ptr(a[k]) for k in ("q", "k", "v", "beta", "g", "bx", "wx",
                                                       "Ub", "Uw", "Vb", "Vw", "S0")],
            _ptr(o), _ptr(S_T), _ptr(S_chunks), _ptr(gb), _ptr(gw),
            nthreads if nthreads else default_threads())
    _check(st, fn_name)
    out = {"o": o, "S_T": S_T}
    if want_chunks:
        out["S_chunks"] = S_chunks
    if want_gates:
        out["gate_b"] = gb
        out["gate_w"] = gw
    return out


def fwd_serial(inp, L, want_chunks=False, want_gates=False, nthreads=None):
    """Token-serial definition of the layer (Eq. carve_state, staleness rule of Alg. carve_fwd)."""
    return _fwd("cref_fwd_serial", inp, L, want_chunks, want_gates, nthreads)


def fwd_chunked(inp, L, want_chunks=False, want_gates=False, nthreads=None):
    """Chunked WY form of the same layer (Sec. WY-form intra-chunk solve)."""
    return _fwd("cref_fwd_chunked", inp, L, want_chunks, want_gates, nthreads)


def baseline_fwd(inp, L=None, nthreads=None):
    """Memory-blind key-axis gated delta recurrence (gates from bx, wx only)."""
    lib = _load()
    d = dims_of(inp, L if L else inp["q"].shape[1])
    a = {k: _f64(inp.get(k)) for k in ("q", "k", "v", "beta", "g", "bx", "wx", "S0")}
    o = np.zeros((d.B, d.T, d.H, d.Dv))
    S_T = np.zeros((d.B, d.H, d.Dv, d.Dk))
    st = lib.cref_baseline_fwd(ctypes.byref(d), *[_ptr(a[k]) for k in ("q", "k", "v", "beta", "g",
                                                                     "bx", "wx", "S0")],
                               _ptr(o), _ptr(S_T), nthreads if nthreads else default_threads())
    _check(st, "cref_baseline_fwd")
    return {"o": o, "S_T": S_T}


def bwd(inp, L, dO, dS_T=None, nthreads=None):
    """Exact reverse mode of ``fwd_serial`` for the loss <dO, o> + <dS_T, S_T>."""
    lib = _load()
    d = dims_of(inp, L)
    a = {k: _f64(inp.get(k)) for k in ("q", "k", "v", "beta", "g", "bx", "wx", "Ub", "Uw", "Vb", "Vw", "S0")}
    dO = _f64(dO)
    dS_T = _f64(dS_T)
    B, T, H, Dk, Dv, R = d.B, d.T, d.H, d.Dk, d.Dv, d.R
    out = {
        "dq": np.zeros((B, T, H, Dk)), "dk": np.zeros((B, T, H, Dk)), "dv": np.zeros((B, T, H, Dv)),
        "dbeta": np.zeros((B, T, H)), "dg": np.zeros((B, T, H, Dk)), "dbx": np.zeros((B, T, H, Dk)),
        "dwx": np.zeros((B, T, H, Dv)), "dUb": np.zeros((R, Dv)), "dUw": np.zeros((R, Dv)),
        "dVb": np.zeros((Dk, R)), "dVw": np.zeros((Dv, R)), "dS0": np.zeros((B, H, Dv, Dk)),
    }
    st = lib.cref_bwd(ctypes.byref(d), *[_ptr(a[k]) for k in ("q", "k", "v", "beta", "g", "bx", "wx",
                                                            "Ub", "Uw", "Vb", "Vw", "S0")],
                      _ptr(dO), _ptr(dS_T),
                      *[_ptr(out[k]) for k in ("dq", "dk", "dv", "dbeta", "dg", "dbx", "dwx",
                                               "dUb", "dUw", "dVb", "dVw", "dS0")],
                      nthreads if nthreads else default_threads())
    _check(st, "cref_bwd")
    return out


def decay_gate(f, A, tau, L=1):
    """g = -exp(A) * softplus(f + tau) (Eq. decay_gate); f [B,T,H,Dk], A and tau [H,Dk]."""
    lib = _load()
    f = _f64(f)
    B, T, H, Dk = f.shape
    d = _Dims(B, T, H, Dk, Dk, 1, L)
    g = np.zeros_like(f)
    _check(lib.cref_decay_gate(ctypes.byref(d), _ptr(f), _ptr(_f64(A)), _ptr(_f64(tau)), _ptr(g)), "cref_decay_gate")
    return g


def decay_gate_bwd(f, A, tau, dg):
    """Reverse mode of ``decay_gate``: returns (df, dA, dtau)."""
    lib = _load()
    f = _f64(f)
    B, T, H, Dk = f.shape
    d = _Dims(B, T, H, Dk, Dk, 1, 1)
    df = np.zeros_like(f)
    dA = np.zeros((H, Dk))
    dtau = np.zeros((H, Dk))
    _check(lib.cref_decay_gate_bwd(ctypes.byref(d), _ptr(f), _ptr(_f64(A)), _ptr(_f64(tau)), _ptr(_f64(dg)),
                                   _ptr(df), _ptr(dA), _ptr(dtau)), "cref_decay_gate_bwd")
    return df, dA, dtau


def _with_gate(inp):
    """The ungated inputs of the gated layer: g from (f, A, tau) by Eq. decay_gate."""
    out = dict(inp)
    out["g"] = decay_gate(inp["f"], inp["A"], inp["tau_f"])
    return out


def fwd_gated(inp, L, want_chunks=False, nthreads=None):
    """The layer with the decay gate computed from its raw logit f (Sec. decay_gate)."""
    return fwd_serial(_with_gate(inp), L, want_chunks=want_chunks, nthreads=nthreads)


def bwd_gated(inp, L, dO, dS_T=None, nthreads=None):
    """Reverse mode of ``fwd_gated``: the gradients of ``bwd`` with dg replaced by
    df, dA, dtau (chain rule through Eq. decay_gate)."""
    out = bwd(_with_gate(inp), L, dO, dS_T, nthreads=nthreads)
    out["df"], out["dA"], out["dtau"] = decay_gate_bwd(inp["f"], inp["A"], inp["tau_f"], out.pop("dg"))
    return out


def scalar_write_inputs(inp):
    """The inputs of the full layer that define the scalar write gate (Sec. scalar
    write gate, ablation rows of Table attribution): a per-head logit wx [B,T,H],
    w_t = sigmoid(wx_t) on every one of the Dv value channels, and no content
    term on the write side.  The full layer gives exactly that with wx repeated
    along the value axis and Uw = Vw = 0 (then Vw tau_w = 0 whatever tau_w is).
    Any Uw, Vw in ``inp`` are ignored."""
    out = dict(inp)
    wx = _f64(inp["wx"])
    Dv = np.shape(inp["v"])[-1]
    R = np.shape(inp["Ub"])[0]
    out["wx"] = np.repeat(wx[..., None], Dv, axis=-1)
    out["Uw"] = np.zeros((R, Dv))
    out["Vw"] = np.zeros((Dv, R))
    return out


def fwd_sw(inp, L, want_chunks=False, nthreads=None):
    """The layer with the scalar write gate; the decay is g, or (when ``inp``
    holds f) formed from f, A, tau_f by Eq. decay_gate."""
    x = scalar_write_inputs(inp)
    if inp.get("f") is not None:
        return fwd_gated(x, L, want_chunks=want_chunks, nthreads=nthreads)
    return fwd_serial(x, L, want_chunks=want_chunks, nthreads=nthreads)


def bwd_sw(inp, L, dO, dS_T=None, nthreads=None):
    """Reverse mode of ``fwd_sw``: dwx [B,T,H] is the sum over the value
    channels of the full layer's dwx (the logit is shared by all of them);
    there is no dUw, dVw.  dg, or df, dA, dtau when ``inp`` holds f."""
    x = scalar_write_inputs(inp)
    if inp.get("f") is not None:
        out = bwd_gated(x, L, dO, dS_T, nthreads=nthreads)
    else:
        out = bwd(x, L, dO, dS_T, nthreads=nthreads)
    out["dwx"] = out["dwx"].sum(axis=-1)
    del out["dUw"], out["dVw"]
    return out


# ---- input activations (Sec. input projections, Fig. carve_block): queries and
# keys go through SiLU then L2 normalisation over d_k, values through SiLU ----
L2_EPS = 1e-6   # x / sqrt(|x|^2 + eps); the paper gives no epsilon


def silu(x):
    x = _f64(x)
    return x / (1.0 + np.exp(-x))


def silu_grad(x):
    x = _f64(x)
    s = 1.0 / (1.0 + np.exp(-x))
    return s * (1.0 + x * (1.0 - s))


def act_qk(xr):
    """q = SiLU(q_raw) / sqrt(|SiLU(q_raw)|^2 + eps), per (token, head) over the last axis."""
    s = silu(xr)
    return s / np.sqrt(np.sum(s * s, axis=-1, keepdims=True) + L2_EPS)


def act_qk_bwd(xr, dy):
    """Reverse mode of ``act_qk``: with s = SiLU(x), n = sqrt(|s|^2 + eps), y = s / n,
    ds = (dy - y (y . dy)) / n and dx = ds * SiLU'(x)."""
    s = silu(xr)
    n = np.sqrt(np.sum(s * s, axis=-1, keepdims=True) + L2_EPS)
    y = s / n
    dy = _f64(dy)
    ds = (dy - y * np.sum(y * dy, axis=-1, keepdims=True)) / n
    return ds * silu_grad(xr)


def act_inputs(inp):
    """The layer's q, k, v from the raw projections held in ``inp`` (q, k, v)."""
    out = dict(inp)
    out["q"] = act_qk(inp["q"])
    out["k"] = act_qk(inp["k"])
    out["v"] = silu(inp["v"])
    return out


def fwd_act(inp, L, want_chunks=False, nthreads=None):
    """The layer fed the raw projections q, k, v (activations inside the layer)."""
    return fwd_serial(act_inputs(inp), L, want_chunks=want_chunks, nthreads=nthreads)


def bwd_act(inp, L, dO, dS_T=None, nthreads=None):
    """Reverse mode of ``fwd_act``: dq, dk, dv with respect to the raw projections."""
    out = bwd(act_inputs(inp), L, dO, dS_T, nthreads=nthreads)
    out["dq"] = act_qk_bwd(inp["q"], out["dq"])
    out["dk"] = act_qk_bwd(inp["k"], out["dk"])
    out["dv"] = out["dv"] * silu_grad(inp["v"])
    return out


# ---- output RMS normalisation (the step that closes Alg. carve_fwd:
# y = W_O RMSNorm(reshape(o)); W_O is a plain GEMM and not part of this) ----
RMSNORM_EPS = 1e-6   # the paper gives no epsilon


def rmsnorm(o, weight, eps=RMSNORM_EPS):
    """RMSNorm of reshape(o): every token's H*Dv values (o [B,T,H,Dv]) divided by
    their root mean square sqrt(mean(x^2) + eps), times weight [H*Dv]."""
    o = _f64(o)
    B, T, H, Dv = o.shape
    x = o.reshape(B, T, H * Dv)
    ms = np.mean(x * x, axis=-1, keepdims=True)
    y = x / np.sqrt(ms + eps) * _f64(weight)
    return y.reshape(B, T, H, Dv)


def rmsnorm_bwd(o, weight, dy, eps=RMSNORM_EPS):
    """Reverse mode of ``rmsnorm`` for the loss <dy, y>, derived from the
    definition: with r = (mean(x^2) + eps)^(-1/2), n = x r and dn = dy * weight,
    dr/dx_i = -r^3 x_i / N, so d_o = r dn - x r^3 <dn, x> / N = r (dn - n <dn, n> / N);
    dweight = sum over the rows of dy * n.  Returns (d_o, dweight)."""
    o = _f64(o)
    B, T, H, Dv = o.shape
    N = H * Dv
    x = o.reshape(-1, N)
    g = _f64(dy).reshape(-1, N)
    w = _f64(weight)
    r = 1.0 / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps)
    n = x * r
    dn = g * w
    dx = r * (dn - n * np.sum(dn * n, axis=-1, keepdims=True) / N)
    dw = np.sum(g * n, axis=0)
    return dx.reshape(B, T, H, Dv), dw
