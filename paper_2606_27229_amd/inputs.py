"""Seeded synthetic inputs for the chunked CARVE layer.

This module only draws random numbers and shapes them: it holds none of the
layer's arithmetic.  It is the one generator shared by the tests, the smoke
check and the benchmark, so every consumer sees identical arrays.

Recipe (distributions of the paper's 1.3B-scale layer inputs, Sec. 4.1):
  q, k   ~ N(0,1), each (token, head) row L2-normalised over d_k
  v      ~ N(0,1)
  beta   = sigmoid(N(0,1))                       per (token, head)
  g      = logsigmoid(N(mu,1))                   key-axis log-decay, always f32
  bx     ~ N(-mu,1)   so log(1 - sigmoid(bx)) has the law of g
  wx     ~ N(0,1)
  Ub, Uw ~ N(0, s_u^2) of shape [R, Dv]          (default s_u = 0.02)
  Vb     ~ N(0, s_u^2) of shape [Dk, R], Vw of shape [Dv, R]
  S0     = 0, or N(0, s0^2) of shape [B, H, Dv, Dk]
  dO     ~ N(0,1) of shape [B, T, H, Dv];  dS_T = 0 unless asked for
With the decay gate computed from its raw logit (gated=True; Sec. decay_gate,
g = -exp(A) softplus(f + tau_f)) three more arrays are drawn after the others
(so every other array is unchanged) and g is left out:
  f      ~ N(0,1) of shape [B, T, H, Dk]         token dtype
  A      ~ N(0, 0.1^2) of shape [H, Dk]          f32 log-amplitudes
  tau_f  ~ N(-mu, 0.1^2) of shape [H, Dk]        f32 biases
so that f + tau_f ~ N(-mu, 1.01) and g is close in law to logsigmoid(N(mu,1)).
With the scalar write gate (scalar_write=True; Sec. scalar write gate) the
per-head write logit is drawn last (after the gated arrays, if any), replacing
the per-channel one, and Uw, Vw are left out:
  wx     ~ N(0,1) of shape [B, T, H]             token dtype
With the input activations inside the layer (act=True; SiLU then L2-norm on
queries and keys, SiLU on values) the raw projections are drawn last and
replace q, k, v:
  q, k   ~ N(0,1) of shape [B, T, H, Dk], v ~ N(0,1) of shape [B, T, H, Dv]
Token tensors of a bf16 workload are rounded to bf16 (round to nearest even)
and the rounded values are what every consumer receives; g, the parameters
and the states stay f32.
"""
from __future__ import annotations

from dataclasses import dataclass, replace

import numpy as np


@dataclass(frozen=True)
class Workload:
    name: str
    B: int
    H: int
    T: int
    Dk: int
    Dv: int
    L: int
    R: int
    dtype: str            # "f32" or "bf16": dtype of the token tensors
    mu: float             # location of the decay / erase logits
    s0: float = 0.0       # std of the initial state (0 = zero state)
    u_std: float = 0.02   # std of the content projections
    backward: bool = True

    def with_(self, **kw) -> "Workload":
        return replace(self, **kw)

    @property
    def tokens(self) -> int:
        return self.B * self.T


# The paper-shaped workloads.  "layer_1p3b_T4096" at L=64 is the headline.
WORKLOADS = {
    "tiny_fp32": Workload("tiny_fp32", B=1, H=1, T=256, Dk=32, Dv=32, L=64, R=4, dtype="f32",
                          mu=2.0, backward=False),
    "layer_fp32": Workload("layer_fp32", B=2, H=4, T=1024, Dk=64, Dv=64, L=64, R=16, dtype="f32",
                           mu=2.0, s0=0.1),
    "layer_1p3b_T2048": Workload("layer_1p3b_T2048", B=8, H=16, T=2048, Dk=128, Dv=128, L=64, R=32,
                                 dtype="bf16", mu=3.0),
    "long_seq_T16384": Workload("long_seq_T16384", B=2, H=16, T=16384, Dk=128, Dv=128, L=64, R=32,
                                dtype="bf16", mu=3.0),
    "layer_1p3b_T4096": Workload("layer_1p3b_T4096", B=4, H=16, T=4096, Dk=128, Dv=128, L=64, R=32,
                                 dtype="bf16", mu=3.0),
}
HEADLINE = "layer_1p3b_T4096"
CHUNK_SWEEP = (16, 32, 64, 128)


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even); returns float32."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    r = ((u + 0x7FFF + lsb) >> 16) << 16
    out = r.astype(np.uint32).view(np.float32)
    nan = np.isnan(x)
    if nan.any():
        out = out.copy()
        out[nan] = np.nan
    return out


def _normal(rng, shape, std=1.0, mean=0.0):
    x = rng.standard_normal(size=shape, dtype=np.float32)
    if std != 1.0:
        x *= np.float32(std)
    if mean != 0.0:
        x += np.float32(mean)
    return x


def _l2_rows(x):
    n = np.sqrt(np.sum(x.astype(np.float64) ** 2, axis=-1, keepdims=True))
    return (x / np.maximum(n, 1e-12)).astype(np.float32)


def _sigmoid(x):
    return (1.0 / (1.0 + np.exp(-x.astype(np.float64)))).astype(np.float32)


def _logsigmoid(x):
    x = x.astype(np.float64)
    return (np.minimum(x, 0.0) - np.log1p(np.exp(-np.abs(x)))).astype(np.float32)


def make_inputs(w: Workload, seed: int = 0, *, zero_content: bool = False,
                dS_T: bool = False, bx_mean: float | None = None, gated: bool = False,
                scalar_write: bool = False, act: bool = False) -> dict:
    """Draw one seeded input set for workload ``w``.

    zero_content: Ub = Uw = 0 (the memory-blind special case).
    bx_mean:      override the erase-logit location (erase-heavy stress uses 0).
    gated:        raw decay logits f with per-head A, tau_f instead of g.
    scalar_write: a per-head write logit wx [B,T,H] and no Uw, Vw.
    act:          q, k, v are raw projections (the layer applies the activations).
    """
    rng = np.random.Generator(np.random.PCG64(seed))
    B, T, H, Dk, Dv, R = w.B, w.T, w.H, w.Dk, w.Dv, w.R
    q = _l2_rows(_normal(rng, (B, T, H, Dk)))
    k = _l2_rows(_normal(rng, (B, T, H, Dk)))
    v = _normal(rng, (B, T, H, Dv))
    beta = _sigmoid(_normal(rng, (B, T, H)))
    g = _logsigmoid(_normal(rng, (B, T, H, Dk), mean=w.mu))
    bx = _normal(rng, (B, T, H, Dk), mean=-w.mu if bx_mean is None else bx_mean)
    wx = _normal(rng, (B, T, H, Dv))
    Ub = _normal(rng, (R, Dv), std=w.u_std)
    Uw = _normal(rng, (R, Dv), std=w.u_std)
    Vb = _normal(rng, (Dk, R), std=w.u_std)
    Vw = _normal(rng, (Dv, R), std=w.u_std)
    if zero_content:
        Ub = np.zeros_like(Ub)
        Uw = np.zeros_like(Uw)
    S0 = _normal(rng, (B, H, Dv, Dk), std=w.s0) if w.s0 > 0 else None
    dO = _normal(rng, (B, T, H, Dv))
    dST = _normal(rng, (B, H, Dv, Dk)) if dS_T else None
    if w.dtype == "bf16":
        q, k, v, beta, bx, wx, dO = (round_bf16(a) for a in (q, k, v, beta, bx, wx, dO))
    out = {"q": q, "k": k, "v": v, "beta": beta, "g": g, "bx": bx, "wx": wx,
           "Ub": Ub, "Uw": Uw, "Vb": Vb, "Vw": Vw, "S0": S0, "dO": dO, "dS_T": dST}
    if gated:
        f = _normal(rng, (B, T, H, Dk))
        out["A"] = _normal(rng, (H, Dk), std=0.1)
        out["tau_f"] = _normal(rng, (H, Dk), std=0.1, mean=-w.mu)
        out["f"] = round_bf16(f) if w.dtype == "bf16" else f
        out["g"] = None
    if scalar_write:
        wxs = _normal(rng, (B, T, H))
        out["wx"] = round_bf16(wxs) if w.dtype == "bf16" else wxs
        out["Uw"] = None
        out["Vw"] = None
    if act:
        raw = [_normal(rng, (B, T, H, Dk)), _normal(rng, (B, T, H, Dk)), _normal(rng, (B, T, H, Dv))]
        if w.dtype == "bf16":
            raw = [round_bf16(a) for a in raw]
        out["q"], out["k"], out["v"] = raw
    return out
