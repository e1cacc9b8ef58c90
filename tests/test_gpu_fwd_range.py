"""Forward (and backward from the forward's own chunk states) at the edges of
the numerical range, through the C ABI, against the CPU oracle.

A forward WY block of 64 tokens takes one exponent reference per key channel
while every channel keeps its log retention over the block above -160, and
per-tile references (one per 16-token tile, with the products across tiles
formed from operands no larger than the raw token values) otherwise.  These
cases drive the second mode:

- hard erase: erase logits near +8 on 16 of the 128 key channels, about -8 of
  log retention per token there (-128 per 16-token tile, -512 per block), so
  every block takes per-tile references; default layer (L = 64, 128) and the
  gate-in-kernel variant;
- concentrated erases: on 16 channels three tokens of every 16-token tile carry
  an erase logit of 40 (about -40 each, -120 per tile, at random positions);
- mixed blocks: erase logits swinging between 1.9 and 2.7 on 16 channels put
  the block sums of those channels on both sides of -160, so blocks of both
  modes follow each other along the sequence (checked on the oracle's gates);
- hard erase at the headline launch (B=4 H=16 T=4096), on sampled slices.

Bar: bf16 inputs with f32 state and accumulation, max-rel <= 2e-2 per tensor.
"""
import numpy as np
import pytest
import torch

from oracle import oracle as orc
from paper_2606_27229_amd import carve
from paper_2606_27229_amd.inputs import Workload, make_inputs, round_bf16
from tests.gpu_util import host, max_rel, to_gpu

pytestmark = pytest.mark.gpu

TOL = {"bf16": 2e-2, "f32": 1e-4}
GRADS = ("dq", "dk", "dv", "dbeta", "dg", "dbx", "dwx", "dUb", "dUw", "dVb", "dVw", "dS0")
GATED_GRADS = ("dq", "dk", "dv", "dbeta", "df", "dA", "dtau", "dbx", "dwx", "dUb", "dUw", "dVb", "dVw", "dS0")


def _w(**kw):
    base = dict(name="range", B=1, H=2, T=256, Dk=128, Dv=128, L=64, R=32, dtype="bf16", mu=3.0, s0=0.2,
                u_std=0.05)
    base.update(kw)
    return Workload(**base)


def _set_bx(inp, w, bx):
    out = dict(inp)
    out["bx"] = round_bf16(bx.astype(np.float32)) if w.dtype == "bf16" else bx.astype(np.float32)
    return out


def _channels(rng, w, nch=16):
    return rng.choice(w.Dk, size=nch, replace=False)


def _hard_erase(inp, w, seed, loc=8.0, scale=0.5):
    rng = np.random.Generator(np.random.PCG64(seed))
    chans = _channels(rng, w)
    bx = np.array(inp["bx"], dtype=np.float32, copy=True)
    bx[..., chans] = loc + scale * rng.standard_normal(bx[..., chans].shape)
    return _set_bx(inp, w, bx)


def _spikes(inp, w, seed, per_tile=3, value=40.0):
    rng = np.random.Generator(np.random.PCG64(seed))
    chans = _channels(rng, w)
    bx = np.array(inp["bx"], dtype=np.float32, copy=True)
    for b in range(w.B):
        for h in range(w.H):
            for ch in chans:
                for t0 in range(0, w.T, 16):
                    pos = t0 + rng.choice(16, size=per_tile, replace=False)
                    bx[b, pos, h, ch] = value
    return _set_bx(inp, w, bx)


def _report(errs, got, tol=TOL["bf16"]):
    for key, val in got.items():
        assert np.all(np.isfinite(val)), key
    print("max-rel errors:", {k: float("%.3g" % e) for k, e in errs.items()}, flush=True)
    bad = {k: e for k, e in errs.items() if not e <= tol}
    assert not bad, bad


def _run_default(inp, L, dtype=torch.bfloat16):
    x = to_gpu(inp, dtype)
    o, S_T, S_chunks = carve.chunk_fwd(x["q"], x["k"], x["v"], x["beta"], x["g"], x["bx"], x["wx"],
                                       x["Ub"], x["Uw"], x["Vb"], x["Vw"], x["S0"], L=L)
    gr = carve.chunk_bwd(x["q"], x["k"], x["v"], x["beta"], x["g"], x["bx"], x["wx"], x["Ub"], x["Uw"],
                         x["Vb"], x["Vw"], S_chunks, x["dO"], x["dS_T"], L=L)
    torch.cuda.synchronize()
    got = {"o": host(o), "S_T": host(S_T), "S_chunks": host(S_chunks)}
    got.update({k: host(gr[k]) for k in GRADS})
    return got


def _check_default(inp, L, rf=None, dtype="bf16"):
    got = _run_default(inp, L, torch.bfloat16 if dtype == "bf16" else torch.float32)
    rf = rf if rf is not None else orc.fwd_serial(inp, L, want_chunks=True)
    rb = orc.bwd(inp, L, inp["dO"], inp["dS_T"])
    errs = {k: max_rel(got[k], rf[k]) for k in ("o", "S_T", "S_chunks")}
    errs.update({k: max_rel(got[k], rb[k]) for k in GRADS})
    _report(errs, got, TOL[dtype])


# (dtype, d, L): the forward blocks are 64 tokens wide except at bf16 d = 128
# L = 32 and f32 d = 64 (32 tokens: two tiles per block)
@pytest.mark.parametrize("dtype,D,L", [("bf16", 128, 64), ("bf16", 128, 128), ("bf16", 128, 32),
                                       ("bf16", 64, 64), ("f32", 32, 64), ("f32", 64, 64)])
def test_fwd_bwd_hard_erase(dtype, D, L):
    w = _w(L=L, Dk=D, Dv=D, dtype=dtype)
    print(f"case forward hard erase {dtype} D={D} L={L}", flush=True)
    inp = _hard_erase(make_inputs(w, seed=400 + L + D, dS_T=True), w, seed=L + D)
    _check_default(inp, L, dtype=dtype)


def test_fwd_bwd_hard_erase_gated():
    w = _w(L=64)
    L = w.L
    print("case forward hard erase gated bf16 D=128 L=64", flush=True)
    inp = _hard_erase(make_inputs(w, seed=460, dS_T=True, gated=True), w, seed=461)
    x = to_gpu(inp, torch.bfloat16)
    args = (x["q"], x["k"], x["v"], x["beta"], x["f"], x["A"], x["tau_f"], x["bx"], x["wx"],
            x["Ub"], x["Uw"], x["Vb"], x["Vw"])
    o, S_T, S_chunks = carve.chunk_fwd_gated(*args, x["S0"], L=L)
    gr = carve.chunk_bwd_gated(*args, S_chunks, x["dO"], x["dS_T"], L=L)
    torch.cuda.synchronize()
    rf = orc.fwd_gated(inp, L, want_chunks=True)
    rb = orc.bwd_gated(inp, L, inp["dO"], inp["dS_T"])
    got = {"o": host(o), "S_T": host(S_T), "S_chunks": host(S_chunks)}
    got.update({k: host(gr[k]) for k in GATED_GRADS})
    errs = {k: max_rel(got[k], rf[k]) for k in ("o", "S_T", "S_chunks")}
    errs.update({k: max_rel(got[k], rb[k]) for k in GATED_GRADS})
    _report(errs, got)


def test_fwd_bwd_concentrated_erases():
    w = _w(L=64)
    print("case forward concentrated erases bf16 D=128 L=64", flush=True)
    inp = _spikes(make_inputs(w, seed=470, dS_T=True), w, seed=471)
    _check_default(inp, w.L)


def test_fwd_bwd_mixed_blocks():
    w = _w(L=64, T=512)
    print("case forward mixed blocks bf16 D=128 L=64 T=512", flush=True)
    # erase logit location swinging between 1.9 and 2.7 over 256 tokens
    loc = (2.3 + 0.4 * np.sin(2 * np.pi * np.arange(w.T) / 256))[None, :, None, None]
    inp = _hard_erase(make_inputs(w, seed=480, dS_T=True), w, seed=481, loc=loc, scale=0.3)
    rf = orc.fwd_serial(inp, w.L, want_chunks=True, want_gates=True)
    # log retention per token and channel, summed over each 64-token block
    lr = inp["g"].astype(np.float64) + np.log1p(-rf["gate_b"])
    sums = lr.reshape(w.B, w.T // 64, 64, w.H, w.Dk).sum(axis=2).min(axis=-1)
    print("block minima over channels:", np.round(sums, 1).tolist(), flush=True)
    assert np.any(sums < -165) and np.any(sums > -155), "the inputs do not mix both block modes"
    _check_default(inp, w.L, rf=rf)


def test_fwd_bwd_hard_erase_full_size_sampled():
    """The headline launch (B=4 H=16 T=4096 d=128 r=32 L=64) with hard-erase
    channels in every (batch, head), every block on per-tile references;
    checked on two sampled (batch, head) slices, the parameter gradients with
    the upstream gradients zeroed outside them (so the full-size sums must
    equal the oracle's sums over the samples)."""
    from paper_2606_27229_amd.inputs import WORKLOADS
    from tests.test_gpu_fullsize import PARAM_GRADS, TOKEN_GRADS, _slice
    w = WORKLOADS["layer_1p3b_T4096"].with_(L=64)
    print(f"case forward hard erase full size B={w.B} H={w.H} T={w.T}", flush=True)
    inp = _hard_erase(make_inputs(w, seed=490, dS_T=True), w, seed=491)
    samples = [(0, 0), (w.B - 1, w.H - 1)]
    keep = np.zeros((w.B, w.H), dtype=bool)
    for b, h in samples:
        keep[b, h] = True
    inp["dO"] = inp["dO"] * keep[:, None, :, None]
    inp["dS_T"] = inp["dS_T"] * keep[:, :, None, None]
    x = to_gpu(inp, torch.bfloat16)
    o, S_T, S_chunks = carve.chunk_fwd(x["q"], x["k"], x["v"], x["beta"], x["g"], x["bx"], x["wx"], x["Ub"],
                                       x["Uw"], x["Vb"], x["Vw"], x["S0"], L=w.L)
    gr = carve.chunk_bwd(x["q"], x["k"], x["v"], x["beta"], x["g"], x["bx"], x["wx"], x["Ub"], x["Uw"],
                         x["Vb"], x["Vw"], S_chunks, x["dO"], x["dS_T"], L=w.L)
    torch.cuda.synchronize()
    del x
    ref_params = {key: 0.0 for key in PARAM_GRADS}
    errs, got = {}, {}
    for b, h in samples:
        s = _slice(inp, b, h)
        rf = orc.fwd_serial(s, w.L, want_chunks=True)
        rb = orc.bwd(s, w.L, s["dO"], s["dS_T"])
        for key, val in (("o", o[b:b + 1, :, h:h + 1]), ("S_T", S_T[b:b + 1, h:h + 1]),
                         ("S_chunks", S_chunks[b:b + 1, h:h + 1])):
            got[f"{key}[{b},{h}]"] = host(val)
            errs[f"{key}[{b},{h}]"] = max_rel(got[f"{key}[{b},{h}]"], rf[key])
        for key in TOKEN_GRADS:
            got[f"{key}[{b},{h}]"] = host(gr[key][b:b + 1, :, h:h + 1])
            errs[f"{key}[{b},{h}]"] = max_rel(got[f"{key}[{b},{h}]"], rb[key])
        got[f"dS0[{b},{h}]"] = host(gr["dS0"][b:b + 1, h:h + 1])
        errs[f"dS0[{b},{h}]"] = max_rel(got[f"dS0[{b},{h}]"], rb["dS0"])
        for key in PARAM_GRADS:
            ref_params[key] = ref_params[key] + rb[key]
    for key in PARAM_GRADS:
        got[key] = host(gr[key])
        errs[key] = max_rel(got[key], ref_params[key])
    _report(errs, got)
