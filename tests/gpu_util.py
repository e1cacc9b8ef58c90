"""Helpers shared by the GPU parity tests (no arithmetic of the layer here)."""
import numpy as np
import torch

INPUT_KEYS = ("q", "k", "v", "beta", "g", "bx", "wx", "Ub", "Uw", "Vb", "Vw", "S0")
F32_KEYS = ("g", "A", "tau_f", "Ub", "Uw", "Vb", "Vw", "S0", "dS_T")


def to_gpu(inp, dtype, device="cuda"):
    """numpy inputs (already bf16-rounded where needed) -> GPU tensors."""
    out = {}
    for key, val in inp.items():
        if val is None:
            out[key] = None
            continue
        t = torch.from_numpy(np.ascontiguousarray(val, dtype=np.float32))
        if key not in F32_KEYS:
            t = t.to(dtype)
        out[key] = t.to(device).contiguous()
    return out


def max_rel(x, ref):
    """max_i |x_i - ref_i| / max_i |ref_i| (the per-tensor error measure)."""
    x = np.asarray(x, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    den = np.max(np.abs(ref))
    if den == 0:
        return float(np.max(np.abs(x)))
    return float(np.max(np.abs(x - ref)) / den)


def host(t):
    return t.detach().float().cpu().numpy()
