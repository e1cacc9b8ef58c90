"""The allocation-free entry point carve_rmsnorm_bwd_noalloc (static per-device
scratch) against carve_rmsnorm_bwd (caller's workspace) through the C ABI: two
calls in a row, the second with a smaller input; outputs bitwise equal."""
import numpy as np
import pytest
import torch

from paper_2606_27229_amd import carve
from paper_2606_27229_amd.inputs import round_bf16

pytestmark = pytest.mark.gpu


def _case(B, T, H, Dv, dt, seed):
    rng = np.random.Generator(np.random.PCG64(seed))
    o = rng.standard_normal((B, T, H, Dv), dtype=np.float32)
    dy = rng.standard_normal((B, T, H, Dv), dtype=np.float32)
    w = (1.0 + 0.1 * rng.standard_normal(H * Dv)).astype(np.float32)
    if dt == torch.bfloat16:
        o, dy = round_bf16(o), round_bf16(dy)
    return (torch.from_numpy(o).to(dt).cuda(), torch.from_numpy(w).cuda(), torch.from_numpy(dy).to(dt).cuda())


def test_noalloc_matches_workspace_entry_point():
    cases = [(4, 1024, 16, 128, torch.bfloat16, 1), (2, 37, 2, 64, torch.float32, 2)]
    for B, T, H, Dv, dt, seed in cases:
        print(f"case noalloc rmsnorm bwd B={B} T={T} H={H} Dv={Dv} {dt}", flush=True)
        o, w, dy = _case(B, T, H, Dv, dt, seed)
        ref_do, ref_dw = carve.rmsnorm_bwd(o, w, dy)
        d_o = torch.full_like(o, float("nan"))
        dw = torch.full((H * Dv,), float("nan"), device="cuda")
        carve.rmsnorm_bwd_noalloc(o, w, dy, d_o, dw)
        torch.cuda.synchronize()
        assert torch.equal(d_o, ref_do)
        assert torch.equal(dw, ref_dw)
        assert torch.isfinite(dw).all() and torch.isfinite(d_o.float()).all()
