"""Host-side checks of the C ABI: the library loads, exports every symbol
include/carve.h declares, and validation errors come back before any HIP
call (no GPU needed)."""
import ctypes
import os
import re

import pytest

from paper_2606_27229_amd import carve

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_symbols():
    text = open(os.path.join(ROOT, "include", "carve.h")).read()
    decl = r"^\s*(?:const\s+char\s*\*|int|size_t|void)\s*(carve_[a-z_]+)\s*\("
    return sorted(set(re.findall(decl, text, flags=re.M)))


def test_header_declares_the_binding_symbols():
    assert sorted(carve.SYMBOLS) == _declared_symbols()


def test_library_exports_every_declared_symbol():
    lib = carve.load_library()
    for name in _declared_symbols():
        assert hasattr(lib, name), name


def test_status_strings():
    lib = carve.load_library()
    for st in range(0, -8, -1):
        assert lib.carve_status_string(st)
    assert "unknown" not in carve.status_string(-7)
    assert carve.status_string(0) == "ok"


def _dims(**kw):
    base = dict(B=1, T=128, H=2, Dk=64, Dv=64, R=16, L=64, dtype=carve.CARVE_BF16)
    base.update(kw)
    return carve.Dims(**base)


@pytest.mark.parametrize("kw,expect", [
    (dict(T=100), -2), (dict(B=0), -2), (dict(Dk=48, Dv=48), -3), (dict(Dk=64, Dv=32), -3),
    (dict(R=65), -3), (dict(L=8, T=128), -3), (dict(dtype=7), -3),
])
def test_forward_validation(kw, expect):
    lib = carve.load_library()
    d = _dims(**kw)
    fake = ctypes.c_void_p(4096)  # never dereferenced: validation fails first
    st = lib.carve_chunk_fwd(ctypes.byref(d), *([fake] * 12), fake, None, None, None, 0, None)
    assert st == expect


def test_forward_null_and_alignment():
    lib = carve.load_library()
    d = _dims()
    fake = ctypes.c_void_p(4096)
    st = lib.carve_chunk_fwd(ctypes.byref(d), None, *([fake] * 11), fake, None, None, None, 0, None)
    assert st == -1
    bad = ctypes.c_void_p(4096 + 4)
    st = lib.carve_chunk_fwd(ctypes.byref(d), bad, *([fake] * 11), fake, None, None, None, 0, None)
    assert st == -4


def test_backward_workspace_checks():
    lib = carve.load_library()
    d = _dims()
    need = lib.carve_workspace_size(ctypes.byref(d), 1)
    assert need > 0
    assert lib.carve_workspace_size(ctypes.byref(_dims(T=100)), 1) == 0
    # distinct fake addresses far apart so no range overlaps
    ptrs = [ctypes.c_void_p(1 << 40 | (i << 32)) for i in range(28)]
    st = lib.carve_chunk_bwd(ctypes.byref(d), *ptrs[:26], None, 0, None)
    assert st == -5
    st = lib.carve_chunk_bwd(ctypes.byref(d), *ptrs[:26], ptrs[26], need - 1, None)
    assert st == -5


def test_aliasing_output_rejected():
    lib = carve.load_library()
    d = _dims()
    ptrs = [ctypes.c_void_p(1 << 40 | (i << 32)) for i in range(16)]
    args = ptrs[:12] + [ptrs[0]]  # o aliases q
    st = lib.carve_chunk_fwd(ctypes.byref(d), *args, None, None, None, 0, None)
    assert st == -3


def test_profile_hook_validation():
    """The measurement hook copies at most 16 handles and rejects bad arguments
    without touching HIP; capacity 0 disarms it."""
    lib = carve.load_library()
    assert lib.carve_profile_events(None, 0) == 0
    assert lib.carve_profile_events(None, 3) == -1
    arr = (ctypes.c_void_p * 17)(*([4096] * 17))
    assert lib.carve_profile_events(arr, -1) == -1
    assert lib.carve_profile_events(arr, 17) == -3
    # an armed hook is cleared by the next call even when that call fails in
    # validation: after a rejected forward, nothing stays armed (the handles
    # here are fake and would fault if ever recorded)
    assert lib.carve_profile_events(arr, 2) == 0
    d = _dims(T=100)
    fake = ctypes.c_void_p(4096)
    assert lib.carve_chunk_fwd(ctypes.byref(d), *([fake] * 12), fake, None, None, None, 0, None) == -2
    assert lib.carve_profile_events(None, 0) == 0


def test_wait_hooks_host():
    """The wait-bound test hook round-trips on the calling thread (negative:
    the default, 2^20 polls); the timeout status query rejects NULL arguments
    and dims no backward accepts before any HIP call."""
    lib = carve.load_library()
    default = 1 << 20
    assert lib.carve_set_ready_wait_limit(0) == default
    assert lib.carve_set_ready_wait_limit(7) == 0
    assert lib.carve_set_ready_wait_limit(-1) == 7
    assert lib.carve_set_ready_wait_limit(-5) == default
    assert lib.carve_set_ready_wait_limit(-1) == default
    d = _dims()
    out = ctypes.c_int(5)
    fake = ctypes.c_void_p(4096)
    assert lib.carve_bwd_wait_status(None, fake, None, ctypes.byref(out)) == -1
    assert lib.carve_bwd_wait_status(ctypes.byref(d), None, None, ctypes.byref(out)) == -1
    assert lib.carve_bwd_wait_status(ctypes.byref(d), fake, None, None) == -1
    assert lib.carve_bwd_wait_status(ctypes.byref(_dims(T=100)), fake, None, ctypes.byref(out)) == -2
    assert out.value == 5


def test_gated_forward_validation():
    """carve_chunk_fwd_gated: NULL f / A / tau_f, bad shapes and misalignment
    are rejected before any HIP call."""
    lib = carve.load_library()
    d = _dims()
    fake = ctypes.c_void_p(4096)
    # q, k, v, beta, f, A, tau_f, bx, wx, Ub, Uw, Vb, Vw, S0, o, S_T, S_chunks, ws, bytes, stream
    args = [fake] * 13 + [None, fake, None, None, None, 0, None]
    for null_at in (4, 5, 6):   # f, A, tau_f
        a = list(args)
        a[null_at] = None
        assert lib.carve_chunk_fwd_gated(ctypes.byref(d), *a) == -1, null_at
    assert lib.carve_chunk_fwd_gated(ctypes.byref(_dims(T=100)), *args) == -2
    a = list(args)
    a[5] = ctypes.c_void_p(4096 + 4)   # A misaligned
    assert lib.carve_chunk_fwd_gated(ctypes.byref(d), *a) == -4


def test_gated_backward_workspace_and_aliasing():
    lib = carve.load_library()
    d = _dims()
    need = lib.carve_workspace_size(ctypes.byref(d), 1)
    # distinct fake addresses far apart: 31 tensors before dS0, workspace
    ptrs = [ctypes.c_void_p(1 << 40 | (i << 32)) for i in range(34)]
    st = lib.carve_chunk_bwd_gated(ctypes.byref(d), *ptrs[:30], None, 0, None)
    assert st == -5
    st = lib.carve_chunk_bwd_gated(ctypes.byref(d), *ptrs[:30], ptrs[30], need - 1, None)
    assert st == -5
    a = list(ptrs[:30])
    a[20] = a[4]          # df aliases f
    st = lib.carve_chunk_bwd_gated(ctypes.byref(d), *a, ptrs[30], need, None)
    assert st == -3
    a = list(ptrs[:30])
    a[21] = None          # dA missing
    st = lib.carve_chunk_bwd_gated(ctypes.byref(d), *a, ptrs[30], need, None)
    assert st == -1


def test_scalar_write_forward_validation():
    """carve_chunk_fwd_sw: exactly one decay form (g, or f with A and tau_f),
    shapes and alignment are checked before any HIP call."""
    lib = carve.load_library()
    d = _dims()
    fake = ctypes.c_void_p(4096)
    # q, k, v, beta, g, f, A, tau_f, bx, wx, Ub, Vb, S0, o, S_T, S_chunks, ws, bytes, stream
    g_form = [fake] * 5 + [None, None, None] + [fake] * 4 + [None, fake, None, None, None, 0, None]
    f_form = [fake] * 4 + [None] + [fake] * 7 + [None, fake, None, None, None, 0, None]
    neither = list(g_form); neither[4] = None
    assert lib.carve_chunk_fwd_sw(ctypes.byref(d), *neither) == -1
    both = list(f_form); both[4] = fake
    assert lib.carve_chunk_fwd_sw(ctypes.byref(d), *both) == -7
    for null_at in (6, 7, 9, 10, 11):   # A, tau_f, wx, Ub, Vb
        a = list(f_form); a[null_at] = None
        assert lib.carve_chunk_fwd_sw(ctypes.byref(d), *a) == -1, null_at
    assert lib.carve_chunk_fwd_sw(ctypes.byref(_dims(T=100)), *g_form) == -2
    a = list(g_form); a[9] = ctypes.c_void_p(4096 + 2)   # wx misaligned
    assert lib.carve_chunk_fwd_sw(ctypes.byref(d), *a) == -4


def test_scalar_write_backward_validation():
    lib = carve.load_library()
    d = _dims()
    need = lib.carve_workspace_size(ctypes.byref(d), 1)
    ptrs = [ctypes.c_void_p(1 << 40 | (i << 32)) for i in range(30)]
    # q k v beta g f A tau bx wx Ub Vb S_chunks dO dS_T dq dk dv dbeta dg df dA dtau dbx dwx dUb dVb dS0
    g_form = list(ptrs[:28])
    for i in (5, 6, 7, 20, 21, 22):
        g_form[i] = None
    ws = ptrs[28]
    assert lib.carve_chunk_bwd_sw(ctypes.byref(d), *g_form, None, 0, None) == -5
    assert lib.carve_chunk_bwd_sw(ctypes.byref(d), *g_form, ws, need - 1, None) == -5
    a = list(g_form); a[19] = None                     # dg missing
    assert lib.carve_chunk_bwd_sw(ctypes.byref(d), *a, ws, need, None) == -1
    a = list(g_form); a[24] = a[15]                    # dwx aliases dq
    assert lib.carve_chunk_bwd_sw(ctypes.byref(d), *a, ws, need, None) == -3
    a = list(g_form); a[5] = ptrs[5]                   # g and f both given
    assert lib.carve_chunk_bwd_sw(ctypes.byref(d), *a, ws, need, None) == -7
    f_form = list(ptrs[:28]); f_form[4] = None; f_form[19] = None
    a = list(f_form); a[22] = None                     # dtau missing
    assert lib.carve_chunk_bwd_sw(ctypes.byref(d), *a, ws, need, None) == -1


@pytest.mark.parametrize("D,R,L,dt", [(128, 32, 64, carve.CARVE_BF16), (64, 16, 32, carve.CARVE_F32),
                                      (32, 40, 16, carve.CARVE_F32)])
def test_backward_workspace_holds_the_chunk_records(D, R, L, dt):
    """The backward workspace holds one record per chunk with at least the fold
    F (2RP x D), tau (L x 2RP) and the block start states (L/16 x D x D) in the
    token dtype and dF (2RP x D) in f32, RP = R rounded up to 32."""
    lib = carve.load_library()
    B, T, H = 2, 4 * L, 3
    d = carve.Dims(B, T, H, D, D, R, L, dt)
    e = 2 if dt == carve.CARVE_BF16 else 4
    RP = (R + 31) // 32 * 32
    per = 2 * RP * D * e + L * 2 * RP * e + (L // 16) * D * D * e + 2 * RP * D * 4
    assert lib.carve_workspace_size(ctypes.byref(d), 1) >= B * H * (T // L) * per


def test_rmsnorm_validation():
    lib = carve.load_library()
    fake = ctypes.c_void_p(4096)
    d = _dims(H=64, Dv=128)            # N = 8192 bf16: too long a row
    assert lib.carve_rmsnorm_fwd(ctypes.byref(d), fake, fake, 1e-6, fake, None) == -3
    assert lib.carve_rmsnorm_workspace_size(ctypes.byref(d)) == 0
    d = _dims(T=100)                   # T need not be a multiple of L for the norm
    assert lib.carve_rmsnorm_workspace_size(ctypes.byref(d)) > 0
    assert lib.carve_rmsnorm_fwd(ctypes.byref(d), None, fake, 1e-6, fake, None) == -1
    assert lib.carve_rmsnorm_fwd(ctypes.byref(d), fake, fake, -1.0, fake, None) == -7
    assert lib.carve_rmsnorm_fwd(ctypes.byref(d), fake, fake, float("nan"), fake, None) == -7
    assert lib.carve_rmsnorm_fwd(ctypes.byref(d), ctypes.c_void_p(4098), fake, 1e-6, fake, None) == -4
    assert lib.carve_rmsnorm_fwd(ctypes.byref(d), fake, fake, 1e-6, fake, None) == -3   # y aliases o
    ws = lib.carve_rmsnorm_workspace_size(ctypes.byref(d))
    assert lib.carve_rmsnorm_bwd(ctypes.byref(d), ctypes.c_void_p(1 << 20), ctypes.c_void_p(2 << 20), 1e-6,
                                 ctypes.c_void_p(3 << 20), ctypes.c_void_p(4 << 20), ctypes.c_void_p(5 << 20),
                                 ctypes.c_void_p(6 << 20), ws - 1, None) == -5
    d = _dims(B=0)
    assert lib.carve_rmsnorm_fwd(ctypes.byref(d), fake, fake, 1e-6, ctypes.c_void_p(8192), None) == -2
