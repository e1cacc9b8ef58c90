"""Thin Python binding of libcarve (C ABI in include/carve.h).

Argument marshalling only: tensors are allocated with PyTorch on the GPU,
their device pointers and the current HIP stream are handed to the C entry
points, and every step of the layer runs in the HIP kernels.  There is no
fallback: if libcarve.so is missing or a tensor is not a contiguous GPU
tensor of the right dtype, the call raises.
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libcarve.so")

CARVE_F32, CARVE_BF16 = 0, 1
SYMBOLS = ("carve_chunk_fwd", "carve_chunk_bwd", "carve_chunk_fwd_gated", "carve_chunk_bwd_gated",
           "carve_chunk_fwd_sw", "carve_chunk_bwd_sw", "carve_chunk_fwd_act", "carve_chunk_bwd_act",
           "carve_rmsnorm_fwd", "carve_rmsnorm_bwd", "carve_rmsnorm_workspace_size", "carve_rmsnorm_bwd_noalloc",
           "carve_workspace_size", "carve_status_string", "carve_profile_events", "carve_bwd_wait_status",
           "carve_set_ready_wait_limit")


class Dims(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int), ("T", ctypes.c_int), ("H", ctypes.c_int), ("Dk", ctypes.c_int),
                ("Dv", ctypes.c_int), ("R", ctypes.c_int), ("L", ctypes.c_int), ("dtype", ctypes.c_int)]


class CarveError(RuntimeError):
    def __init__(self, fn, status, msg):
        super().__init__(f"{fn} failed with status {status}: {msg}")
        self.status = status


_lib = None


def load_library(path: str = LIB_PATH):
    """Load libcarve.so (no GPU needed).  Raises if it has not been built."""
    global _lib
    if _lib is not None and path == LIB_PATH:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} not found: build it with paper_2606_27229_amd.build.build()")
    lib = ctypes.CDLL(path)
    vp, fp, sz = ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t
    D = ctypes.POINTER(Dims)
    lib.carve_workspace_size.argtypes = [D, ctypes.c_int]
    lib.carve_workspace_size.restype = sz
    lib.carve_status_string.argtypes = [ctypes.c_int]
    lib.carve_status_string.restype = ctypes.c_char_p
    lib.carve_chunk_fwd.argtypes = [D] + [vp] * 7 + [fp] * 5 + [vp, fp, fp, vp, sz, vp]
    lib.carve_chunk_fwd.restype = ctypes.c_int
    lib.carve_chunk_bwd.argtypes = [D] + [vp] * 7 + [fp] * 5 + [vp, fp] + [vp] * 12 + [vp, sz, vp]
    lib.carve_chunk_bwd.restype = ctypes.c_int
    lib.carve_chunk_fwd_gated.argtypes = [D] + [vp] * 5 + [fp] * 2 + [vp] * 2 + [fp] * 5 + [vp, fp, fp, vp, sz, vp]
    lib.carve_chunk_fwd_gated.restype = ctypes.c_int
    lib.carve_chunk_bwd_gated.argtypes = ([D] + [vp] * 5 + [fp] * 2 + [vp] * 2 + [fp] * 5 + [vp, fp]
                                          + [vp] * 5 + [fp] * 2 + [vp] * 2 + [fp] * 5 + [vp, sz, vp])
    lib.carve_chunk_bwd_gated.restype = ctypes.c_int
    lib.carve_chunk_fwd_sw.argtypes = [D] + [vp] * 4 + [fp, vp, fp, fp, vp, vp, fp, fp, fp, vp, fp, fp, vp, sz, vp]
    lib.carve_chunk_fwd_sw.restype = ctypes.c_int
    lib.carve_chunk_bwd_sw.argtypes = ([D] + [vp] * 4 + [fp, vp, fp, fp, vp, vp, fp, fp, fp, vp, fp]
                                       + [vp] * 4 + [fp, vp, fp, fp, vp, vp, fp, fp, fp, vp, sz, vp])
    lib.carve_chunk_bwd_sw.restype = ctypes.c_int
    lib.carve_chunk_fwd_act.argtypes = lib.carve_chunk_fwd.argtypes
    lib.carve_chunk_fwd_act.restype = ctypes.c_int
    lib.carve_chunk_bwd_act.argtypes = lib.carve_chunk_bwd.argtypes
    lib.carve_chunk_bwd_act.restype = ctypes.c_int
    lib.carve_rmsnorm_fwd.argtypes = [D, vp, fp, ctypes.c_float, vp, vp]
    lib.carve_rmsnorm_fwd.restype = ctypes.c_int
    lib.carve_rmsnorm_bwd.argtypes = [D, vp, fp, ctypes.c_float, vp, vp, fp, vp, sz, vp]
    lib.carve_rmsnorm_bwd.restype = ctypes.c_int
    lib.carve_rmsnorm_bwd_noalloc.argtypes = [D, vp, fp, ctypes.c_float, vp, vp, fp, vp]
    lib.carve_rmsnorm_bwd_noalloc.restype = ctypes.c_int
    lib.carve_rmsnorm_workspace_size.argtypes = [D]
    lib.carve_rmsnorm_workspace_size.restype = sz
    lib.carve_profile_events.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_int]
    lib.carve_profile_events.restype = ctypes.c_int
    lib.carve_bwd_wait_status.argtypes = [D, vp, vp, ctypes.POINTER(ctypes.c_int)]
    lib.carve_bwd_wait_status.restype = ctypes.c_int
    lib.carve_set_ready_wait_limit.argtypes = [ctypes.c_int]
    lib.carve_set_ready_wait_limit.restype = ctypes.c_int
    if path == LIB_PATH:
        _lib = lib
    return lib


def status_string(st: int) -> str:
    return load_library().carve_status_string(st).decode()


def profile_events(events) -> None:
    """Arm the next chunk_fwd / chunk_bwd call on this thread to record the
    given torch.cuda.Event objects at its kernel-launch boundaries (measurement
    only).  The events must already exist on the device (record each once)."""
    arr = (ctypes.c_void_p * len(events))(*[e.cuda_event for e in events])
    _check("carve_profile_events", load_library().carve_profile_events(arr, len(events)))


def bwd_wait_status(dims: Dims, workspace, stream=None) -> bool:
    """Whether an adjoint wave's bounded wait for a chunk record ran out in the
    last backward made with this workspace (synchronises the stream)."""
    out = ctypes.c_int(0)
    _check("carve_bwd_wait_status", load_library().carve_bwd_wait_status(
        ctypes.byref(dims), _ptr(workspace, "workspace"), _stream(stream), ctypes.byref(out)))
    return bool(out.value)


def set_ready_wait_limit(polls: int) -> int:
    """Test hook: the bound of the backward's record wait for calls on this
    thread (negative: the default).  Returns the previous bound."""
    return int(load_library().carve_set_ready_wait_limit(int(polls)))


def make_dims(B, T, H, Dk, Dv, R, L, dtype) -> Dims:
    return Dims(B, T, H, Dk, Dv, R, L, CARVE_BF16 if dtype == torch.bfloat16 else CARVE_F32)


def workspace_size(dims: Dims, backward: bool) -> int:
    return int(load_library().carve_workspace_size(ctypes.byref(dims), 1 if backward else 0))


def _ptr(t, name, dtype=None, shape=None):
    if t is None:
        return None
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a GPU tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    return t.data_ptr()


def _stream(stream):
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


def _check(fn, st):
    if st != 0:
        raise CarveError(fn, st, status_string(st))


def chunk_fwd(q, k, v, beta, g, bx, wx, Ub, Uw, Vb, Vw, S0=None, *, L=64, want_chunks=True,
              want_state=True, out=None, stream=None, act=False):
    """Forward of the chunked CARVE layer.

    Shapes: q, k, bx, g [B,T,H,Dk]; v, wx [B,T,H,Dv]; beta [B,T,H]; Ub, Uw [R,Dv];
    Vb [Dk,R]; Vw [Dv,R]; S0 [B,H,Dv,Dk] or None.  Returns (o, S_T, S_chunks).
    ``out`` may hold preallocated {"o", "S_T", "S_chunks"} tensors.  act=True:
    q, k, v are the raw projections and the kernels apply SiLU (+ L2 norm for
    q, k) (carve_chunk_fwd_act).
    """
    lib = load_library()
    B, T, H, Dk = q.shape
    Dv = v.shape[-1]
    R = Ub.shape[0]
    dt = q.dtype
    f32 = torch.float32
    dims = make_dims(B, T, H, Dk, Dv, R, L, dt)
    out = dict(out or {})
    o = out.get("o")
    if o is None:
        o = torch.empty((B, T, H, Dv), dtype=dt, device=q.device)
    S_T = out.get("S_T") if "S_T" in out else (torch.empty((B, H, Dv, Dk), dtype=f32, device=q.device) if want_state else None)
    S_chunks = out.get("S_chunks") if "S_chunks" in out else (
        torch.empty((B, H, T // L, Dv, Dk), dtype=f32, device=q.device) if want_chunks else None)
    fn = "carve_chunk_fwd_act" if act else "carve_chunk_fwd"
    st = getattr(lib, fn)(
        ctypes.byref(dims), _ptr(q, "q", dt, (B, T, H, Dk)), _ptr(k, "k", dt, (B, T, H, Dk)),
        _ptr(v, "v", dt, (B, T, H, Dv)), _ptr(beta, "beta", dt, (B, T, H)), _ptr(g, "g", f32, (B, T, H, Dk)),
        _ptr(bx, "bx", dt, (B, T, H, Dk)), _ptr(wx, "wx", dt, (B, T, H, Dv)),
        _ptr(Ub, "Ub", f32, (R, Dv)), _ptr(Uw, "Uw", f32, (R, Dv)), _ptr(Vb, "Vb", f32, (Dk, R)),
        _ptr(Vw, "Vw", f32, (Dv, R)), _ptr(S0, "S0", f32, (B, H, Dv, Dk)),
        _ptr(o, "o", dt, (B, T, H, Dv)), _ptr(S_T, "S_T", f32), _ptr(S_chunks, "S_chunks", f32),
        None, 0, _stream(stream))
    _check(fn, st)
    return o, S_T, S_chunks


def chunk_bwd(q, k, v, beta, g, bx, wx, Ub, Uw, Vb, Vw, S_chunks, dO, dS_T=None, *, L=64,
              want_dS0=True, out=None, workspace=None, stream=None, act=False):
    """Backward of the chunked CARVE layer for loss <dO, o> + <dS_T, S_T>.

    Returns a dict with dq, dk, dv, dbeta, dg, dbx, dwx, dUb, dUw, dVb, dVw, dS0.
    act=True: the backward of chunk_fwd(act=True) (gradients of the raw q, k, v).
    """
    lib = load_library()
    B, T, H, Dk = q.shape
    Dv = v.shape[-1]
    R = Ub.shape[0]
    dt = q.dtype
    f32 = torch.float32
    dev = q.device
    dims = make_dims(B, T, H, Dk, Dv, R, L, dt)
    res = dict(out or {})
    spec = {"dq": ((B, T, H, Dk), dt), "dk": ((B, T, H, Dk), dt), "dv": ((B, T, H, Dv), dt),
            "dbeta": ((B, T, H), dt), "dg": ((B, T, H, Dk), f32), "dbx": ((B, T, H, Dk), dt),
            "dwx": ((B, T, H, Dv), dt), "dUb": ((R, Dv), f32), "dUw": ((R, Dv), f32),
            "dVb": ((Dk, R), f32), "dVw": ((Dv, R), f32)}
    if want_dS0:
        spec["dS0"] = ((B, H, Dv, Dk), f32)
    for name, (shape, dtype) in spec.items():
        if res.get(name) is None:
            res[name] = torch.empty(shape, dtype=dtype, device=dev)
    ws_bytes = workspace_size(dims, True)
    if workspace is None and ws_bytes:
        workspace = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    ws_ptr = _ptr(workspace, "workspace") if workspace is not None else None
    ws_len = workspace.numel() * workspace.element_size() if workspace is not None else 0
    fn = "carve_chunk_bwd_act" if act else "carve_chunk_bwd"
    st = getattr(lib, fn)(
        ctypes.byref(dims), _ptr(q, "q", dt, (B, T, H, Dk)), _ptr(k, "k", dt, (B, T, H, Dk)),
        _ptr(v, "v", dt, (B, T, H, Dv)), _ptr(beta, "beta", dt, (B, T, H)), _ptr(g, "g", f32, (B, T, H, Dk)),
        _ptr(bx, "bx", dt, (B, T, H, Dk)), _ptr(wx, "wx", dt, (B, T, H, Dv)),
        _ptr(Ub, "Ub", f32, (R, Dv)), _ptr(Uw, "Uw", f32, (R, Dv)), _ptr(Vb, "Vb", f32, (Dk, R)),
        _ptr(Vw, "Vw", f32, (Dv, R)), _ptr(S_chunks, "S_chunks", f32, (B, H, T // L, Dv, Dk)),
        _ptr(dO, "dO", dt, (B, T, H, Dv)), _ptr(dS_T, "dS_T", f32, (B, H, Dv, Dk)),
        *[_ptr(res[n], n) for n in ("dq", "dk", "dv", "dbeta", "dg", "dbx", "dwx", "dUb", "dUw", "dVb", "dVw")],
        _ptr(res.get("dS0"), "dS0"), ws_ptr, ws_len, _stream(stream))
    _check(fn, st)
    return res


def chunk_fwd_gated(q, k, v, beta, f, A, tau_f, bx, wx, Ub, Uw, Vb, Vw, S0=None, *, L=64,
                    want_chunks=True, want_state=True, out=None, stream=None):
    """Forward with the decay computed in the kernels from its raw logit f
    (g = -exp(A) softplus(f + tau_f)).  f [B,T,H,Dk] has the token dtype; A and
    tau_f are f32 [H,Dk].  Returns (o, S_T, S_chunks)."""
    lib = load_library()
    B, T, H, Dk = q.shape
    Dv = v.shape[-1]
    R = Ub.shape[0]
    dt = q.dtype
    f32 = torch.float32
    dims = make_dims(B, T, H, Dk, Dv, R, L, dt)
    out = dict(out or {})
    o = out.get("o")
    if o is None:
        o = torch.empty((B, T, H, Dv), dtype=dt, device=q.device)
    S_T = out.get("S_T") if "S_T" in out else (torch.empty((B, H, Dv, Dk), dtype=f32, device=q.device) if want_state else None)
    S_chunks = out.get("S_chunks") if "S_chunks" in out else (
        torch.empty((B, H, T // L, Dv, Dk), dtype=f32, device=q.device) if want_chunks else None)
    st = lib.carve_chunk_fwd_gated(
        ctypes.byref(dims), _ptr(q, "q", dt, (B, T, H, Dk)), _ptr(k, "k", dt, (B, T, H, Dk)),
        _ptr(v, "v", dt, (B, T, H, Dv)), _ptr(beta, "beta", dt, (B, T, H)), _ptr(f, "f", dt, (B, T, H, Dk)),
        _ptr(A, "A", f32, (H, Dk)), _ptr(tau_f, "tau_f", f32, (H, Dk)),
        _ptr(bx, "bx", dt, (B, T, H, Dk)), _ptr(wx, "wx", dt, (B, T, H, Dv)),
        _ptr(Ub, "Ub", f32, (R, Dv)), _ptr(Uw, "Uw", f32, (R, Dv)), _ptr(Vb, "Vb", f32, (Dk, R)),
        _ptr(Vw, "Vw", f32, (Dv, R)), _ptr(S0, "S0", f32, (B, H, Dv, Dk)),
        _ptr(o, "o", dt, (B, T, H, Dv)), _ptr(S_T, "S_T", f32), _ptr(S_chunks, "S_chunks", f32),
        None, 0, _stream(stream))
    _check("carve_chunk_fwd_gated", st)
    return o, S_T, S_chunks


def chunk_bwd_gated(q, k, v, beta, f, A, tau_f, bx, wx, Ub, Uw, Vb, Vw, S_chunks, dO, dS_T=None, *, L=64,
                    want_dS0=True, out=None, workspace=None, stream=None):
    """Backward of ``chunk_fwd_gated``: the gradients of ``chunk_bwd`` with dg
    replaced by df (token dtype), dA and dtau ([H,Dk] f32)."""
    lib = load_library()
    B, T, H, Dk = q.shape
    Dv = v.shape[-1]
    R = Ub.shape[0]
    dt = q.dtype
    f32 = torch.float32
    dev = q.device
    dims = make_dims(B, T, H, Dk, Dv, R, L, dt)
    res = dict(out or {})
    spec = {"dq": ((B, T, H, Dk), dt), "dk": ((B, T, H, Dk), dt), "dv": ((B, T, H, Dv), dt),
            "dbeta": ((B, T, H), dt), "df": ((B, T, H, Dk), dt), "dA": ((H, Dk), f32), "dtau": ((H, Dk), f32),
            "dbx": ((B, T, H, Dk), dt), "dwx": ((B, T, H, Dv), dt), "dUb": ((R, Dv), f32),
            "dUw": ((R, Dv), f32), "dVb": ((Dk, R), f32), "dVw": ((Dv, R), f32)}
    if want_dS0:
        spec["dS0"] = ((B, H, Dv, Dk), f32)
    for name, (shape, dtype) in spec.items():
        if res.get(name) is None:
            res[name] = torch.empty(shape, dtype=dtype, device=dev)
    ws_bytes = workspace_size(dims, True)
    if workspace is None and ws_bytes:
        workspace = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    ws_ptr = _ptr(workspace, "workspace") if workspace is not None else None
    ws_len = workspace.numel() * workspace.element_size() if workspace is not None else 0
    st = lib.carve_chunk_bwd_gated(
        ctypes.byref(dims), _ptr(q, "q", dt, (B, T, H, Dk)), _ptr(k, "k", dt, (B, T, H, Dk)),
        _ptr(v, "v", dt, (B, T, H, Dv)), _ptr(beta, "beta", dt, (B, T, H)), _ptr(f, "f", dt, (B, T, H, Dk)),
        _ptr(A, "A", f32, (H, Dk)), _ptr(tau_f, "tau_f", f32, (H, Dk)),
        _ptr(bx, "bx", dt, (B, T, H, Dk)), _ptr(wx, "wx", dt, (B, T, H, Dv)),
        _ptr(Ub, "Ub", f32, (R, Dv)), _ptr(Uw, "Uw", f32, (R, Dv)), _ptr(Vb, "Vb", f32, (Dk, R)),
        _ptr(Vw, "Vw", f32, (Dv, R)), _ptr(S_chunks, "S_chunks", f32, (B, H, T // L, Dv, Dk)),
        _ptr(dO, "dO", dt, (B, T, H, Dv)), _ptr(dS_T, "dS_T", f32, (B, H, Dv, Dk)),
        *[_ptr(res[n], n) for n in ("dq", "dk", "dv", "dbeta", "df", "dA", "dtau", "dbx", "dwx",
                                    "dUb", "dUw", "dVb", "dVw")],
        _ptr(res.get("dS0"), "dS0"), ws_ptr, ws_len, _stream(stream))
    _check("carve_chunk_bwd_gated", st)
    return res


def chunk_fwd_sw(q, k, v, beta, bx, wx, Ub, Vb, S0=None, *, g=None, f=None, A=None, tau_f=None, L=64,
                 want_chunks=True, want_state=True, out=None, stream=None):
    """Forward with the scalar write gate: wx [B,T,H] (one logit per token and
    head, w = sigmoid(wx) on every value channel), no Uw, Vw.  The decay is g
    (f32 [B,T,H,Dk]) or, with g=None, formed in the kernels from f, A, tau_f.
    Returns (o, S_T, S_chunks)."""
    lib = load_library()
    B, T, H, Dk = q.shape
    Dv = v.shape[-1]
    R = Ub.shape[0]
    dt = q.dtype
    f32 = torch.float32
    dims = make_dims(B, T, H, Dk, Dv, R, L, dt)
    out = dict(out or {})
    o = out.get("o")
    if o is None:
        o = torch.empty((B, T, H, Dv), dtype=dt, device=q.device)
    S_T = out.get("S_T") if "S_T" in out else (torch.empty((B, H, Dv, Dk), dtype=f32, device=q.device) if want_state else None)
    S_chunks = out.get("S_chunks") if "S_chunks" in out else (
        torch.empty((B, H, T // L, Dv, Dk), dtype=f32, device=q.device) if want_chunks else None)
    st = lib.carve_chunk_fwd_sw(
        ctypes.byref(dims), _ptr(q, "q", dt, (B, T, H, Dk)), _ptr(k, "k", dt, (B, T, H, Dk)),
        _ptr(v, "v", dt, (B, T, H, Dv)), _ptr(beta, "beta", dt, (B, T, H)), _ptr(g, "g", f32, (B, T, H, Dk)),
        _ptr(f, "f", dt, (B, T, H, Dk)), _ptr(A, "A", f32, (H, Dk)), _ptr(tau_f, "tau_f", f32, (H, Dk)),
        _ptr(bx, "bx", dt, (B, T, H, Dk)), _ptr(wx, "wx", dt, (B, T, H)),
        _ptr(Ub, "Ub", f32, (R, Dv)), _ptr(Vb, "Vb", f32, (Dk, R)), _ptr(S0, "S0", f32, (B, H, Dv, Dk)),
        _ptr(o, "o", dt, (B, T, H, Dv)), _ptr(S_T, "S_T", f32), _ptr(S_chunks, "S_chunks", f32),
        None, 0, _stream(stream))
    _check("carve_chunk_fwd_sw", st)
    return o, S_T, S_chunks


def chunk_bwd_sw(q, k, v, beta, bx, wx, Ub, Vb, S_chunks, dO, dS_T=None, *, g=None, f=None, A=None, tau_f=None,
                 L=64, want_dS0=True, out=None, workspace=None, stream=None):
    """Backward of ``chunk_fwd_sw``: dq, dk, dv, dbeta, dbx, dwx [B,T,H], dUb,
    dVb, dS0, and dg (g given) or df, dA, dtau (f given)."""
    lib = load_library()
    B, T, H, Dk = q.shape
    Dv = v.shape[-1]
    R = Ub.shape[0]
    dt = q.dtype
    f32 = torch.float32
    dev = q.device
    dims = make_dims(B, T, H, Dk, Dv, R, L, dt)
    res = dict(out or {})
    spec = {"dq": ((B, T, H, Dk), dt), "dk": ((B, T, H, Dk), dt), "dv": ((B, T, H, Dv), dt),
            "dbeta": ((B, T, H), dt), "dbx": ((B, T, H, Dk), dt), "dwx": ((B, T, H), dt),
            "dUb": ((R, Dv), f32), "dVb": ((Dk, R), f32)}
    if f is None:
        spec["dg"] = ((B, T, H, Dk), f32)
    else:
        spec.update({"df": ((B, T, H, Dk), dt), "dA": ((H, Dk), f32), "dtau": ((H, Dk), f32)})
    if want_dS0:
        spec["dS0"] = ((B, H, Dv, Dk), f32)
    for name, (shape, dtype) in spec.items():
        if res.get(name) is None:
            res[name] = torch.empty(shape, dtype=dtype, device=dev)
    ws_bytes = workspace_size(dims, True)
    if workspace is None and ws_bytes:
        workspace = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    ws_ptr = _ptr(workspace, "workspace") if workspace is not None else None
    ws_len = workspace.numel() * workspace.element_size() if workspace is not None else 0
    st = lib.carve_chunk_bwd_sw(
        ctypes.byref(dims), _ptr(q, "q", dt, (B, T, H, Dk)), _ptr(k, "k", dt, (B, T, H, Dk)),
        _ptr(v, "v", dt, (B, T, H, Dv)), _ptr(beta, "beta", dt, (B, T, H)), _ptr(g, "g", f32, (B, T, H, Dk)),
        _ptr(f, "f", dt, (B, T, H, Dk)), _ptr(A, "A", f32, (H, Dk)), _ptr(tau_f, "tau_f", f32, (H, Dk)),
        _ptr(bx, "bx", dt, (B, T, H, Dk)), _ptr(wx, "wx", dt, (B, T, H)),
        _ptr(Ub, "Ub", f32, (R, Dv)), _ptr(Vb, "Vb", f32, (Dk, R)),
        _ptr(S_chunks, "S_chunks", f32, (B, H, T // L, Dv, Dk)),
        _ptr(dO, "dO", dt, (B, T, H, Dv)), _ptr(dS_T, "dS_T", f32, (B, H, Dv, Dk)),
        *[_ptr(res.get(n), n) for n in ("dq", "dk", "dv", "dbeta", "dg", "df", "dA", "dtau", "dbx", "dwx",
                                        "dUb", "dVb", "dS0")],
        ws_ptr, ws_len, _stream(stream))
    _check("carve_chunk_bwd_sw", st)
    return res


RMSNORM_EPS = 1e-6


def _norm_dims(o):
    B, T, H, Dv = o.shape
    # only B, T, H, Dv and dtype are read by the norm entry points
    return make_dims(B, T, H, Dv, Dv, 1, 1, o.dtype)


def rmsnorm_fwd(o, weight, *, eps=RMSNORM_EPS, out=None, stream=None):
    """Output RMS normalisation of the layer output o [B,T,H,Dv] over each
    token's H*Dv values (Alg. carve_fwd's last step, without W_O):
    y = o / sqrt(mean(o^2) + eps) * weight, weight [H*Dv] f32."""
    lib = load_library()
    B, T, H, Dv = o.shape
    dims = _norm_dims(o)
    y = out if out is not None else torch.empty_like(o)
    st = lib.carve_rmsnorm_fwd(ctypes.byref(dims), _ptr(o, "o", o.dtype, (B, T, H, Dv)),
                               _ptr(weight, "weight", torch.float32, (H * Dv,)), float(eps),
                               _ptr(y, "y", o.dtype, (B, T, H, Dv)), _stream(stream))
    _check("carve_rmsnorm_fwd", st)
    return y


def rmsnorm_bwd(o, weight, dy, *, eps=RMSNORM_EPS, out=None, workspace=None, stream=None):
    """Backward of ``rmsnorm_fwd`` for loss <dy, y>: returns (d_o, dweight)."""
    lib = load_library()
    B, T, H, Dv = o.shape
    dims = _norm_dims(o)
    res = dict(out or {})
    d_o = res.get("d_o")
    if d_o is None:
        d_o = torch.empty_like(o)
    dw = res.get("dweight")
    if dw is None:
        dw = torch.empty((H * Dv,), dtype=torch.float32, device=o.device)
    ws_bytes = int(lib.carve_rmsnorm_workspace_size(ctypes.byref(dims)))
    if workspace is None:
        workspace = torch.empty(max(ws_bytes, 16), dtype=torch.uint8, device=o.device)
    ws_len = workspace.numel() * workspace.element_size()
    st = lib.carve_rmsnorm_bwd(ctypes.byref(dims), _ptr(o, "o", o.dtype, (B, T, H, Dv)),
                               _ptr(weight, "weight", torch.float32, (H * Dv,)), float(eps),
                               _ptr(dy, "dy", o.dtype, (B, T, H, Dv)), _ptr(d_o, "d_o", o.dtype, (B, T, H, Dv)),
                               _ptr(dw, "dweight", torch.float32, (H * Dv,)), _ptr(workspace, "workspace"),
                               ws_len, _stream(stream))
    _check("carve_rmsnorm_bwd", st)
    return d_o, dw


def rmsnorm_bwd_noalloc(o, weight, dy, d_o, dweight, *, eps=RMSNORM_EPS, stream=None):
    """``rmsnorm_bwd`` through the entry point that allocates nothing (its
    scratch is the library's static per-device array): the caller passes the
    outputs d_o (like o) and dweight ([H*Dv] f32)."""
    lib = load_library()
    B, T, H, Dv = o.shape
    dims = _norm_dims(o)
    st = lib.carve_rmsnorm_bwd_noalloc(ctypes.byref(dims), _ptr(o, "o", o.dtype, (B, T, H, Dv)),
                                       _ptr(weight, "weight", torch.float32, (H * Dv,)), float(eps),
                                       _ptr(dy, "dy", o.dtype, (B, T, H, Dv)),
                                       _ptr(d_o, "d_o", o.dtype, (B, T, H, Dv)),
                                       _ptr(dweight, "dweight", torch.float32, (H * Dv,)), _stream(stream))
    _check("carve_rmsnorm_bwd_noalloc", st)
    return d_o, dweight
