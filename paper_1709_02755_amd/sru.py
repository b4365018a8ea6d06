"""Thin Python binding of libsru.so (argument marshalling only).

Every step of the layer runs in the HIP library; this module checks tensor
devices/dtypes/shapes, allocates outputs with torch (device memory and
streams are torch's job here) and passes raw pointers through ctypes.  There
is no fallback: if the library cannot be loaded, every call raises.
"""

from __future__ import annotations

import ctypes
import os
import threading

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
# SRU_LIBRARY names another build of the same library (e.g. the host-side
# sanitizer build the ABI tests run against); it must exist
LIB_PATH = os.environ.get("SRU_LIBRARY") or os.path.join(_PKG, "libsru.so")

SRU_OK = 0
DIR_FWD, DIR_REV, DIR_BI = 0, 1, 2
GEMM_FP32, GEMM_BF16 = 0, 1
OP_NT, OP_NN, OP_TN = 0, 1, 2

_lock = threading.Lock()
_lib = None

_P = ctypes.c_void_p
_I = ctypes.c_int
_S = ctypes.c_size_t

# name -> (restype, argtypes); mirrors include/sru.h
_SIGNATURES = {
    "sru_status_string": (ctypes.c_char_p, [_I]),
    "sru_last_hip_error": (_I, []),
    "sru_version": (_I, []),
    "sru_forward_workspace_bytes": (_S, [_I] * 6),
    "sru_backward_workspace_bytes": (_S, [_I] * 6),
    "sru_forward": (_I, [_P] * 7 + [_I] * 5 + [_P, _I, _P] + [_P] * 4 + [_P] * 3
                    + [_P, _S, _P]),
    "sru_forward_noalloc": (_I, [_P] * 7 + [_I] * 5 + [_P, _I, _P] + [_P] * 4 + [_P] * 3
                            + [_P]),
    "sru_backward": (_I, [_P] * 7 + [_I] * 5 + [_P, _I, _P] + [_P] * 4 + [_P] * 7 + [_P] * 2
                     + [_P, _S, _P]),
    "sru_gemm_workspace_bytes": (_S, [_I] * 5),
    "sru_gemm": (_I, [_I] * 5 + [_P, _I, _P, _I, _P, _I] + [_P, _S, _P]),
    "sru_scan_forward_workspace_bytes": (_S, [_I] * 5),
    "sru_scan_forward": (_I, [_P] * 7 + [_I] * 5 + [_P, _P] + [_P] * 3 + [_P] + [_P, _S, _P]),
    "sru_scan_backward_workspace_bytes": (_S, [_I] * 5),
    "sru_scan_backward": (_I, [_P] * 10 + [_I] * 5 + [_P, _P] + [_P] * 7 + [_P, _S, _P]),
    "sru_forward_lowrank_workspace_bytes": (_S, [_I] * 7),
    "sru_backward_lowrank_workspace_bytes": (_S, [_I] * 7),
    "sru_forward_lowrank": (_I, [_P] * 8 + [_I] * 6 + [_P, _I, _P] + [_P] * 5 + [_P] * 3
                            + [_P, _S, _P]),
    "sru_backward_lowrank": (_I, [_P] * 8 + [_I] * 6 + [_P, _I, _P] + [_P] * 5 + [_P] * 8
                             + [_P] * 2 + [_P, _S, _P]),
    "sru_round_bf16": (_I, [_P, _S, _P, _P]),
    "sru_forward_fused_available": (_I, [_I] * 6),
    "sru_timing_begin": (_I, [_P, _I]),
    "sru_timing_end": (_I, []),
    "sru_timing_label": (ctypes.c_char_p, [_I]),
}


class SruError(RuntimeError):
    pass


RESET_PREV, RESET_NEW = 0, 1
RECURRENCE_GATED, RECURRENCE_LINEAR = 0, 1


class Options(ctypes.Structure):
    """sru_options: highway_scale (alpha, Sec. 3.2), reset_state
    (RESET_PREV: Eq. 3; RESET_NEW: Algorithm 1's order) and recurrence
    (RECURRENCE_LINEAR: v * c removed from both gates, ablation (1) of
    Sec. 4.5; v_f, v_r may then be None and have no gradient)."""
    _fields_ = [("highway_scale", ctypes.c_float), ("reset_state", ctypes.c_int),
                ("recurrence", ctypes.c_int)]


def _options(highway_scale=1.0, reset_new=False, linear=False):
    """NULL for Eq. 1-4 as printed, else a pointer to an sru_options."""
    if highway_scale == 1.0 and not reset_new and not linear:
        return None
    return ctypes.byref(Options(float(highway_scale), RESET_NEW if reset_new else RESET_PREV,
                                RECURRENCE_LINEAR if linear else RECURRENCE_GATED))


def lib():
    """Load libsru.so (building it first only if it has never been built)."""
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(LIB_PATH):
                if os.environ.get("SRU_LIBRARY"):
                    raise OSError(f"SRU_LIBRARY={LIB_PATH} does not exist")
                from . import build as _build
                _build.build()
            h = ctypes.CDLL(LIB_PATH)
            for name, (res, args) in _SIGNATURES.items():
                fn = getattr(h, name)
                fn.restype = res
                fn.argtypes = args
            _lib = h
    return _lib


def exported_symbols():
    return list(_SIGNATURES)


def _check(status: int, what: str):
    if status != SRU_OK:
        msg = lib().sru_status_string(status).decode()
        if status == 5:
            msg += f" (hipError {lib().sru_last_hip_error()})"
        raise SruError(f"{what}: {msg}")


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _on_gpu(t):
    return t.is_cuda


def _req(t, name, shape, dtype=torch.float32, optional=False, device=None):
    """A GPU tensor of this shape and dtype, contiguous, on `device` (if given)."""
    if t is None:
        if optional:
            return
        raise ValueError(f"{name} is required")
    if not isinstance(t, torch.Tensor):
        raise ValueError(f"{name} must be a torch tensor")
    if not _on_gpu(t):
        raise ValueError(f"{name} must be a GPU tensor")
    if device is not None and t.device != device:
        raise ValueError(f"{name} is on {t.device}, expected {device}")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")


def _req_out(out, specs, device):
    """Check the caller-supplied output buffers of `out` against
    name -> (shape, dtype, required)."""
    for name, (shape, dtype, required) in specs.items():
        _req(out.get(name), name, shape, dtype=dtype, optional=not required, device=device)


def _ws(ws, need, device):
    """(workspace tensor or None, its size in bytes).  A caller's workspace
    must be a contiguous uint8 GPU tensor on `device`; its real size is what
    the library is told, so the library's own size check applies."""
    if ws is None:
        if not need:
            return None, 0
        ws = workspace(need, device)
    _req(ws, "ws", (ws.numel(),), dtype=torch.uint8, device=device)
    return ws, ws.numel() * ws.element_size()


def dims(X, W):
    L, B, d_in = X.shape
    ndir, k, d, _ = W.shape
    return L, B, d_in, d, ndir, k


def _check_params(X, W, v_f, v_r, b_f, b_r, c0, direction, mask, gemm_dtype=GEMM_FP32):
    for n, t, nd in (("X", X, 3), ("W", W, 4)):
        if not isinstance(t, torch.Tensor) or t.dim() != nd:
            raise ValueError(f"{n} must be a {nd}-d tensor")
    _req(X, "X", tuple(X.shape))
    L, B, d_in, d, ndir, k = dims(X, W)
    want_nd = 2 if direction == DIR_BI else 1
    if ndir != want_nd or k != (3 if d_in == d else 4):
        raise ValueError(f"W shape {tuple(W.shape)} does not fit d_in={d_in}, direction={direction}")
    dv = X.device
    # bf16 products take the weights already rounded as a bfloat16 W
    w_dtype = torch.bfloat16 if W.dtype == torch.bfloat16 else torch.float32
    if w_dtype == torch.bfloat16 and gemm_dtype != GEMM_BF16:
        raise ValueError("a bfloat16 W needs bf16 products (gemm_dtype=GEMM_BF16)")
    _req(W, "W", (ndir, k, d, d_in), dtype=w_dtype, device=dv)
    for n, t in (("v_f", v_f), ("v_r", v_r)):
        _req(t, n, (ndir, d), optional=True, device=dv)  # the library reports a missing v
    for n, t in (("b_f", b_f), ("b_r", b_r)):
        _req(t, n, (ndir, d), device=dv)
    _req(c0, "c0", (B, ndir * d), optional=True, device=dv)
    _req(mask, "mask", (L, B), dtype=torch.uint8, optional=True, device=dv)
    return L, B, d_in, d, ndir, k


def _weights(W, W_bf16):
    """(W, W_bf16) as the library takes them: a bfloat16 W is the rounded
    weights, passed as W_bf16 with W = NULL."""
    if W.dtype != torch.bfloat16:
        return W, W_bf16
    if W_bf16 is not None:
        raise ValueError("W is already bfloat16: pass no W_bf16 beside it")
    return None, W


def forward_workspace_bytes(L, B, d_in, d, direction, gemm_dtype):
    return lib().sru_forward_workspace_bytes(L, B, d_in, d, direction, gemm_dtype)


def backward_workspace_bytes(L, B, d_in, d, direction, gemm_dtype):
    return lib().sru_backward_workspace_bytes(L, B, d_in, d, direction, gemm_dtype)


def workspace(nbytes, device):
    return torch.empty(max(int(nbytes), 1), dtype=torch.uint8, device=device)


def fused_available(L, B, d_in, d, direction, gemm_dtype):
    """Whether forward() can run without U and C (fused projection + scan)."""
    return bool(lib().sru_forward_fused_available(L, B, d_in, d, direction, gemm_dtype))


def forward(X, W, v_f, v_r, b_f, b_r, c0=None, direction=DIR_FWD, mask=None,
            gemm_dtype=GEMM_FP32, store_c=True, out=None, ws=None, X_bf16=None,
            highway_scale=1.0, reset_new=False, linear=False, keep_u=True):
    """One layer forward; returns dict(U, H, C, c_last) (C None without store_c).

    keep_u=False with store_c=False: U is not kept either, where
    fused_available() allows it (U is then None).

    bf16 GEMMs only: X_bf16 (torch.bfloat16, X rounded) replaces the
    rounding of X; entries W_bf16 / H_bf16 of `out` (bfloat16 tensors), if
    present, receive Wcat and H rounded to bf16.  W itself may be bfloat16:
    the weights already rounded (e.g. by round_bf16, held across inference
    calls), read as they are; `out` then takes no W_bf16."""
    L, B, d_in, d, ndir, k = _check_params(X, W, v_f, v_r, b_f, b_r, c0, direction, mask,
                                           gemm_dtype)
    dv = X.device
    _req(X_bf16, "X_bf16", (L, B, d_in), dtype=torch.bfloat16, optional=True, device=dv)
    if out is None:
        no_u = not keep_u and not store_c and fused_available(L, B, d_in, d, direction,
                                                                gemm_dtype)
        out = dict(U=None if no_u else torch.empty((L, B, ndir, k, d), device=dv),
                   H=torch.empty((L, B, ndir * d), device=dv),
                   C=torch.empty((L, B, ndir * d), device=dv) if store_c else None,
                   c_last=torch.empty((B, ndir * d), device=dv))
    f32, b16 = torch.float32, torch.bfloat16
    _req_out(out, dict(U=((L, B, ndir, k, d), f32, False), H=((L, B, ndir * d), f32, True),
                       C=((L, B, ndir * d), f32, False), c_last=((B, ndir * d), f32, False),
                       W_bf16=(tuple(W.shape), b16, False),
                       H_bf16=((L, B, ndir * d), b16, False)), dv)
    Wf, Wb = _weights(W, out.get("W_bf16"))
    ws, nbytes = _ws(ws, forward_workspace_bytes(L, B, d_in, d, direction, gemm_dtype), dv)
    st = lib().sru_forward(_ptr(X), _ptr(Wf), _ptr(v_f), _ptr(v_r), _ptr(b_f), _ptr(b_r),
                           _ptr(c0), L, B, d_in, d, direction, _ptr(mask), gemm_dtype,
                           _options(highway_scale, reset_new, linear),
                           _ptr(out.get("U")), _ptr(out["H"]), _ptr(out.get("C")),
                           _ptr(out.get("c_last")), _ptr(X_bf16), _ptr(Wb),
                           _ptr(out.get("H_bf16")), _ptr(ws), nbytes, _stream())
    _check(st, "sru_forward")
    return out


NOALLOC_SCRATCH_BYTES = 128 << 20


def forward_noalloc(X, W, v_f, v_r, b_f, b_r, c0=None, direction=DIR_FWD, mask=None,
                    gemm_dtype=GEMM_FP32, out=None, X_bf16=None, highway_scale=1.0,
                    reset_new=False, linear=False):
    """forward() through sru_forward_noalloc: the library takes its workspace
    from a static device array instead of a caller buffer.  `out` (as for
    forward(); U may be None where fused_available() says so and C is None)
    is required too, so the call allocates nothing."""
    L, B, d_in, d, ndir, k = _check_params(X, W, v_f, v_r, b_f, b_r, c0, direction, mask,
                                           gemm_dtype)
    dv = X.device
    _req(X_bf16, "X_bf16", (L, B, d_in), dtype=torch.bfloat16, optional=True, device=dv)
    if out is None:
        raise ValueError("forward_noalloc needs caller-owned outputs (out)")
    f32, b16 = torch.float32, torch.bfloat16
    _req_out(out, dict(U=((L, B, ndir, k, d), f32, False), H=((L, B, ndir * d), f32, True),
                       C=((L, B, ndir * d), f32, False), c_last=((B, ndir * d), f32, False),
                       W_bf16=(tuple(W.shape), b16, False),
                       H_bf16=((L, B, ndir * d), b16, False)), dv)
    Wf, Wb = _weights(W, out.get("W_bf16"))
    st = lib().sru_forward_noalloc(_ptr(X), _ptr(Wf), _ptr(v_f), _ptr(v_r), _ptr(b_f),
                                   _ptr(b_r), _ptr(c0), L, B, d_in, d, direction, _ptr(mask),
                                   gemm_dtype, _options(highway_scale, reset_new, linear),
                                   _ptr(out.get("U")), _ptr(out["H"]), _ptr(out.get("C")),
                                   _ptr(out.get("c_last")), _ptr(X_bf16), _ptr(Wb),
                                   _ptr(out.get("H_bf16")), _stream())
    _check(st, "sru_forward_noalloc")
    return out


def backward(X, W, v_f, v_r, b_f, b_r, U, C, dH, c0=None, dc_last=None, direction=DIR_FWD,
             mask=None, gemm_dtype=GEMM_FP32, want_dc0=True, out=None, ws=None, X_bf16=None,
             W_bf16=None, highway_scale=1.0, reset_new=False, linear=False):
    """One layer backward; returns dict(dX, dW, dv_f, dv_r, db_f, db_r, dc0).

    bf16 GEMMs only: X_bf16 / W_bf16 (bfloat16 roundings of X and Wcat, as
    forward() writes them) replace the library's own rounding; a bfloat16 W
    (the weights held rounded) takes W_bf16's place.  dW is fp32 either way."""
    L, B, d_in, d, ndir, k = _check_params(X, W, v_f, v_r, b_f, b_r, c0, direction, mask,
                                           gemm_dtype)
    dv = X.device
    _req(X_bf16, "X_bf16", (L, B, d_in), dtype=torch.bfloat16, optional=True, device=dv)
    _req(W_bf16, "W_bf16", tuple(W.shape), dtype=torch.bfloat16, optional=True, device=dv)
    _req(U, "U", (L, B, ndir, k, d), device=dv)
    _req(C, "C", (L, B, ndir * d), device=dv)
    _req(dH, "dH", (L, B, ndir * d), device=dv)
    _req(dc_last, "dc_last", (B, ndir * d), optional=True, device=dv)
    if out is None:
        out = dict(dX=torch.empty_like(X), dW=torch.empty(tuple(W.shape), device=dv),
                   dv_f=None if linear else torch.empty((ndir, d), device=dv),
                   dv_r=None if linear else torch.empty((ndir, d), device=dv),
                   db_f=torch.empty((ndir, d), device=dv), db_r=torch.empty((ndir, d), device=dv),
                   dc0=torch.empty((B, ndir * d), device=dv) if want_dc0 else None)
    f32 = torch.float32
    vec = ((ndir, d), f32, False)
    _req_out(out, dict(dX=(tuple(X.shape), f32, True), dW=(tuple(W.shape), f32, True),
                       dv_f=vec, dv_r=vec, db_f=((ndir, d), f32, True),
                       db_r=((ndir, d), f32, True), dc0=((B, ndir * d), f32, False)), dv)
    Wf, Wb = _weights(W, W_bf16)
    ws, nbytes = _ws(ws, backward_workspace_bytes(L, B, d_in, d, direction, gemm_dtype), dv)
    st = lib().sru_backward(_ptr(X), _ptr(Wf), _ptr(v_f), _ptr(v_r), _ptr(b_f), _ptr(b_r),
                            _ptr(c0), L, B, d_in, d, direction, _ptr(mask), gemm_dtype,
                            _options(highway_scale, reset_new, linear),
                            _ptr(U), _ptr(C), _ptr(dH), _ptr(dc_last),
                            _ptr(out["dX"]), _ptr(out["dW"]), _ptr(out.get("dv_f")),
                            _ptr(out.get("dv_r")), _ptr(out["db_f"]), _ptr(out["db_r"]),
                            _ptr(out.get("dc0")), _ptr(X_bf16), _ptr(Wb), _ptr(ws), nbytes,
                            _stream())
    _check(st, "sru_backward")
    return out


def _check_lowrank(X, Q, P, v_f, v_r, b_f, b_r, c0, mask):
    """Shapes, dtypes and device of a low-rank layer's inputs."""
    for n, t, nd in (("X", X, 3), ("Q", Q, 2), ("P", P, 4)):
        if not isinstance(t, torch.Tensor) or t.dim() != nd:
            raise ValueError(f"{n} must be a {nd}-d tensor")
    L, B, d_in = X.shape
    ndir, k, d, dp = P.shape
    dv = X.device
    _req(X, "X", (L, B, d_in))
    _req(Q, "Q", (d_in, dp), device=dv)
    _req(P, "P", (ndir, k, d, dp), device=dv)
    for n, t in (("v_f", v_f), ("v_r", v_r)):
        _req(t, n, (ndir, d), optional=True, device=dv)
    for n, t in (("b_f", b_f), ("b_r", b_r)):
        _req(t, n, (ndir, d), device=dv)
    _req(c0, "c0", (B, ndir * d), optional=True, device=dv)
    _req(mask, "mask", (L, B), dtype=torch.uint8, optional=True, device=dv)
    return L, B, d_in, d, dp, ndir, k


def forward_lowrank(X, Q, P, v_f, v_r, b_f, b_r, c0=None, direction=DIR_FWD, mask=None,
                    gemm_dtype=GEMM_FP32, store_c=True, out=None, ws=None, highway_scale=1.0,
                    reset_new=False, linear=False, X_bf16=None):
    """Layer with Wcat = P Q^T (Sec. 4.4); Q [d_in, dp], P [ndir, k, d, dp].
    Returns dict(T, U, H, C, c_last); T = X Q is needed by the backward.

    bf16 GEMMs only: X_bf16 replaces the rounding of X; entries T_bf16 /
    H_bf16 of `out` (bfloat16 tensors), if present, receive T and H rounded
    to bf16."""
    L, B, d_in, d, dp, ndir, k = _check_lowrank(X, Q, P, v_f, v_r, b_f, b_r, c0, mask)
    dv = X.device
    _req(X_bf16, "X_bf16", (L, B, d_in), dtype=torch.bfloat16, optional=True, device=dv)
    if out is None:
        out = dict(T=torch.empty((L, B, dp), device=dv),
                   U=torch.empty((L, B, ndir, k, d), device=dv),
                   H=torch.empty((L, B, ndir * d), device=dv),
                   C=torch.empty((L, B, ndir * d), device=dv) if store_c else None,
                   c_last=torch.empty((B, ndir * d), device=dv))
    f32, b16 = torch.float32, torch.bfloat16
    _req_out(out, dict(T=((L, B, dp), f32, True), U=((L, B, ndir, k, d), f32, True),
                       H=((L, B, ndir * d), f32, True), C=((L, B, ndir * d), f32, False),
                       c_last=((B, ndir * d), f32, False), T_bf16=((L, B, dp), b16, False),
                       H_bf16=((L, B, ndir * d), b16, False)), dv)
    need = lib().sru_forward_lowrank_workspace_bytes(L, B, d_in, d, dp, direction, gemm_dtype)
    ws, nbytes = _ws(ws, need, dv)
    st = lib().sru_forward_lowrank(_ptr(X), _ptr(Q), _ptr(P), _ptr(v_f), _ptr(v_r), _ptr(b_f),
                                   _ptr(b_r), _ptr(c0), L, B, d_in, d, dp, direction, _ptr(mask),
                                   gemm_dtype, _options(highway_scale, reset_new, linear), _ptr(out["T"]),
                                   _ptr(out["U"]), _ptr(out["H"]), _ptr(out.get("C")),
                                   _ptr(out.get("c_last")), _ptr(X_bf16), _ptr(out.get("T_bf16")),
                                   _ptr(out.get("H_bf16")), _ptr(ws), nbytes, _stream())
    _check(st, "sru_forward_lowrank")
    return out


def backward_lowrank(X, Q, P, v_f, v_r, b_f, b_r, T, U, C, dH, c0=None, dc_last=None,
                     direction=DIR_FWD, mask=None, gemm_dtype=GEMM_FP32, want_dc0=True, out=None,
                     ws=None, highway_scale=1.0, reset_new=False, linear=False, X_bf16=None,
                     T_bf16=None):
    """Backward of forward_lowrank; returns dict(dX, dQ, dP, dv_f, dv_r, db_f,
    db_r, dc0).  bf16 GEMMs only: X_bf16 / T_bf16 (the roundings of X and T,
    as forward_lowrank writes them) replace the library's own rounding."""
    L, B, d_in, d, dp, ndir, k = _check_lowrank(X, Q, P, v_f, v_r, b_f, b_r, c0, mask)
    dv = X.device
    _req(X_bf16, "X_bf16", (L, B, d_in), dtype=torch.bfloat16, optional=True, device=dv)
    _req(T_bf16, "T_bf16", (L, B, dp), dtype=torch.bfloat16, optional=True, device=dv)
    _req(T, "T", (L, B, dp), device=dv)
    _req(U, "U", (L, B, ndir, k, d), device=dv)
    _req(C, "C", (L, B, ndir * d), device=dv)
    _req(dH, "dH", (L, B, ndir * d), device=dv)
    _req(dc_last, "dc_last", (B, ndir * d), optional=True, device=dv)
    if out is None:
        out = dict(dX=torch.empty_like(X), dQ=torch.empty_like(Q), dP=torch.empty_like(P),
                   dv_f=None if linear else torch.empty((ndir, d), device=dv),
                   dv_r=None if linear else torch.empty((ndir, d), device=dv),
                   db_f=torch.empty((ndir, d), device=dv), db_r=torch.empty((ndir, d), device=dv),
                   dc0=torch.empty((B, ndir * d), device=dv) if want_dc0 else None)
    f32 = torch.float32
    vec = ((ndir, d), f32, False)
    _req_out(out, dict(dX=(tuple(X.shape), f32, True), dQ=(tuple(Q.shape), f32, True),
                       dP=(tuple(P.shape), f32, True), dv_f=vec, dv_r=vec,
                       db_f=((ndir, d), f32, True), db_r=((ndir, d), f32, True),
                       dc0=((B, ndir * d), f32, False)), dv)
    need = lib().sru_backward_lowrank_workspace_bytes(L, B, d_in, d, dp, direction, gemm_dtype)
    ws, nbytes = _ws(ws, need, dv)
    st = lib().sru_backward_lowrank(_ptr(X), _ptr(Q), _ptr(P), _ptr(v_f), _ptr(v_r), _ptr(b_f),
                                    _ptr(b_r), _ptr(c0), L, B, d_in, d, dp, direction,
                                    _ptr(mask), gemm_dtype, _options(highway_scale, reset_new, linear),
                                    _ptr(T), _ptr(U), _ptr(C), _ptr(dH), _ptr(dc_last),
                                    _ptr(out["dX"]), _ptr(out["dQ"]), _ptr(out["dP"]),
                                    _ptr(out.get("dv_f")), _ptr(out.get("dv_r")), _ptr(out["db_f"]),
                                    _ptr(out["db_r"]), _ptr(out.get("dc0")), _ptr(X_bf16),
                                    _ptr(T_bf16), _ptr(ws), nbytes, _stream())
    _check(st, "sru_backward_lowrank")
    return out


def round_bf16(src, out=None):
    """bf16 (RNE) copy of an fp32 tensor, as the bf16 companions expect."""
    if not isinstance(src, torch.Tensor):
        raise ValueError("src must be a torch tensor")
    _req(src, "src", tuple(src.shape))
    if out is None:
        out = torch.empty(tuple(src.shape), dtype=torch.bfloat16, device=src.device)
    _req(out, "out", tuple(src.shape), dtype=torch.bfloat16, device=src.device)
    _check(lib().sru_round_bf16(_ptr(src), src.numel(), _ptr(out), _stream()), "sru_round_bf16")
    return out


def gemm(op, A, B, M, N, K, gemm_dtype=GEMM_FP32, C=None, ws=None):
    """C[M,N] for op NT (A[M,K] B[N,K]^T), NN (A[M,K] B[K,N]) or TN (A[K,M]^T B[K,N])."""
    a_shape = (K, M) if op == OP_TN else (M, K)
    b_shape = (N, K) if op == OP_NT else (K, N)
    _req(A, "A", a_shape)
    dv = A.device
    _req(B, "B", b_shape, device=dv)
    if C is None:
        C = torch.empty((M, N), device=dv)
    _req(C, "C", (M, N), device=dv)
    ws, nbytes = _ws(ws, lib().sru_gemm_workspace_bytes(op, M, N, K, gemm_dtype), dv)
    st = lib().sru_gemm(op, gemm_dtype, M, N, K, _ptr(A), a_shape[1], _ptr(B), b_shape[1],
                        _ptr(C), N, _ptr(ws), nbytes, _stream())
    _check(st, "sru_gemm")
    return C


def _check_scan_params(U, v_f, v_r, b_f, b_r, c0, mask):
    if not isinstance(U, torch.Tensor) or U.dim() != 5:
        raise ValueError("U must be a 5-d tensor [L, B, ndir, k, d]")
    L, B, ndir, k, d = U.shape
    _req(U, "U", (L, B, ndir, k, d))
    dv = U.device
    for n, t in (("v_f", v_f), ("v_r", v_r)):
        _req(t, n, (ndir, d), optional=True, device=dv)
    for n, t in (("b_f", b_f), ("b_r", b_r)):
        _req(t, n, (ndir, d), device=dv)
    _req(c0, "c0", (B, ndir * d), optional=True, device=dv)
    _req(mask, "mask", (L, B), dtype=torch.uint8, optional=True, device=dv)
    return L, B, ndir, k, d


def scan_forward(U, X, v_f, v_r, b_f, b_r, c0=None, direction=DIR_FWD, mask=None,
                 store_c=True, out=None, ws=None, highway_scale=1.0, reset_new=False,
                 linear=False):
    L, B, ndir, k, d = _check_scan_params(U, v_f, v_r, b_f, b_r, c0, mask)
    dv = U.device
    if k == 4 and X is None:
        raise ValueError("pass X (or its shape via d_in) for k = 4")
    if X is not None:
        if not isinstance(X, torch.Tensor) or X.dim() != 3:
            raise ValueError("X must be a 3-d tensor [L, B, d_in]")
        _req(X, "X", (L, B, X.shape[2]), device=dv)
    d_in = X.shape[2] if X is not None else d
    if out is None:
        out = dict(H=torch.empty((L, B, ndir * d), device=dv),
                   C=torch.empty((L, B, ndir * d), device=dv) if store_c else None,
                   c_last=torch.empty((B, ndir * d), device=dv))
    f32 = torch.float32
    _req_out(out, dict(H=((L, B, ndir * d), f32, True), C=((L, B, ndir * d), f32, False),
                       c_last=((B, ndir * d), f32, False),
                       H_bf16=((L, B, ndir * d), torch.bfloat16, False)), dv)
    need = lib().sru_scan_forward_workspace_bytes(L, B, d_in, d, direction)
    ws, nbytes = _ws(ws, need, dv)
    st = lib().sru_scan_forward(_ptr(U), _ptr(X), _ptr(v_f), _ptr(v_r), _ptr(b_f), _ptr(b_r),
                                _ptr(c0), L, B, d_in, d, direction, _ptr(mask),
                                _options(highway_scale, reset_new, linear),
                                _ptr(out["H"]), _ptr(out.get("C")), _ptr(out.get("c_last")),
                                _ptr(out.get("H_bf16")), _ptr(ws), nbytes, _stream())
    _check(st, "sru_scan_forward")
    return out


def scan_backward(U, X, C, dH, v_f, v_r, b_f, b_r, c0=None, dc_last=None, direction=DIR_FWD,
                  mask=None, d_in=None, out=None, ws=None, highway_scale=1.0, reset_new=False,
                  linear=False):
    L, B, ndir, k, d = _check_scan_params(U, v_f, v_r, b_f, b_r, c0, mask)
    dv = U.device
    if X is not None:
        if not isinstance(X, torch.Tensor) or X.dim() != 3:
            raise ValueError("X must be a 3-d tensor [L, B, d_in]")
        _req(X, "X", (L, B, X.shape[2]), device=dv)
    if d_in is None:
        d_in = X.shape[2] if X is not None else d
    _req(C, "C", (L, B, ndir * d), device=dv)
    _req(dH, "dH", (L, B, ndir * d), device=dv)
    _req(dc_last, "dc_last", (B, ndir * d), optional=True, device=dv)
    if out is None:
        out = dict(dU=torch.empty_like(U),
                   dxh=torch.empty((L, B, ndir, d), device=dv) if k == 3 else None,
                   dv_f=None if linear else torch.empty((ndir, d), device=dv),
                   dv_r=None if linear else torch.empty((ndir, d), device=dv),
                   db_f=torch.empty((ndir, d), device=dv), db_r=torch.empty((ndir, d), device=dv),
                   dc0=torch.empty((B, ndir * d), device=dv))
    f32 = torch.float32
    vec = ((ndir, d), f32, False)
    _req_out(out, dict(dU=((L, B, ndir, k, d), f32, True), dxh=((L, B, ndir, d), f32, False),
                       dv_f=vec, dv_r=vec, db_f=((ndir, d), f32, True),
                       db_r=((ndir, d), f32, True), dc0=((B, ndir * d), f32, False)), dv)
    need = lib().sru_scan_backward_workspace_bytes(L, B, d_in, d, direction)
    ws, nbytes = _ws(ws, need, dv)
    st = lib().sru_scan_backward(_ptr(U), _ptr(X), _ptr(C), _ptr(dH), _ptr(dc_last),
                                 _ptr(v_f), _ptr(v_r), _ptr(b_f), _ptr(b_r), _ptr(c0),
                                 L, B, d_in, d, direction, _ptr(mask),
                                 _options(highway_scale, reset_new, linear),
                                 _ptr(out["dU"]), _ptr(out.get("dxh")), _ptr(out.get("dv_f")),
                                 _ptr(out.get("dv_r")), _ptr(out["db_f"]), _ptr(out["db_r"]),
                                 _ptr(out.get("dc0")), _ptr(ws), nbytes, _stream())
    _check(st, "sru_scan_backward")
    return out


class Stack:
    """Stacked SRU layers (layer l+1 reads layer l's H) with preallocated
    buffers, for the multi-layer forward + backward step.

    `layers` holds per-layer dicts of GPU tensors v_f, v_r, b_f, b_r and
    either W (dense) or Q, P (the low-rank projection, Wcat = P Q^T).
    With bf16 GEMMs each layer's forward also writes bf16 copies of H (below
    the top layer) and of Wcat (dense) or T (low-rank): the next layer's
    projection and the backward products read those instead of rounding the
    same values again.  Without a backward pass, store_c=False skips the
    states C (inference).  With bf16 GEMMs a dense layer's W may be held in
    bfloat16 (rounded once, e.g. for inference): it is then read as it is.
    """

    def __init__(self, layers, L, B, d_in, d, direction, gemm_dtype, device, backward=True,
                 highway_scale=1.0, reset_new=False, store_c=True, linear=False):
        self.layers = layers
        self.variant = dict(highway_scale=highway_scale, reset_new=reset_new, linear=linear)
        self.L, self.B, self.d, self.direction, self.gemm_dtype = L, B, d, direction, gemm_dtype
        ndir = 2 if direction == DIR_BI else 1
        self.ndir = ndir
        self.fw = []
        self.bw = []
        ws_bytes = 0
        for li, p in enumerate(layers):
            din = d_in if li == 0 else ndir * d
            low = "Q" in p
            k = (p["P"] if low else p["W"]).shape[1]
            keep_c = store_c or backward  # the backward reads C
            # inference: dense layers run the fused projection + scan where
            # available, which keeps no U
            no_u = (not keep_c and not low and
                    fused_available(L, B, din, d, direction, gemm_dtype))
            o = dict(U=None if no_u else torch.empty((L, B, ndir, k, d), device=device),
                     H=torch.empty((L, B, ndir * d), device=device),
                     C=torch.empty((L, B, ndir * d), device=device) if keep_c else None,
                     c_last=torch.empty((B, ndir * d), device=device))
            bf = dict(dtype=torch.bfloat16, device=device)
            if low:
                dp = p["Q"].shape[1]
                o["T"] = torch.empty((L, B, dp), device=device)
                if gemm_dtype == GEMM_BF16:
                    o["T_bf16"] = torch.empty((L, B, dp), **bf)
            elif gemm_dtype == GEMM_BF16 and p["W"].dtype != torch.bfloat16:
                o["W_bf16"] = torch.empty(tuple(p["W"].shape), **bf)
            if gemm_dtype == GEMM_BF16 and li + 1 < len(layers):
                o["H_bf16"] = torch.empty((L, B, ndir * d), **bf)  # the next layer's operand
            self.fw.append(o)
            if backward:
                g = dict(dX=torch.empty((L, B, din), device=device),
                         dv_f=None if linear else torch.empty((ndir, d), device=device),
                         dv_r=None if linear else torch.empty((ndir, d), device=device),
                         db_f=torch.empty((ndir, d), device=device),
                         db_r=torch.empty((ndir, d), device=device), dc0=None)
                if low:
                    g["dQ"] = torch.empty_like(p["Q"])
                    g["dP"] = torch.empty_like(p["P"])
                    ws_bytes = max(ws_bytes, lib().sru_backward_lowrank_workspace_bytes(
                        L, B, din, d, dp, direction, gemm_dtype))
                else:
                    g["dW"] = torch.empty(tuple(p["W"].shape), device=device)
                    ws_bytes = max(ws_bytes, backward_workspace_bytes(L, B, din, d, direction,
                                                                      gemm_dtype))
                self.bw.append(g)
            if low:
                ws_bytes = max(ws_bytes, lib().sru_forward_lowrank_workspace_bytes(
                    L, B, din, d, dp, direction, gemm_dtype))
            else:
                ws_bytes = max(ws_bytes, forward_workspace_bytes(L, B, din, d, direction,
                                                                 gemm_dtype))
        self.ws = workspace(ws_bytes, device)
        # bf16 products: the first layer's input is rounded once per step and
        # the copy serves its forward and its backward
        self.xb0 = (torch.empty((L, B, d_in), dtype=torch.bfloat16, device=device)
                    if gemm_dtype == GEMM_BF16 else None)

    def forward(self, X, mask=None):
        x, xb = X, None
        if self.xb0 is not None:
            xb = round_bf16(X, self.xb0)
        for p, o in zip(self.layers, self.fw):
            v = (p["v_f"], p["v_r"], p["b_f"], p["b_r"], None, self.direction, mask,
                 self.gemm_dtype)
            if "Q" in p:
                forward_lowrank(x, p["Q"], p["P"], *v, out=o, ws=self.ws, X_bf16=xb,
                                **self.variant)
            else:
                forward(x, p["W"], *v, out=o, ws=self.ws, X_bf16=xb, **self.variant)
            x, xb = o["H"], o.get("H_bf16")
        return x

    def backward(self, X, dH, mask=None):
        """Backward of the last forward(), which must have run on the same X."""
        g = dH
        for li in range(len(self.layers) - 1, -1, -1):
            p, o, b = self.layers[li], self.fw[li], self.bw[li]
            x = X if li == 0 else self.fw[li - 1]["H"]
            v = (p["v_f"], p["v_r"], p["b_f"], p["b_r"])
            xb = self.xb0 if li == 0 else self.fw[li - 1].get("H_bf16")
            if "Q" in p:
                backward_lowrank(x, p["Q"], p["P"], *v, o["T"], o["U"], o["C"], g, None, None,
                                 self.direction, mask, self.gemm_dtype, want_dc0=False, out=b,
                                 ws=self.ws, X_bf16=xb, T_bf16=o.get("T_bf16"), **self.variant)
            else:
                backward(x, p["W"], *v, o["U"], o["C"], g, None, None, self.direction, mask,
                         self.gemm_dtype, want_dc0=False, out=b, ws=self.ws, X_bf16=xb,
                         W_bf16=o.get("W_bf16"), **self.variant)
            g = b["dX"]
        return g

    def step(self, X, dH=None, mask=None):
        """One forward (+ backward, if the stack has one) pass."""
        self.forward(X, mask)
        if self.bw:
            self.backward(X, dH, mask)

    def capture(self, X, dH=None, mask=None):
        """Record one step into a HIP graph (torch.cuda.CUDAGraph).

        The library allocates, frees and synchronises nothing and issues no
        memset, so a whole step records as plain kernel nodes.  Replaying the
        graph runs the step again on whatever X, dH and mask then hold (the
        same tensors, updated in place), with no per-kernel launch cost.  The
        graph reads and writes this stack's buffers: do not run the stack
        eagerly and replay the graph concurrently."""
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            self.step(X, dH, mask)  # warm-up outside the capture
        torch.cuda.current_stream().wait_stream(side)
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            self.step(X, dH, mask)
        return graph
