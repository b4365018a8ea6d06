"""C-ABI contract checks that need no GPU: the library loads, exports every
symbol include/sru.h declares, and rejects invalid arguments before anything
is enqueued (no compute call is made here)."""

import ctypes
import os
import re

import pytest

from paper_1709_02755_amd import sru

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "sru.h")

OK, E_NULL, E_SHAPE, E_FLAG, E_WS, E_HIP, E_ALIGN = range(7)
FAKE = ctypes.c_void_p(0x10000)        # never dereferenced: validation fails first
FAKE_MIS = ctypes.c_void_p(0x10002)    # not 4-byte aligned


def declared_symbols():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"SRU_API\s+[\w\s\*]+?\b(sru_\w+)\s*\(", text)))


def test_library_loads_and_exports_every_declared_symbol():
    lib = sru.lib()
    names = declared_symbols()
    assert len(names) >= 12
    for n in names:
        assert hasattr(lib, n), n
    assert sorted(sru.exported_symbols()) == names


def test_version_and_status_strings():
    lib = sru.lib()
    assert lib.sru_version() >> 16 == 1
    for code in range(7):
        s = lib.sru_status_string(code).decode()
        assert s.startswith("SRU_")
    assert lib.sru_status_string(99).decode() == "unknown sru_status"


def _fwd(lib, **kw):
    a = dict(X=FAKE, W=FAKE, v_f=FAKE, v_r=FAKE, b_f=FAKE, b_r=FAKE, c0=None, L=4, B=2, d_in=8,
             d=8, direction=0, mask=None, gemm=0, opts=None, U=FAKE, H=FAKE, C=FAKE,
             c_last=None, Xb=None, Wb=None, Hb=None, ws=None, ws_bytes=0)
    a.update(kw)
    return lib.sru_forward(a["X"], a["W"], a["v_f"], a["v_r"], a["b_f"], a["b_r"], a["c0"],
                           a["L"], a["B"], a["d_in"], a["d"], a["direction"], a["mask"],
                           a["gemm"], a["opts"], a["U"], a["H"], a["C"], a["c_last"], a["Xb"], a["Wb"],
                           a["Hb"], a["ws"], a["ws_bytes"], None)


def _bwd(lib, **kw):
    a = dict(X=FAKE, W=FAKE, v_f=FAKE, v_r=FAKE, b_f=FAKE, b_r=FAKE, c0=None, L=4, B=2, d_in=8,
             d=8, direction=0, mask=None, gemm=0, opts=None, U=FAKE, C=FAKE, dH=FAKE,
             dc_last=None,
             dX=FAKE, dW=FAKE, dv_f=FAKE, dv_r=FAKE, db_f=FAKE, db_r=FAKE, dc0=None, Xb=None,
             Wb=None, ws=None, ws_bytes=0)
    a.update(kw)
    return lib.sru_backward(a["X"], a["W"], a["v_f"], a["v_r"], a["b_f"], a["b_r"], a["c0"],
                            a["L"], a["B"], a["d_in"], a["d"], a["direction"], a["mask"],
                            a["gemm"], a["opts"], a["U"], a["C"], a["dH"], a["dc_last"], a["dX"], a["dW"],
                            a["dv_f"], a["dv_r"], a["db_f"], a["db_r"], a["dc0"], a["Xb"],
                            a["Wb"], a["ws"], a["ws_bytes"], None)


@pytest.mark.parametrize("field", ["X", "W", "v_f", "v_r", "b_f", "b_r", "U", "H"])
def test_forward_rejects_null_required_pointer(field):
    assert _fwd(sru.lib(), **{field: None}) == E_NULL


@pytest.mark.parametrize("kw", [dict(L=0), dict(B=0), dict(d=0), dict(d_in=-1),
                                dict(L=1 << 20, B=1 << 12), dict(d=1 << 30, d_in=1 << 30)])
def test_forward_rejects_bad_shape(kw):
    assert _fwd(sru.lib(), **kw) == E_SHAPE


@pytest.mark.parametrize("kw", [dict(direction=3), dict(direction=-1), dict(gemm=2)])
def test_forward_rejects_bad_flag(kw):
    assert _fwd(sru.lib(), **kw) == E_FLAG


def test_forward_rejects_misaligned_pointer():
    assert _fwd(sru.lib(), H=FAKE_MIS) == E_ALIGN


@pytest.mark.parametrize("field", ["Xb", "Wb", "Hb"])
def test_forward_bf16_companions_checked(field):
    lib = sru.lib()
    # only with bf16 GEMMs
    assert _fwd(lib, **{field: FAKE}) == E_FLAG
    # 16-byte aligned (checked before the workspace)
    assert _fwd(lib, gemm=1, **{field: ctypes.c_void_p(0x10008)}) == E_ALIGN
    assert _fwd(lib, gemm=1, **{field: FAKE}) == E_WS


@pytest.mark.parametrize("field", ["Xb", "Wb"])
def test_backward_bf16_companions_checked(field):
    lib = sru.lib()
    assert _bwd(lib, **{field: FAKE}) == E_FLAG
    assert _bwd(lib, gemm=1, **{field: ctypes.c_void_p(0x10008)}) == E_ALIGN
    assert _bwd(lib, gemm=1, **{field: FAKE}) == E_WS


@pytest.mark.parametrize("field", ["X", "W", "U", "C", "dH", "dX", "dW", "dv_f", "db_r"])
def test_backward_rejects_null_required_pointer(field):
    assert _bwd(sru.lib(), **{field: None}) == E_NULL


def test_backward_requires_workspace():
    lib = sru.lib()
    need = lib.sru_backward_workspace_bytes(4, 2, 8, 8, 0, 0)
    assert need > 0
    assert _bwd(lib) == E_WS
    assert _bwd(lib, ws=FAKE, ws_bytes=need - 1) == E_WS
    # a large enough but misaligned workspace
    assert _bwd(lib, ws=ctypes.c_void_p(0x10040), ws_bytes=need) == E_ALIGN


def test_workspace_queries():
    lib = sru.lib()
    assert lib.sru_forward_workspace_bytes(4, 2, 8, 8, 0, 0) == 0
    assert lib.sru_forward_workspace_bytes(0, 2, 8, 8, 0, 0) == 0
    assert lib.sru_backward_workspace_bytes(4, 2, 8, 8, 7, 0) == 0
    # dU (M*N floats) plus dxh plus partials, each 256-aligned
    L, B, d = 16, 4, 32
    need = lib.sru_backward_workspace_bytes(L, B, d, d, 2, 0)
    assert need >= 4 * (L * B * 2 * 3 * d + L * B * 2 * d + 4 * B * 2 * d)
    assert need % 256 == 0
    # bf16 and fp32 sizes are both valid; k = 4 has no dxh buffer
    assert lib.sru_backward_workspace_bytes(L, B, 2 * d, d, 2, 1) > 0


def test_gemm_argument_checks():
    lib = sru.lib()
    g = lib.sru_gemm
    assert g(3, 0, 4, 4, 4, FAKE, 4, FAKE, 4, FAKE, 4, None, 0, None) == E_FLAG
    assert g(0, 5, 4, 4, 4, FAKE, 4, FAKE, 4, FAKE, 4, None, 0, None) == E_FLAG
    assert g(0, 0, 0, 4, 4, FAKE, 4, FAKE, 4, FAKE, 4, None, 0, None) == E_SHAPE
    assert g(0, 0, 4, 4, 8, FAKE, 4, FAKE, 8, FAKE, 4, None, 0, None) == E_SHAPE   # lda < K
    assert g(2, 0, 4, 4, 8, FAKE, 3, FAKE, 4, FAKE, 4, None, 0, None) == E_SHAPE   # TN: lda < M
    assert g(0, 0, 4, 4, 4, None, 4, FAKE, 4, FAKE, 4, None, 0, None) == E_NULL
    assert g(0, 0, 4, 4, 4, FAKE_MIS, 4, FAKE, 4, FAKE, 4, None, 0, None) == E_ALIGN
    # a long TN reduction is split and then needs workspace
    need = lib.sru_gemm_workspace_bytes(2, 512, 512, 1 << 16, 0)
    assert need > 0
    assert g(2, 0, 512, 512, 1 << 16, FAKE, 512, FAKE, 512, FAKE, 512, None, 0, None) == E_WS


def test_scan_argument_checks():
    lib = sru.lib()
    f = lib.sru_scan_forward
    assert f(FAKE, None, FAKE, FAKE, FAKE, FAKE, None, 4, 2, 8, 8, 0, None, None, FAKE, None,
             None, None, None, 0, None) == E_NULL          # k = 3 needs X
    assert f(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None, 4, 2, 8, 8, 9, None, None, FAKE, None,
             None, None, None, 0, None) == E_FLAG
    assert f(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None, 4, 2, 8, 8, 0, None, None, FAKE, None,
             None, ctypes.c_void_p(0x10001), None, 0, None) == E_ALIGN  # bf16 H: 2-byte aligned
    b = lib.sru_scan_backward
    args = [FAKE, FAKE, FAKE, FAKE, None, FAKE, FAKE, FAKE, FAKE, None, 4, 2, 16, 8, 0, None,
            None, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None, None, 0, None]
    assert b(*args) == E_SHAPE                             # k = 4 takes no dxh
    args[18] = None
    assert b(*args) == E_WS


@pytest.mark.parametrize("alpha,reset", [(float("nan"), 0), (float("inf"), 0), (1.0, 2),
                                         (1.0, -1)])
def test_invalid_options_rejected(alpha, reset):
    lib = sru.lib()
    bad = ctypes.byref(sru.Options(alpha, reset))
    assert _fwd(lib, opts=bad) == E_FLAG
    assert _bwd(lib, opts=bad) == E_FLAG


def test_valid_options_pass_validation():
    # a valid options struct is read and the call proceeds to the next check
    lib = sru.lib()
    ok = ctypes.byref(sru.Options(3.0 ** 0.5, sru.RESET_NEW))
    assert _fwd(lib, opts=ok, H=FAKE_MIS) == E_ALIGN
    assert _bwd(lib, opts=ok) == E_WS


@pytest.mark.parametrize("recurrence", [2, -1])
def test_invalid_recurrence_rejected(recurrence):
    lib = sru.lib()
    bad = ctypes.byref(sru.Options(1.0, sru.RESET_PREV, recurrence))
    assert _fwd(lib, opts=bad) == E_FLAG
    assert _bwd(lib, opts=bad) == E_FLAG


def test_linear_recurrence_needs_no_v():
    """Ablation (1) has no v: v_f, v_r, dv_f, dv_r may be NULL (the calls go
    on to the next check); the gated recurrence still requires them."""
    lib = sru.lib()
    lin = ctypes.byref(sru.Options(1.0, sru.RESET_PREV, sru.RECURRENCE_LINEAR))
    assert _fwd(lib, opts=lin, v_f=None, v_r=None, H=FAKE_MIS) == E_ALIGN
    assert _bwd(lib, opts=lin, v_f=None, v_r=None, dv_f=None, dv_r=None) == E_WS
    assert _fwd(lib, v_f=None, v_r=None) == E_NULL
    assert _bwd(lib, dv_r=None) == E_NULL
    assert lib.sru_scan_forward(FAKE, FAKE, None, None, FAKE, FAKE, None, 4, 2, 8, 8, 0, None,
                                lin, FAKE_MIS, None, None, None, None, 0, None) == E_ALIGN
    # few lanes: the linear scans cut time into segments and need scratch,
    # which the gated scan does not
    need = lib.sru_scan_forward_workspace_bytes(4000, 2, 64, 64, 0)
    assert need > 0 and need % 256 == 0
    fargs = [FAKE, FAKE, None, None, FAKE, FAKE, None, 4000, 2, 64, 64, 0, None, lin, FAKE, None,
             None, None, None, 0, None]
    assert lib.sru_scan_forward(*fargs) == E_WS
    fargs[18], fargs[19] = FAKE_MIS, need
    assert lib.sru_scan_forward(*fargs) == E_ALIGN      # 256-byte aligned workspace
    # many lanes: one segment, no scratch
    assert lib.sru_scan_forward_workspace_bytes(64, 64, 1024, 1024, 0) == 0
    args = [FAKE, FAKE, FAKE, FAKE, None, None, None, FAKE, FAKE, None, 4, 2, 8, 8, 0, None,
            lin, FAKE, FAKE, None, None, FAKE, FAKE, None, None, 0, None]
    assert lib.sru_scan_backward(*args) == E_WS


def test_lowrank_argument_checks():
    lib = sru.lib()
    f = lib.sru_forward_lowrank

    def fwd(**kw):
        a = dict(L=4, B=2, d_in=8, d=8, dp=8, direction=0, gemm=0, T=FAKE, Xb=None, Tb=None,
                 Hb=None, ws=None, ws_bytes=0)
        a.update(kw)
        return f(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None, a["L"], a["B"], a["d_in"], a["d"],
                 a["dp"], a["direction"], None, a["gemm"], None, a["T"], FAKE, FAKE, FAKE, None,
                 a["Xb"], a["Tb"], a["Hb"], a["ws"], a["ws_bytes"], None)
    assert fwd(Tb=FAKE) == E_FLAG              # bf16 companions need bf16 products
    assert fwd(gemm=1, Tb=ctypes.c_void_p(0x10008)) == E_ALIGN  # 16-byte aligned
    assert fwd(dp=0) == E_SHAPE
    assert fwd(gemm=1, dp=6) == E_SHAPE        # bf16 products need dp % 8 == 0
    assert fwd(gemm=1, d_in=12) == E_SHAPE
    assert fwd(T=None) == E_NULL
    assert fwd(direction=5) == E_FLAG
    need = lib.sru_forward_lowrank_workspace_bytes(4, 2, 8, 8, 8, 0, 1)
    assert need > 0 and lib.sru_forward_lowrank_workspace_bytes(4, 2, 8, 8, 8, 0, 0) == 0
    assert fwd(gemm=1) == E_WS
    assert lib.sru_backward_lowrank_workspace_bytes(4, 2, 8, 8, 8, 0, 0) > 0
    assert lib.sru_backward_lowrank_workspace_bytes(4, 2, 8, 8, 0, 0, 0) == 0
    b = lib.sru_backward_lowrank
    args = [FAKE] * 7 + [None, 4, 2, 8, 8, 8, 0, None, 0, None] + [FAKE] * 4 + [None] + \
        [FAKE] * 7 + [None] + [FAKE, None, None, 0, None]
    assert b(*args) == E_FLAG                   # X_bf16 with fp32 products
    args[-5] = None
    assert b(*args) == E_WS


def test_round_bf16_argument_checks():
    lib = sru.lib()
    f = lib.sru_round_bf16
    assert f(None, 0, None, None) == OK                       # nothing to do
    assert f(None, 8, FAKE, None) == E_NULL
    assert f(FAKE, 8, ctypes.c_void_p(0x10008), None) == E_ALIGN
    assert f(ctypes.c_void_p(0x20000), 8, ctypes.c_void_p(0x20010), None) == E_SHAPE  # overlap


def test_forward_without_u_needs_the_fused_path():
    lib = sru.lib()
    assert lib.sru_forward_fused_available(4, 2, 128, 64, 0, 1) == 1
    assert lib.sru_forward_fused_available(4, 2, 128, 64, 0, 0) == 0  # fp32 products
    assert lib.sru_forward_fused_available(4, 2, 64, 64, 0, 1) == 1   # k = 3
    assert lib.sru_forward_fused_available(4, 2, 60, 64, 0, 1) == 0   # d_in % 8
    assert lib.sru_forward_fused_available(4, 2, 64, 32, 0, 1) == 0   # d % 64
    assert lib.sru_forward_fused_available(128, 2, 128, 64, 0, 1) == 1
    assert lib.sru_forward_fused_available(129, 2, 128, 64, 0, 1) == 0  # L > 128, 1 tile
    assert lib.sru_forward_fused_available(1024, 32, 1024, 1024, 0, 1) == 1  # 256 tiles
    # U omitted: fp32 products, or C kept, leave U required
    assert _fwd(lib, d_in=128, d=64, U=None, C=None) == E_NULL
    assert _fwd(lib, d_in=128, d=64, gemm=1, U=None, C=FAKE) == E_NULL
    # bf16, C omitted: U may be omitted (the call goes on to the workspace check)
    assert _fwd(lib, d_in=128, d=64, gemm=1, U=None, C=None) == E_WS


def test_missing_library_fails_loudly(monkeypatch, tmp_path):
    """With no library and no way to build one, the binding raises; there is
    no other path to the results (no CPU fallback)."""
    from paper_1709_02755_amd import build as build_mod

    def no_build():
        raise RuntimeError("hipcc unavailable")

    monkeypatch.delenv("SRU_LIBRARY", raising=False)
    monkeypatch.setattr(sru, "_lib", None)
    monkeypatch.setattr(sru, "LIB_PATH", str(tmp_path / "libsru.so"))
    monkeypatch.setattr(build_mod, "build", no_build)
    with pytest.raises(RuntimeError, match="hipcc unavailable"):
        sru.lib()
    (tmp_path / "libsru.so").write_bytes(b"not a shared object")
    with pytest.raises(OSError):
        sru.lib()


def _fwd_noalloc(lib, **kw):
    a = dict(X=FAKE, W=FAKE, v_f=FAKE, v_r=FAKE, b_f=FAKE, b_r=FAKE, c0=None, L=4, B=2, d_in=8,
             d=8, direction=0, mask=None, gemm=0, opts=None, U=FAKE, H=FAKE, C=FAKE,
             c_last=None, Xb=None, Wb=None, Hb=None)
    a.update(kw)
    return lib.sru_forward_noalloc(a["X"], a["W"], a["v_f"], a["v_r"], a["b_f"], a["b_r"],
                                   a["c0"], a["L"], a["B"], a["d_in"], a["d"], a["direction"],
                                   a["mask"], a["gemm"], a["opts"], a["U"], a["H"], a["C"],
                                   a["c_last"], a["Xb"], a["Wb"], a["Hb"], None)


def test_noalloc_forward_refuses_what_its_scratch_cannot_hold():
    """The allocation-free forward takes its workspace from a fixed array of
    SRU_NOALLOC_SCRATCH_BYTES; a shape whose forward workspace is larger is
    refused before any HIP call (so this runs without a GPU), and so are
    invalid sizes and flags."""
    lib = sru.lib()
    text = open(HEADER).read()
    assert "#define SRU_NOALLOC_SCRATCH_BYTES (128u << 20)" in text
    assert sru.NOALLOC_SCRATCH_BYTES == 128 << 20
    # bf16: the forward workspace holds X and Wcat in bf16
    L, B, d = 1024, 128, 1024
    need = lib.sru_forward_workspace_bytes(L, B, d, d, 0, 1)
    assert need > sru.NOALLOC_SCRATCH_BYTES
    assert _fwd_noalloc(lib, L=L, B=B, d_in=d, d=d, gemm=1) == E_WS
    assert _fwd_noalloc(lib, L=0) == E_SHAPE
    assert _fwd_noalloc(lib, direction=7) == E_FLAG
    assert _fwd_noalloc(lib, gemm=9) == E_FLAG


def test_weights_held_in_bf16():
    """bf16 products may take the weights already rounded: W = NULL with
    W_bf16 given (the calls go on to the next check).  A NULL W without
    W_bf16, or with fp32 products, is still a missing pointer."""
    lib = sru.lib()
    assert _fwd(lib, W=None, Wb=FAKE, gemm=1, H=FAKE_MIS) == E_ALIGN
    assert _bwd(lib, W=None, Wb=FAKE, gemm=1) == E_WS
    assert _fwd(lib, W=None, gemm=1) == E_NULL
    assert _bwd(lib, W=None, gemm=1) == E_NULL
    assert _fwd(lib, W=None, Wb=FAKE, gemm=0) == E_NULL
    assert _bwd(lib, W=None, Wb=FAKE, gemm=0) == E_NULL
