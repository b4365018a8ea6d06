"""Argument checks of the Python binding, on the CPU.

Every wrapper must reject a bad tensor (host memory, wrong dtype, wrong
shape, not contiguous, another device) with ValueError before the library is
called, and must tell the library the caller's real workspace size.  Host
tensors stand in for device tensors here by switching off the binding's
"is it on the GPU" test only; a stub library records which entry points are
reached, so a compute call is never made."""

import pytest
import torch

from paper_1709_02755_amd import sru

F32 = torch.float32


class StubLib:
    """Workspace queries answer; compute calls are recorded, not run."""

    def __init__(self, ws=4096):
        self.calls = []
        self.ws = ws

    def __getattr__(self, name):
        if name.endswith("workspace_bytes"):
            return lambda *a: self.ws
        if name == "sru_forward_fused_available":
            return lambda *a: 0

        def call(*a):
            self.calls.append((name, a))
            return 0
        return call


@pytest.fixture
def stub(monkeypatch):
    lib = StubLib()
    monkeypatch.setattr(sru, "_lib", lib)
    monkeypatch.setattr(sru, "_on_gpu", lambda t: True)
    monkeypatch.setattr(sru, "_stream", lambda: None)
    return lib


def z(*shape, dtype=F32):
    return torch.zeros(shape, dtype=dtype)


L, B, D = 4, 3, 8


def layer(ndir=1, k=3, d_in=D):
    return dict(X=z(L, B, d_in), W=z(ndir, k, D, d_in), v_f=z(ndir, D), v_r=z(ndir, D),
                b_f=z(ndir, D), b_r=z(ndir, D))


def bad_variants(t):
    """Ways a tensor argument can be wrong, each with a label."""
    yield "dtype", t.to(torch.float64)
    yield "shape", torch.zeros(tuple(t.shape[:-1]) + (t.shape[-1] + 1,), dtype=t.dtype)
    if t.dim() >= 2 and t.shape[-1] > 1 and t.shape[-2] > 1:
        yield "strided", torch.zeros(tuple(t.shape[:-2]) + (t.shape[-1], t.shape[-2]),
                                     dtype=t.dtype).transpose(-1, -2)
    yield "not a tensor", t.float().numpy()


def run_forward(a):
    return sru.forward(a["X"], a["W"], a["v_f"], a["v_r"], a["b_f"], a["b_r"], c0=a.get("c0"),
                       mask=a.get("mask"), out=a.get("out"), ws=a.get("ws"),
                       X_bf16=a.get("X_bf16"), gemm_dtype=a.get("gemm", sru.GEMM_FP32))


def fwd_args():
    a = layer()
    a["c0"] = z(B, D)
    a["mask"] = z(L, B, dtype=torch.uint8)
    return a


def test_forward_accepts_valid_arguments(stub):
    run_forward(fwd_args())
    assert [c[0] for c in stub.calls] == ["sru_forward"]


@pytest.mark.parametrize("name", ["X", "W", "v_f", "b_f", "b_r", "c0", "mask"])
def test_forward_rejects_bad_inputs(stub, name):
    for why, bad in bad_variants(fwd_args()[name]):
        if name == "mask" and why == "dtype":
            bad = bad.to(torch.int64)
        a = fwd_args()
        a[name] = bad
        with pytest.raises(ValueError):
            run_forward(a)
    assert stub.calls == []


@pytest.mark.parametrize("name,shape,dtype", [
    ("U", (L, B, 1, 3, D), F32), ("H", (L, B, D), F32), ("C", (L, B, D), F32),
    ("c_last", (B, D), F32), ("W_bf16", (1, 3, D, D), torch.bfloat16),
    ("H_bf16", (L, B, D), torch.bfloat16)])
def test_forward_rejects_bad_outputs(stub, name, shape, dtype):
    good = dict(U=z(L, B, 1, 3, D), H=z(L, B, D), C=z(L, B, D), c_last=z(B, D))
    for why, bad in bad_variants(z(*shape, dtype=dtype)):
        a = fwd_args()
        a["out"] = dict(good, **{name: bad})
        with pytest.raises(ValueError):
            run_forward(a)
    a = fwd_args()
    a["out"] = dict(good, **{name: z(*shape, dtype=dtype)})
    run_forward(a)  # the right buffer is accepted
    assert [c[0] for c in stub.calls] == ["sru_forward"]


def test_forward_rejects_bad_workspace(stub):
    for bad in (z(64), z(8, 8, dtype=torch.uint8), z(128, dtype=torch.uint8)[::2]):
        a = fwd_args()
        a["ws"] = bad
        with pytest.raises(ValueError):
            run_forward(a)
    assert stub.calls == []


def test_workspace_size_passed_is_the_callers(stub):
    """The library is told the size of the buffer it gets, not the size it
    asked for, so its own check of the workspace applies."""
    a = fwd_args()
    a["ws"] = z(100, dtype=torch.uint8)
    run_forward(a)
    args = stub.calls[-1][1]
    assert args[-2] == 100
    X, W = z(L, B, D), z(1, 3, D, D)
    U, C, dH = z(L, B, 1, 3, D), z(L, B, D), z(L, B, D)
    p = [z(1, D) for _ in range(4)]
    sru.backward(X, W, *p, U, C, dH, ws=z(77, dtype=torch.uint8))
    assert stub.calls[-1][0] == "sru_backward" and stub.calls[-1][1][-2] == 77
    sru.gemm(sru.OP_NT, z(5, 4), z(6, 4), 5, 6, 4, ws=z(33, dtype=torch.uint8))
    assert stub.calls[-1][0] == "sru_gemm" and stub.calls[-1][1][-2] == 33


def test_backward_rejects_bad_arguments(stub):
    X, W = z(L, B, D), z(1, 3, D, D)
    p = [z(1, D) for _ in range(4)]
    base = dict(U=z(L, B, 1, 3, D), C=z(L, B, D), dH=z(L, B, D), dc_last=z(B, D),
                X_bf16=z(L, B, D, dtype=torch.bfloat16),
                W_bf16=z(1, 3, D, D, dtype=torch.bfloat16))

    def run(**kw):
        a = dict(base, **kw)
        return sru.backward(X, W, *p, a["U"], a["C"], a["dH"], dc_last=a["dc_last"],
                            X_bf16=a["X_bf16"], W_bf16=a["W_bf16"], out=a.get("out"))
    run()
    for name in base:
        for why, bad in bad_variants(base[name]):
            with pytest.raises(ValueError):
                run(**{name: bad})
    good = dict(dX=z(L, B, D), dW=z(1, 3, D, D), dv_f=z(1, D), dv_r=z(1, D), db_f=z(1, D),
                db_r=z(1, D), dc0=z(B, D))
    for name in good:
        for why, bad in bad_variants(good[name]):
            with pytest.raises(ValueError):
                run(out=dict(good, **{name: bad}))
    assert [c[0] for c in stub.calls] == ["sru_backward"]


def test_lowrank_calls_check_every_tensor(stub):
    dp = 4
    X, Q, P = z(L, B, D), z(D, dp), z(1, 3, D, dp)
    p = [z(1, D) for _ in range(4)]
    sru.forward_lowrank(X, Q, P, *p)
    base = dict(X=X, Q=Q, P=P, T=z(L, B, dp), U=z(L, B, 1, 3, D), C=z(L, B, D), dH=z(L, B, D),
                c0=z(B, D), dc_last=z(B, D), X_bf16=z(L, B, D, dtype=torch.bfloat16),
                T_bf16=z(L, B, dp, dtype=torch.bfloat16), v_f=p[0], b_r=p[3],
                mask=z(L, B, dtype=torch.uint8))

    def run(**kw):
        a = dict(base, **kw)
        return sru.backward_lowrank(a["X"], a["Q"], a["P"], a["v_f"], p[1], p[2], a["b_r"],
                                    a["T"], a["U"], a["C"], a["dH"], c0=a["c0"],
                                    dc_last=a["dc_last"], mask=a["mask"], X_bf16=a["X_bf16"],
                                    T_bf16=a["T_bf16"])
    run()
    n = len(stub.calls)
    for name in base:
        for why, bad in bad_variants(base[name]):
            if name == "mask" and why == "dtype":
                bad = bad.to(torch.int64)
            with pytest.raises(ValueError):
                run(**{name: bad})
    assert len(stub.calls) == n
    assert [c[0] for c in stub.calls] == ["sru_forward_lowrank", "sru_backward_lowrank"]


def test_scan_calls_check_every_tensor(stub):
    U = z(L, B, 1, 3, D)
    p = [z(1, D) for _ in range(4)]
    X = z(L, B, D)
    sru.scan_forward(U, X, *p)
    sru.scan_backward(U, X, z(L, B, D), z(L, B, D), *p)
    n = len(stub.calls)
    for why, bad in bad_variants(U):
        with pytest.raises(ValueError):
            sru.scan_forward(bad, X, *p)
    for why, bad in bad_variants(X):
        if why == "shape":
            bad = z(L, B + 1, D)
        with pytest.raises(ValueError):
            sru.scan_forward(U, bad, *p)
        with pytest.raises(ValueError):
            sru.scan_backward(U, bad, z(L, B, D), z(L, B, D), *p)
    for name in ("C", "dH"):
        for why, bad in bad_variants(z(L, B, D)):
            a = dict(C=z(L, B, D), dH=z(L, B, D))
            a[name] = bad
            with pytest.raises(ValueError):
                sru.scan_backward(U, X, a["C"], a["dH"], *p)
    for why, bad in bad_variants(z(L, B, D)):
        with pytest.raises(ValueError):
            sru.scan_forward(U, X, *p, out=dict(H=bad))
    for why, bad in bad_variants(z(L, B, 1, 3, D)):
        with pytest.raises(ValueError):
            sru.scan_backward(U, X, z(L, B, D), z(L, B, D), *p,
                              out=dict(dU=bad, db_f=z(1, D), db_r=z(1, D)))
    assert len(stub.calls) == n


def test_gemm_and_round_check_their_tensors(stub):
    A, Bm = z(5, 4), z(6, 4)
    sru.gemm(sru.OP_NT, A, Bm, 5, 6, 4)
    sru.round_bf16(z(10))
    n = len(stub.calls)
    for why, bad in bad_variants(A):
        with pytest.raises(ValueError):
            sru.gemm(sru.OP_NT, bad, Bm, 5, 6, 4)
    for why, bad in bad_variants(z(5, 6)):
        with pytest.raises(ValueError):
            sru.gemm(sru.OP_NT, A, Bm, 5, 6, 4, C=bad)
    with pytest.raises(ValueError):
        sru.round_bf16(z(10), out=z(10))
    assert len(stub.calls) == n


def test_host_tensors_rejected_without_the_seam(monkeypatch):
    """Without the stand-in, host tensors are refused before the library."""
    lib = StubLib()
    monkeypatch.setattr(sru, "_lib", lib)
    a = fwd_args()
    with pytest.raises(ValueError, match="GPU"):
        run_forward(a)
    assert lib.calls == []


def test_undersized_workspace_reaches_the_library_check(monkeypatch):
    """The real library refuses a workspace smaller than it needs
    (SRU_E_WORKSPACE) before it enqueues anything; the binding must pass the
    buffer's true size for that check to see it."""
    monkeypatch.setattr(sru, "_on_gpu", lambda t: True)
    monkeypatch.setattr(sru, "_stream", lambda: None)
    X, W = z(L, B, D), z(1, 3, D, D)
    p = [z(1, D) for _ in range(4)]
    U, C, dH = z(L, B, 1, 3, D), z(L, B, D), z(L, B, D)
    need = sru.backward_workspace_bytes(L, B, D, D, sru.DIR_FWD, sru.GEMM_FP32)
    assert need > 256
    small = torch.zeros(need - 256, dtype=torch.uint8)
    with pytest.raises(sru.SruError, match="WORKSPACE"):
        sru.backward(X, W, *p, U, C, dH, ws=small)
    need_f = sru.forward_workspace_bytes(L, B, D, D, sru.DIR_FWD, sru.GEMM_BF16)
    with pytest.raises(sru.SruError, match="WORKSPACE"):
        sru.forward(X, W, *p, gemm_dtype=sru.GEMM_BF16,
                    ws=torch.zeros(need_f - 256, dtype=torch.uint8))


def test_bf16_weights_passed_as_the_rounded_input(stub):
    """A bfloat16 W (weights held rounded) goes to the library as W_bf16 with
    W = NULL; it needs bf16 products and takes no second W_bf16; dW stays
    fp32."""
    a = fwd_args()
    Wb = z(1, 3, D, D, dtype=torch.bfloat16)
    a["W"], a["gemm"] = Wb, sru.GEMM_BF16
    run_forward(a)
    name, args = stub.calls[-1]
    assert name == "sru_forward" and args[1] is None and args[20].value == Wb.data_ptr()
    with pytest.raises(ValueError, match="bf16 products"):
        run_forward(dict(a, gemm=sru.GEMM_FP32))
    with pytest.raises(ValueError, match="already bfloat16"):
        run_forward(dict(a, out=dict(H=z(L, B, D), W_bf16=z(1, 3, D, D, dtype=torch.bfloat16))))
    X, p = a["X"], [z(1, D) for _ in range(4)]
    bw = sru.backward(X, Wb, *p, z(L, B, 1, 3, D), z(L, B, D), z(L, B, D),
                      gemm_dtype=sru.GEMM_BF16)
    name, args = stub.calls[-1]
    assert name == "sru_backward" and args[1] is None and args[27].value == Wb.data_ptr()
    assert bw["dW"].dtype == F32
    with pytest.raises(ValueError, match="already bfloat16"):
        sru.backward(X, Wb, *p, z(L, B, 1, 3, D), z(L, B, D), z(L, B, D),
                     gemm_dtype=sru.GEMM_BF16, W_bf16=Wb)
    assert [c[0] for c in stub.calls] == ["sru_forward", "sru_backward"]
